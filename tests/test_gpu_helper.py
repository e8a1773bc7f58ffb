"""The binding's `allreduce` helper: in-place results equal the oracle, one
cached plan per shape, settings and stream, and a bounded cache."""
from __future__ import annotations

import numpy as np
import pytest

from tests.gpu_helpers import assert_ranks_equal, draw, oracle_bits, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ar():
    import torch

    import paper_2603_11438_amd as ar

    assert torch.cuda.is_available()
    torch.cuda.set_device(0)
    ar.lib()
    ar.ar_set_tuner(None)
    return ar


def test_allreduce_helper_results_and_cache(ar):
    import torch

    ar.release_plans()
    x = draw(8, 5003, "f32", "uniform", seed=61)
    ts = to_device(x, "f32")
    p1 = ar.allreduce(ts)
    torch.cuda.synchronize()
    assert_ranks_equal(ts, oracle_bits(x, "f32"), "f32", "helper auto")
    # the same key reuses the plan; another stream or protocol gets its own
    ts = to_device(x, "f32")
    assert ar.allreduce(ts) is p1
    torch.cuda.synchronize()
    assert_ranks_equal(ts, oracle_bits(x, "f32"), "f32", "helper auto, cached plan")
    side = torch.cuda.Stream()
    ts = to_device(x, "f32")
    side.wait_stream(torch.cuda.current_stream())
    p2 = ar.allreduce(ts, stream=side)
    side.synchronize()
    assert p2 is not p1
    assert_ranks_equal(ts, oracle_bits(x, "f32"), "f32", "helper auto, side stream")
    xb = draw(3, 777, "bf16", "normal", seed=62)
    tb = to_device(xb, "bf16")
    p3 = ar.allreduce(tb, proto="ll", nchannels=2)
    torch.cuda.synchronize()
    assert p3 not in (p1, p2)
    assert_ranks_equal(tb, oracle_bits(xb, "bf16"), "bf16", "helper ll bf16")
    ar.release_plans()
    assert not ar._plan_cache


def test_allreduce_helper_cache_is_bounded(ar):
    import torch

    ar.release_plans()
    for i in range(ar._PLAN_CACHE_MAX + 5):
        count = 64 + i
        x = draw(2, count, "f32", "uniform", seed=700 + i)
        ts = to_device(x, "f32")
        ar.allreduce(ts, proto="simple", nchannels=1)
        torch.cuda.synchronize()
        assert_ranks_equal(ts, oracle_bits(x, "f32"), "f32", f"helper count {count}")
        assert len(ar._plan_cache) <= ar._PLAN_CACHE_MAX
    assert len(ar._plan_cache) == 5
    ar.release_plans()
    assert not ar._plan_cache
