"""Python binding of libar: simulated-ring AllReduce for AMD MI355X (gfx950).

A thin ctypes layer over the C ABI in include/ar.h.  The functions named
``ar_*`` mirror the C entry points one to one; ``Plan`` and ``allreduce``
wrap them for torch tensors.  Every step of the AllReduce runs in the HIP
library; torch only provides device memory and streams.  If the library has
not been built (``__graft_entry__.build()`` or ``python -m
paper_2603_11438_amd._build``), loading fails with an error: there is no
fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "_lib", "libar.so")

# ---- constants (include/ar.h) -------------------------------------------
AR_VERSION = 4  # the interface revision include/ar.h declares
AR_FLOAT32, AR_BFLOAT16 = 0, 1
AR_PROTO_AUTO, AR_PROTO_LL, AR_PROTO_LL128, AR_PROTO_SIMPLE = -1, 0, 1, 2
AR_COLL_ALLREDUCE, AR_COLL_REDUCESCATTER, AR_COLL_ALLGATHER = 0, 1, 2
COLLS = {"allreduce": AR_COLL_ALLREDUCE, "reducescatter": AR_COLL_REDUCESCATTER, "allgather": AR_COLL_ALLGATHER}
AR_PLACE_RANK_SPREAD, AR_PLACE_CHANNEL_LOCAL = 0, 1
(AR_OK, AR_ERR_ARG, AR_ERR_UNSUPPORTED, AR_ERR_NOMEM, AR_ERR_HIP, AR_ERR_OCCUPANCY,
 AR_ERR_TIMEOUT, AR_ERR_STATE, AR_ERR_SCRATCH) = range(9)
AR_NOALLOC_SCRATCH_BYTES = 16 << 20
AR_DEBUG_SKIP_POST, AR_DEBUG_JITTER, AR_DEBUG_CHECK_LINES, AR_DEBUG_TRACE = 1, 2, 4, 8
TRACE_FIELDS = ("t_begin", "t_recv", "polls", "t_issued", "t_drained", "t_posted", "msg", "kind")
AR_PLAN_PROFILE, AR_PLAN_FIFO_ONLY, AR_PLAN_LL128_ORDERED = 1, 2, 4
AR_ALGO_AUTO, AR_ALGO_RING, AR_ALGO_DIRECT = 0, 1, 2
ALGOS = {"auto": AR_ALGO_AUTO, "ring": AR_ALGO_RING, "direct": AR_ALGO_DIRECT}
ALGO_NAMES = {v: k for k, v in ALGOS.items()}
AR_MAX_RANKS, AR_MAX_CHANNELS, AR_MAX_WAVES = 16, 256, 16

PROTOS = {"ll": AR_PROTO_LL, "ll128": AR_PROTO_LL128, "simple": AR_PROTO_SIMPLE, "auto": AR_PROTO_AUTO}
PROTO_NAMES = {v: k for k, v in PROTOS.items()}
DTYPES = {"f32": AR_FLOAT32, "bf16": AR_BFLOAT16}
DTYPE_NAMES = {v: k for k, v in DTYPES.items()}
ELEM_BYTES = {AR_FLOAT32: 4, AR_BFLOAT16: 2}


class ar_plan_desc(ctypes.Structure):
    _fields_ = [("nranks", ctypes.c_int), ("dtype", ctypes.c_int), ("count", ctypes.c_size_t),
                ("proto", ctypes.c_int), ("nchannels", ctypes.c_int), ("chunk_bytes", ctypes.c_size_t),
                ("fifo_depth", ctypes.c_int), ("nwaves", ctypes.c_int), ("placement", ctypes.c_int),
                ("timeout_us", ctypes.c_uint32), ("debug_flags", ctypes.c_uint32),
                ("max_channels", ctypes.c_int), ("comm_id", ctypes.c_uint64), ("flags", ctypes.c_uint32),
                ("algo", ctypes.c_int), ("coll", ctypes.c_int), ("direct_unroll", ctypes.c_int)]


class ar_plan_info(ctypes.Structure):
    _fields_ = [("nranks", ctypes.c_int), ("dtype", ctypes.c_int), ("proto", ctypes.c_int),
                ("nchannels", ctypes.c_int), ("nwaves", ctypes.c_int), ("fifo_depth", ctypes.c_int),
                ("placement", ctypes.c_int), ("grid", ctypes.c_int), ("block", ctypes.c_int),
                ("count", ctypes.c_size_t), ("seg_elems", ctypes.c_size_t), ("chan_elems", ctypes.c_size_t),
                ("chunk_elems", ctypes.c_size_t), ("wave_elems", ctypes.c_size_t), ("nchunks", ctypes.c_size_t),
                ("slot_bytes", ctypes.c_size_t), ("fifo_bytes", ctypes.c_size_t), ("flag_bytes", ctypes.c_size_t),
                ("msgs_per_run", ctypes.c_uint64), ("wire_bytes_per_run", ctypes.c_uint64), ("algo", ctypes.c_int),
                ("coll", ctypes.c_int), ("peer_direct", ctypes.c_int), ("direct_unroll", ctypes.c_int)]

    def as_dict(self) -> dict:
        d = {name: getattr(self, name) for name, _ in self._fields_}
        d["proto_name"] = PROTO_NAMES.get(d["proto"], str(d["proto"]))
        d["algo_name"] = ALGO_NAMES.get(d["algo"], str(d["algo"]))
        d["dtype_name"] = DTYPE_NAMES.get(d["dtype"], str(d["dtype"]))
        return d


class ar_debug_stats(ctypes.Structure):
    _fields_ = [("lines_checked", ctypes.c_uint64), ("lines_first_read", ctypes.c_uint64),
                ("lines_bad", ctypes.c_uint64)]


class ar_tune_ctx(ctypes.Structure):
    _fields_ = [("coll", ctypes.c_int), ("msg_bytes", ctypes.c_size_t), ("nranks", ctypes.c_int),
                ("dtype", ctypes.c_int), ("max_channels", ctypes.c_int), ("comm_id", ctypes.c_uint64)]


class ar_tune_out(ctypes.Structure):
    _fields_ = [("proto", ctypes.c_int), ("nchannels", ctypes.c_int), ("chunk_bytes", ctypes.c_size_t),
                ("nwaves", ctypes.c_int), ("algo", ctypes.c_int), ("direct_parts", ctypes.c_int),
                ("direct_nwaves", ctypes.c_int), ("direct_unroll", ctypes.c_int)]


class ar_latency_state(ctypes.Structure):
    _fields_ = [("comm_id", ctypes.c_uint64), ("latency_ns", ctypes.c_uint64), ("nchannels", ctypes.c_int),
                ("samples", ctypes.c_uint64)]


class ar_adaptive_cfg(ctypes.Structure):
    _fields_ = [("min_channels", ctypes.c_int), ("max_channels", ctypes.c_int), ("ramp_calls", ctypes.c_uint32),
                ("backoff_ratio", ctypes.c_uint32), ("proto", ctypes.c_int)]


class ar_reload_stats(ctypes.Structure):
    _fields_ = [("validate_ns", ctypes.c_uint64), ("swap_ns", ctypes.c_uint64), ("drain_ns", ctypes.c_uint64),
                ("probes", ctypes.c_uint64)]


ar_tuner_fn = ctypes.CFUNCTYPE(ctypes.c_int, ctypes.POINTER(ar_tune_ctx), ctypes.POINTER(ar_tune_out),
                               ctypes.c_void_p)

# Every symbol include/ar.h declares, with (restype, argtypes).
_P = ctypes.c_void_p
SIGNATURES = {
    "ar_plan": (_P, [ctypes.c_int, ctypes.c_size_t, ctypes.c_int, ctypes.c_int, ctypes.c_int]),
    "ar_plan_ex": (_P, [ctypes.POINTER(ar_plan_desc)]),
    "ar_run": (ctypes.c_int, [_P, ctypes.POINTER(_P), _P]),
    "ar_run_oop": (ctypes.c_int, [_P, ctypes.POINTER(_P), ctypes.POINTER(_P), _P]),
    "ar_run_noalloc": (ctypes.c_int, [ctypes.POINTER(ar_plan_desc), ctypes.POINTER(_P), ctypes.POINTER(_P), _P]),
    "ar_plan_status": (ctypes.c_int, [_P]),
    "ar_plan_reset": (ctypes.c_int, [_P]),
    "ar_plan_poison": (ctypes.c_int, [_P, _P]),
    "ar_destroy": (None, [_P]),
    "ar_plan_debug_stats": (ctypes.c_int, [_P, ctypes.POINTER(ar_debug_stats)]),
    "ar_plan_debug_trace": (ctypes.c_int, [_P, _P, ctypes.c_size_t]),
    "ar_plan_get_info": (ctypes.c_int, [_P, ctypes.POINTER(ar_plan_info)]),
    "ar_plan_workspace_bytes": (ctypes.c_size_t, [_P]),
    "ar_plan_geometry": (ctypes.c_int, [ctypes.POINTER(ar_plan_desc), ctypes.POINTER(ar_plan_info)]),
    "ar_set_tuner": (ctypes.c_int, [ar_tuner_fn, _P]),
    "ar_reload_tuner": (ctypes.c_int, [ar_tuner_fn, _P, ctypes.POINTER(ar_reload_stats)]),
    "ar_tune": (ctypes.c_int, [ctypes.POINTER(ar_tune_ctx), ctypes.POINTER(ar_tune_out)]),
    "ar_tuner_table": (ctypes.c_int, [ctypes.POINTER(ar_tune_ctx), ctypes.POINTER(ar_tune_out), _P]),
    "ar_tuner_fixed_default": (ctypes.c_int, [ctypes.POINTER(ar_tune_ctx), ctypes.POINTER(ar_tune_out), _P]),
    "ar_tuner_noop": (ctypes.c_int, [ctypes.POINTER(ar_tune_ctx), ctypes.POINTER(ar_tune_out), _P]),
    "ar_profile_record": (ctypes.c_int, [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int]),
    "ar_profile_lookup": (ctypes.c_int, [ctypes.c_uint64, ctypes.POINTER(ar_latency_state)]),
    "ar_profile_clear": (None, []),
    "ar_tuner_adaptive": (ctypes.c_int, [ctypes.POINTER(ar_tune_ctx), ctypes.POINTER(ar_tune_out), _P]),
    "ar_tuner_size_adaptive": (ctypes.c_int, [ctypes.POINTER(ar_tune_ctx), ctypes.POINTER(ar_tune_out), _P]),
    "ar_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "ar_last_error": (ctypes.c_int, []),
    "ar_version": (ctypes.c_int, []),
    "ar_debug_bf16_round": (ctypes.c_int, [_P, _P, ctypes.c_size_t, _P]),
}

_lib = None


class ARError(RuntimeError):
    def __init__(self, code: int, what: str = ""):
        self.code = code
        msg = ar_strerror(code) if _lib is not None else f"error {code}"
        super().__init__(f"{what}: {msg} (code {code})" if what else f"{msg} (code {code})")


def lib() -> ctypes.CDLL:
    """Load libar.so.  Raises if it has not been built: there is no fallback."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"libar is not built ({LIB_PATH} missing); run __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


# ---- one-to-one wrappers of the C entry points ---------------------------

def ar_strerror(code: int) -> str:
    return lib().ar_strerror(code).decode()


def ar_last_error() -> int:
    return lib().ar_last_error()


def ar_version() -> int:
    return lib().ar_version()


def _check(rc: int, what: str):
    if rc != AR_OK:
        raise ARError(rc, what)


def make_desc(nranks: int, count: int, dtype="f32", proto="auto", nchannels: int = 0, chunk_bytes: int = 0,
              fifo_depth: int = 0, nwaves: int = 0, placement: int = 0, timeout_us: int = 0,
              debug_flags: int = 0, max_channels: int = 0, comm_id: int = 0, flags: int = 0,
              algo="auto", coll="allreduce", direct_unroll: int = 0) -> ar_plan_desc:
    d = ar_plan_desc()
    d.nranks = nranks
    d.dtype = DTYPES[dtype] if isinstance(dtype, str) else dtype
    d.count = count
    d.proto = PROTOS[proto] if isinstance(proto, str) else (AR_PROTO_AUTO if proto is None else proto)
    d.nchannels = nchannels
    d.chunk_bytes = chunk_bytes
    d.fifo_depth = fifo_depth
    d.nwaves = nwaves
    d.placement = placement
    d.timeout_us = timeout_us
    d.debug_flags = debug_flags
    d.max_channels = max_channels
    d.comm_id = comm_id
    d.flags = flags
    d.algo = ALGOS[algo] if isinstance(algo, str) else algo
    d.coll = COLLS[coll] if isinstance(coll, str) else coll
    d.direct_unroll = direct_unroll
    return d


def ar_plan_geometry(desc: ar_plan_desc) -> dict:
    """Host-only geometry of a plan description (no GPU needed)."""
    info = ar_plan_info()
    _check(lib().ar_plan_geometry(ctypes.byref(desc), ctypes.byref(info)), "ar_plan_geometry")
    return info.as_dict()


def ar_tune(msg_bytes: int, nranks: int = 8, dtype="f32", max_channels: int = AR_MAX_CHANNELS,
            coll: int = AR_COLL_ALLREDUCE, comm_id: int = 0) -> dict:
    ctx = ar_tune_ctx(coll, msg_bytes, nranks, DTYPES[dtype] if isinstance(dtype, str) else dtype,
                      max_channels, comm_id)
    out = ar_tune_out()
    _check(lib().ar_tune(ctypes.byref(ctx), ctypes.byref(out)), "ar_tune")
    return {"proto": out.proto, "proto_name": PROTO_NAMES[out.proto], "nchannels": out.nchannels,
            "chunk_bytes": out.chunk_bytes, "nwaves": out.nwaves, "algo": out.algo,
            "algo_name": ALGO_NAMES[out.algo], "direct_parts": out.direct_parts,
            "direct_nwaves": out.direct_nwaves, "direct_unroll": out.direct_unroll}


_BUILTIN_TUNERS = {"table": "ar_tuner_table", "fixed_default": "ar_tuner_fixed_default", "noop": "ar_tuner_noop",
                   "adaptive": "ar_tuner_adaptive", "size_adaptive": "ar_tuner_size_adaptive"}


def ar_tuner_raw(name: str, msg_bytes: int, nranks: int = 8, dtype="f32", max_channels: int = AR_MAX_CHANNELS,
                 coll: int = AR_COLL_ALLREDUCE, comm_id: int = 0) -> dict:
    """Call one built-in tuner directly (no validation, no defaults filled
    in): what the policy itself answers.  Fields it leaves alone keep the
    no-opinion values (AUTO, 0)."""
    ctx = ar_tune_ctx(coll, msg_bytes, nranks, DTYPES[dtype] if isinstance(dtype, str) else dtype,
                      max_channels, comm_id)
    out = ar_tune_out(AR_PROTO_AUTO, 0, 0, 0, AR_ALGO_AUTO, 0, 0, 0)
    rc = getattr(lib(), _BUILTIN_TUNERS[name])(ctypes.byref(ctx), ctypes.byref(out), None)
    return {"rc": rc, "proto": out.proto, "nchannels": out.nchannels, "chunk_bytes": out.chunk_bytes,
            "nwaves": out.nwaves, "algo": out.algo, "direct_parts": out.direct_parts,
            "direct_nwaves": out.direct_nwaves, "direct_unroll": out.direct_unroll}


_tuner_refs = []  # keep ctypes callbacks alive while installed


def _tuner_callback(fn):
    L = lib()
    if fn == "adaptive":
        return ctypes.cast(L.ar_tuner_adaptive, ar_tuner_fn)
    if fn == "size_adaptive":
        return ctypes.cast(L.ar_tuner_size_adaptive, ar_tuner_fn)
    if fn is None or fn == "table":
        cb = ctypes.cast(L.ar_tuner_table, ar_tuner_fn)
    elif fn == "fixed_default":
        cb = ctypes.cast(L.ar_tuner_fixed_default, ar_tuner_fn)
    elif fn == "noop":
        cb = ctypes.cast(L.ar_tuner_noop, ar_tuner_fn)
    else:
        pyfn = fn

        def _trampoline(ctx_p, out_p, user):
            c = ctx_p.contents
            res = pyfn({"coll": c.coll, "msg_bytes": c.msg_bytes, "nranks": c.nranks, "dtype": c.dtype,
                        "max_channels": c.max_channels, "comm_id": c.comm_id})
            if res is None:
                return -1
            o = out_p.contents
            o.proto = int(res.get("proto", AR_PROTO_AUTO))
            o.nchannels = int(res.get("nchannels", 0))
            o.chunk_bytes = int(res.get("chunk_bytes", 0))
            o.nwaves = int(res.get("nwaves", 0))
            o.algo = int(res.get("algo", AR_ALGO_AUTO))
            o.direct_parts = int(res.get("direct_parts", 0))
            o.direct_nwaves = int(res.get("direct_nwaves", 0))
            o.direct_unroll = int(res.get("direct_unroll", 0))
            return int(res.get("rc", 0))

        cb = ar_tuner_fn(_trampoline)
    _tuner_refs.append(cb)
    return cb


_adaptive_cfgs = []


def ar_set_tuner(fn=None, adaptive: Optional[dict] = None):
    """Install a tuner: None (built-in table), a name ("table", "fixed_default",
    "noop", "adaptive"), or a Python callable fn(ctx: dict) -> dict | None.
    For "adaptive", `adaptive` may override ar_adaptive_cfg fields."""
    user = None
    if fn == "adaptive" and adaptive:
        cfg = ar_adaptive_cfg(2, 12, 9000, 4, AR_PROTO_SIMPLE)
        for k, v in adaptive.items():
            setattr(cfg, k, v)
        _adaptive_cfgs.append(cfg)
        user = ctypes.cast(ctypes.byref(cfg), ctypes.c_void_p)
    _check(lib().ar_set_tuner(_tuner_callback(fn), user), "ar_set_tuner")


def ar_profile_record(comm_id: int, latency_ns: int, nchannels: int) -> None:
    _check(lib().ar_profile_record(comm_id, latency_ns, nchannels), "ar_profile_record")


def ar_profile_lookup(comm_id: int) -> Optional[dict]:
    st = ar_latency_state()
    if lib().ar_profile_lookup(comm_id, ctypes.byref(st)) != AR_OK:
        return None
    return {"comm_id": st.comm_id, "latency_ns": st.latency_ns, "nchannels": st.nchannels, "samples": st.samples}


def ar_profile_clear() -> None:
    lib().ar_profile_clear()


def ar_reload_tuner(fn=None) -> dict:
    """Checked hot reload; raises ARError(AR_ERR_ARG) and keeps the current
    tuner if the candidate answers malformed decisions on the probe grid."""
    st = ar_reload_stats()
    _check(lib().ar_reload_tuner(_tuner_callback(fn), None, ctypes.byref(st)), "ar_reload_tuner")
    return {"validate_ns": st.validate_ns, "swap_ns": st.swap_ns, "drain_ns": st.drain_ns, "probes": st.probes}


# ---- torch-facing helpers -------------------------------------------------

def _stream_ptr(stream) -> Optional[int]:
    import torch

    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _ptr_array(tensors: Sequence) -> ctypes.Array:
    arr = (ctypes.c_void_p * max(len(tensors), 1))()
    for i, t in enumerate(tensors):
        arr[i] = t.data_ptr()
    return arr


_TORCH_DT = None


def _dtype_of(t) -> int:
    import torch

    if t.dtype == torch.float32:
        return AR_FLOAT32
    if t.dtype == torch.bfloat16:
        return AR_BFLOAT16
    raise TypeError(f"unsupported dtype {t.dtype}")


class Plan:
    """An AllReduce plan: geometry, FIFOs and flags for one (N, count, dtype)."""

    def __init__(self, nranks: int, count: int, dtype="f32", proto="auto", nchannels: int = 0,
                 chunk_bytes: int = 0, fifo_depth: int = 0, nwaves: int = 0, placement: int = 0,
                 timeout_us: int = 0, debug_flags: int = 0, comm_id: int = 0, flags: int = 0, algo="auto",
                 coll="allreduce", direct_unroll: int = 0):
        self.desc = make_desc(nranks, count, dtype, proto, nchannels, chunk_bytes, fifo_depth, nwaves,
                              placement, timeout_us, debug_flags, 0, comm_id, flags, algo, coll, direct_unroll)
        L = lib()
        h = L.ar_plan_ex(ctypes.byref(self.desc))
        if not h:
            raise ARError(L.ar_last_error(), "ar_plan_ex")
        self._h = ctypes.c_void_p(h)
        info = ar_plan_info()
        _check(L.ar_plan_get_info(self._h, ctypes.byref(info)), "ar_plan_get_info")
        self.info = info.as_dict()

    @property
    def handle(self):
        return self._h

    def run(self, tensors: Sequence, stream=None) -> None:
        """In-place collective over a list of N device tensors (each the full buffer)."""
        self._check_tensors(tensors, self._full)
        rc = lib().ar_run(self._h, _ptr_array(tensors), _stream_ptr(stream))
        _check(rc, "ar_run")

    def run_oop(self, send: Sequence, recv: Sequence, stream=None) -> None:
        coll = self.info["coll"]
        self._check_tensors(send, self.info["count"] if coll == AR_COLL_ALLGATHER else self._full)
        self._check_tensors(recv, self.info["count"] if coll == AR_COLL_REDUCESCATTER else self._full)
        rc = lib().ar_run_oop(self._h, _ptr_array(send), _ptr_array(recv), _stream_ptr(stream))
        _check(rc, "ar_run_oop")

    def bind(self, send: Sequence, recv: Optional[Sequence] = None, stream=None):
        """Check the buffers once and return a callable that launches the
        collective on them with one C call: in place on `send` when recv is
        None, else out of place.  For tight loops and timing: the returned
        callable keeps the tensors alive, and they must keep their storage
        while it is used; once the plan is destroyed a call raises."""
        coll = self.info["coll"]
        if recv is None:
            self._check_tensors(send, self._full)
        else:
            self._check_tensors(send, self.info["count"] if coll == AR_COLL_ALLGATHER else self._full)
            self._check_tensors(recv, self.info["count"] if coll == AR_COLL_REDUCESCATTER else self._full)
        sp = _ptr_array(send)
        rp = None if recv is None else _ptr_array(recv)
        st = _stream_ptr(stream)
        L = lib()
        keep = (list(send), None if recv is None else list(recv))
        plan = self

        if recv is None:
            def call():
                rc = L.ar_run(plan._h, sp, st)
                if rc:
                    _check(rc, "ar_run")
        else:
            def call():
                rc = L.ar_run_oop(plan._h, sp, rp, st)
                if rc:
                    _check(rc, "ar_run_oop")
        call.tensors = keep
        return call

    @property
    def _full(self) -> int:
        c = self.info["count"]
        return c if self.info["coll"] == AR_COLL_ALLREDUCE else c * self.info["nranks"]

    def _check_tensors(self, tensors, numel):
        n, dt = self.info["nranks"], self.info["dtype"]
        if len(tensors) != n:
            raise ValueError(f"expected {n} tensors, got {len(tensors)}")
        for t in tensors:
            if not t.is_cuda or not t.is_contiguous() or t.numel() != numel or _dtype_of(t) != dt:
                raise ValueError("each tensor must be a contiguous device tensor of the collective's size and dtype")

    def status(self) -> int:
        return lib().ar_plan_status(self._h)

    def reset(self) -> None:
        _check(lib().ar_plan_reset(self._h), "ar_plan_reset")

    def poison(self, stream=None) -> None:
        _check(lib().ar_plan_poison(self._h, _stream_ptr(stream)), "ar_plan_poison")

    def debug_stats(self) -> dict:
        """Line-check counts of AR_DEBUG_CHECK_LINES (after synchronising)."""
        st = ar_debug_stats()
        _check(lib().ar_plan_debug_stats(self._h, ctypes.byref(st)), "ar_plan_debug_stats")
        return {"lines_checked": st.lines_checked, "lines_first_read": st.lines_first_read,
                "lines_bad": st.lines_bad}

    def set_trace(self, buf) -> None:
        """Give an AR_DEBUG_TRACE plan its record buffer (a device tensor,
        kept alive by the plan; None stops tracing)."""
        self._trace_buf = buf
        ptr = None if buf is None else buf.data_ptr()
        nbytes = 0 if buf is None else buf.numel() * buf.element_size()
        _check(lib().ar_plan_debug_trace(self._h, ptr, nbytes), "ar_plan_debug_trace")

    @property
    def workspace_bytes(self) -> int:
        return lib().ar_plan_workspace_bytes(self._h)

    def destroy(self) -> None:
        if getattr(self, "_h", None) is not None and self._h.value:
            lib().ar_destroy(self._h)
            self._h = ctypes.c_void_p(0)

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.destroy()

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


_plan_cache = {}
_PLAN_CACHE_MAX = 64


def release_plans() -> None:
    """Free every plan `allreduce` has cached (after waiting for the device,
    since a cached plan may still be in flight on some stream)."""
    import torch

    if _plan_cache:
        torch.cuda.synchronize()
    for plan in _plan_cache.values():
        plan.destroy()
    _plan_cache.clear()


def allreduce(tensors: Sequence, proto="auto", nchannels: int = 0, chunk_bytes: int = 0, stream=None, **kw):
    """In-place sum AllReduce of N equal-shape device tensors (one per simulated rank).

    Plans are cached per shape, settings and stream: a plan must never be in
    flight on two streams at once (its FIFOs and flags are shared by all its
    runs), so calls on different streams use different plans.  The cache
    holds at most 64 plans; a call that would add one more first frees them
    all (release_plans), which waits for the device."""
    if not tensors:
        raise ValueError("need at least one tensor")
    t0 = tensors[0]
    dt = DTYPE_NAMES[_dtype_of(t0)]
    key = (len(tensors), t0.numel(), dt, proto, nchannels, chunk_bytes, tuple(sorted(kw.items())),
           _stream_ptr(stream))
    plan = _plan_cache.get(key)
    if plan is None:
        if len(_plan_cache) >= _PLAN_CACHE_MAX:
            release_plans()
        plan = Plan(len(tensors), t0.numel(), dt, proto, nchannels, chunk_bytes, **kw)
        _plan_cache[key] = plan
    plan.run(tensors, stream)
    return plan


def run_noalloc(send: Sequence, recv: Optional[Sequence] = None, stream=None, **desc_kw) -> None:
    """ar_run_noalloc on torch tensors: the collective desc_kw describes
    (make_desc's keywords; nranks, count and dtype come from the tensors),
    in place on `send` when recv is None.  Allocates no device memory: the
    ring uses the library's static scratch."""
    if not send:
        raise ValueError("need at least one tensor")
    coll = desc_kw.get("coll", "allreduce")
    coll = COLLS[coll] if isinstance(coll, str) else coll
    n = len(send)
    t0 = send[0]
    if recv is None:
        if coll == AR_COLL_ALLREDUCE:
            recv = send
            count = t0.numel()
        elif coll == AR_COLL_REDUCESCATTER:
            count = t0.numel() // n
            recv = [t.view(-1)[r * count:(r + 1) * count] for r, t in enumerate(send)]
        else:
            count = t0.numel() // n
            recv, send = send, [t.view(-1)[r * count:(r + 1) * count] for r, t in enumerate(send)]
    else:
        count = t0.numel() if coll != AR_COLL_REDUCESCATTER else t0.numel() // n
    d = make_desc(n, count, DTYPE_NAMES[_dtype_of(t0)], **desc_kw)
    full = count if coll == AR_COLL_ALLREDUCE else count * n
    send_n = count if coll == AR_COLL_ALLGATHER else full
    recv_n = count if coll == AR_COLL_REDUCESCATTER else full
    if len(send) != n or len(recv) != n:
        raise ValueError(f"expected {n} send and {n} recv tensors")
    for t, numel in [(t, send_n) for t in send] + [(t, recv_n) for t in recv]:
        if not t.is_cuda or not t.is_contiguous() or _dtype_of(t) != d.dtype or t.numel() != numel:
            raise ValueError("each tensor must be a contiguous device tensor of the collective's size and dtype")
    rc = lib().ar_run_noalloc(ctypes.byref(d), _ptr_array(send), _ptr_array(recv), _stream_ptr(stream))
    _check(rc, "ar_run_noalloc")


def ar_debug_bf16_round(x, stream=None):
    """Device bf16 rounding of a float32 device tensor; returns int16 bit patterns."""
    import torch

    out = torch.empty(x.numel(), dtype=torch.int16, device=x.device)
    _check(lib().ar_debug_bf16_round(x.data_ptr(), out.data_ptr(), x.numel(), _stream_ptr(stream)),
           "ar_debug_bf16_round")
    return out


def bus_bandwidth(msg_bytes: int, seconds: float, nranks: int) -> float:
    """busBW in GB/s (1e9 B/s): (S / t) * 2(N-1)/N for AllReduce."""
    if seconds <= 0:
        return float("inf")
    return msg_bytes / seconds * 2.0 * (nranks - 1) / nranks / 1e9


def alg_bandwidth(msg_bytes: int, seconds: float) -> float:
    return msg_bytes / seconds / 1e9


def ring_bytes(msg_bytes: int, nranks: int, dtype="f32", proto="simple", peer_direct: bool = False) -> float:
    """Bytes the ring formulation moves through global memory per AllReduce.

    Through FIFOs: every rank reads its input and writes its output (2 N S),
    and every element crosses 2(N-1) links, each written to a FIFO once and
    read once: N-1 crossings carry an fp32 partial, N-1 the finished value,
    scaled by the protocol's wire factor (LL 2, LL128 128/120, Simple 1).

    The peer-direct Simple ring (peer_direct), per element of a segment: the
    second rank reads the chain start's input and its own and writes an fp32
    partial (2e + 4); each of the N-3 further middle ranks reads a partial
    and its input and writes a partial (8 + e); the owner reads a partial
    and its input and writes its own and the next rank's output (4 + 3e);
    each of the N-2 forwarding ranks reads its output and writes the next
    rank's (2e); the last rank moves nothing.  With two ranks the owner is
    the second rank: it reads both inputs and writes both outputs (4e).

    The peer-direct LL and LL128 rings only start their chains with the
    peer read: the first hop's partial line is neither written nor read,
    2 * 4 * w bytes fewer per element than through the FIFOs."""
    e = 4 if dtype == "f32" else 2
    count = msg_bytes // e
    if peer_direct and proto == "simple" and nranks >= 2:
        if nranks == 2:
            return float(count * 4 * e)
        per_elem = (2 * e + 4) + (nranks - 3) * (8 + e) + (4 + 3 * e) + (nranks - 2) * 2 * e
        return float(count * per_elem)
    wf = {"simple": 1.0, "ll": 2.0, "ll128": 128.0 / 120.0}[proto]
    wire = count * (nranks - 1) * (4 + e) * wf
    total = 2.0 * nranks * msg_bytes + 2.0 * wire
    if peer_direct and proto in ("ll", "ll128") and nranks >= 2:
        total -= count * 2 * 4 * wf
    return total


def compulsory_bytes(msg_bytes: int, nranks: int) -> float:
    """Lower bound for any AllReduce of N buffers in one memory: read and write each once."""
    return 2.0 * nranks * msg_bytes
