/*
 * Plain-C CPU oracle for the simulated-ring AllReduce (sum) -- TEST
 * INFRASTRUCTURE.  Used by the tests and by the benchmark's CPU-baseline
 * leg only; the HIP library never links or calls it and shares no code
 * with it.
 *
 * It computes the same thing as ring_oracle.py: AllReduce-sum over N rank
 * buffers (paper, section 2 and section 5.3, Table 2), with every element
 * reduced along its segment-major ring chain:
 *
 *   A   = 16 / element bytes, seg = roundup(ceil(count / N), A)
 *   segment s = [s*seg, min((s+1)*seg, count))
 *   acc = x_s[i]; acc += x_{s+1}[i]; ... ; acc += x_{s+N-1}[i]   (mod N)
 *
 * in IEEE binary32 round-to-nearest-even with subnormals kept.  bf16 inputs
 * are widened exactly, summed in fp32 and rounded to bf16 once (RNE, NaN ->
 * 0x7FC0).
 *
 * Build: gcc -O2 -fno-fast-math -ffp-contract=off -fopenmp -shared -fPIC.
 * The optional thread count splits the elements of a segment across OpenMP
 * threads; each element's chain is still one thread's sequential loop, so
 * the order of additions, and hence every bit, is independent of it.
 */
#include <stddef.h>
#include <stdint.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

uint64_t ring_oracle_segment(int nranks, uint64_t count, int elem_bytes)
{
    if (nranks < 1 || (elem_bytes != 2 && elem_bytes != 4)) return 0;
    uint64_t a = 16u / (uint64_t)elem_bytes;
    uint64_t per = (count + (uint64_t)nranks - 1) / (uint64_t)nranks;
    return (per + a - 1) / a * a;
}

static float bf16_widen(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

static uint16_t bf16_round(float f)
{
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;
    uint32_t lsb = (u >> 16) & 1u;
    return (uint16_t)((u + 0x7FFFu + lsb) >> 16);
}

/* y[i] for all i; x[r] points at rank r's count floats. */
int ring_oracle_f32(const float *const *x, float *y, int nranks, uint64_t count,
                    int nthreads)
{
    if (nranks < 1 || !x || (count && !y)) return -1;
    uint64_t seg = ring_oracle_segment(nranks, count, 4);
    for (int s = 0; s < nranks; ++s) {
        uint64_t lo = (uint64_t)s * seg;
        uint64_t hi = lo + seg < count ? lo + seg : count;
        if (lo >= hi) continue;
        int64_t n = (int64_t)(hi - lo);
#pragma omp parallel for schedule(static) num_threads(nthreads > 0 ? nthreads : 1) if (nthreads > 1)
        for (int64_t k = 0; k < n; ++k) {
            uint64_t i = lo + (uint64_t)k;
            float acc = x[s][i];
            for (int j = 1; j < nranks; ++j) acc = acc + x[(s + j) % nranks][i];
            y[i] = acc;
        }
    }
    return 0;
}

/* bf16 bits in and out; fp32 chain, one rounding. */
int ring_oracle_bf16(const uint16_t *const *x, uint16_t *y, int nranks,
                     uint64_t count, int nthreads)
{
    if (nranks < 1 || !x || (count && !y)) return -1;
    uint64_t seg = ring_oracle_segment(nranks, count, 2);
    for (int s = 0; s < nranks; ++s) {
        uint64_t lo = (uint64_t)s * seg;
        uint64_t hi = lo + seg < count ? lo + seg : count;
        if (lo >= hi) continue;
        int64_t n = (int64_t)(hi - lo);
#pragma omp parallel for schedule(static) num_threads(nthreads > 0 ? nthreads : 1) if (nthreads > 1)
        for (int64_t k = 0; k < n; ++k) {
            uint64_t i = lo + (uint64_t)k;
            float acc = bf16_widen(x[s][i]);
            for (int j = 1; j < nranks; ++j) acc = acc + bf16_widen(x[(s + j) % nranks][i]);
            y[i] = bf16_round(acc);
        }
    }
    return 0;
}

int ring_oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
