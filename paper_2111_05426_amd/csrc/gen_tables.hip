// gen_tables.hip -- the random-program workload, generated on the GPU.
//
// One lane per candidate writes its op records in program order, straight
// into the op-major / candidate-fastest table layout (coalesced stores).
//
// Every random decision is a pure function of (seed, candidate, op, field):
// draw f of op j of candidate c is output number c*2^32 + j*32 + f + 1 of
// SplitMix64 (Steele, Lea & Flood, OOPSLA 2014) seeded with `seed`, i.e.
// mix(seed + n * 0x9E3779B97F4A7C15).  Fields:
//   0 op kind: floor(hi32 * 10 / 2^32): 0..6 compute, 7..8 send, 9 all-reduce
//   1 device a: uniform in [0, n_dev)
//   2 send: destination a + 1 + uniform[0, n_dev - 1) mod n_dev;
//     all-reduce: index into the ascending list of masks with >= 2 bits
//   3 compute FLOPs, log-uniform in [1e6, 1e12]
//   4 compute / all-reduce bytes, log-uniform in [1e3, 1e9]
//   5 compute / send: free one of device a's live buffers (top bit = coin,
//     low 32 bits pick the buffer uniformly; the last buffer moves into the
//     hole)
//   6 compute: allocate a new buffer on a (top bit = coin, if a has < 16)
//   7 size of the new buffer (compute) or of the message (send), log-uniform
//     in [1e3, 1e9] bytes; a send's message becomes a live buffer of the
//     destination when the destination has < 16
// Log-uniform in [lo, hi]: 2^t rounded once to fp32, t = log2(lo) + u
// (log2(hi) - log2(lo)) with u the top 53 bits of the draw over 2^53 and
// the logarithms taken as the nearest doubles; 2^t = 2^floor(t) e^(y),
// y = (t - floor(t)) ln 2, e^y summed as its Taylor series up to y^13
// (Horner form, fp64, no contraction: the oracle computes the same bits).
#include "internal.h"

namespace dsim {
namespace {

constexpr int kGenBlock = 64;
constexpr int kSlots = 16;

struct GenArgs {
    uint64_t seed;
    int64_t n_cand;
    int32_t n_ops, n_dev;
    uint32_t *code;
    float *flops;
    float *bytes;
    uint32_t *alloc;
    uint32_t *freeb;
    uint32_t *n_ops_out;
};

__device__ __forceinline__ uint64_t splitmix_at(uint64_t seed, uint64_t n)
{
    uint64_t z = seed + n * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__device__ __forceinline__ uint32_t pick(uint64_t r, uint32_t n)
{
    return (uint32_t)(((r >> 32) * (uint64_t)n) >> 32);
}

// base-2 logarithms of the bounds (nearest doubles)
constexpr double kLog2_1e3 = 0x1.3ee7b471b3a95p+3, kLog2_1e6 = 0x1.3ee7b471b3a95p+4;
constexpr double kLog2_1e9 = 0x1.de5b8eaa8d7e0p+4, kLog2_1e12 = 0x1.3ee7b471b3a95p+5;

__device__ __forceinline__ float log_uniform(uint64_t r, double log2_lo, double log2_hi)
{
    // 1 / k! for k = 13 down to 0
    constexpr double c[14] = {0x1.6124613a86d09p-33, 0x1.1eed8eff8d898p-29, 0x1.ae64567f544e4p-26,
                              0x1.27e4fb7789f5cp-22, 0x1.71de3a556c734p-19, 0x1.a01a01a01a01ap-16,
                              0x1.a01a01a01a01ap-13, 0x1.6c16c16c16c17p-10, 0x1.1111111111111p-7,
                              0x1.5555555555555p-5, 0x1.5555555555555p-3, 0.5, 1.0, 1.0};
    const double u = (double)(r >> 11) * 0x1p-53;
    const double t = log2_lo + u * (log2_hi - log2_lo);
    const double n = floor(t);
    const double y = (t - n) * 0x1.62e42fefa39efp-1;
    double e = c[0];
#pragma unroll
    for (int k = 1; k < 14; ++k) e = e * y + c[k];
    return (float)ldexp(e, (int)n);
}

__global__ __launch_bounds__(kGenBlock) void k_gen_tables(const GenArgs g)
{
    __shared__ uint32_t s_buf[8][kSlots][kGenBlock];
    __shared__ uint32_t s_cnt[8][kGenBlock];
    __shared__ uint32_t s_masks[256];
    __shared__ uint32_t s_nmasks;

    const int tid = threadIdx.x;
    if (tid == 0) {
        uint32_t n = 0;
        for (uint32_t mask = 0; mask < (1u << g.n_dev); ++mask)
            if (__popc(mask) >= 2) s_masks[n++] = mask;
        s_nmasks = n;
    }
    for (int d = 0; d < 8; ++d) s_cnt[d][tid] = 0;
    __syncthreads();
    const int64_t cand = (int64_t)blockIdx.x * kGenBlock + tid;
    if (cand >= g.n_cand) return;

    const uint64_t c = (uint64_t)cand;
    const uint64_t seed = g.seed;
    const uint32_t nd = (uint32_t)g.n_dev;
    const uint32_t n_masks = s_nmasks;
    const size_t N = (size_t)g.n_cand;

    for (int32_t j = 0; j < g.n_ops; ++j) {
        const uint64_t base = (c << 32) + ((uint64_t)j << 5) + 1u;
        const uint32_t kd = pick(splitmix_at(seed, base + 0), 10u);
        const uint32_t a = pick(splitmix_at(seed, base + 1), nd);
        uint32_t al = 0, fr = 0, code;
        float fl = 0.f, by;
        if (kd < 9u) {
            const uint64_t r5 = splitmix_at(seed, base + 5);
            const uint32_t na = s_cnt[a][tid];
            if ((r5 >> 63) && na > 0u) {
                const uint32_t i = (uint32_t)(((r5 & 0xffffffffull) * (uint64_t)na) >> 32);
                fr = s_buf[a][i][tid];
                s_buf[a][i][tid] = s_buf[a][na - 1u][tid];
                s_cnt[a][tid] = na - 1u;
            }
        }
        if (kd < 7u) {
            const uint64_t r6 = splitmix_at(seed, base + 6);
            code = a << 8;
            fl = log_uniform(splitmix_at(seed, base + 3), kLog2_1e6, kLog2_1e12);
            by = log_uniform(splitmix_at(seed, base + 4), kLog2_1e3, kLog2_1e9);
            const uint32_t na = s_cnt[a][tid];
            if ((r6 >> 63) && na < (uint32_t)kSlots) {
                al = (uint32_t)log_uniform(splitmix_at(seed, base + 7), kLog2_1e3, kLog2_1e9);
                s_buf[a][na][tid] = al;
                s_cnt[a][tid] = na + 1u;
            }
        } else if (kd < 9u) {
            const uint32_t b = (a + 1u + pick(splitmix_at(seed, base + 2), nd - 1u)) % nd;
            const uint32_t msg = (uint32_t)log_uniform(splitmix_at(seed, base + 7), kLog2_1e3, kLog2_1e9);
            code = 1u | (a << 8) | (b << 16);
            by = (float)msg;
            const uint32_t nb = s_cnt[b][tid];
            if (nb < (uint32_t)kSlots) {
                al = msg;
                s_buf[b][nb][tid] = msg;
                s_cnt[b][tid] = nb + 1u;
            }
        } else {
            const uint32_t mask = s_masks[pick(splitmix_at(seed, base + 2), n_masks)];
            code = 2u | (mask << 16);
            by = log_uniform(splitmix_at(seed, base + 4), kLog2_1e3, kLog2_1e9);
        }
        const size_t o = (size_t)j * N + (size_t)cand;
        __builtin_nontemporal_store(code, g.code + o);
        __builtin_nontemporal_store(fl, g.flops + o);
        __builtin_nontemporal_store(by, g.bytes + o);
        __builtin_nontemporal_store(al, g.alloc + o);
        __builtin_nontemporal_store(fr, g.freeb + o);
    }
    if (g.n_ops_out) g.n_ops_out[cand] = (uint32_t)g.n_ops;
}

}  // namespace

dsim_status launch_gen_tables(uint64_t seed, int64_t n_cand, int32_t n_ops, int32_t n_dev,
                              uint32_t *code, float *flops, float *bytes, uint32_t *alloc,
                              uint32_t *freeb, uint32_t *n_ops_out, hipStream_t s)
{
    if (n_cand == 0) return DSIM_OK;
    GenArgs g{seed, n_cand, n_ops, n_dev, code, flops, bytes, alloc, freeb, n_ops_out};
    const int64_t blocks = (n_cand + kGenBlock - 1) / kGenBlock;
    hipLaunchKernelGGL(k_gen_tables, dim3((unsigned)blocks), dim3(kGenBlock), 0, s, g);
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? DSIM_OK : hip_fail(e, "gen_tables launch");
}

}  // namespace dsim
