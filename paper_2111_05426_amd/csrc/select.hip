// select.hip -- feasibility filter and ordered top-k over the candidates.
//
// Selection of Sec. 5.2: drop candidates whose peak exceeds the per-device
// memory cap (or whose status is non-zero), rank the rest by predicted time
// (makespan ascending, ties to the lower index), keep the first k.
//
// Two passes.  Pass 1: block b owns a contiguous chunk and extracts its k
// smallest (makespan, index) keys in order, round r selecting the smallest
// key strictly greater than round r-1's with a block-wide min reduction
// (the chunk is re-read per round; k <= 64 and chunks are small, so the
// passes stay within L2; chunks shrink to 256 keys while fewer than 256
// blocks would run).  Pass 2: one block merges the blocks' ascending
// k-lists, round r taking the least of the lists' heads.  The order is a
// total order on (makespan, index), so the result does not depend on the
// launch shape.
#include "internal.h"

#include <math.h>

namespace dsim {
namespace {

constexpr int kSelBlock = 256;
constexpr int64_t kChunk = 4096;
constexpr int64_t kMinChunk = 256;
constexpr int kMaxBlocks = 2048;
constexpr int kFillBlocks = 256;   // one chunk per CU at least, while chunks stay >= kMinChunk

struct Key {
    double mk;
    int64_t idx;
};

__device__ __forceinline__ bool key_less(double am, int64_t ai, double bm, int64_t bi)
{
    return am < bm || (am == bm && ai < bi);
}

// block-wide argmin of (m, i); returns the winner in every thread: a
// butterfly over each wavefront's lanes, then the wavefronts' winners
__device__ Key block_min(double m, int64_t i, double *s_m, int64_t *s_i)
{
    constexpr int kWaves = kSelBlock / 64;
    for (int o = 32; o > 0; o >>= 1) {
        const double om = __shfl_xor(m, o, 64);
        const int64_t oi = __shfl_xor(i, o, 64);
        if (key_less(om, oi, m, i)) {
            m = om;
            i = oi;
        }
    }
    if ((threadIdx.x & 63) == 0) {
        s_m[threadIdx.x / 64] = m;
        s_i[threadIdx.x / 64] = i;
    }
    __syncthreads();
    Key k{s_m[0], s_i[0]};
    for (int v = 1; v < kWaves; ++v)
        if (key_less(s_m[v], s_i[v], k.mk, k.idx)) k = Key{s_m[v], s_i[v]};
    __syncthreads();
    return k;
}

constexpr int64_t kNone = INT64_MAX;

__global__ __launch_bounds__(kSelBlock) void k_select_chunks(const double *mk, const uint64_t *pk,
                                                             const int32_t *st, int64_t n, uint64_t cap,
                                                             int k, int64_t chunk, Key *ws)
{
    __shared__ double s_m[kSelBlock];
    __shared__ int64_t s_i[kSelBlock];
    const int64_t lo = (int64_t)blockIdx.x * chunk;
    const int64_t hi = lo + chunk < n ? lo + chunk : n;
    double pm = -HUGE_VAL;
    int64_t pi = -1;
    for (int r = 0; r < k; ++r) {
        double bm = HUGE_VAL;
        int64_t bi = kNone;
        for (int64_t i = lo + threadIdx.x; i < hi; i += kSelBlock) {
            if (st[i] != 0) continue;
            if (cap != 0 && pk[i] > cap) continue;
            const double m = mk[i];
            if (!key_less(pm, pi, m, i)) continue;
            if (key_less(m, i, bm, bi)) {
                bm = m;
                bi = i;
            }
        }
        const Key best = block_min(bm, bi, s_m, s_i);
        if (threadIdx.x == 0) {
            ws[(int64_t)blockIdx.x * k + r].mk = best.mk;
            ws[(int64_t)blockIdx.x * k + r].idx = best.idx == kNone ? -1 : best.idx;
        }
        pm = best.mk;
        pi = best.idx;
        if (best.idx == kNone) {
            for (int q = r + 1; q < k && threadIdx.x == 0; ++q) {
                ws[(int64_t)blockIdx.x * k + q].mk = HUGE_VAL;
                ws[(int64_t)blockIdx.x * k + q].idx = -1;
            }
            break;
        }
    }
}

// Pass 2: the blocks' lists are ascending, so round r's key is the least
// of the lists' heads; each thread holds the heads of its lists (list q
// at thread q mod kSelBlock) and the owner of the winning head advances it.
constexpr int kListsPerThread = kMaxBlocks / kSelBlock;
__global__ __launch_bounds__(kSelBlock) void k_select_merge(const Key *ws, int64_t nl, int k,
                                                            int64_t *out_idx, double *out_mk,
                                                            int32_t *out_found)
{
    __shared__ double s_m[kSelBlock];
    __shared__ int64_t s_i[kSelBlock];
    int head[kListsPerThread];
    double hm[kListsPerThread];
    int64_t hi[kListsPerThread];
#pragma unroll
    for (int j = 0; j < kListsPerThread; ++j) {
        const int64_t q = threadIdx.x + (int64_t)j * kSelBlock;
        head[j] = 0;
        hm[j] = HUGE_VAL;
        hi[j] = kNone;
        if (q < nl && ws[q * k].idx >= 0) {
            hm[j] = ws[q * k].mk;
            hi[j] = ws[q * k].idx;
        }
    }
    int found = 0;
    for (int r = 0; r < k; ++r) {
        double bm = HUGE_VAL;
        int64_t bi = kNone;
#pragma unroll
        for (int j = 0; j < kListsPerThread; ++j)
            if (key_less(hm[j], hi[j], bm, bi)) {
                bm = hm[j];
                bi = hi[j];
            }
        const Key best = block_min(bm, bi, s_m, s_i);
        if (threadIdx.x == 0) {
            out_idx[r] = best.idx == kNone ? -1 : best.idx;
            out_mk[r] = best.idx == kNone ? HUGE_VAL : best.mk;
        }
        if (best.idx == kNone) continue;
        found = r + 1;
#pragma unroll
        for (int j = 0; j < kListsPerThread; ++j)
            if (hi[j] == best.idx) {   // indices are unique: this thread's list holds the winner
                const int64_t q = threadIdx.x + (int64_t)j * kSelBlock;
                ++head[j];
                hm[j] = HUGE_VAL;
                hi[j] = kNone;
                if (head[j] < k && ws[q * k + head[j]].idx >= 0) {
                    hm[j] = ws[q * k + head[j]].mk;
                    hi[j] = ws[q * k + head[j]].idx;
                }
            }
    }
    if (threadIdx.x == 0) *out_found = found;
}

int64_t n_chunks(int64_t n, int64_t *chunk)
{
    int64_t c = kChunk;
    while ((n + c - 1) / c > kMaxBlocks) c *= 2;
    while (c > kMinChunk && (n + c - 1) / c < kFillBlocks) c /= 2;
    *chunk = c;
    const int64_t b = (n + c - 1) / c;
    return b > 0 ? b : 1;
}

}  // namespace

size_t argmin_workspace(int64_t n, int32_t k)
{
    int64_t chunk;
    return (size_t)n_chunks(n, &chunk) * (size_t)k * sizeof(Key);
}

dsim_status launch_argmin(const double *mk, const uint64_t *pk, const int32_t *st, int64_t n,
                          uint64_t cap, int32_t k, void *ws, int64_t *out_idx, double *out_mk,
                          int32_t *out_found, hipStream_t s)
{
    int64_t chunk;
    const int64_t blocks = n_chunks(n, &chunk);
    Key *w = static_cast<Key *>(ws);
    hipLaunchKernelGGL(k_select_chunks, dim3((unsigned)blocks), dim3(kSelBlock), 0, s, mk, pk, st, n,
                       cap, k, chunk, w);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "select_chunks launch");
    hipLaunchKernelGGL(k_select_merge, dim3(1), dim3(kSelBlock), 0, s, w, blocks, k, out_idx, out_mk, out_found);
    e = hipGetLastError();
    return e == hipSuccess ? DSIM_OK : hip_fail(e, "select_merge launch");
}

}  // namespace dsim
