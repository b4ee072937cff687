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
// passes stay within L2).  Pass 2: one block applies the same rounds to the
// blocks' k-lists.  The order is a total order on (makespan, index), so the
// result does not depend on the launch shape.
#include "internal.h"

#include <math.h>

namespace dsim {
namespace {

constexpr int kSelBlock = 256;
constexpr int64_t kChunk = 4096;
constexpr int kMaxBlocks = 2048;

struct Key {
    double mk;
    int64_t idx;
};

__device__ __forceinline__ bool key_less(double am, int64_t ai, double bm, int64_t bi)
{
    return am < bm || (am == bm && ai < bi);
}

// block-wide argmin of (m, i); returns the winner in every thread
__device__ Key block_min(double m, int64_t i, double *s_m, int64_t *s_i)
{
    const int tid = threadIdx.x;
    s_m[tid] = m;
    s_i[tid] = i;
    __syncthreads();
    for (int w = kSelBlock / 2; w > 0; w >>= 1) {
        if (tid < w && key_less(s_m[tid + w], s_i[tid + w], s_m[tid], s_i[tid])) {
            s_m[tid] = s_m[tid + w];
            s_i[tid] = s_i[tid + w];
        }
        __syncthreads();
    }
    Key k{s_m[0], s_i[0]};
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

__global__ __launch_bounds__(kSelBlock) void k_select_merge(const Key *ws, int64_t m, int k,
                                                            int64_t *out_idx, double *out_mk,
                                                            int32_t *out_found)
{
    __shared__ double s_m[kSelBlock];
    __shared__ int64_t s_i[kSelBlock];
    double pm = -HUGE_VAL;
    int64_t pi = -1;
    int found = 0;
    for (int r = 0; r < k; ++r) {
        double bm = HUGE_VAL;
        int64_t bi = kNone;
        for (int64_t q = threadIdx.x; q < m; q += kSelBlock) {
            const int64_t i = ws[q].idx;
            if (i < 0) continue;
            const double v = ws[q].mk;
            if (!key_less(pm, pi, v, i)) continue;
            if (key_less(v, i, bm, bi)) {
                bm = v;
                bi = i;
            }
        }
        const Key best = block_min(bm, bi, s_m, s_i);
        if (threadIdx.x == 0) {
            out_idx[r] = best.idx == kNone ? -1 : best.idx;
            out_mk[r] = best.idx == kNone ? HUGE_VAL : best.mk;
        }
        if (best.idx != kNone) found = r + 1;
        pm = best.mk;
        pi = best.idx;
    }
    if (threadIdx.x == 0) *out_found = found;
}

int64_t n_chunks(int64_t n, int64_t *chunk)
{
    int64_t c = kChunk;
    while ((n + c - 1) / c > kMaxBlocks) c *= 2;
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
    hipLaunchKernelGGL(k_select_merge, dim3(1), dim3(kSelBlock), 0, s, w, blocks * (int64_t)k, k,
                       out_idx, out_mk, out_found);
    e = hipGetLastError();
    return e == hipSuccess ? DSIM_OK : hip_fail(e, "select_merge launch");
}

}  // namespace dsim
