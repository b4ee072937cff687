// parametric.hip -- simulate the D/H/P/K transform without building op lists.
//
// Each candidate gets a segment of W = 2^ceil(log2 P) lanes of a wavefront,
// one lane per pipeline stage; segments of equal width share wavefronts
// (64 / W candidates each).  A lane expands, on the fly and in program order,
// the ops of its stage of the distributed program the transform of Sec. 4
// produces (ops in model.h) and simulates them with the semantics of Sec. 2.1
// and the cost model of Sec. 3.3:
//   * synchronous 1F1B (training) or forward-only (inference) per stage;
//   * the global order is slot by slot: every stage runs its next block if
//     the block's input was produced in an earlier slot (the stages of a slot
//     touch disjoint devices, so they run in parallel lanes); then the slot's
//     Sends run in ascending order of source stage, a serial chain of
//     max-plus steps across neighbouring lanes (DPP wave shifts); the weight
//     update follows the last slot;
//   * every replica (d, h) of a stage runs the same ops at the same times, so
//     one replica per stage is walked: a collective over the H ranks or the
//     D replicas starts at the stage's own clock and costs the ring
//     all-reduce of its full group; a Send synchronises two stage clocks.
//
// The layers of a stage repeat one op sequence (for the MLP with H > 1, one
// column/row layer pair), so each lane records that sequence's op costs once
// per microbatch size and direction (LDS, [entry][lane]) together with its
// memory summary (net bytes, peak above the starting live bytes, op counts),
// and walks a block's layers as a chain of fp64 adds over the recorded costs.
// Adding the same costs in the same order gives the same rounding as the op
// by op walk, and the memory summary is exact integer arithmetic.  Ops outside
// the repeating part (embedding, LM head, loss, the stage's first MLP layer in
// backward, the last layer in inference) and backward blocks of microbatch 0
// (which have no gradient accumulation) are walked op by op.
//
// A counting-sort pre-pass groups the candidates by segment width into a
// temporary permutation (stable, so the grid's own order keeps wavefronts
// uniform in K).
#include "model.h"

namespace dsim {
namespace {

constexpr int kLanes = 64;
constexpr int kClasses = 7;       // segment widths 1, 2, 4, ..., 64
constexpr int kScanBlock = 256;
constexpr int kPat2 = 12;         // pattern capacity per direction, in double2

// pattern sizes (double2 entries) per model family
template <bool TF> struct PatSize;
template <> struct PatSize<true> {
    static constexpr int F2 = 7;    // 12 compute ops + 2 all-reduces
    static constexpr int B2 = 12;   // 17 compute + 4 accumulations + 2 all-reduces
};
template <> struct PatSize<false> {
    static constexpr int F2 = 3;    // column layer (2 ops) + row layer (3)
    static constexpr int B2 = 5;    // row layer (4 ops) + column layer (5)
};

struct ParArgs {
    dsim_model m;
    const dsim_strategy *cand;
    int64_t n_cand;
    int32_t row_width;
    int32_t p_bound;
    const uint32_t *perm;   // candidates grouped by segment class
    const uint32_t *meta;   // [0,8) class totals, [8,16) first perm index, [16,24) first lane
    double *makespan;
    double *finish;
    uint64_t *peak;
    uint64_t *cand_peak;
    uint64_t *n_ops;
    uint64_t *walked;
    int32_t *status;
    CostConsts c;
};

__device__ __forceinline__ int seg_class(const dsim_strategy &st, int p_bound)
{
    const int P = st.P;
    if (P < 1 || P > p_bound) return 0;
    int j = 0;
    while ((1 << j) < P) ++j;
    return j;
}

// ---------------------------------------------------------------------------
// Sinks
// ---------------------------------------------------------------------------
// The lane's stage replica, op by op.
struct Walk {
    const Ctx &x;
    double clk;
    int64_t live, peak;
    uint64_t walked, nops;

    __device__ __forceinline__ void local(uint64_t fl, uint64_t by, uint64_t al, uint64_t fr)
    {
        clk = clk + cost_local(x, fl, by);
        live += (int64_t)al;
        peak = live > peak ? live : peak;
        live -= (int64_t)fr;
        walked += 1;
        nops += x.mult_dev;
    }
    __device__ __forceinline__ void ar_tp(uint64_t by)
    {
        if (x.H <= 1) return;
        clk = clk + cost_ar_tp(x, by);
        walked += 1;
        nops += x.mult_tp;
    }
    __device__ __forceinline__ void ar_dp(uint64_t by)
    {
        if (x.D <= 1) return;
        clk = clk + cost_ar_dp(x, by);
        walked += 1;
        nops += x.mult_dp;
    }
};

// Memory and op-count summary of one repeating unit.
struct Summary {
    int64_t delta;     // live bytes after the unit minus before
    int64_t top;       // max over the unit's ops of (live after alloc) minus live before
    uint64_t walked;   // ops walked per unit
    uint64_t nops;     // program ops per unit
};

// Records a unit's op costs into the lane's LDS pattern and summarises it.
struct Record {
    const Ctx &x;
    double *base;      // entry j at base[(j / 2) * 2 * kLanes + (j & 1)]
    int n;
    int64_t cur, top;
    uint64_t walked, nops;

    __device__ __forceinline__ void put(double c)
    {
        base[(n >> 1) * 2 * kLanes + (n & 1)] = c;
        ++n;
    }
    __device__ __forceinline__ void local(uint64_t fl, uint64_t by, uint64_t al, uint64_t fr)
    {
        put(cost_local(x, fl, by));
        const int64_t a = cur + (int64_t)al;
        top = a > top ? a : top;
        cur = a - (int64_t)fr;
        walked += 1;
        nops += x.mult_dev;
    }
    __device__ __forceinline__ void ar_tp(uint64_t by)
    {
        if (x.H <= 1) return;
        put(cost_ar_tp(x, by));
        walked += 1;
        nops += x.mult_tp;
    }
    __device__ __forceinline__ void ar_dp(uint64_t by)
    {
        if (x.D <= 1) return;
        put(cost_ar_dp(x, by));
        walked += 1;
        nops += x.mult_dp;
    }
};

// The repeating unit: one transformer layer; one MLP layer (H = 1) or one
// column/row pair (H > 1), in the block's walk order.  Records with
// accumulation (microbatches >= 1), outside every stage boundary.
template <bool TF>
__device__ void record_unit(const Ctx &x, bool bwd, uint64_t m, double *base, Summary &out)
{
    Record r{x, base, 0, 0, 0, 0, 0};
    if (TF) {
        const TfSz z = tf_sizes(x, m);
        if (bwd) tf_layer_bwd(x, r, z, true);
        else tf_layer_fwd(x, r, z);
    } else if (bwd) {
        if (x.H > 1) {
            mlp_layer_bwd(x, r, m, kRow, false, false, true);
            mlp_layer_bwd(x, r, m, kCol, false, false, true);
        } else {
            mlp_layer_bwd(x, r, m, kPlain, false, false, true);
        }
    } else {
        if (x.H > 1) {
            mlp_layer_fwd(x, r, m, kCol, false);
            mlp_layer_fwd(x, r, m, kRow, false);
        } else {
            mlp_layer_fwd(x, r, m, kPlain, false);
        }
    }
    while (r.n < 2 * PatSize<TF>::B2) r.put(0.0);   // x + 0.0 == x for the clocks
    out.delta = r.cur;
    out.top = r.top;
    out.walked = r.walked;
    out.nops = r.nops;
}

// n repetitions of a unit: clocks by the recorded adds, memory in closed form
template <int N2>
__device__ __forceinline__ void walk_units(Walk &w, const double2 *pp, const Summary &sm, int n)
{
    if (n <= 0) return;
    double2 r[N2];
#pragma unroll
    for (int j = 0; j < N2; ++j) r[j] = pp[j * kLanes];
    double clk = w.clk;
    for (int u = 0; u < n; ++u) {
#pragma unroll
        for (int j = 0; j < N2; ++j) {
            clk = clk + r[j].x;
            clk = clk + r[j].y;
        }
    }
    w.clk = clk;
    // unit u starts at live + u * delta; its highest point is that plus top
    const int64_t hi = w.live + sm.top + (sm.delta > 0 ? (int64_t)(n - 1) * sm.delta : 0);
    w.peak = hi > w.peak ? hi : w.peak;
    w.live += (int64_t)n * sm.delta;
    w.walked += (uint64_t)n * sm.walked;
    w.nops += (uint64_t)n * sm.nops;
}

// ---------------------------------------------------------------------------
// Cross-lane helpers
// ---------------------------------------------------------------------------
// lane i receives lane i-1's value (0 at lane 0) / lane i+1's (0 at lane 63)
__device__ __forceinline__ int shr1(int v) { return __builtin_amdgcn_update_dpp(0, v, 0x138, 0xf, 0xf, true); }
__device__ __forceinline__ int shl1(int v) { return __builtin_amdgcn_update_dpp(0, v, 0x130, 0xf, 0xf, true); }
__device__ __forceinline__ double shr1(double v)
{
    return __hiloint2double(shr1(__double2hiint(v)), shr1(__double2loint(v)));
}
__device__ __forceinline__ double shl1(double v)
{
    return __hiloint2double(shl1(__double2hiint(v)), shl1(__double2loint(v)));
}
__device__ __forceinline__ uint64_t shr1(uint64_t v)
{
    return ((uint64_t)(uint32_t)shr1((int)(v >> 32)) << 32) | (uint32_t)shr1((int)(uint32_t)v);
}
__device__ __forceinline__ uint64_t shl1(uint64_t v)
{
    return ((uint64_t)(uint32_t)shl1((int)(v >> 32)) << 32) | (uint32_t)shl1((int)(uint32_t)v);
}

__device__ __forceinline__ uint64_t ballot(bool b) { return __ballot(b); }

// OR of the W-bit segments of a wave mask, in the low W bits
__device__ __forceinline__ uint64_t fold_segments(uint64_t m, int W)
{
    for (int sh = 32; sh >= W; sh >>= 1) m |= m >> sh;
    return W == 64 ? m : (m & ((1ull << W) - 1));
}

template <class T, class Op>
__device__ __forceinline__ T seg_reduce(T v, int W, Op op)
{
    for (int o = 1; o < W; o <<= 1) v = op(v, __shfl_xor(v, o, kLanes));
    return v;
}

// ---------------------------------------------------------------------------
// The simulation kernel
// ---------------------------------------------------------------------------
template <bool TF>
__global__ __launch_bounds__(kLanes) void k_parametric(const ParArgs g)
{
    constexpr int F2 = PatSize<TF>::F2, B2 = PatSize<TF>::B2;
    __shared__ double2 s_pat[2][kPat2][kLanes];   // [backward][entry pair][lane]

    const int lane = threadIdx.x;
    const uint32_t gl = blockIdx.x * (uint32_t)kLanes;
    if (gl >= g.meta[16 + kClasses]) return;      // beyond the last class (whole wave)
    int cls = 0;
    while (cls + 1 < kClasses && gl >= g.meta[16 + cls + 1]) ++cls;
    const int W = 1 << cls;
    const uint32_t local = gl + lane - g.meta[16 + cls];
    const uint32_t slot = local >> cls;
    const int li = (int)(local & (uint32_t)(W - 1));   // stage of this lane
    const int64_t c = slot < g.meta[cls] ? (int64_t)g.perm[g.meta[8 + cls] + slot] : -1;

    const dsim_model &M = g.m;
    Ctx x = {};
    bool ok = false;
    if (c >= 0) {
        const dsim_strategy st = g.cand[c];
        ok = strategy_ok(M, st.D, st.H, st.P, st.K) && st.P <= g.p_bound && st.P <= W && st.K <= kMaxK;
        if (ok) make_ctx(M, g.c, st, x);
    }
    const int P = ok ? x.P : 0;
    const int s = li;
    bool live_stage = s < P;
    int32_t status = (c >= 0 && !ok) ? DSIM_ST_BAD_STRATEGY : 0;

    Walk w{x, 0.0, 0, 0, 0, 0};
    int pos = 0, nf = 0, nb = 0, len = 0;
    int pat_f = -1, pat_b = -1;   // microbatch size class each pattern was recorded for
    Summary sum_f{}, sum_b{};
    if (live_stage) {
        const int64_t r0 = (int64_t)resident(x, s);
        w.live = r0;
        w.peak = r0;
        len = x.train ? 2 * x.K : x.K;
        // microbatch splits before the pipeline
        if (x.K > 1) {
            if (s == 0) split(x, w);
            if (x.train && s == x.P - 1) split(x, w);
        }
    }
    const uint64_t segmask = W == 64 ? ~0ull : (((1ull << W) - 1) << (lane & ~(W - 1)));

    for (;;) {
        const bool active = live_stage && pos < len;
        const uint64_t act_mask = ballot(active);
        if (act_mask == 0) break;
        const int nf_left = shr1(nf), nb_right = shl1(nb);   // slot-start counters
        bool bwd = false, ready = false;
        int k = 0;
        if (active) {
            block_at(x, s, pos, bwd, k);
            ready = !bwd ? (s == 0 || nf_left > k) : (s == x.P - 1 ? nf > k : nb_right > k);
        }
        const uint64_t rdy_mask = ballot(ready);
        if ((act_mask & segmask) != 0 && (rdy_mask & segmask) == 0) {
            // no stage can proceed: impossible for 1F1B, stops the candidate
            status |= DSIM_ST_BAD_STRATEGY;
            live_stage = false;
        }
        const bool all_fwd = ballot(ready && bwd) == 0;

        if (ready) {
            const int d = bwd ? 1 : 0;
            const uint64_t m = mb_rows(x, k);
            const int mc = (uint64_t)k < x.mr ? 1 : 0;
            double2 *pp = &s_pat[d][0][lane];
            if (bwd && k == 0) {
                block_bwd(x, w, s, k);   // no accumulation: op by op
            } else {
                if ((bwd ? pat_b : pat_f) != mc) {
                    Summary t;
                    record_unit<TF>(x, bwd, m, reinterpret_cast<double *>(pp), t);
                    if (bwd) {
                        sum_b = t;
                        pat_b = mc;
                    } else {
                        sum_f = t;
                        pat_f = mc;
                    }
                }
                const Summary sm = bwd ? sum_b : sum_f;
                const int nl = stage_nl(x, s);
                if (TF) {
                    const TfSz z = tf_sizes(x, m);
                    if (!bwd && s == 0) tf_fwd_first(x, w, z);
                    if (bwd && s == x.P - 1) tf_bwd_last(x, w, z, true);
                    if (all_fwd) walk_units<F2>(w, pp, sm, nl);
                    else walk_units<B2>(w, pp, sm, nl);
                    if (!bwd && s == x.P - 1) tf_fwd_last(x, w, z);
                    if (bwd && s == 0) tf_bwd_first(x, w, z, true);
                } else {
                    const int per = x.H > 1 ? 2 : 1;
                    const int units = nl / per;
                    const int l0 = stage_l0(x, s);
                    if (!bwd) {
                        const bool dead = !x.train && s == x.P - 1;
                        if (all_fwd) walk_units<F2>(w, pp, sm, units - (dead ? 1 : 0));
                        else walk_units<B2>(w, pp, sm, units - (dead ? 1 : 0));
                        if (dead) {
                            for (int i = l0 + nl - per; i < l0 + nl; ++i)
                                mlp_layer_fwd(x, w, m, mlp_kind(x, i), i == x.L - 1);
                        }
                    } else {
                        if (s == x.P - 1) mlp_loss(x, w, m);
                        walk_units<B2>(w, pp, sm, units - 1);
                        for (int i = l0 + per - 1; i >= l0; --i)
                            mlp_layer_bwd(x, w, m, mlp_kind(x, i), i == l0, i == 0, true);
                    }
                }
            }
            ++pos;
            if (bwd) ++nb;
            else ++nf;
        }

        // the slot's sends, ascending by source stage
        int sdir = 0;
        double scost = 0.0;
        uint64_t ssz = 0, sfre = 0;
        if (ready && ((!bwd && s < x.P - 1) || (bwd && s > 0))) {
            sdir = bwd ? -1 : 1;
            send_size(x, s, k, bwd, ssz, sfre);
            scost = cost_send(x, ssz);
        }
        const int l_dir = shr1(sdir), r_dir = shl1(sdir);
        const double l_cost = shr1(scost), r_cost = shl1(scost);
        const uint64_t l_sz = shr1(ssz), r_sz = shl1(ssz);
        const bool from_left = live_stage && s >= 1 && l_dir == 1;
        const bool from_right = live_stage && s + 1 < P && r_dir == -1;
        uint64_t steps = fold_segments(ballot(sdir != 0), W);
        while (steps != 0) {
            const int st = __builtin_ctzll(steps);
            steps &= steps - 1;
            const double cl = shr1(w.clk), cr = shl1(w.clk);
            const bool src = s == st && sdir != 0;
            const bool tl = s == st + 1 && from_left;
            const bool tr = s == st - 1 && from_right;
            const double a = ((src && sdir < 0) || tl) ? cl : cr;
            const double mx = a > w.clk ? a : w.clk;
            const double e = mx + (src ? scost : (tl ? l_cost : r_cost));
            if (src || tl || tr) w.clk = e;
        }
        if (live_stage) {
            if (from_left) {
                w.live += (int64_t)l_sz;
                w.peak = w.live > w.peak ? w.live : w.peak;
            }
            if (sdir != 0) {
                w.live -= (int64_t)sfre;
                w.walked += 1;
                w.nops += x.mult_dev;
            }
            if (from_right) {
                w.live += (int64_t)r_sz;
                w.peak = w.live > w.peak ? w.live : w.peak;
            }
        }
    }
    if (live_stage && x.train && status == 0) weight_update(x, w, s);

    // per-candidate results: reductions over the segment
    const bool contributes = s < P && status == 0;
    const double mk = seg_reduce(contributes ? w.clk : 0.0, W, [](double a, double b) { return a > b ? a : b; });
    const uint64_t cp = seg_reduce(contributes ? (uint64_t)w.peak : 0ull, W,
                                   [](uint64_t a, uint64_t b) { return a > b ? a : b; });
    const uint64_t nops = seg_reduce(contributes ? w.nops : 0ull, W, [](uint64_t a, uint64_t b) { return a + b; });
    const uint64_t walked = seg_reduce(contributes ? w.walked : 0ull, W,
                                       [](uint64_t a, uint64_t b) { return a + b; });
    status = seg_reduce(status, W, [](int32_t a, int32_t b) { return a | b; });
    if (c < 0) return;
    const bool valid = status == 0;
    if (s == 0) {
        int32_t st = status;
        if (valid && g.c.cap != 0 && cp > g.c.cap) st |= DSIM_ST_OVER_CAP;
        g.makespan[c] = valid ? mk : 0.0;
        g.cand_peak[c] = valid ? cp : 0;
        g.status[c] = st;
        if (g.n_ops) g.n_ops[c] = valid ? nops : 0;
        if (g.walked) g.walked[c] = valid ? walked : 0;
    }
    const bool mine = valid && s < P;
    if (g.finish) {
        double *row = g.finish + (size_t)c * g.row_width;
        for (int j = s; j < g.row_width; j += W) row[j] = (mine && j == s) ? w.clk : 0.0;
    }
    if (g.peak) {
        uint64_t *row = g.peak + (size_t)c * g.row_width;
        for (int j = s; j < g.row_width; j += W) row[j] = (mine && j == s) ? (uint64_t)w.peak : 0;
    }
}

// ---------------------------------------------------------------------------
// Pre-pass: stable counting sort of the candidates by segment class
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kScanBlock) void k_class_count(const dsim_strategy *cand, int64_t n, int p_bound,
                                                           uint32_t *counts)
{
    __shared__ uint32_t s_cnt[8];
    if (threadIdx.x < 8) s_cnt[threadIdx.x] = 0;
    __syncthreads();
    const int64_t c = (int64_t)blockIdx.x * kScanBlock + threadIdx.x;
    if (c < n) atomicAdd(&s_cnt[seg_class(cand[c], p_bound)], 1u);
    __syncthreads();
    if (threadIdx.x < 8) counts[(size_t)blockIdx.x * 8 + threadIdx.x] = s_cnt[threadIdx.x];
}

// counts[b][j] -> exclusive prefix over blocks b, per class j; meta as in
// ParArgs.  One block.
__global__ __launch_bounds__(kScanBlock) void k_class_scan(uint32_t *counts, int64_t nb, uint32_t *meta)
{
    __shared__ uint32_t s_v[kScanBlock];
    __shared__ uint32_t s_total[8];
    const int t = threadIdx.x;
    for (int j = 0; j < kClasses; ++j) {
        uint32_t carry = 0;
        for (int64_t b0 = 0; b0 < nb; b0 += kScanBlock) {
            const int64_t b = b0 + t;
            const uint32_t v = b < nb ? counts[(size_t)b * 8 + j] : 0;
            s_v[t] = v;
            __syncthreads();
            for (int o = 1; o < kScanBlock; o <<= 1) {
                const uint32_t add = t >= o ? s_v[t - o] : 0;
                __syncthreads();
                s_v[t] += add;
                __syncthreads();
            }
            if (b < nb) counts[(size_t)b * 8 + j] = carry + s_v[t] - v;
            carry += s_v[kScanBlock - 1];
            __syncthreads();
        }
        if (t == 0) s_total[j] = carry;
        __syncthreads();
    }
    if (t == 0) {
        uint32_t rank = 0, lane = 0;
        for (int j = 0; j < kClasses; ++j) {
            meta[j] = s_total[j];
            meta[8 + j] = rank;
            meta[16 + j] = lane;
            rank += s_total[j];
            lane += ((s_total[j] << j) + kLanes - 1) / kLanes * kLanes;
        }
        meta[kClasses] = 0;
        meta[8 + kClasses] = rank;
        meta[16 + kClasses] = lane;
    }
}

__global__ __launch_bounds__(kScanBlock) void k_class_scatter(const dsim_strategy *cand, int64_t n, int p_bound,
                                                             const uint32_t *offsets, const uint32_t *meta,
                                                             uint32_t *perm)
{
    constexpr int kWaves = kScanBlock / kLanes;
    __shared__ uint32_t s_wcnt[kWaves][8];
    const int t = threadIdx.x, wv = t / kLanes, lane = t % kLanes;
    const int64_t c = (int64_t)blockIdx.x * kScanBlock + t;
    const int j = c < n ? seg_class(cand[c], p_bound) : kClasses;
    const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
    uint32_t rank = 0;
    for (int jj = 0; jj < kClasses; ++jj) {
        const uint64_t b = __ballot(j == jj);
        if (lane == 0) s_wcnt[wv][jj] = (uint32_t)__popcll(b);
        if (j == jj) rank = (uint32_t)__popcll(b & below);
    }
    __syncthreads();
    if (j < kClasses) {
        for (int v = 0; v < wv; ++v) rank += s_wcnt[v][j];
        perm[meta[8 + j] + offsets[(size_t)blockIdx.x * 8 + j] + rank] = (uint32_t)c;
    }
}

}  // namespace

dsim_status launch_parametric(const dsim_model &m, const dsim_strategy *cand, int64_t n_cand, const CostConsts &c,
                              const dsim_results &r, hipStream_t s)
{
    if (n_cand > (int64_t)0x7fffffff)
        return fail(DSIM_ERANGE, "parametric: at most 2^31 - 1 candidates per call");
    ParArgs g;
    g.m = m;
    g.cand = cand;
    g.n_cand = n_cand;
    g.row_width = r.row_width;
    int pb = r.row_width > 0 ? r.row_width : kMaxStages;
    if (pb > kMaxStages) pb = kMaxStages;
    if (pb > m.n_layers) pb = m.n_layers;
    g.p_bound = pb;
    int wmax = 1;
    while (wmax < pb) wmax <<= 1;
    g.makespan = r.makespan;
    g.finish = r.finish;
    g.peak = r.peak;
    g.cand_peak = r.cand_peak;
    g.n_ops = r.n_ops;
    g.walked = r.walked_ops;
    g.status = r.status;
    g.c = c;

    // temporary: per-block class counts, class table, permutation
    const int64_t nb = (n_cand + kScanBlock - 1) / kScanBlock;
    const size_t counts_b = (size_t)nb * 8 * sizeof(uint32_t), meta_b = 32 * sizeof(uint32_t);
    const size_t perm_b = (size_t)n_cand * sizeof(uint32_t);
    void *ws = nullptr;
    hipError_t e = hipMallocAsync(&ws, counts_b + meta_b + perm_b, s);
    if (e != hipSuccess) return hip_fail(e, "parametric: temporary buffer");
    uint32_t *counts = static_cast<uint32_t *>(ws);
    uint32_t *meta = counts + (size_t)nb * 8;
    uint32_t *perm = meta + 32;
    g.perm = perm;
    g.meta = meta;

    hipLaunchKernelGGL(k_class_count, dim3((unsigned)nb), dim3(kScanBlock), 0, s, cand, n_cand, pb, counts);
    hipLaunchKernelGGL(k_class_scan, dim3(1), dim3(kScanBlock), 0, s, counts, nb, meta);
    hipLaunchKernelGGL(k_class_scatter, dim3((unsigned)nb), dim3(kScanBlock), 0, s, cand, n_cand, pb,
                       (const uint32_t *)counts, (const uint32_t *)meta, perm);
    // every class's lanes round up to whole wavefronts: at most one partial
    // wavefront per class beyond n * wmax lanes
    const int64_t waves = (n_cand * wmax + kLanes - 1) / kLanes + kClasses;
    if (m.family == DSIM_MLP)
        hipLaunchKernelGGL(k_parametric<false>, dim3((unsigned)waves), dim3(kLanes), 0, s, g);
    else
        hipLaunchKernelGGL(k_parametric<true>, dim3((unsigned)waves), dim3(kLanes), 0, s, g);
    e = hipGetLastError();
    const hipError_t e2 = hipFreeAsync(ws, s);
    if (e != hipSuccess) return hip_fail(e, "parametric launch");
    if (e2 != hipSuccess) return hip_fail(e2, "parametric: temporary buffer release");
    return DSIM_OK;
}

}  // namespace dsim
