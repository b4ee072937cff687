// parametric.hip -- simulate the D/H/P/K transform without building op lists.
//
// One lane per candidate.  The lane expands, on the fly and in program order,
// the distributed program the transform of Sec. 4 produces (Fig. 2 is its
// P = 2, K = 2 instance) and simulates it with the semantics of Sec. 2.1 and
// the cost model of Sec. 3.3:
//   * pipeline stages hold contiguous layer ranges (L = q*P + r: the first r
//     stages get q + 1 layers) and run synchronous 1F1B: w = min(P-1-s, K)
//     warm-up forwards, then forward/backward pairs, then w backwards;
//   * the global order is slot by slot: every stage, ascending, runs its next
//     block if the block's input was produced in an earlier slot, then the
//     slot's Sends run ascending by source stage; the weight update follows;
//   * every replica (d, h) of a stage runs the same ops at the same times, so
//     the lane walks one replica per stage: a collective over the H ranks or
//     the D replicas starts at the stage's own clock and costs the ring
//     all-reduce of its full group; a Send synchronises two stage clocks.
// Live memory follows def/use liveness of the transform's tensors, written
// here in closed form: every op allocates its outputs, the peak is sampled,
// then the tensors whose last use is this op are freed.
//
// Stage state (clock, live and peak bytes, schedule counters) lives in LDS,
// laid out [stage][lane] with one 64-lane wavefront per workgroup; the
// per-op arithmetic stays in VGPRs.
#include "internal.h"

namespace dsim {
namespace {

constexpr int kLanes = 64;
constexpr int kMaxStages = 64;
constexpr int kMaxK = 16383;
constexpr uint16_t kNoBlock = 0xffffu;

struct ParArgs {
    dsim_model m;
    const dsim_strategy *cand;
    int64_t n_cand;
    int32_t row_width;
    int32_t p_bound;
    double *makespan;
    double *finish;
    uint64_t *peak;
    uint64_t *cand_peak;
    uint64_t *n_ops;
    uint64_t *walked;
    int32_t *status;
    CostConsts c;
};

// Per-candidate constants.
struct Ctx {
    int D, H, P, K, L, q, r;
    bool train, mlp;
    int mode;
    uint64_t e, d, dff, seq, vocab, heads, rows, mq, mr;
    uint64_t dH, FH, Vh, aH;
    double inv_f, inv_b, inv_l, lat, launch;
    double arl_h, arc_h, arl_d, arc_d;
    uint64_t mult_dev, mult_tp, mult_dp;
};

// One stage's running state while a block of its ops is walked.
struct Acc {
    double clk;
    uint64_t live, peak;
};

struct Counters {
    uint64_t walked, nops;
};

__device__ __forceinline__ uint64_t umax(uint64_t a, uint64_t b) { return a > b ? a : b; }

// local compute op on every replica of the stage
__device__ __forceinline__ void op_local(const Ctx &x, Acc &a, Counters &n, uint64_t flops, uint64_t bytes,
                                         uint64_t alloc, uint64_t fre)
{
    const double tf = (double)flops * x.inv_f;
    const double tb = (double)bytes * x.inv_b;
    a.clk = a.clk + (x.launch + (tf > tb ? tf : tb));
    a.live += alloc;
    a.peak = umax(a.peak, a.live);
    a.live -= fre;
    n.walked += 1;
    n.nops += x.mult_dev;
}

// all-reduce over the H ranks of each data replica (in place)
__device__ __forceinline__ void op_ar_tp(const Ctx &x, Acc &a, Counters &n, uint64_t bytes)
{
    if (x.H <= 1) return;
    a.clk = a.clk + (x.arl_h + x.arc_h * ((double)bytes * x.inv_l));
    n.walked += 1;
    n.nops += x.mult_tp;
}

// all-reduce over the D replicas of each tensor rank (in place)
__device__ __forceinline__ void op_ar_dp(const Ctx &x, Acc &a, Counters &n, uint64_t bytes)
{
    if (x.D <= 1) return;
    a.clk = a.clk + (x.arl_d + x.arc_d * ((double)bytes * x.inv_l));
    n.walked += 1;
    n.nops += x.mult_dp;
}

__device__ __forceinline__ uint64_t mb_rows(const Ctx &x, int k)
{
    return x.mq + ((uint64_t)k < x.mr ? 1u : 0u);
}

__device__ __forceinline__ int stage_l0(const Ctx &x, int s) { return s * x.q + (s < x.r ? s : x.r); }
__device__ __forceinline__ int stage_nl(const Ctx &x, int s) { return x.q + (s < x.r ? 1 : 0); }

// ---------------------------------------------------------------------------
// MLP (Fig. 2: @dense = Gemm + Relu): with H > 1 even layers are
// column-parallel (W: d x d/H), odd layers row-parallel (W: d/H x d) with an
// all-reduce of their output; dX of column-parallel layers is all-reduced in
// the backward pass (layer 0's dX is computed and discarded).
// ---------------------------------------------------------------------------
__device__ __forceinline__ void mlp_dims(const Ctx &x, int i, uint64_t &din, uint64_t &dout, bool &row)
{
    const bool col = x.H > 1 && (i & 1) == 0;
    row = x.H > 1 && (i & 1) == 1;
    din = row ? x.d / (uint64_t)x.H : x.d;
    dout = col ? x.d / (uint64_t)x.H : x.d;
}

__device__ void mlp_fwd(const Ctx &x, Acc &a, Counters &n, int s, int k)
{
    const uint64_t m = mb_rows(x, k), e = x.e;
    const int l0 = stage_l0(x, s), l1 = l0 + stage_nl(x, s);
    for (int i = l0; i < l1; ++i) {
        uint64_t din, dout;
        bool row;
        mlp_dims(x, i, din, dout, row);
        // Gemm: the layer input dies here in inference (it is kept for the
        // weight gradient in training)
        op_local(x, a, n, 2 * m * din * dout, e * (m * din + din * dout + m * dout), e * m * dout,
                 x.train ? 0 : e * m * din);
        if (row) op_ar_tp(x, a, n, e * m * dout);
        // Relu frees the pre-activation; the last layer's output has no use
        // in inference
        const bool dead_out = !x.train && i == x.L - 1;
        op_local(x, a, n, m * dout, 2 * e * m * dout, e * m * dout, e * m * dout + (dead_out ? e * m * dout : 0));
    }
}

__device__ void mlp_bwd(const Ctx &x, Acc &a, Counters &n, int s, int k)
{
    const uint64_t m = mb_rows(x, k), e = x.e;
    const int l0 = stage_l0(x, s), l1 = l0 + stage_nl(x, s);
    if (s == x.P - 1) op_local(x, a, n, 3 * m * x.d, 3 * e * m * x.d, e * m * x.d, e * m * x.d);   // loss grad, y_k dies
    for (int i = l1 - 1; i >= l0; --i) {
        uint64_t din, dout;
        bool row;
        mlp_dims(x, i, din, dout, row);
        // ReluGrad(da, a): both die
        op_local(x, a, n, m * dout, 3 * e * m * dout, e * m * dout, 2 * e * m * dout);
        // weight gradient; the stage's input dies at its first layer
        op_local(x, a, n, 2 * m * din * dout, e * (m * din + m * dout + din * dout), e * din * dout,
                 i == l0 ? e * m * din : 0);
        if (k >= 1) op_local(x, a, n, din * dout, 3 * e * din * dout, 0, e * din * dout);   // accumulate
        // input gradient; dh dies; layer 0's dX has no use
        op_local(x, a, n, 2 * m * din * dout, e * (m * dout + din * dout + m * din), e * m * din,
                 e * m * dout + (i == 0 ? e * m * din : 0));
        if (!row && x.H > 1 && i != 0) op_ar_tp(x, a, n, e * m * din);
    }
}

// bytes of the activation a stage sends forward / backward
__device__ __forceinline__ uint64_t mlp_act_out(const Ctx &x, int s, int k)
{
    uint64_t din, dout;
    bool row;
    mlp_dims(x, stage_l0(x, s) + stage_nl(x, s) - 1, din, dout, row);
    return x.e * mb_rows(x, k) * dout;
}

__device__ __forceinline__ uint64_t mlp_grad_out(const Ctx &x, int s, int k)
{
    uint64_t din, dout;
    bool row;
    mlp_dims(x, stage_l0(x, s), din, dout, row);
    return x.e * mb_rows(x, k) * din;
}

// ---------------------------------------------------------------------------
// Transformer (GPT-2-shaped decoder, Megatron tensor parallelism: QKV and
// fc1 column-parallel, out-proj and fc2 row-parallel with an all-reduce of
// their output; vocabulary-parallel embedding and LM head, ceil(V/H) rows per
// rank).
// ---------------------------------------------------------------------------
struct TfSz {
    uint64_t m, T, ACT, QKV, OH, S2, FF, LOG, ST, IDS;
};

__device__ __forceinline__ TfSz tf_sizes(const Ctx &x, int k)
{
    TfSz z;
    z.m = mb_rows(x, k);
    z.T = z.m * x.seq;
    z.ACT = x.e * z.T * x.d;
    z.QKV = x.e * z.T * 3 * x.dH;
    z.OH = x.e * z.T * x.dH;
    z.S2 = x.e * z.m * x.aH * x.seq * x.seq;
    z.FF = x.e * z.T * x.FH;
    z.LOG = x.e * z.T * x.Vh;
    z.ST = 12 * z.T;
    z.IDS = 4 * z.T;
    return z;
}

__device__ void tf_fwd(const Ctx &x, Acc &a, Counters &n, int s, int k)
{
    const TfSz z = tf_sizes(x, k);
    const uint64_t T = z.T, d = x.d, dH = x.dH, FH = x.FH, e = x.e, S = x.seq;
    const bool tr = x.train;
    if (s == 0) {
        op_local(x, a, n, T * d, 2 * z.ACT + z.IDS, z.ACT, tr ? 0 : z.IDS);   // embedding; ids die in inference
        op_ar_tp(x, a, n, z.ACT);
    }
    const int nl = stage_nl(x, s);
    for (int i = 0; i < nl; ++i) {
        op_local(x, a, n, 8 * T * d, 2 * z.ACT, z.ACT, 0);                                               // LN1
        op_local(x, a, n, 2 * T * d * 3 * dH, e * (T * d + d * 3 * dH + T * 3 * dH), z.QKV, tr ? 0 : z.ACT);  // QKV
        op_local(x, a, n, 2 * T * S * dH, 2 * z.OH + z.S2, z.S2, 0);                                     // scores
        op_local(x, a, n, 5 * z.m * x.aH * S * S, 2 * z.S2, z.S2, z.S2);                                 // softmax
        op_local(x, a, n, 2 * T * S * dH, z.S2 + 2 * z.OH, z.OH, tr ? 0 : z.S2 + z.QKV);                // P.V
        op_local(x, a, n, 2 * T * dH * d, e * (T * dH + dH * d + T * d), z.ACT, tr ? 0 : z.OH);          // out-proj
        op_ar_tp(x, a, n, z.ACT);
        op_local(x, a, n, T * d, 3 * z.ACT, z.ACT, tr ? z.ACT : 2 * z.ACT);                             // residual
        op_local(x, a, n, 8 * T * d, 2 * z.ACT, z.ACT, 0);                                               // LN2
        op_local(x, a, n, 2 * T * d * FH, e * (T * d + d * FH + T * FH), z.FF, tr ? 0 : z.ACT);          // fc1
        op_local(x, a, n, 8 * T * FH, 2 * z.FF, z.FF, tr ? 0 : z.FF);                                   // GeLU
        op_local(x, a, n, 2 * T * FH * d, e * (T * FH + FH * d + T * d), z.ACT, tr ? 0 : z.FF);          // fc2
        op_ar_tp(x, a, n, z.ACT);
        op_local(x, a, n, T * d, 3 * z.ACT, z.ACT, tr ? z.ACT : 2 * z.ACT);                             // residual
    }
    if (s == x.P - 1) {
        op_local(x, a, n, 8 * T * d, 2 * z.ACT, z.ACT, tr ? 0 : z.ACT);                                  // final LN
        op_local(x, a, n, 2 * T * d * x.Vh, e * (T * d + d * x.Vh + T * x.Vh), z.LOG,
                 tr ? 0 : z.ACT + z.LOG);                                                                // LM head
    }
}

__device__ void tf_bwd(const Ctx &x, Acc &a, Counters &n, int s, int k)
{
    const TfSz z = tf_sizes(x, k);
    const uint64_t T = z.T, d = x.d, dH = x.dH, FH = x.FH, e = x.e, S = x.seq, Vh = x.Vh;
    const bool acc = k >= 1;
    if (s == x.P - 1) {
        op_local(x, a, n, 3 * T * Vh, z.LOG + z.ST, z.ST, 0);                                 // loss statistics
        op_ar_tp(x, a, n, z.ST);
        op_local(x, a, n, 2 * T * Vh, 2 * z.LOG + z.ST + z.IDS, z.LOG, z.LOG + z.ST + z.IDS); // dlogits
        op_local(x, a, n, 2 * T * d * Vh, e * (T * Vh + d * Vh + T * d), z.ACT, 0);           // LM head dX
        op_ar_tp(x, a, n, z.ACT);
        op_local(x, a, n, 2 * T * d * Vh, e * (T * d + T * Vh + d * Vh), e * d * Vh, z.ACT + z.LOG);  // LM head dW
        if (acc) op_local(x, a, n, d * Vh, 3 * e * d * Vh, 0, e * d * Vh);
        op_local(x, a, n, 8 * T * d, 3 * z.ACT, z.ACT, 2 * z.ACT);                           // final LN grad
    }
    const int nl = stage_nl(x, s);
    for (int i = 0; i < nl; ++i) {
        op_local(x, a, n, 2 * T * FH * d, e * (T * d + FH * d + T * FH), z.FF, 0);            // fc2 dX
        op_local(x, a, n, 2 * T * FH * d, e * (T * FH + T * d + FH * d), e * FH * d, z.FF);   // fc2 dW
        if (acc) op_local(x, a, n, FH * d, 3 * e * FH * d, 0, e * FH * d);
        op_local(x, a, n, 8 * T * FH, 3 * z.FF, z.FF, 2 * z.FF);                              // GeLU grad
        op_local(x, a, n, 2 * T * d * FH, e * (T * FH + d * FH + T * d), z.ACT, 0);           // fc1 dX
        op_ar_tp(x, a, n, z.ACT);
        op_local(x, a, n, 2 * T * d * FH, e * (T * d + T * FH + d * FH), e * d * FH, z.ACT + z.FF);  // fc1 dW
        if (acc) op_local(x, a, n, d * FH, 3 * e * d * FH, 0, e * d * FH);
        op_local(x, a, n, 8 * T * d, 3 * z.ACT, z.ACT, 2 * z.ACT);                            // LN2 grad
        op_local(x, a, n, T * d, 3 * z.ACT, z.ACT, 2 * z.ACT);                                // residual merge
        op_local(x, a, n, 2 * T * dH * d, e * (T * d + dH * d + T * dH), z.OH, 0);            // out-proj dX
        op_local(x, a, n, 2 * T * dH * d, e * (T * dH + T * d + dH * d), e * dH * d, z.OH);   // out-proj dW
        if (acc) op_local(x, a, n, dH * d, 3 * e * dH * d, 0, e * dH * d);
        op_local(x, a, n, 4 * T * S * dH, 2 * z.S2 + 3 * z.OH, z.S2 + z.QKV, z.OH);           // P.V grads
        op_local(x, a, n, 5 * z.m * x.aH * S * S, 3 * z.S2, z.S2, 2 * z.S2);                  // softmax grad
        op_local(x, a, n, 4 * T * S * dH, z.S2 + 4 * z.OH, 0, z.S2 + z.QKV);                  // Q.K^T grads
        op_local(x, a, n, 2 * T * 3 * dH * d, e * (T * 3 * dH + 3 * dH * d + T * d), z.ACT, 0);  // QKV dX
        op_ar_tp(x, a, n, z.ACT);
        op_local(x, a, n, 2 * T * d * 3 * dH, e * (T * d + T * 3 * dH + d * 3 * dH), e * d * 3 * dH,
                 z.ACT + z.QKV);                                                               // QKV dW
        if (acc) op_local(x, a, n, d * 3 * dH, 3 * e * d * 3 * dH, 0, e * d * 3 * dH);
        op_local(x, a, n, 8 * T * d, 3 * z.ACT, z.ACT, 2 * z.ACT);                            // LN1 grad
        op_local(x, a, n, T * d, 3 * z.ACT, z.ACT, 2 * z.ACT);                                // residual merge
    }
    if (s == 0) {
        op_local(x, a, n, T * d, z.ACT + z.IDS + e * Vh * d, e * Vh * d, z.ACT + z.IDS);      // embedding dW
        if (acc) op_local(x, a, n, Vh * d, 3 * e * Vh * d, 0, e * Vh * d);
    }
}

// ---------------------------------------------------------------------------
// Optimizer, inputs, splits and the weight update
// ---------------------------------------------------------------------------
__device__ __forceinline__ void opt_cost(const Ctx &x, uint64_t N, uint64_t &flops, uint64_t &bytes)
{
    if (x.mode == DSIM_TRAIN_SGD) {
        flops = 2 * N;
        bytes = 3 * x.e * N;
    } else if (x.mode == DSIM_TRAIN_ADAM) {
        flops = 12 * N;
        bytes = 7 * x.e * N;
    } else {
        flops = 12 * N;
        bytes = 28 * N;
    }
}

__device__ __forceinline__ uint64_t opt_state(const Ctx &x, uint64_t N)
{
    if (!x.train) return 0;
    if (x.mode == DSIM_TRAIN_ADAM) return 2 * x.e * N;
    if (x.mode == DSIM_TRAIN_ADAM_MIXED) return 12 * N;
    return 0;
}

__device__ __forceinline__ void wu_param(const Ctx &x, Acc &a, Counters &n, uint64_t N)
{
    op_ar_dp(x, a, n, x.e * N);
    uint64_t fl, by;
    opt_cost(x, N, fl, by);
    op_local(x, a, n, fl, by, 0, x.e * N);   // the gradient dies
}

__device__ void weight_update(const Ctx &x, Acc &a, Counters &n, int s)
{
    const int l0 = stage_l0(x, s), nl = stage_nl(x, s);
    if (x.mlp) {
        for (int i = l0; i < l0 + nl; ++i) {
            uint64_t din, dout;
            bool row;
            mlp_dims(x, i, din, dout, row);
            wu_param(x, a, n, din * dout);
        }
        return;
    }
    const uint64_t d = x.d;
    if (s == 0) wu_param(x, a, n, x.Vh * d);
    for (int i = 0; i < nl; ++i) {
        wu_param(x, a, n, d * 3 * x.dH);
        wu_param(x, a, n, x.dH * d);
        wu_param(x, a, n, d * x.FH);
        wu_param(x, a, n, x.FH * d);
    }
    if (s == x.P - 1) wu_param(x, a, n, d * x.Vh);
}

// bytes of one row (sequence) of the stage-0 input / last-stage target
__device__ __forceinline__ uint64_t input_row(const Ctx &x) { return x.mlp ? x.e * x.d : 4 * x.seq; }

__device__ uint64_t resident(const Ctx &x, int s)
{
    const int l0 = stage_l0(x, s), nl = stage_nl(x, s);
    uint64_t N = 0;
    if (x.mlp) {
        for (int i = l0; i < l0 + nl; ++i) {
            uint64_t din, dout;
            bool row;
            mlp_dims(x, i, din, dout, row);
            N += din * dout;
        }
    } else {
        N = (uint64_t)nl * (x.d * 3 * x.dH + x.dH * x.d + x.d * x.FH + x.FH * x.d);
        if (s == 0) N += x.Vh * x.d;
        if (s == x.P - 1) N += x.d * x.Vh;
    }
    uint64_t b = x.e * N + opt_state(x, N);
    if (s == 0) b += input_row(x) * x.rows;
    if (s == x.P - 1 && x.train) b += input_row(x) * x.rows;
    return b;
}

__device__ __forceinline__ void split(const Ctx &x, Acc &a, Counters &n)
{
    const uint64_t whole = input_row(x) * x.rows;
    op_local(x, a, n, 0, 2 * whole, whole, whole);
}

// ---------------------------------------------------------------------------
// The kernel
// ---------------------------------------------------------------------------
__device__ bool strategy_ok(const dsim_model &m, int D, int H, int P, int K)
{
    if (D < 1 || H < 1 || P < 1 || K < 1) return false;
    const int64_t B = m.global_batch;
    if (B % D != 0 || (int64_t)K > B / D || P > m.n_layers) return false;
    if (m.family == DSIM_MLP) {
        if (m.d_model % H != 0) return false;
        if (H > 1) {
            const int q = m.n_layers / P, r = m.n_layers % P;
            if ((q & 1) != 0 && r < P) return false;          // stages with q layers
            if (r > 0 && ((q + 1) & 1) != 0) return false;    // stages with q + 1 layers
        }
        return true;
    }
    return m.n_heads % H == 0 && m.d_model % H == 0 && m.d_ff % H == 0;
}

// position `pos` of stage s's block sequence -> (is_backward, microbatch)
__device__ __forceinline__ void block_at(const Ctx &x, int s, int pos, bool &bwd, int &k)
{
    if (!x.train) {
        bwd = false;
        k = pos;
        return;
    }
    const int w = (x.P - 1 - s) < x.K ? (x.P - 1 - s) : x.K;
    if (pos < w) {
        bwd = false;
        k = pos;
    } else if (pos < w + 2 * (x.K - w)) {
        const int j = pos - w;
        bwd = (j & 1) != 0;
        k = bwd ? (j - 1) / 2 : w + j / 2;
    } else {
        bwd = true;
        k = pos - w - (x.K - w);
    }
}

__global__ __launch_bounds__(kLanes) void k_parametric(const ParArgs g)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int lane = threadIdx.x;
    const int PB = g.p_bound;
    double *s_clk = reinterpret_cast<double *>(smem);
    uint64_t *s_live = reinterpret_cast<uint64_t *>(s_clk + PB * kLanes);
    uint64_t *s_peak = s_live + PB * kLanes;
    uint16_t *s_pos = reinterpret_cast<uint16_t *>(s_peak + PB * kLanes);
    uint16_t *s_nf = s_pos + PB * kLanes;
    uint16_t *s_nb = s_nf + PB * kLanes;
    uint16_t *s_em = s_nb + PB * kLanes;
#define AT(s) ((s) * kLanes + lane)

    const int64_t c = (int64_t)blockIdx.x * kLanes + lane;
    if (c >= g.n_cand) return;
    const dsim_strategy st = g.cand[c];
    const dsim_model &M = g.m;
    int32_t status = 0;
    const bool ok = strategy_ok(M, st.D, st.H, st.P, st.K) && st.P <= PB && st.K <= kMaxK;

    Ctx x;
    x.D = st.D; x.H = st.H; x.P = st.P; x.K = st.K;
    x.L = M.n_layers;
    x.mlp = M.family == DSIM_MLP;
    x.mode = M.mode;
    x.train = M.mode != DSIM_INFER;
    double mk = 0.0;
    uint64_t cp = 0;
    Counters n{0, 0};
    if (!ok) {
        status = DSIM_ST_BAD_STRATEGY;
    } else {
        x.q = x.L / x.P;
        x.r = x.L % x.P;
        x.e = (uint64_t)M.elem_bytes;
        x.d = (uint64_t)M.d_model;
        x.dff = (uint64_t)M.d_ff;
        x.seq = (uint64_t)M.seq_len;
        x.vocab = (uint64_t)M.vocab;
        x.heads = (uint64_t)M.n_heads;
        x.rows = (uint64_t)M.global_batch / (uint64_t)x.D;
        x.mq = x.rows / (uint64_t)x.K;
        x.mr = x.rows % (uint64_t)x.K;
        x.dH = x.d / (uint64_t)x.H;
        x.FH = x.mlp ? 0 : x.dff / (uint64_t)x.H;
        x.Vh = x.mlp ? 0 : (x.vocab + (uint64_t)x.H - 1) / (uint64_t)x.H;
        x.aH = x.mlp ? 0 : x.heads / (uint64_t)x.H;
        x.inv_f = g.c.inv_f;
        x.inv_b = g.c.inv_b;
        x.inv_l = g.c.inv_l;
        x.lat = g.c.lat;
        x.launch = g.c.launch;
        {
            const double ah = 2.0 * (double)(x.H - 1), ad = 2.0 * (double)(x.D - 1);
            x.arl_h = ah * x.lat;
            x.arc_h = ah / (double)x.H;
            x.arl_d = ad * x.lat;
            x.arc_d = ad / (double)x.D;
        }
        x.mult_dev = (uint64_t)x.D * (uint64_t)x.H;
        x.mult_tp = (uint64_t)x.D;
        x.mult_dp = (uint64_t)x.H;

        for (int s = 0; s < x.P; ++s) {
            const uint64_t r0 = resident(x, s);
            s_clk[AT(s)] = 0.0;
            s_live[AT(s)] = r0;
            s_peak[AT(s)] = r0;
            s_pos[AT(s)] = 0;
            s_nf[AT(s)] = 0;
            s_nb[AT(s)] = 0;
        }
        // microbatch splits before the pipeline
        if (x.K > 1) {
            Acc a{s_clk[AT(0)], s_live[AT(0)], s_peak[AT(0)]};
            split(x, a, n);
            s_clk[AT(0)] = a.clk; s_live[AT(0)] = a.live; s_peak[AT(0)] = a.peak;
            if (x.train) {
                const int t = x.P - 1;
                Acc b{s_clk[AT(t)], s_live[AT(t)], s_peak[AT(t)]};
                split(x, b, n);
                s_clk[AT(t)] = b.clk; s_live[AT(t)] = b.live; s_peak[AT(t)] = b.peak;
            }
        }
        const int len = x.train ? 2 * x.K : x.K;
        // slots
        for (;;) {
            bool left = false, any = false;
            uint16_t prev_nf0 = 0;
            for (int s = 0; s < x.P; ++s) {
                uint16_t pos = s_pos[AT(s)], nf = s_nf[AT(s)], nb = s_nb[AT(s)];
                const uint16_t nf0 = nf;
                uint16_t em = kNoBlock;
                if (pos < len) {
                    left = true;
                    bool bwd;
                    int k;
                    block_at(x, s, pos, bwd, k);
                    bool ready;
                    if (!bwd) ready = s == 0 || prev_nf0 > k;
                    else ready = (s == x.P - 1) ? nf0 > k : s_nb[AT(s + 1)] > k;
                    if (ready) {
                        Acc a{s_clk[AT(s)], s_live[AT(s)], s_peak[AT(s)]};
                        if (x.mlp) {
                            if (bwd) mlp_bwd(x, a, n, s, k);
                            else mlp_fwd(x, a, n, s, k);
                        } else {
                            if (bwd) tf_bwd(x, a, n, s, k);
                            else tf_fwd(x, a, n, s, k);
                        }
                        s_clk[AT(s)] = a.clk; s_live[AT(s)] = a.live; s_peak[AT(s)] = a.peak;
                        ++pos;
                        if (bwd) ++nb;
                        else ++nf;
                        em = (uint16_t)((k << 1) | (bwd ? 1 : 0));
                        any = true;
                    }
                }
                s_pos[AT(s)] = pos;
                s_nf[AT(s)] = nf;
                s_nb[AT(s)] = nb;
                s_em[AT(s)] = em;
                prev_nf0 = nf0;
            }
            if (!left) break;
            if (!any) {   // cannot happen for 1F1B; guarantees termination
                status |= DSIM_ST_BAD_STRATEGY;
                break;
            }
            // the slot's sends, ascending by source stage
            for (int s = 0; s < x.P; ++s) {
                const uint16_t em = s_em[AT(s)];
                if (em == kNoBlock) continue;
                const bool bwd = em & 1;
                const int k = em >> 1;
                if (!bwd && s == x.P - 1) continue;
                if (bwd && s == 0) continue;
                const int t = bwd ? s - 1 : s + 1;
                uint64_t sz, fre;
                if (x.mlp) {
                    sz = bwd ? mlp_grad_out(x, s, k) : mlp_act_out(x, s, k);
                    fre = (bwd || !x.train) ? sz : 0;
                } else {
                    sz = x.e * mb_rows(x, k) * x.seq * x.d;
                    fre = sz;
                }
                const double c0 = s_clk[AT(s)], c1 = s_clk[AT(t)];
                double start = 0.0;
                start = c0 > start ? c0 : start;
                start = c1 > start ? c1 : start;
                const double end = start + (x.lat + (double)sz * x.inv_l);
                s_clk[AT(s)] = end;
                s_clk[AT(t)] = end;
                const uint64_t lt = s_live[AT(t)] + sz;
                s_live[AT(t)] = lt;
                s_peak[AT(t)] = umax(s_peak[AT(t)], lt);
                s_live[AT(s)] -= fre;
                n.walked += 1;
                n.nops += x.mult_dev;
            }
        }
        if (x.train) {
            for (int s = 0; s < x.P; ++s) {
                Acc a{s_clk[AT(s)], s_live[AT(s)], s_peak[AT(s)]};
                weight_update(x, a, n, s);
                s_clk[AT(s)] = a.clk; s_live[AT(s)] = a.live; s_peak[AT(s)] = a.peak;
            }
        }
        for (int s = 0; s < x.P; ++s) {
            const double cl = s_clk[AT(s)];
            const uint64_t pk = s_peak[AT(s)];
            mk = cl > mk ? cl : mk;
            cp = umax(cp, pk);
        }
        if (g.c.cap != 0 && cp > g.c.cap) status |= DSIM_ST_OVER_CAP;
    }
    g.makespan[c] = mk;
    g.cand_peak[c] = cp;
    g.status[c] = status;
    if (g.n_ops) g.n_ops[c] = n.nops;
    if (g.walked) g.walked[c] = n.walked;
    const int P = ok ? x.P : 0;
    if (g.finish) {
        double *row = g.finish + (size_t)c * g.row_width;
        for (int s = 0; s < g.row_width; ++s) row[s] = s < P ? s_clk[AT(s)] : 0.0;
    }
    if (g.peak) {
        uint64_t *row = g.peak + (size_t)c * g.row_width;
        for (int s = 0; s < g.row_width; ++s) row[s] = s < P ? s_peak[AT(s)] : 0;
    }
#undef AT
}

}  // namespace

dsim_status launch_parametric(const dsim_model &m, const dsim_strategy *cand, int64_t n_cand, const CostConsts &c,
                              const dsim_results &r, hipStream_t s)
{
    ParArgs g;
    g.m = m;
    g.cand = cand;
    g.n_cand = n_cand;
    g.row_width = r.row_width;
    int pb = r.row_width > 0 ? r.row_width : kMaxStages;
    if (pb > kMaxStages) pb = kMaxStages;
    if (pb > m.n_layers) pb = m.n_layers;
    g.p_bound = pb;
    g.makespan = r.makespan;
    g.finish = r.finish;
    g.peak = r.peak;
    g.cand_peak = r.cand_peak;
    g.n_ops = r.n_ops;
    g.walked = r.walked_ops;
    g.status = r.status;
    g.c = c;
    const size_t lds = (size_t)pb * kLanes * (3 * sizeof(uint64_t) + 4 * sizeof(uint16_t));
    int dev = 0, lds_max = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
    if (e != hipSuccess) return hip_fail(e, "parametric: device query");
    if (lds > (size_t)lds_max)
        return fail(DSIM_ERANGE, "parametric: %d pipeline stages need %zu bytes of LDS, the device allows %d "
                    "(lower results.row_width)", pb, lds, lds_max);
    if (lds > 65536) {
        e = hipFuncSetAttribute(reinterpret_cast<const void *>(k_parametric),
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return hip_fail(e, "parametric: LDS attribute");
    }
    const int64_t blocks = (n_cand + kLanes - 1) / kLanes;
    hipLaunchKernelGGL(k_parametric, dim3((unsigned)blocks), dim3(kLanes), lds, s, g);
    e = hipGetLastError();
    return e == hipSuccess ? DSIM_OK : hip_fail(e, "parametric launch");
}

}  // namespace dsim
