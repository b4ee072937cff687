// model.h -- the ops of the D/H/P/K transform, written once for every
// consumer in the library.
//
// The transform of Sec. 4 (Fig. 2 is its P = 2, K = 2 instance) turns a model
// and a strategy into one straight-line distributed program.  The functions
// here produce that program's ops for one pipeline stage, in program order,
// and hand each to a sink:
//
//   o.local(flops, bytes, alloc, free)  compute op on every replica of the
//                                        stage: allocate `alloc` bytes of
//                                        outputs, then free `free` bytes of
//                                        tensors whose last use this is
//   o.mm(flops, bytes, alloc, free, k) the same for a matrix multiplication
//                                        of reduction length k (the empirical
//                                        MatMul cost applies)
//   o.ar_tp(bytes)                       all-reduce over the H ranks of each
//                                        data replica (emitted only if H > 1)
//   o.ar_dp(bytes)                       all-reduce over the D replicas of
//                                        each tensor rank (only if D > 1)
//   o.bcast(bytes, grp)                  ZeRO: the owner of parameter group
//                                        grp broadcasts a weight of `bytes`
//                                        over the D replicas of each tensor
//                                        rank; the next o.local is the op that
//                                        reads it, after which the other
//                                        replicas' copies die
//   o.reduce(bytes, grp)                 ZeRO: every replica's gradient of
//                                        group grp is reduced onto the owner
//                                        (which allocates the reduced tensor;
//                                        the gradients die there)
//   o.owner_local(fl, by, al, fr, grp)   ZeRO: compute op on the owner of
//                                        group grp only (its optimizer step)
//   o.handover(bytes)                    overlap: the last microbatch has
//                                        finished a weight gradient of
//                                        `bytes`; every replica hands it to
//                                        its GPU's communication stream (a
//                                        Send between the GPU's two streams,
//                                        allocating nothing), whose D
//                                        replicas then all-reduce it there
//   o.handback(bytes)                    overlap: the reduced gradient comes
//                                        back to the computation stream
//                                        (again a Send allocating nothing)
//
// Sinks: the parametric simulator (one replica per stage), the per-layer
// cost recorder and the table materialiser.  Memory follows def/use
// liveness, in closed form per op: outputs are allocated, the peak is
// sampled, then tensors at their last use are freed (a value with no use is
// freed by the op that defines it).
#pragma once

#include "internal.h"

namespace dsim {

constexpr int kMaxStages = 64;

// Per-candidate constants.
struct Ctx {
    int D, H, P, K, L, q, r;
    bool train, mlp;
    int mode;
    int schedule;   // DSIM_SCHED_1F1B or DSIM_SCHED_GPIPE
    bool rc;        // activation recomputation (training only)
    bool zero;      // ZeRO partitioning (training only, D > 1)
    bool ov;        // gradient all-reduce on the communication streams (training only, D > 1)
    uint64_t e, d, dff, seq, vocab, heads, rows, mq, mr;
    uint64_t dH, FH, Vh, aH, hd;   // hd: one attention head's width
    double inv_f, inv_b, inv_l, lat, launch;
    double inv_l_h, inv_l_d;   // 1 / bandwidth of the tensor- / data-parallel groups' link
    double lat_d;              // latency of the data-parallel groups' link
    double arl_h, arc_h, arl_d, arc_d;
    double chl_d;   // (D - 1) * lat: latency part of a broadcast / reduce over the D replicas
    bool mm;        // matrix multiplications take the regression
                    // max(mmf, ((mm0 + mm1 * flops) + mm2 * bytes) + mm3 * k)
    double mm0, mm1, mm2, mm3, mmf;
    double st_lat, st_inv_l;   // a Send between the two streams of one GPU
    uint64_t mult_dev, mult_tp, mult_dp;
};

// Preconditions of the transform (evenly divisible batch, heads and hidden
// sizes; K <= rows per replica; P <= layers; with H > 1 every MLP stage holds
// whole column/row layer pairs).
__device__ inline bool strategy_ok(const dsim_model &m, int D, int H, int P, int K)
{
    if (D < 1 || H < 1 || P < 1 || K < 1) return false;
    if ((int64_t)D * H * P > kMaxDevices) return false;
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

// M: the model (dsim_model, in any address space); c: the device constants
template <class MM, class CC>
__device__ inline void make_ctx(const MM &M, const CC &c, const dsim_strategy &st, Ctx &x)
{
    x.D = st.D;
    x.H = st.H;
    x.P = st.P;
    x.K = st.K;
    x.L = M.n_layers;
    x.mlp = M.family == DSIM_MLP;
    x.mode = M.mode;
    x.schedule = M.schedule;
    x.train = M.mode != DSIM_INFER;
    x.rc = x.train && M.recompute != 0;
    x.zero = x.train && M.zero != 0 && x.D > 1;
    x.ov = x.train && M.overlap != 0 && x.D > 1;
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
    x.hd = x.mlp ? 0 : x.d / x.heads;
    x.inv_f = c.inv_f;
    x.inv_b = c.inv_b;
    x.inv_l = c.inv_l;
    x.lat = c.lat;
    x.launch = c.launch;
    // with nodes (placement uniform, see placement_ok) a tensor-parallel
    // group leaves its node iff H > node size, a data-parallel group iff its
    // stage's D*H devices do and D > 1
    const bool net_h = c.node > 0 && x.H > c.node;
    const bool net_d = c.node > 0 && x.D > 1 && x.D * x.H > c.node;
    const double lat_h = net_h ? c.net_lat : c.lat;
    x.lat_d = net_d ? c.net_lat : c.lat;
    x.inv_l_h = net_h ? c.net_inv_l : c.inv_l;
    x.inv_l_d = net_d ? c.net_inv_l : c.inv_l;
    const double ah = 2.0 * (double)(x.H - 1), ad = 2.0 * (double)(x.D - 1);
    x.arl_h = ah * lat_h;
    x.arc_h = ah / (double)x.H;
    x.arl_d = ad * x.lat_d;
    x.arc_d = ad / (double)x.D;
    x.chl_d = (double)(x.D - 1) * x.lat_d;
    x.mm = c.mm != 0;
    x.mm0 = c.mm_c0;
    x.mm1 = c.mm_c1;
    x.mm2 = c.mm_c2;
    x.mm3 = c.mm_c3;
    x.mmf = c.mm_floor;
    x.st_lat = c.st_lat;
    x.st_inv_l = c.st_inv_l;
    x.mult_dev = (uint64_t)x.D * (uint64_t)x.H;
    x.mult_tp = (uint64_t)x.D;
    x.mult_dp = (uint64_t)x.H;
}

// Op costs (Sec. 3.3 roofline form, ring all-reduce of the whole group).
__device__ __forceinline__ double cost_local(const Ctx &x, uint64_t flops, uint64_t bytes)
{
    const double tf = (double)flops * x.inv_f;
    const double tb = (double)bytes * x.inv_b;
    return x.launch + (tf > tb ? tf : tb);
}
__device__ __forceinline__ double cost_ar_tp(const Ctx &x, uint64_t bytes)
{
    return x.arl_h + x.arc_h * ((double)bytes * x.inv_l_h);
}
__device__ __forceinline__ double cost_ar_dp(const Ctx &x, uint64_t bytes)
{
    return x.arl_d + x.arc_d * ((double)bytes * x.inv_l_d);
}
__device__ __forceinline__ double cost_send(const Ctx &x, uint64_t bytes)
{
    return x.lat + (double)bytes * x.inv_l;
}
// a matrix multiplication of reduction length k: the empirical regression of
// Sec. 4 when the device model carries one, the roofline otherwise
__device__ __forceinline__ double cost_mm(const Ctx &x, uint64_t flops, uint64_t bytes, uint64_t k)
{
    if (!x.mm) return cost_local(x, flops, bytes);
    const double c = ((x.mm0 + x.mm1 * (double)flops) + x.mm2 * (double)bytes) + x.mm3 * (double)k;
    return x.mmf > c ? x.mmf : c;
}
// a Send between the two streams of one GPU (overlap)
__device__ __forceinline__ double cost_stream(const Ctx &x, uint64_t bytes)
{
    return x.st_lat + (double)bytes * x.st_inv_l;
}
// broadcast / reduce over the D replicas (ZeRO, Fig. 9): a pipelined chain,
// D - 1 link latencies plus the bytes crossing one link once
__device__ __forceinline__ double cost_chain_d(const Ctx &x, uint64_t bytes)
{
    return x.chl_d + (double)bytes * x.inv_l_d;
}

// Nodes of `node` devices must cut every tensor-parallel group, data-parallel
// group and stage alike: node and D*H, and node and H, divide one another.
__device__ __forceinline__ bool placement_ok(int node, int D, int H)
{
    if (node <= 0) return true;
    const int DH = D * H;
    return (node % DH == 0 || DH % node == 0) && (node % H == 0 || H % node == 0);
}

// whether the Sends between stage s and stage t (= s +- 1) cross nodes:
// replica r of stage s is device s*D*H + r, and uniform placement makes the
// answer the same for every r
__device__ __forceinline__ bool send_spans(int node, int D, int H, int s, int t)
{
    if (node <= 0) return false;
    const int DH = D * H;
    return (s * DH) / node != (t * DH) / node;
}

// Uneven microbatches: the first rows % K get one extra row.
__device__ __forceinline__ uint64_t mb_rows(const Ctx &x, int k)
{
    return x.mq + ((uint64_t)k < x.mr ? 1u : 0u);
}

// Contiguous stages: L = q*P + r, the first r stages get q + 1 layers.
__device__ __forceinline__ int stage_l0(const Ctx &x, int s) { return s * x.q + (s < x.r ? s : x.r); }
__device__ __forceinline__ int stage_nl(const Ctx &x, int s) { return x.q + (s < x.r ? 1 : 0); }

// ---------------------------------------------------------------------------
// MLP (Fig. 2: @dense = Gemm + Relu).  With H > 1 even layers are
// column-parallel (W: d x d/H), odd layers row-parallel (W: d/H x d) with an
// all-reduce of their output; dX of column-parallel layers is all-reduced in
// the backward pass (layer 0's dX is computed and discarded).
// ---------------------------------------------------------------------------
enum MlpKind { kPlain = 0, kCol = 1, kRow = 2 };

__device__ __forceinline__ int mlp_kind(const Ctx &x, int i) { return x.H <= 1 ? kPlain : ((i & 1) ? kRow : kCol); }

// ZeRO parameter group of MLP layer i: the layer, or with H > 1 its
// column/row pair
__device__ __forceinline__ int mlp_group(const Ctx &x, int i) { return x.H > 1 ? i / 2 : i; }

__device__ __forceinline__ void mlp_dims(const Ctx &x, int kind, uint64_t &din, uint64_t &dout)
{
    din = kind == kRow ? x.d / (uint64_t)x.H : x.d;
    dout = kind == kCol ? x.d / (uint64_t)x.H : x.d;
}

// One layer's forward.  free_in: the layer input dies at the Gemm (inference,
// and layers after the first under recomputation; otherwise the weight
// gradient reads it); dead_out: the model's last layer in inference, whose
// output has no use; grp: the layer's parameter group.
template <class S>
__device__ __forceinline__ void mlp_layer_fwd(const Ctx &x, S &o, uint64_t m, int kind, bool free_in, bool dead_out,
                                              int grp)
{
    const uint64_t e = x.e;
    uint64_t din, dout;
    mlp_dims(x, kind, din, dout);
    o.bcast(e * din * dout, grp);
    o.mm(2 * m * din * dout, e * (m * din + din * dout + m * dout), e * m * dout, free_in ? e * m * din : 0, din);
    if (kind == kRow) o.ar_tp(e * m * dout);
    // Relu frees the pre-activation
    o.local(m * dout, 2 * e * m * dout, e * m * dout, e * m * dout + (dead_out ? e * m * dout : 0));
}

// One layer's backward.  frees_input: the stage's first layer, where the
// stage input dies at the weight gradient; layer0: the model's first layer,
// whose dX has no use and is not all-reduced; grp: the parameter group;
// last: the stage's last backward block under overlap, which hands every
// finished weight gradient over.
template <class S>
__device__ __forceinline__ void mlp_layer_bwd(const Ctx &x, S &o, uint64_t m, int kind, bool frees_input,
                                              bool layer0, bool acc, int grp, bool last = false)
{
    const uint64_t e = x.e;
    uint64_t din, dout;
    mlp_dims(x, kind, din, dout);
    o.local(m * dout, 3 * e * m * dout, e * m * dout, 2 * e * m * dout);                 // ReluGrad: da and a die
    o.mm(2 * m * din * dout, e * (m * din + m * dout + din * dout), e * din * dout,
         frees_input ? e * m * din : 0, m);                                             // weight gradient
    if (acc) o.local(din * dout, 3 * e * din * dout, 0, e * din * dout);                // accumulate
    if (last) o.handover(e * din * dout);
    o.bcast(e * din * dout, grp);
    o.mm(2 * m * din * dout, e * (m * dout + din * dout + m * din), e * m * din,
         e * m * dout + (layer0 ? e * m * din : 0), dout);                              // input gradient
    if (kind != kRow && x.H > 1 && !layer0) o.ar_tp(e * m * din);
}

template <class S>
__device__ __forceinline__ void mlp_loss(const Ctx &x, S &o, uint64_t m)
{
    const uint64_t e = x.e;
    o.local(3 * m * x.d, 3 * e * m * x.d, e * m * x.d, e * m * x.d);   // loss gradient; y_k dies
}

// bytes of the activation a stage sends forward / the gradient it sends back
// for a microbatch of m rows
__device__ __forceinline__ uint64_t mlp_act_out(const Ctx &x, int s, uint64_t m)
{
    uint64_t din, dout;
    mlp_dims(x, mlp_kind(x, stage_l0(x, s) + stage_nl(x, s) - 1), din, dout);
    return x.e * m * dout;
}

__device__ __forceinline__ uint64_t mlp_grad_out(const Ctx &x, int s, uint64_t m)
{
    uint64_t din, dout;
    mlp_dims(x, mlp_kind(x, stage_l0(x, s)), din, dout);
    return x.e * m * din;
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

__device__ __forceinline__ TfSz tf_sizes(const Ctx &x, uint64_t m)
{
    TfSz z;
    z.m = m;
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

// ZeRO parameter groups of the transformer in model order: the embedding,
// layer i, the LM head
__device__ __forceinline__ int tf_group_layer(int i) { return i + 1; }
__device__ __forceinline__ int tf_group_head(const Ctx &x) { return x.L + 1; }

// stage 0, before its layers: embedding
template <class S>
__device__ __forceinline__ void tf_fwd_first(const Ctx &x, S &o, const TfSz &z)
{
    const uint64_t T = z.T, d = x.d;
    o.bcast(x.e * x.Vh * d, 0);
    o.local(T * d, 2 * z.ACT + z.IDS, z.ACT, x.train ? 0 : z.IDS);   // ids die in inference
    o.ar_tp(z.ACT);
}

// One layer's forward.  save: the activations the layer's backward reads
// stay live (training without recomputation, and the replay); keep_in: the
// layer input stays live (save, or the checkpoint of a recomputed stage);
// full = false stops after GeLU (the replay of a stage's last layer, whose
// output nothing reads); grp: the layer's parameter group.
template <class S>
__device__ __forceinline__ void tf_layer_fwd(const Ctx &x, S &o, const TfSz &z, bool save, bool keep_in, bool full,
                                             int grp)
{
    const uint64_t T = z.T, d = x.d, dH = x.dH, FH = x.FH, e = x.e, S_ = x.seq;
    o.local(8 * T * d, 2 * z.ACT, z.ACT, 0);                                                  // LN1
    o.bcast(e * d * 3 * dH, grp);
    o.mm(2 * T * d * 3 * dH, e * (T * d + d * 3 * dH + T * 3 * dH), z.QKV, save ? 0 : z.ACT, d);  // QKV
    o.mm(2 * T * S_ * dH, 2 * z.OH + z.S2, z.S2, 0, x.hd);                                 // scores
    o.local(5 * z.m * x.aH * S_ * S_, 2 * z.S2, z.S2, z.S2);                                  // softmax
    o.mm(2 * T * S_ * dH, z.S2 + 2 * z.OH, z.OH, save ? 0 : z.S2 + z.QKV, S_);            // P.V
    o.bcast(e * dH * d, grp);
    o.mm(2 * T * dH * d, e * (T * dH + dH * d + T * d), z.ACT, save ? 0 : z.OH, dH);       // out-proj
    o.ar_tp(z.ACT);
    o.local(T * d, 3 * z.ACT, z.ACT, keep_in ? z.ACT : 2 * z.ACT);                           // residual
    o.local(8 * T * d, 2 * z.ACT, z.ACT, 0);                                                  // LN2
    o.bcast(e * d * FH, grp);
    o.mm(2 * T * d * FH, e * (T * d + d * FH + T * FH), z.FF, save ? 0 : z.ACT, d);        // fc1
    o.local(8 * T * FH, 2 * z.FF, z.FF, save ? 0 : z.FF);                                    // GeLU
    if (!full) return;
    o.bcast(e * FH * d, grp);
    o.mm(2 * T * FH * d, e * (T * FH + FH * d + T * d), z.ACT, save ? 0 : z.FF, FH);       // fc2
    o.ar_tp(z.ACT);
    o.local(T * d, 3 * z.ACT, z.ACT, save ? z.ACT : 2 * z.ACT);                              // residual
}

// last stage, after its layers: final LN and LM head
template <class S>
__device__ __forceinline__ void tf_fwd_last(const Ctx &x, S &o, const TfSz &z)
{
    const uint64_t T = z.T, d = x.d, e = x.e;
    const bool tr = x.train;
    o.local(8 * T * d, 2 * z.ACT, z.ACT, tr ? 0 : z.ACT);                                  // final LN
    o.bcast(e * d * x.Vh, tf_group_head(x));
    o.mm(2 * T * d * x.Vh, e * (T * d + d * x.Vh + T * x.Vh), z.LOG, tr ? 0 : z.ACT + z.LOG, d);  // LM head
}

// last stage, before its layers' backward: loss, LM head and final LN grads
template <class S>
__device__ __forceinline__ void tf_bwd_last(const Ctx &x, S &o, const TfSz &z, bool acc, bool last = false)
{
    const uint64_t T = z.T, d = x.d, e = x.e, Vh = x.Vh;
    o.local(3 * T * Vh, z.LOG + z.ST, z.ST, 0);                                   // loss statistics
    o.ar_tp(z.ST);
    o.local(2 * T * Vh, 2 * z.LOG + z.ST + z.IDS, z.LOG, z.LOG + z.ST + z.IDS);   // dlogits
    o.bcast(e * d * Vh, tf_group_head(x));
    o.mm(2 * T * d * Vh, e * (T * Vh + d * Vh + T * d), z.ACT, 0, Vh);         // LM head dX
    o.ar_tp(z.ACT);
    o.mm(2 * T * d * Vh, e * (T * d + T * Vh + d * Vh), e * d * Vh, z.ACT + z.LOG, T);  // LM head dW
    if (acc) o.local(d * Vh, 3 * e * d * Vh, 0, e * d * Vh);
    if (last) o.handover(e * d * Vh);
    o.local(8 * T * d, 3 * z.ACT, z.ACT, 2 * z.ACT);                             // final LN grad
}

template <class S>
__device__ __forceinline__ void tf_layer_bwd(const Ctx &x, S &o, const TfSz &z, bool acc, int grp, bool last = false)
{
    const uint64_t T = z.T, d = x.d, dH = x.dH, FH = x.FH, e = x.e, S_ = x.seq;
    o.bcast(e * FH * d, grp);
    o.mm(2 * T * FH * d, e * (T * d + FH * d + T * FH), z.FF, 0, d);          // fc2 dX
    o.mm(2 * T * FH * d, e * (T * FH + T * d + FH * d), e * FH * d, z.FF, T);  // fc2 dW
    if (acc) o.local(FH * d, 3 * e * FH * d, 0, e * FH * d);
    if (last) o.handover(e * FH * d);
    o.local(8 * T * FH, 3 * z.FF, z.FF, 2 * z.FF);                                // GeLU grad
    o.bcast(e * d * FH, grp);
    o.mm(2 * T * d * FH, e * (T * FH + d * FH + T * d), z.ACT, 0, FH);         // fc1 dX
    o.ar_tp(z.ACT);
    o.mm(2 * T * d * FH, e * (T * d + T * FH + d * FH), e * d * FH, z.ACT + z.FF, T);  // fc1 dW
    if (acc) o.local(d * FH, 3 * e * d * FH, 0, e * d * FH);
    if (last) o.handover(e * d * FH);
    o.local(8 * T * d, 3 * z.ACT, z.ACT, 2 * z.ACT);                              // LN2 grad
    o.local(T * d, 3 * z.ACT, z.ACT, 2 * z.ACT);                                  // residual merge
    o.bcast(e * dH * d, grp);
    o.mm(2 * T * dH * d, e * (T * d + dH * d + T * dH), z.OH, 0, d);          // out-proj dX
    o.mm(2 * T * dH * d, e * (T * dH + T * d + dH * d), e * dH * d, z.OH, T);  // out-proj dW
    if (acc) o.local(dH * d, 3 * e * dH * d, 0, e * dH * d);
    if (last) o.handover(e * dH * d);
    o.mm(4 * T * S_ * dH, 2 * z.S2 + 3 * z.OH, z.S2 + z.QKV, z.OH, x.hd + S_);  // P.V grads: dP over hd, dV over S
    o.local(5 * z.m * x.aH * S_ * S_, 3 * z.S2, z.S2, 2 * z.S2);                  // softmax grad
    o.mm(4 * T * S_ * dH, z.S2 + 4 * z.OH, 0, z.S2 + z.QKV, 2 * S_);          // Q.K^T grads: dQ, dK over S
    o.bcast(e * d * 3 * dH, grp);
    o.mm(2 * T * 3 * dH * d, e * (T * 3 * dH + 3 * dH * d + T * d), z.ACT, 0, 3 * dH);  // QKV dX
    o.ar_tp(z.ACT);
    o.mm(2 * T * d * 3 * dH, e * (T * d + T * 3 * dH + d * 3 * dH), e * d * 3 * dH, z.ACT + z.QKV, T);  // QKV dW
    if (acc) o.local(d * 3 * dH, 3 * e * d * 3 * dH, 0, e * d * 3 * dH);
    if (last) o.handover(e * d * 3 * dH);
    o.local(8 * T * d, 3 * z.ACT, z.ACT, 2 * z.ACT);                              // LN1 grad
    o.local(T * d, 3 * z.ACT, z.ACT, 2 * z.ACT);                                  // residual merge
}

// stage 0, after its layers' backward: embedding gradient
template <class S>
__device__ __forceinline__ void tf_bwd_first(const Ctx &x, S &o, const TfSz &z, bool acc, bool last = false)
{
    const uint64_t T = z.T, d = x.d, e = x.e, Vh = x.Vh;
    o.local(T * d, z.ACT + z.IDS + e * Vh * d, e * Vh * d, z.ACT + z.IDS);        // embedding dW
    if (acc) o.local(Vh * d, 3 * e * Vh * d, 0, e * Vh * d);
    if (last) o.handover(e * Vh * d);
}

// ---------------------------------------------------------------------------
// Whole blocks (one microbatch's forward or backward on one stage), op by op
// ---------------------------------------------------------------------------
template <class S>
__device__ __forceinline__ void block_fwd(const Ctx &x, S &o, int s, int k)
{
    const uint64_t m = mb_rows(x, k);
    if (x.mlp) {
        const int l0 = stage_l0(x, s), l1 = l0 + stage_nl(x, s);
        for (int i = l0; i < l1; ++i)
            mlp_layer_fwd(x, o, m, mlp_kind(x, i), !x.train || (x.rc && i > l0), !x.train && i == x.L - 1,
                          mlp_group(x, i));
        return;
    }
    const TfSz z = tf_sizes(x, m);
    if (s == 0) tf_fwd_first(x, o, z);
    const int nl = stage_nl(x, s), l0 = stage_l0(x, s);
    const bool save = x.train && !x.rc;
    for (int i = 0; i < nl; ++i) tf_layer_fwd(x, o, z, save, save || (x.rc && i == 0), true, tf_group_layer(l0 + i));
    if (s == x.P - 1) tf_fwd_last(x, o, z);
}

// (under overlap the stage's last backward block, microbatch K - 1, hands
// each weight gradient over as soon as it is finished)
template <class S>
__device__ __forceinline__ void block_bwd(const Ctx &x, S &o, int s, int k)
{
    const uint64_t m = mb_rows(x, k);
    const bool acc = k >= 1;
    const bool last = x.ov && k == x.K - 1;
    if (x.mlp) {
        const int l0 = stage_l0(x, s), l1 = l0 + stage_nl(x, s);
        if (s == x.P - 1) mlp_loss(x, o, m);
        if (x.rc)   // replay every layer but the last from the checkpoint
            for (int i = l0; i < l1 - 1; ++i) mlp_layer_fwd(x, o, m, mlp_kind(x, i), false, false, mlp_group(x, i));
        for (int i = l1 - 1; i >= l0; --i)
            mlp_layer_bwd(x, o, m, mlp_kind(x, i), i == l0, i == 0, acc, mlp_group(x, i), last);
        return;
    }
    const TfSz z = tf_sizes(x, m);
    if (s == x.P - 1) tf_bwd_last(x, o, z, acc, last);
    const int nl = stage_nl(x, s), l0 = stage_l0(x, s);
    if (x.rc)   // replay the layers from the checkpoint, the last one up to its GeLU
        for (int i = 0; i < nl; ++i) tf_layer_fwd(x, o, z, true, true, i < nl - 1, tf_group_layer(l0 + i));
    for (int i = nl - 1; i >= 0; --i) tf_layer_bwd(x, o, z, acc, tf_group_layer(l0 + i), last);
    if (s == 0) tf_bwd_first(x, o, z, acc, last);
}

// ---------------------------------------------------------------------------
// Optimizer, resident memory, splits and the weight update
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

// one parameter tensor of group grp: all-reduce its gradient over the D
// replicas, then the optimizer op (in place), after which the gradient dies.
// ZeRO: reduce the gradients onto the owner (they die there), whose
// optimizer op consumes the reduced gradient.  Overlap: the gradient was
// all-reduced on the communication streams; it comes back first.
template <class S>
__device__ __forceinline__ void wu_param(const Ctx &x, S &o, uint64_t N, int grp)
{
    uint64_t fl, by;
    opt_cost(x, N, fl, by);
    if (x.zero) {
        o.reduce(x.e * N, grp);
        o.owner_local(fl, by, 0, x.e * N, grp);
        return;
    }
    if (x.ov) o.handback(x.e * N);
    else o.ar_dp(x.e * N);
    o.local(fl, by, 0, x.e * N);
}

// after the stage's last backward, layer by layer in ascending order
template <class S>
__device__ __forceinline__ void weight_update(const Ctx &x, S &o, int s)
{
    const int l0 = stage_l0(x, s), nl = stage_nl(x, s);
    if (x.mlp) {
        for (int i = l0; i < l0 + nl; ++i) {
            uint64_t din, dout;
            mlp_dims(x, mlp_kind(x, i), din, dout);
            wu_param(x, o, din * dout, mlp_group(x, i));
        }
        return;
    }
    const uint64_t d = x.d;
    if (s == 0) wu_param(x, o, x.Vh * d, 0);
    for (int i = 0; i < nl; ++i) {
        const int g = tf_group_layer(l0 + i);
        wu_param(x, o, d * 3 * x.dH, g);
        wu_param(x, o, x.dH * d, g);
        wu_param(x, o, d * x.FH, g);
        wu_param(x, o, x.FH * d, g);
    }
    if (s == x.P - 1) wu_param(x, o, d * x.Vh, tf_group_head(x));
}

// bytes of one row (sequence) of the stage-0 input / last-stage target
__device__ __forceinline__ uint64_t input_row(const Ctx &x) { return x.mlp ? x.e * x.d : 4 * x.seq; }

// bytes of the replica's input rows (stage 0) and targets (last stage,
// training), resident from t = 0
__device__ __forceinline__ uint64_t resident_inputs(const Ctx &x, int s)
{
    uint64_t b = 0;
    if (s == 0) b += input_row(x) * x.rows;
    if (s == x.P - 1 && x.train) b += input_row(x) * x.rows;
    return b;
}

// bytes resident on a device of stage s at t = 0 without ZeRO: weight
// shard, optimizer state, the replica's inputs
__device__ __forceinline__ uint64_t resident(const Ctx &x, int s)
{
    const int l0 = stage_l0(x, s), nl = stage_nl(x, s);
    uint64_t N = 0;
    if (x.mlp) {
        for (int i = l0; i < l0 + nl; ++i) {
            uint64_t din, dout;
            mlp_dims(x, mlp_kind(x, i), din, dout);
            N += din * dout;
        }
    } else {
        N = (uint64_t)nl * (x.d * 3 * x.dH + x.dH * x.d + x.d * x.FH + x.FH * x.d);
        if (s == 0) N += x.Vh * x.d;
        if (s == x.P - 1) N += x.d * x.Vh;
    }
    return x.e * N + opt_state(x, N) + resident_inputs(x, s);
}

// ---------------------------------------------------------------------------
// ZeRO ownership (Fig. 9): the parameter groups of stage s are a contiguous
// range of the model order (transformer: the embedding on stage 0, layer
// groups l0+1 .. l1, the head L+1 on the last stage; MLP: its layers or
// column/row pairs), and group g belongs to data replica g mod D.
// ---------------------------------------------------------------------------
struct ZStage {
    int gl_lo, gl_hi;     // layer groups of the stage [gl_lo, gl_hi)
    bool emb, head;       // holds the embedding (group 0) / the LM head (group L+1)
    int g_head;
    uint64_t GL, GE;      // resident bytes (weights + optimizer state) of a layer group / the embedding or head
    uint64_t rmax, rsec;  // largest owned bytes over the D replicas; over the replicas other than `arg`
    int arg;
};

// groups g in [lo, hi) with g mod D == d (0 <= d < D)
__device__ __forceinline__ int64_t count_mod(int lo, int hi, int d, int D)
{
    auto upto = [&](int n) -> int64_t { return n > d ? (int64_t)(n - d - 1) / D + 1 : 0; };
    return hi > lo ? upto(hi) - upto(lo) : 0;
}

// bytes of weights and optimizer state that replica d owns on stage s
__device__ __forceinline__ uint64_t z_owned(const Ctx &x, const ZStage &z, int d)
{
    uint64_t b = (uint64_t)count_mod(z.gl_lo, z.gl_hi, d, x.D) * z.GL;
    if (z.emb && d == 0) b += z.GE;
    if (z.head && z.g_head % x.D == d) b += z.GE;
    return b;
}

__device__ inline void z_stage(const Ctx &x, int s, ZStage &z)
{
    const int l0 = stage_l0(x, s), l1 = l0 + stage_nl(x, s);
    uint64_t NL, NE = 0;
    if (x.mlp) {
        z.gl_lo = mlp_group(x, l0);
        z.gl_hi = mlp_group(x, l1 - 1) + 1;
        NL = x.H > 1 ? 2 * x.d * (x.d / (uint64_t)x.H) : x.d * x.d;
        z.emb = z.head = false;
    } else {
        z.gl_lo = tf_group_layer(l0);
        z.gl_hi = tf_group_layer(l1 - 1) + 1;
        NL = x.d * 3 * x.dH + x.dH * x.d + x.d * x.FH + x.FH * x.d;
        NE = x.Vh * x.d;
        z.emb = s == 0;
        z.head = s == x.P - 1;
    }
    z.g_head = x.L + 1;
    z.GL = x.e * NL + opt_state(x, NL);
    z.GE = x.e * NE + opt_state(x, NE);
    // the replicas that own something here are the owners of the stage's
    // first min(D, #groups) groups; the others own nothing
    const int g_lo = z.emb ? 0 : z.gl_lo, g_hi = z.head ? z.g_head + 1 : z.gl_hi;
    const int n_own = (g_hi - g_lo) < x.D ? (g_hi - g_lo) : x.D;
    uint64_t m1 = 0, m2 = 0;
    int a1 = -1;
    for (int j = 0; j < n_own; ++j) {
        const int d = (g_lo + j) % x.D;
        const uint64_t b = z_owned(x, z, d);
        if (a1 < 0 || b > m1) {
            m2 = a1 < 0 ? 0 : m1;
            m1 = b;
            a1 = d;
        } else if (b > m2) {
            m2 = b;
        }
    }
    // a replica owning nothing has 0 bytes, already the floor of m2
    z.rmax = m1;
    z.rsec = m2;
    z.arg = a1;
}

// K > 1: split the replica's whole input (stage 0) or target (last stage)
// into microbatches; a copy whose source dies
template <class S>
__device__ __forceinline__ void split(const Ctx &x, S &o)
{
    const uint64_t whole = input_row(x) * x.rows;
    o.local(0, 2 * whole, whole, whole);
}

// ---------------------------------------------------------------------------
// Block order of a stage: forward-only (inference); synchronous 1F1B; GPipe
// ---------------------------------------------------------------------------
// position `pos` of stage s's block sequence -> (is_backward, microbatch)
__device__ __forceinline__ void block_at(const Ctx &x, int s, int pos, bool &bwd, int &k)
{
    if (!x.train) {
        bwd = false;
        k = pos;
        return;
    }
    if (x.schedule == DSIM_SCHED_GPIPE) {   // all forwards, then all backwards
        bwd = pos >= x.K;
        k = bwd ? pos - x.K : pos;
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

// bytes sent after a block of m rows, and the bytes the sender frees
__device__ __forceinline__ void send_size(const Ctx &x, int s, uint64_t m, bool bwd, uint64_t &sz, uint64_t &fre)
{
    if (x.mlp) {
        sz = bwd ? mlp_grad_out(x, s, m) : mlp_act_out(x, s, m);
        fre = (bwd || !x.train) ? sz : 0;
    } else {
        sz = x.e * m * x.seq * x.d;
        fre = sz;
    }
}

}  // namespace dsim
