// parametric.hip -- simulate the D/H/P/K transform without building op lists.
//
// Each candidate gets a segment of W = 2^ceil(log2 P) lanes of a wavefront,
// one lane per pipeline stage; segments of equal width share wavefronts
// (64 / W candidates each).  A lane expands, on the fly and in program order,
// the ops of its stage of the distributed program the transform of Sec. 4
// produces (ops in model.h) and simulates them with the semantics of Sec. 2.1
// and the cost model of Sec. 3.3:
//   * synchronous 1F1B or GPipe (training), forward-only (inference) per
//     stage;
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
//   * with ZeRO (Fig. 9) the replicas still run the same ops at the same
//     times, except that only a parameter's owner runs its optimizer op; the
//     next gradient reduce waits for it, so the stage's latest device finishes
//     at the lane's clock.  Their memory differs: each holds only the groups
//     it owns and a copy of every other weight while an op reads it.  The
//     lane tracks the live bytes that do not depend on ownership plus the
//     largest owned resident, and each block kind's highest point is taken
//     as the maximum over the replicas in closed form (see zero_block).
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
#include <mutex>
#include <type_traits>

#include "model.h"

namespace dsim {
namespace {

constexpr int kLanes = 64;
constexpr int kClasses = 7;       // segment widths 1, 2, 4, ..., 64
constexpr int kScanBlock = 256;

// Recorded block program of one lane and direction, in double2 entries:
// ops before the repeating units, one unit, ops after the units.  The
// regions are sized for the larger (backward) block; forward blocks use the
// F_* prefix of each region.
template <bool TF, bool Z> struct Shape;
template <> struct Shape<true, false> {
    static constexpr int PRE2 = 4;    // last stage backward: loss .. final LN grad (8 ops)
    static constexpr int U2 = 12;     // one layer backward: 17 compute + 4 accumulations + 2 all-reduces
    static constexpr int SUF2 = 1;    // stage 0 backward: embedding grad + accumulation
    static constexpr int F_PRE2 = 1;  // stage 0 forward: embedding + all-reduce
    static constexpr int F_U2 = 7;    // one layer forward: 12 compute + 2 all-reduces
    static constexpr int F_SUF2 = 1;  // last stage forward: final LN + LM head
};
template <> struct Shape<false, false> {
    static constexpr int PRE2 = 1;    // last stage backward: loss gradient
    static constexpr int U2 = 5;      // row layer (4 ops) + column layer (5) backward
    static constexpr int SUF2 = 5;    // the stage's first unit backward (frees the stage input)
    static constexpr int F_PRE2 = 0;
    static constexpr int F_U2 = 3;    // column layer (2 ops) + row layer (3) forward
    static constexpr int F_SUF2 = 3;  // the model's last unit in inference (dead output)
};
// ZeRO adds one broadcast before every op that reads a weight
template <> struct Shape<true, true> {
    static constexpr int PRE2 = 5;    // 8 ops + 1 broadcast
    static constexpr int U2 = 14;     // 22 ops + 4 broadcasts
    static constexpr int SUF2 = 2;    // the forward suffix is the larger one here
    static constexpr int F_PRE2 = 2;  // 2 ops + 1 broadcast
    static constexpr int F_U2 = 9;    // 14 ops + 4 broadcasts
    static constexpr int F_SUF2 = 2;  // 2 ops + 1 broadcast
};
template <> struct Shape<false, true> {
    static constexpr int PRE2 = 1;
    static constexpr int U2 = 6;      // 9 ops + 2 broadcasts
    static constexpr int SUF2 = 6;    // 9 ops + 2 broadcasts
    static constexpr int F_PRE2 = 0;
    static constexpr int F_U2 = 4;    // 5 ops + 2 broadcasts
    static constexpr int F_SUF2 = 3;  // inference only: no ZeRO
};
// a forward block's regions are prefixes of the backward block's
template <class Sh> constexpr bool shape_nested()
{
    return Sh::F_PRE2 <= Sh::PRE2 && Sh::F_U2 <= Sh::U2 && Sh::F_SUF2 <= Sh::SUF2;
}
static_assert(shape_nested<Shape<true, false>>() && shape_nested<Shape<false, false>>() &&
                  shape_nested<Shape<true, true>>() && shape_nested<Shape<false, true>>(),
              "forward regions must fit the backward ones");

// the device-model constants the transform reads (the table format's
// per-group-size rows stay out of the kernel arguments)
struct ParConsts {
    double inv_f, inv_b, inv_l, lat, launch;
    uint64_t cap;
    int32_t mm;
    double mm_c0, mm_c1, mm_c2, mm_c3, mm_floor;
    int32_t node;
    double net_lat, net_inv_l;
    int32_t streams;
    double st_lat, st_inv_l;
};

struct ParArgs {
    dsim_model m;
    const dsim_strategy *cand;
    int64_t n_cand;
    int32_t row_width;
    int32_t p_bound;
    const uint32_t *perm;   // candidates grouped by segment class
    const uint32_t *meta;   // [0,8) class totals, [8,16) first perm index, [16,24) first lane
    int32_t narrow_end;     // classes the narrow launch takes: [0, narrow_end)
    const uint32_t *order;  // the wide launch's wavefronts, longest first
    double *makespan;
    double *finish;
    uint64_t *peak;
    uint64_t *cand_peak;
    uint64_t *n_ops;
    uint64_t *walked;
    int32_t *status;
    ParConsts c;
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
// The lane's stage replica, op by op (splits, the weight update and, under
// overlap, the last backward block).  With ZeRO, live counts the largest
// owned resident and z describes the stage's ownership: a reduce samples the
// owner holding the reduced gradient and the other replicas, then every
// gradient dies; the owner's optimizer op frees the reduced gradient again
// (below that sample).  Under overlap tm is the communication stream's
// clock: a hand-over or hand-back is a Send between the two streams (both
// clocks meet at its end), the all-reduce advances tm alone (every replica's
// communication stream is at the same time).
struct Walk {
    const Ctx &x;
    double clk;
    int64_t live, peak;
    uint64_t walked, nops;
    const ZStage *z;
    double tm = 0.0;

    __device__ __forceinline__ void meet(uint64_t by)
    {
        const double st = clk > tm ? clk : tm;
        clk = st + cost_stream(x, by);
        tm = clk;
    }
    __device__ __forceinline__ void handover(uint64_t by)
    {
        meet(by);
        tm = tm + cost_ar_dp(x, by);
        walked += 2;
        nops += x.mult_dev + x.mult_dp;
    }
    __device__ __forceinline__ void handback(uint64_t by)
    {
        meet(by);
        walked += 1;
        nops += x.mult_dev;
    }

    __device__ __forceinline__ void op(double c, uint64_t al, uint64_t fr)
    {
        clk = clk + c;
        live += (int64_t)al;
        peak = live > peak ? live : peak;
        live -= (int64_t)fr;
        walked += 1;
        nops += x.mult_dev;
    }
    __device__ __forceinline__ void local(uint64_t fl, uint64_t by, uint64_t al, uint64_t fr)
    {
        op(cost_local(x, fl, by), al, fr);
    }
    __device__ __forceinline__ void mm(uint64_t fl, uint64_t by, uint64_t al, uint64_t fr, uint64_t k)
    {
        op(cost_mm(x, fl, by, k), al, fr);
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
    __device__ __forceinline__ void bcast(uint64_t by, int)
    {
        if (!x.zero) return;
        clk = clk + cost_chain_d(x, by);
        walked += 1;
        nops += x.mult_dp;
    }
    __device__ __forceinline__ void reduce(uint64_t by, int grp)
    {
        clk = clk + cost_chain_d(x, by);
        walked += 1;
        nops += x.mult_dp;
        const int o = grp % x.D;
        const int64_t own = (int64_t)z_owned(x, *z, o) + (int64_t)by;
        const int64_t other = (int64_t)(o == z->arg ? z->rsec : z->rmax);
        const int64_t hi = live - (int64_t)z->rmax + (own > other ? own : other);
        peak = hi > peak ? hi : peak;
        live -= (int64_t)by;
    }
    __device__ __forceinline__ void owner_local(uint64_t fl, uint64_t by, uint64_t, uint64_t, int)
    {
        clk = clk + cost_local(x, fl, by);
        walked += 1;
        nops += x.mult_dp;
    }
};

// Records ops' costs into a region of LDS and summarises their memory effect
// relative to the live bytes at the region's start.
struct Record {
    const Ctx &x;
    double *base;      // entry j at base[(j / 2) * step + (j & 1)]
    int step;          // doubles between consecutive entry pairs
    int n;
    int64_t cur, top;  // net bytes so far; max of (bytes after an op's allocation)

    __device__ __forceinline__ void put(double c)
    {
        base[(n >> 1) * step + (n & 1)] = c;
        ++n;
    }
    __device__ __forceinline__ void pad(int entries2)
    {
        while (n < 2 * entries2) put(0.0);   // clock + 0.0 == clock
    }
    __device__ __forceinline__ void op(double c, uint64_t al, uint64_t fr)
    {
        put(c);
        const int64_t a = cur + (int64_t)al;
        top = a > top ? a : top;
        cur = a - (int64_t)fr;
    }
    __device__ __forceinline__ void local(uint64_t fl, uint64_t by, uint64_t al, uint64_t fr)
    {
        op(cost_local(x, fl, by), al, fr);
    }
    __device__ __forceinline__ void mm(uint64_t fl, uint64_t by, uint64_t al, uint64_t fr, uint64_t k)
    {
        op(cost_mm(x, fl, by, k), al, fr);
    }
    __device__ __forceinline__ void ar_tp(uint64_t by)
    {
        if (x.H <= 1) return;
        put(cost_ar_tp(x, by));
    }
    __device__ __forceinline__ void ar_dp(uint64_t by)
    {
        if (x.D <= 1) return;
        put(cost_ar_dp(x, by));
    }
    // a broadcast's cost; with ZeRO the memory summary comes from MemZ
    __device__ __forceinline__ void bcast(uint64_t by, int)
    {
        if (!x.zero) return;
        put(cost_chain_d(x, by));
    }
    __device__ __forceinline__ void reduce(uint64_t by, int) { put(cost_chain_d(x, by)); }
    __device__ __forceinline__ void owner_local(uint64_t fl, uint64_t by, uint64_t, uint64_t, int)
    {
        put(cost_local(x, fl, by));
    }
    // recorded programs hold no last block of an overlapped stage
    __device__ __forceinline__ void handover(uint64_t) {}
    __device__ __forceinline__ void handback(uint64_t) {}
};

// Memory summary only (net bytes, peak above the start), no costs.
struct Mem {
    const Ctx &x;
    int64_t cur, top;
    __device__ __forceinline__ void local(uint64_t, uint64_t, uint64_t al, uint64_t fr)
    {
        const int64_t a = cur + (int64_t)al;
        top = a > top ? a : top;
        cur = a - (int64_t)fr;
    }
    __device__ __forceinline__ void mm(uint64_t fl, uint64_t by, uint64_t al, uint64_t fr, uint64_t)
    {
        local(fl, by, al, fr);
    }
    __device__ __forceinline__ void ar_tp(uint64_t) {}
    __device__ __forceinline__ void ar_dp(uint64_t) {}
    __device__ __forceinline__ void bcast(uint64_t, int) {}
    __device__ __forceinline__ void reduce(uint64_t, int) {}
    __device__ __forceinline__ void owner_local(uint64_t, uint64_t, uint64_t, uint64_t, int) {}
    __device__ __forceinline__ void handover(uint64_t) {}   // allocates nothing
    __device__ __forceinline__ void handback(uint64_t) {}
};

// ZeRO memory summary of ops that read the weights of one parameter group:
// net bytes and the highest point above the start, seen by a replica that
// does not own the group (tn: it holds each broadcast copy from the
// broadcast until the op that reads it) and by the owner (to: no copies).
// Copies die inside the summarised ops, so the net is the same for both.
struct MemZ {
    const Ctx &x;
    int64_t cur, tn, to, pend;
    __device__ __forceinline__ void local(uint64_t, uint64_t, uint64_t al, uint64_t fr)
    {
        const int64_t a = cur + (int64_t)al;
        tn = a + pend > tn ? a + pend : tn;
        to = a > to ? a : to;
        cur = a - (int64_t)fr;
        pend = 0;
    }
    __device__ __forceinline__ void mm(uint64_t fl, uint64_t by, uint64_t al, uint64_t fr, uint64_t)
    {
        local(fl, by, al, fr);
    }
    __device__ __forceinline__ void ar_tp(uint64_t) {}
    __device__ __forceinline__ void ar_dp(uint64_t) {}
    __device__ __forceinline__ void bcast(uint64_t by, int)
    {
        if (!x.zero) return;
        tn = cur + (int64_t)by > tn ? cur + (int64_t)by : tn;
        to = cur > to ? cur : to;
        pend = (int64_t)by;
    }
    __device__ __forceinline__ void reduce(uint64_t, int) {}
    __device__ __forceinline__ void owner_local(uint64_t, uint64_t, uint64_t, uint64_t, int) {}
    __device__ __forceinline__ void handover(uint64_t) {}   // allocates nothing
    __device__ __forceinline__ void handback(uint64_t) {}
};

// Liveness of a forward unit.  kFwdBlock: as in a forward block (training
// keeps what the backward reads; inference and recomputation drop it);
// kFwdFirst: the first unit of a forward block under recomputation (its
// input is the checkpoint); kFwdReplay: the backward block's replay, which
// keeps what the backward reads.  Every variant has the same op costs.
enum FwdLive { kFwdBlock = 0, kFwdFirst = 1, kFwdReplay = 2 };

// The repeating unit of a block for microbatches of m rows: one transformer
// layer; one MLP layer (H = 1) or column/row pair (H > 1), in walk order.
// acc: with gradient accumulation (every backward microbatch but the first).
template <bool TF, class S>
__device__ void record_unit(const Ctx &x, bool bwd, uint64_t m, bool acc, S &r, int live = kFwdBlock)
{
    if (TF) {
        const TfSz z = tf_sizes(x, m);
        if (bwd) {
            tf_layer_bwd(x, r, z, acc, 0);
        } else {
            const bool save = live == kFwdReplay || (live == kFwdBlock && x.train && !x.rc);
            tf_layer_fwd(x, r, z, save, save || live == kFwdFirst, true, 0);
        }
    } else if (bwd) {
        if (x.H > 1) {
            mlp_layer_bwd(x, r, m, kRow, false, false, acc, 0);
            mlp_layer_bwd(x, r, m, kCol, false, false, acc, 0);
        } else {
            mlp_layer_bwd(x, r, m, kPlain, false, false, acc, 0);
        }
    } else {
        // free_in of the unit's first layer and of its second (pair) layer
        const bool fi_rest = live != kFwdReplay && (!x.train || x.rc);
        const bool fi_first = live == kFwdBlock && fi_rest;
        if (x.H > 1) {
            mlp_layer_fwd(x, r, m, kCol, fi_first, false, 0);
            mlp_layer_fwd(x, r, m, kRow, fi_rest, false, 0);
        } else {
            mlp_layer_fwd(x, r, m, kPlain, fi_first, false, 0);
        }
    }
}

// The replay's last, partial unit: a transformer layer up to its GeLU; the
// column layer of the MLP's last pair (H > 1); nothing for H = 1.  Its ops
// are the first ops of a forward unit, with the same costs.
template <bool TF, class S>
__device__ void record_partial(const Ctx &x, uint64_t m, S &r)
{
    if (TF) tf_layer_fwd(x, r, tf_sizes(x, m), true, true, false, 0);
    else if (x.H > 1) mlp_layer_fwd(x, r, m, kCol, false, false, 0);
}

// The ops of stage s's block before (pre) and after (suf) its repeating
// units: embedding, LM head, loss (transformer); loss, the last unit in
// inference and the stage's first unit in backward (MLP).
template <bool TF, class SP, class SS>
__device__ void record_edges(const Ctx &x, int s, bool bwd, uint64_t m, bool acc, SP &rp, SS &rs)
{
    if (TF) {
        const TfSz z = tf_sizes(x, m);
        if (!bwd) {
            if (s == 0) tf_fwd_first(x, rp, z);
            if (s == x.P - 1) tf_fwd_last(x, rs, z);
        } else {
            if (s == x.P - 1) tf_bwd_last(x, rp, z, acc);
            if (s == 0) tf_bwd_first(x, rs, z, acc);
        }
        return;
    }
    const int per = x.H > 1 ? 2 : 1, l0 = stage_l0(x, s), nl = stage_nl(x, s);
    if (!bwd) {
        if (!x.train && s == x.P - 1)
            for (int i = l0 + nl - per; i < l0 + nl; ++i)
                mlp_layer_fwd(x, rs, m, mlp_kind(x, i), true, i == x.L - 1, 0);
    } else {
        if (s == x.P - 1) mlp_loss(x, rp, m);
        for (int i = l0 + per - 1; i >= l0; --i) mlp_layer_bwd(x, rs, m, mlp_kind(x, i), i == l0, i == 0, acc, 0);
    }
}

// memory effect of pre, n units, suf: unit u starts at pre's net + u * ud;
// top >= 0 is enough (the running peak is never below the live bytes)
__device__ __forceinline__ void compose(int64_t pd, int64_t pt, int64_t ud, int64_t ut, int n, int64_t sd,
                                        int64_t st, int64_t &delta, int64_t &top)
{
    int64_t cur = pd, t = pt;
    if (n > 0) {
        const int64_t hi = cur + ut + (ud > 0 ? (int64_t)(n - 1) * ud : 0);
        t = hi > t ? hi : t;
        cur += (int64_t)n * ud;
    }
    t = cur + st > t ? cur + st : t;
    delta = cur + sd;
    top = t;
}

// appends a summary (d2, t2) to (delta, top)
__device__ __forceinline__ void chain(int64_t &delta, int64_t &top, int64_t d2, int64_t t2)
{
    const int64_t t = delta + t2;
    top = t > top ? t : top;
    delta += d2;
}

// pre, a first unit with its own summary, n - 1 units, suf (n >= 1)
__device__ __forceinline__ void compose_first(int64_t pd, int64_t pt, int64_t fd, int64_t ft, int64_t ud, int64_t ut,
                                              int n, int64_t sd, int64_t st, int64_t &delta, int64_t &top)
{
    int64_t d = pd, t = pt;
    chain(d, t, fd, ft);
    compose(d, t, ud, ut, n - 1, sd, st, delta, top);
}

// Units walked per block: every layer (transformer); every layer or layer
// pair (MLP) except the last unit in inference (last stage) and the
// stage's first unit in backward, which the block records separately.
__device__ __forceinline__ int block_units(const dsim_model &M, int P, int H, int s, bool bwd, bool TF)
{
    const int L = M.n_layers, nl = L / P + (s < L % P ? 1 : 0);
    if (TF) return nl;
    const int per = H > 1 ? 2 : 1;
    if (bwd) return nl / per - 1;
    return nl / per - ((M.mode == DSIM_INFER && s == P - 1) ? 1 : 0);
}

// Counts ops (walked and program ops) without simulating them.
struct Count {
    const Ctx &x;
    uint64_t walked, nops;
    __device__ __forceinline__ void local(uint64_t, uint64_t, uint64_t, uint64_t)
    {
        walked += 1;
        nops += x.mult_dev;
    }
    __device__ __forceinline__ void mm(uint64_t fl, uint64_t by, uint64_t al, uint64_t fr, uint64_t)
    {
        local(fl, by, al, fr);
    }
    __device__ __forceinline__ void ar_tp(uint64_t)
    {
        if (x.H <= 1) return;
        walked += 1;
        nops += x.mult_tp;
    }
    __device__ __forceinline__ void ar_dp(uint64_t)
    {
        if (x.D <= 1) return;
        walked += 1;
        nops += x.mult_dp;
    }
    // ZeRO collectives: one per tensor rank
    __device__ __forceinline__ void bcast(uint64_t, int)
    {
        if (!x.zero) return;
        walked += 1;
        nops += x.mult_dp;
    }
    __device__ __forceinline__ void reduce(uint64_t, int)
    {
        walked += 1;
        nops += x.mult_dp;
    }
    __device__ __forceinline__ void owner_local(uint64_t, uint64_t, uint64_t, uint64_t, int)
    {
        walked += 1;
        nops += x.mult_dp;
    }
    // overlap: a hand-over per replica and an all-reduce per tensor rank; a hand-back per replica
    __device__ __forceinline__ void handover(uint64_t)
    {
        walked += 2;
        nops += x.mult_dev + x.mult_dp;
    }
    __device__ __forceinline__ void handback(uint64_t)
    {
        walked += 1;
        nops += x.mult_dev;
    }
};

// ops of stage s's blocks and sends: K forward blocks; in training one
// backward block without and K - 1 with gradient accumulation, the last of
// which hands the gradients over under overlap.  Op counts do not depend on
// the microbatch size.
__device__ __forceinline__ void count_blocks(const Ctx &x, int s, uint64_t &walked, uint64_t &nops)
{
    Count f{x, 0, 0}, b0{x, 0, 0}, b1{x, 0, 0}, bl{x, 0, 0};
    block_fwd(x, f, s, 0);
    const uint64_t K = (uint64_t)x.K;
    const uint64_t fs = s < x.P - 1 ? 1 : 0;   // Send after each forward block
    walked += K * (f.walked + fs);
    nops += K * (f.nops + fs * x.mult_dev);
    if (!x.train) return;
    const uint64_t bs = s > 0 ? 1 : 0;         // Send after each backward block
    walked += K * bs;
    nops += K * bs * x.mult_dev;
    block_bwd(x, b0, s, 0);                    // microbatch 0 (the last one if K = 1)
    walked += b0.walked;
    nops += b0.nops;
    if (K == 1) return;
    block_bwd(x, b1, s, 1);                    // microbatches 1 .. K-2 (K >= 3)
    block_bwd(x, bl, s, x.K - 1);              // microbatch K-1
    walked += (K - 2) * b1.walked + bl.walked;
    nops += (K - 2) * b1.nops + bl.nops;
}

// ---------------------------------------------------------------------------
// ZeRO: one block kind's memory over the D replicas of a stage
// ---------------------------------------------------------------------------
// A run of n equal units (an edge is a run of one): net bytes d per unit,
// highest points tn (a replica that does not own the unit's group) and to
// (its owner) above the unit's start; unit u reads the weights of group
// gs + dir * u (gs < 0: no weight is read).
struct ZSeg {
    int n;
    int64_t d, tn, to;
    int gs, dir;
};

// highest point of a run above its start as replica d sees it (d < 0: a
// replica owning none of the groups).  Unit u starts at u * d; over the
// units a replica owns (u = r mod D) and those it does not, the highest
// start is the last one (d >= 0) or the first one (d < 0).
__device__ __forceinline__ int64_t run_top(const ZSeg &g, int d, int D)
{
    const int n = g.n;
    const int64_t ud = g.d;
    int r = -1;
    if (d >= 0 && g.gs >= 0) {
        r = (g.dir > 0 ? d - g.gs : g.gs - d) % D;
        if (r < 0) r += D;
    }
    int64_t best = INT64_MIN;
    if (ud >= 0) {
        if (r >= 0 && r <= n - 1) {
            const int64_t t = (int64_t)(r + ((n - 1 - r) / D) * D) * ud + g.to;
            best = t > best ? t : best;
        }
        const int un = (r >= 0 && (n - 1) % D == r) ? n - 2 : n - 1;   // D >= 2: n - 2 is not owned
        if (un >= 0) {
            const int64_t t = (int64_t)un * ud + g.tn;
            best = t > best ? t : best;
        }
    } else {
        if (r >= 0 && r <= n - 1) {
            const int64_t t = (int64_t)r * ud + g.to;
            best = t > best ? t : best;
        }
        const int un = r == 0 ? 1 : 0;
        if (un <= n - 1) {
            const int64_t t = (int64_t)un * ud + g.tn;
            best = t > best ? t : best;
        }
    }
    return best;
}

// Highest point of a block of stage s with ZeRO, relative to the live bytes
// at its start counted with the largest owned resident (z.rmax): the maximum
// over replicas d of owned(d) - rmax + the highest point of d's own walk
// through the block's segments (edge ops, replayed units and the partial
// unit under recomputation, units, edge ops).  n: units of the block; n_r:
// replayed units.  The block's net bytes do not depend on ownership.
//
// A replica's walk never rises above that of a replica owning none of the
// segments' groups (A), and reaches A unless it owns every unit at which A is
// reached.  Those units have one owner at most (consecutive groups belong to
// different replicas), so every other replica reaches A, the largest of them
// holding the largest owned resident besides that owner's, and only the
// owner's walk needs composing.
template <bool TF>
__device__ int64_t zero_top(const Ctx &x, int s, const ZStage &z, bool bwd, uint64_t m, bool acc, int n, int n_r)
{
    // five fixed slots (pre edge, first / replayed unit, the replay's partial
    // unit, the units, suf edge); absent ones hold no unit (n = 0).  Every
    // index below is a constant, so the list stays in registers.
    constexpr int kSeg = 5;
    ZSeg seg[kSeg];
#pragma unroll
    for (int i = 0; i < kSeg; ++i) seg[i] = ZSeg{0, 0, 0, 0, -1, 1};
    MemZ pre{x, 0, 0, 0, 0}, suf{x, 0, 0, 0, 0};
    record_edges<TF>(x, s, bwd, m, acc, pre, suf);
    int g_pre = -1, g_suf = -1;
    if (TF) {
        if (!bwd && s == 0) g_pre = 0;
        if (!bwd && s == x.P - 1) g_suf = z.g_head;
        if (bwd && s == x.P - 1) g_pre = z.g_head;
    } else if (bwd) {
        g_suf = z.gl_lo;   // the stage's first unit
    }
    seg[0] = ZSeg{1, pre.cur, pre.tn, pre.to, g_pre, 1};
    if (!bwd) {
        MemZ u{x, 0, 0, 0, 0};
        record_unit<TF>(x, false, m, false, u);
        if (x.rc && n >= 1) {
            MemZ f{x, 0, 0, 0, 0};
            record_unit<TF>(x, false, m, false, f, kFwdFirst);
            seg[1] = ZSeg{1, f.cur, f.tn, f.to, z.gl_lo, 1};
            seg[3] = ZSeg{n - 1, u.cur, u.tn, u.to, z.gl_lo + 1, 1};
        } else {
            seg[3] = ZSeg{n, u.cur, u.tn, u.to, z.gl_lo, 1};
        }
    } else {
        if (x.rc) {
            MemZ u{x, 0, 0, 0, 0}, q{x, 0, 0, 0, 0};
            record_unit<TF>(x, false, m, false, u, kFwdReplay);
            record_partial<TF>(x, m, q);
            seg[1] = ZSeg{n_r, u.cur, u.tn, u.to, z.gl_lo, 1};
            seg[2] = ZSeg{1, q.cur, q.tn, q.to, z.gl_hi - 1, 1};
        }
        MemZ u{x, 0, 0, 0, 0};
        record_unit<TF>(x, true, m, acc, u);
        seg[3] = ZSeg{n, u.cur, u.tn, u.to, z.gl_hi - 1, -1};
    }
    seg[4] = ZSeg{1, suf.cur, suf.tn, suf.to, g_suf, 1};
    const int D = x.D;
    // A, and the owner of the units at which it is reached
    int64_t a_none = INT64_MIN, at = 0;
#pragma unroll
    for (int i = 0; i < kSeg; ++i) {
        if (seg[i].n <= 0) continue;
        const int64_t v = at + run_top(seg[i], -1, D);
        a_none = v > a_none ? v : a_none;
        at += (int64_t)seg[i].n * seg[i].d;
    }
    int owner = -1;
    bool shared = false;   // reached where every replica reaches it
    at = 0;
#pragma unroll
    for (int i = 0; i < kSeg; ++i) {
        if (seg[i].n <= 0) continue;
        if (at + run_top(seg[i], -1, D) == a_none) {
            if (seg[i].gs < 0 || (seg[i].d == 0 && seg[i].n >= 2)) {
                shared = true;
            } else {
                int o = (seg[i].gs + seg[i].dir * (seg[i].d > 0 ? seg[i].n - 1 : 0)) % D;
                if (o < 0) o += D;
                shared = shared || (owner >= 0 && owner != o);
                owner = o;
            }
        }
        at += (int64_t)seg[i].n * seg[i].d;
    }
    if (shared || owner < 0) return a_none;
    int64_t t_o = INT64_MIN;
    at = 0;
#pragma unroll
    for (int i = 0; i < kSeg; ++i) {
        if (seg[i].n <= 0) continue;
        const int64_t v = at + run_top(seg[i], owner, D);
        t_o = v > t_o ? v : t_o;
        at += (int64_t)seg[i].n * seg[i].d;
    }
    const int64_t rmax = (int64_t)z.rmax;
    const int64_t others = (int64_t)(owner == z.arg ? z.rsec : z.rmax) - rmax + a_none;
    const int64_t own = (int64_t)z_owned(x, z, owner) - rmax + t_o;
    return others > own ? others : own;
}

// n repetitions of a unit of costs r: the same value as n * 2 * U2n
// sequential fp64 additions, with far fewer dependent steps.
//
// While the clock t stays in one binade [2^e, 2^(e+1)), it is a multiple
// of ulp = 2^(e-52), and rounding t + c to nearest lands on t plus c rounded
// to a multiple of ulp, whatever t is, unless c sits exactly half way
// between two multiples (then ties-to-even depends on t's last bit).  So
// each unit adds the same whole number I of ulps, and q units add q * I
// exactly, as long as t + q * I ulps stays below 2^(e+1).  The unit that
// crosses into the next binade, tiny clocks and the units of a binade in
// which some cost is a half-way case are added op by op.
template <int U2n>
__device__ __forceinline__ double units_seq(const double2 (&r)[U2n], double clk)
{
#pragma unroll
    for (int j = 0; j < U2n; ++j) {
        clk = clk + r[j].x;
        clk = clk + r[j].y;
    }
    return clk;
}

template <int U2n>
__device__ __forceinline__ double units_exact(const double2 (&r)[U2n], double clk, int n)
{
    while (n > 0) {
        // (an overflowed clock, +inf, stays +inf: op by op, n units)
        if (clk >= 0x1p-500 && clk <= 0x1.fffffffffffffp+1023) {
            const int e = ilogb(clk);
            const double sc = ldexp(1.0, 52 - e);
            const double k = clk * sc;                 // integer in [2^52, 2^53)
            const double room = 0x1p53 - k;            // ulps left in the binade
            double part[U2n];
            bool tie = false;
#pragma unroll
            for (int j = 0; j < U2n; ++j) {
                const double tx = r[j].x * sc, ty = r[j].y * sc;
                const double rx = rint(tx), ry = rint(ty);
                tie = tie || fabs(tx - rx) == 0.5 || fabs(ty - ry) == 0.5;
                part[j] = rx + ry;
            }
            // whole numbers: exact while below 2^53 (larger sums cannot fit)
#pragma unroll
            for (int w = 1; w < U2n; w <<= 1)
#pragma unroll
                for (int j = 0; j + w < U2n; j += 2 * w) part[j] = part[j] + part[j + w];
            const double I = part[0];
            if (tie) {
                // op by op until the clock leaves this binade (ties become
                // half as likely with every binade)
                const double top = ldexp(1.0, e + 1);
                for (; n > 0 && clk < top; --n) clk = units_seq(r, clk);
                continue;
            }
            if (I == 0.0) return clk;
            if ((double)n * I <= room - 1.0) return ldexp(k + (double)n * I, e - 52);
            double q = floor((room - 1.0) / I);
            const double rem = fma(-q, I, room - 1.0);   // exact: |rem| < 2^53
            if (rem < 0.0) q -= 1.0;
            else if (rem >= I) q += 1.0;
            if (q > 0.0) {
                clk = ldexp(k + q * I, e - 52);
                n -= (int)q;
            }
        }
        clk = units_seq(r, clk);   // crosses into the next binade (or a tiny clock)
        --n;
    }
    return clk;
}

// the clock part of a block: pre, n units, suf (entry counts per region;
// PST / UST: double2 stride of the edge / unit entries)
template <int P2, int U2n, int S2, int PST, int UST>
__device__ __forceinline__ double walk3(const double2 *pre, const double2 *unit, const double2 *suf, double clk, int n,
                                        bool fast)
{
#pragma unroll
    for (int j = 0; j < P2; ++j) {
        const double2 v = pre[j * PST];
        clk = clk + v.x;
        clk = clk + v.y;
    }
    double2 r[U2n];
#pragma unroll
    for (int j = 0; j < U2n; ++j) r[j] = unit[j * UST];
    if (fast) {
        clk = units_exact(r, clk, n);
    } else {
        for (int u = 0; u < n; ++u) clk = units_seq(r, clk);
    }
#pragma unroll
    for (int j = 0; j < S2; ++j) {
        const double2 v = suf[j * PST];
        clk = clk + v.x;
        clk = clk + v.y;
    }
    return clk;
}

// the first n entries of a unit program (the replay's partial unit)
template <int UST>
__device__ __forceinline__ double walk_prefix(const double2 *unit, int n, double clk)
{
    for (int j = 0; j < n; ++j) {
        const double2 v = unit[(j >> 1) * UST];
        clk = clk + ((j & 1) ? v.y : v.x);
    }
    return clk;
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

// DPP moves within the wavefront: row_shr:n (0x110 + n, lane i of a row of
// 16 receives lane i - n of the same row), row_bcast:15 (0x142, lane 15 of
// each row into the next row; rows 1 and 3 written) and row_bcast:31 (0x143,
// lane 31 into rows 2 and 3).  Rows outside ROWS, and lanes whose source
// lies outside the row, receive 0.
template <int CTRL, int ROWS> __device__ __forceinline__ int dpp(int v)
{
    return __builtin_amdgcn_update_dpp(0, v, CTRL, ROWS, 0xf, true);
}
template <int CTRL, int ROWS> __device__ __forceinline__ double dpp(double v)
{
    return __hiloint2double(dpp<CTRL, ROWS>(__double2hiint(v)), dpp<CTRL, ROWS>(__double2loint(v)));
}

// Inclusive scan by op over the segments of the wavefront: each lane
// combines the values of its segment from the segment's first lane (spos = 0
// there) up to itself.  Rows of 16 lanes scan first, treating a row's first
// lane as a segment start (shift-and-combine over 2^nlev > the largest spos
// positions); then lanes whose segment began in an earlier row take the
// carries, lane 15 of rows 0 and 2 into rows 1 and 3, then lane 31 into rows
// 2 and 3 (cross: some segment spans a row boundary; nlev and cross are
// uniform).  op is exact and associative on the values met, so the result is
// the plain left-to-right one.
template <class T, class Op>
__device__ __forceinline__ T seg_scan(T v, int spos, int lane, int nlev, bool cross, Op op)
{
    const int rl = lane & 15;
    const int sr = spos < rl ? spos : rl;
    T up;
    if (nlev > 0) {
        up = dpp<0x111, 0xf>(v);
        v = sr >= 1 ? op(v, up) : v;
    }
    if (nlev > 1) {
        up = dpp<0x112, 0xf>(v);
        v = sr >= 2 ? op(v, up) : v;
    }
    if (nlev > 2) {
        up = dpp<0x114, 0xf>(v);
        v = sr >= 4 ? op(v, up) : v;
    }
    if (nlev > 3) {
        up = dpp<0x118, 0xf>(v);
        v = sr >= 8 ? op(v, up) : v;
    }
    if (cross) {
        up = dpp<0x142, 0xa>(v);
        v = ((lane & 16) != 0 && spos > rl) ? op(v, up) : v;
        up = dpp<0x143, 0xc>(v);
        v = (lane >= 32 && spos >= lane - 31) ? op(v, up) : v;
    }
    return v;
}

// max of two clocks, which are never NaN or -0.0: the bare instruction
// (fmax would canonicalize both operands first, two more dependent steps)
__device__ __forceinline__ double max_nn(double a, double b)
{
    double r;
    asm("v_max_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}

// The Sends of one slot as prefix scans, exact.
//
// Along a run of linked Sends (positions r = 0, 1, ... in ascending source
// stage), each Send starts at the later of the clock the previous Send left
// on the shared stage and a clock no earlier Send of the run has touched,
// and every stage it joins ends at start + cost:
//   v_r = fl(max(v_{r-1}, z_r) + w_r),
// z_r being the larger of the Send's own two stage clocks before the slot's
// Sends (a stage without a Send that received one from its left carries
// v_{r-1} on; any other position starts the recurrence afresh).  While every
// v stays in the binade [2^E, 2^(E+1)) of the first one, rounding to nearest
// adds each w_r as the whole number W_r of ulps 2^(E-52) nearest to it,
// whatever v is, unless w_r lies exactly half way between two (then ties to
// even depend on v).  In integer ulps K_r = z_r / ulp, with Q_r = W_0 + ... +
// W_r, the recurrence is then v_r = Q_r + max_{i <= r} (K_i - Q_{i-1}): an
// inclusive sum scan and an inclusive max scan, in exact integer-valued fp64
// (below 2^53), over the positions of each segment.  A position that starts
// afresh starts a segment.  Returns false, changing nothing, if some lane
// leaves those conditions (a first value that is 0, not finite or below
// 2^-1022; a cost that is not finite or a half-way case; a result past the
// binade); the caller then walks the Sends step by step.  nlev: scan levels,
// 2^nlev > the largest position.
__device__ __forceinline__ bool send_scan(double &clk, int sdir, double scost, bool from_left, bool from_right,
                                          int lane, int nlev)
{
    const double cl = shr1(clk), cr = shl1(clk);
    const double z = sdir > 0 ? max_nn(clk, cr) : (sdir < 0 ? max_nn(clk, cl) : clk);
    const bool carry = sdir < 0 || from_left;
    const bool involved = sdir != 0 || from_left || from_right;
    const uint64_t starts = ballot(!carry);
    const uint64_t upto = starts & (lane == 63 ? ~0ull : ((2ull << lane) - 1));
    const int spos = lane - (63 - __builtin_clzll(upto));
    bool bad = false;
    int e = INT_MIN;   // the binade of the segment's first value, at its first lane
    if (!carry) {
        e = 0;
        if (involved) {
            bad = !(z > 0.0 && z <= 0x1.fffffffffffffp+1023);
            if (!bad) e = ilogb(z);
            bad = bad || e < -1022;
        }
    }
    const bool cross = ballot(spos > (lane & 15)) != 0;
    e = seg_scan(e, spos, lane, nlev, cross, [](int a, int b) { return a > b ? a : b; });
    const int sh = 52 - e;
    const double K = ldexp(z, sh);
    double w = 0.0;
    if (sdir != 0) {
        const double t = ldexp(scost, sh);
        w = rint(t);
        bad = bad || !(scost >= 0.0 && scost <= 0x1.fffffffffffffp+1023) || fabs(t - w) == 0.5;
    }
    const double q = seg_scan(w, spos, lane, nlev, cross, [](double a, double b) { return a + b; });
    const double y = seg_scan(K - (q - w), spos, lane, nlev, cross, [](double a, double b) { return a > b ? a : b; });
    const double v = q + y;
    bad = bad || (involved && !(v < 0x1p53));
    if (ballot(bad) != 0) return false;
    const double vd = ldexp(v, -sh);
    const double vr = shl1(vd);
    if (from_right) clk = vr;
    else if (sdir != 0 || from_left) clk = vd;
    return true;
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
// a wavefront whose blocks repeat a unit at least this many times sums the
// repeats binade-wise (units_exact), else unit by unit: below it the walk's
// dependent adds cost less than the binade arithmetic
constexpr int kFastUnits = 12;
constexpr int kScanMinRun = 12;   // the last run position from which the Sends take send_scan
constexpr int kKeys = 6;          // forward: 2 row classes; backward: 2 row classes x accumulation
constexpr int kMaxSegShared = 16; // segments of >= 4 lanes per wavefront

// Per-lane programs (segments of 1 or 2 lanes): each lane records its own
// block program per direction, again whenever the microbatch size class or
// the accumulation changes, with the block's composed memory summary.
template <class Sh> struct LdsLane {
    double2 prog[2][Sh::PRE2 + Sh::U2 + Sh::SUF2][kLanes];
    int64_t sum[2][2][kLanes];   // [backward][delta, top][lane]
};
// Shared programs (segments of >= 4 lanes): the repeating unit does not
// depend on the stage, so each segment records the unit of every key once,
// cooperatively; the stage edges stay per lane (transformer: stages 0 and
// P-1 only).
template <class Sh> struct LdsSeg {
    double2 unit[kMaxSegShared][kKeys][Sh::U2];
    int64_t usum[kMaxSegShared][kKeys][2];
    int64_t xsum[kMaxSegShared][2][6];   // recomputation, per forward key: first unit, replay unit, partial
    double2 edge[2][Sh::PRE2 + Sh::SUF2][kLanes];
    int64_t esum[2][4][kLanes];  // [backward][pre delta, pre top, suf delta, suf top][lane]
};

template <class Sh> union LdsNarrow {
    LdsLane<Sh> a;
    LdsSeg<Sh> b;
};

// Wide segments (>= 16 lanes, transformer): at most 4 segments per
// wavefront, and only stages 0 and P-1 have edge ops, so the edge programs
// are kept per segment; middle stages walk a zero program.  About 7 KB.
// Their stages hold few layers, so the kernel adds units one by one: without
// the binade arithmetic's registers four wavefronts share a SIMD.  With the
// overlapped gradient all-reduce the wide kernel keeps that arithmetic (its
// registers are taken anyway) and also takes segments of 8 lanes (8 per
// wavefront, about 14 KB).
// (ZeRO without recomputation moves its 8-lane segments to the wide launch
// too: its narrow kernel holds 48 KB of LDS, three wavefronts per CU)
template <bool OV, bool ZR> constexpr int first_wide_class() { return (OV || ZR) ? 3 : 4; }
inline int first_wide_class(bool ov, bool zr) { return (ov || zr) ? 3 : 4; }
constexpr int64_t kSplitMinCand = 8192;
template <class Sh, int NS> struct LdsWide {
    double2 unit[NS][kKeys][Sh::U2];
    int64_t usum[NS][kKeys][2];
    int64_t xsum[NS][2][6];
    double2 edge[NS][2][2][Sh::PRE2 + Sh::SUF2];   // [segment][stage 0, P-1][backward]
    int64_t esum[NS][2][2][4];
    double2 zero[Sh::PRE2 + Sh::SUF2];
    int64_t zsum[4];
};

// Records a lane-owned block program of one direction (pre, unit, suf
// regions from pp, lane stride kLanes) and its composed memory summary: n
// units; under recomputation the forward block's first unit keeps its input
// and the backward block replays n_r forward units and the partial unit
// after its pre ops.
template <bool TF, class Sh>
__device__ void record_lane(const Ctx &x, int s, bool bwd, uint64_t m, bool acc, int n, int n_r, double2 *pp,
                            int64_t &delta, int64_t &top)
{
    double *base = reinterpret_cast<double *>(pp);
    Record rp{x, base, 2 * kLanes, 0, 0, 0};
    Record ru{x, base + Sh::PRE2 * 2 * kLanes, 2 * kLanes, 0, 0, 0};
    Record rs{x, base + (Sh::PRE2 + Sh::U2) * 2 * kLanes, 2 * kLanes, 0, 0, 0};
    record_edges<TF>(x, s, bwd, m, acc, rp, rs);
    record_unit<TF>(x, bwd, m, acc, ru);
    rp.pad(Sh::PRE2);
    ru.pad(Sh::U2);
    rs.pad(Sh::SUF2);
    int64_t d = 0, t = 0;
    if (!x.rc || (!bwd && n < 1)) {
        compose(rp.cur, rp.top, ru.cur, ru.top, n, rs.cur, rs.top, d, t);
    } else if (!bwd) {
        Mem f{x, 0, 0};
        record_unit<TF>(x, false, m, false, f, kFwdFirst);
        compose_first(rp.cur, rp.top, f.cur, f.top, ru.cur, ru.top, n, rs.cur, rs.top, d, t);
    } else {
        Mem u{x, 0, 0}, q{x, 0, 0};
        record_unit<TF>(x, false, m, false, u, kFwdReplay);
        record_partial<TF>(x, m, q);
        compose(rp.cur, rp.top, u.cur, u.top, n_r, q.cur, q.top, d, t);
        int64_t d2, t2;
        compose(0, 0, ru.cur, ru.top, n, rs.cur, rs.top, d2, t2);
        chain(d, t, d2, t2);
    }
    delta = d;
    top = t;
}

// WIDE: the launch for wide segments of a transformer; otherwise every class
// of an MLP, or the narrow classes of a transformer.  RC: training with
// activation recomputation; ZR: training with ZeRO; OV: training with the
// gradient all-reduce on the communication streams (separate instantiations
// keep the replay, the broadcasts and the two-stream walk out of the other
// kernels).
// The kernel's argument block (its only argument, at offset 0 of the
// kernarg segment), addressed through a pointer the compiler cannot see
// through.  The recording paths inside the slot loop and the weight update
// after it read the model and the device constants through it: those values
// are then loaded again with scalar loads where they are needed instead of
// being kept live across the loop, where they would not fit the scalar
// registers and would be spilled to vector-register lanes and read back in
// every slot.
template <class T> __device__ __forceinline__ const __attribute__((address_space(4))) T *kernel_args()
{
    auto p = (const __attribute__((address_space(4))) T *)__builtin_amdgcn_kernarg_segment_ptr();
    asm volatile("" : "+s"(p));
    return p;
}

template <bool TF, bool WIDE, bool RC, bool ZR, bool OV>
__device__ __forceinline__ void parametric_body(const ParArgs &g)
{
    using Sh = Shape<TF, ZR>;
    constexpr int PST = WIDE ? 1 : kLanes;   // double2 stride of a lane's edge program
    // at most 64 / 2^(first wide class) segments per wide wavefront
    __shared__ typename std::conditional<WIDE, LdsWide<Sh, (kLanes >> first_wide_class<OV, ZR && !RC>())>, LdsNarrow<Sh>>::type L;

    const int lane = threadIdx.x;
    // the binade-wise unit sums: not in the wide kernels (but in the one
    // with the overlapped all-reduce, whose registers it does not raise)
    constexpr bool kBinadeSums = !WIDE || OV;
    // Wavefronts start longest first, so that short ones fill the tail: the
    // wide launch in the pre-pass's order (by the estimated length of each
    // wavefront), the only launch widest class first, each class from its
    // last wavefront (the strategy grid lists microbatch counts ascending).
    // The narrow launch beside a wide one runs in lane order.  The grid is
    // sized for the worst case; wavefronts beyond the launch's own exit.
    uint32_t blk = 0xffffffffu;
    if constexpr (WIDE) {
        const uint32_t n_wide = (g.meta[16 + kClasses] - g.meta[16 + first_wide_class<OV, ZR && !RC>()]) / (uint32_t)kLanes;
        if (blockIdx.x < n_wide) blk = g.order[blockIdx.x];
    } else {
        const uint32_t nw = g.meta[16 + kClasses] / (uint32_t)kLanes;   // wavefronts holding classes
        if (blockIdx.x < nw) blk = g.narrow_end == kClasses ? nw - 1 - blockIdx.x : blockIdx.x;
    }
    if (blk == 0xffffffffu) return;
    const uint32_t gl = blk * (uint32_t)kLanes;
    int cls = 0;
    while (cls + 1 < kClasses && gl >= g.meta[16 + cls + 1]) ++cls;
    if (WIDE ? cls < first_wide_class<OV, ZR && !RC>() : cls >= g.narrow_end) return;   // the other launch's classes
    const int W = 1 << cls;
    const bool shared = WIDE || W >= 4;
    const uint32_t local = gl + lane - g.meta[16 + cls];
    const uint32_t slot = local >> cls;
    const int s = (int)(local & (uint32_t)(W - 1));   // stage of this lane
    const int seg = lane >> cls;
    const int64_t c = slot < g.meta[cls] ? (int64_t)g.perm[g.meta[8 + cls] + slot] : -1;

    const dsim_model &M = g.m;
    dsim_strategy st = {1, 1, 1, 1};
    bool ok = false;
    if (c >= 0) {
        st = g.cand[c];
        ok = strategy_ok(M, st.D, st.H, st.P, st.K) && st.P <= g.p_bound && st.P <= W && st.K <= kMaxK &&
             placement_ok(g.c.node, st.D, st.H);
    }
    const int P = ok ? st.P : 0, K = st.K;
    const bool train = M.mode != DSIM_INFER;
    bool live_stage = s < P;
    int32_t status = (c >= 0 && !ok) ? DSIM_ST_BAD_STRATEGY : 0;

    double clk = 0.0;
    double clkm = 0.0;   // overlap: the communication stream's clock
    const bool ov_c = OV && train && M.overlap != 0 && st.D > 1;
    int64_t live = 0, peak = 0;
    uint64_t walked = 0, nops = 0;
    uint64_t mq = 0, rb_f = 0, rb_b = 0;   // rows of a short microbatch; Send bytes per row
    int pos = 0, nf = 0, nb = 0, len = 0, mr = 0, n_f = 0, n_b = 0;
    constexpr bool rc = RC;   // the launch checks it against the model
    int n_r = 0, n_part = 0;                     // replayed units, entries of the partial unit
    // ZeRO: the highest point of every block kind over the stage's replicas
    const bool zero_c = ZR && train && M.zero != 0 && st.D > 1;
    __shared__ int64_t s_ztop[ZR ? kKeys : 1][kLanes];
    if (live_stage) {
        Ctx x = {};
        make_ctx(M, g.c, st, x);
        x.mlp = !TF;   // the family is uniform per launch: compiles out the other
        uint64_t res0;
        ZStage zs;
        if (ZR && x.zero) {
            z_stage(x, s, zs);
            res0 = resident_inputs(x, s) + zs.rmax;
        } else {
            res0 = resident(x, s);
        }
        Walk w{x, 0.0, (int64_t)res0, 0, 0, 0, nullptr};
        w.peak = w.live;
        // microbatch splits before the pipeline
        if (x.K > 1) {
            if (s == 0) split(x, w);
            if (x.train && s == x.P - 1) split(x, w);
        }
        clk = w.clk;
        live = w.live;
        peak = w.peak;
        walked = w.walked;
        nops = w.nops;
        len = train ? 2 * K : K;
        mq = x.mq;
        mr = (int)x.mr;
        n_f = block_units(M, P, st.H, s, false, TF);
        n_b = block_units(M, P, st.H, s, true, TF);
        if (rc) {
            const int nl = stage_nl(x, s);
            n_r = TF ? nl - 1 : nl / (st.H > 1 ? 2 : 1) - 1;
            Count c{x, 0, 0};
            record_partial<TF>(x, 1, c);
            n_part = (int)c.walked;
        }
        if constexpr (ZR) {
            if (zero_c) {
                // all six kinds up front: every lane of the wavefront at once
                for (int key = 0; key < kKeys; ++key) {
                    const bool bwd = key >= 2;
                    const int mc = bwd ? ((key - 2) & 1) : key;
                    s_ztop[key][lane] = zero_top<TF>(x, s, zs, bwd, x.mq + (uint64_t)mc, key >= 4, bwd ? n_b : n_f, n_r);
                }
            }
        }
        uint64_t sz, fre;
        send_size(x, s, 1, false, sz, fre);
        rb_f = sz;
        send_size(x, s, 1, true, sz, fre);
        rb_b = sz;
        if constexpr (!WIDE) {
            if (shared) {
                // empty edges unless a later record fills them
                for (int d = 0; d < 2; ++d) {
                    Record e{x, reinterpret_cast<double *>(&L.b.edge[d][0][lane]), 2 * kLanes, 0, 0, 0};
                    e.pad(Sh::PRE2 + Sh::SUF2);
                    for (int f = 0; f < 4; ++f) L.b.esum[d][f][lane] = 0;
                }
            }
        }
    }
    if (shared) {
        if (ok) {
            Ctx x = {};
            make_ctx(kernel_args<ParArgs>()->m, kernel_args<ParArgs>()->c, st, x);
            x.mlp = !TF;
            for (int key = s; key < kKeys; key += W) {
                const bool bwd = key >= 2;
                const int mc = bwd ? ((key - 2) & 1) : key;
                double2 *u;
                int64_t *us;
                if constexpr (WIDE) {
                    u = &L.unit[seg][key][0];
                    us = &L.usum[seg][key][0];
                } else {
                    u = &L.b.unit[seg][key][0];
                    us = &L.b.usum[seg][key][0];
                }
                Record r{x, reinterpret_cast<double *>(u), 2, 0, 0, 0};
                const uint64_t m = x.mq + (uint64_t)mc;
                record_unit<TF>(x, bwd, m, key >= 4, r);
                r.pad(Sh::U2);
                us[0] = r.cur;
                us[1] = r.top;
                if (rc && !bwd) {
                    int64_t *xs;
                    if constexpr (WIDE) xs = &L.xsum[seg][key][0];
                    else xs = &L.b.xsum[seg][key][0];
                    Mem f{x, 0, 0}, u2{x, 0, 0}, q{x, 0, 0};
                    record_unit<TF>(x, false, m, false, f, kFwdFirst);
                    record_unit<TF>(x, false, m, false, u2, kFwdReplay);
                    record_partial<TF>(x, m, q);
                    xs[0] = f.cur;
                    xs[1] = f.top;
                    xs[2] = u2.cur;
                    xs[3] = u2.top;
                    xs[4] = q.cur;
                    xs[5] = q.top;
                }
            }
        }
        if constexpr (WIDE) {
            if (lane < Sh::PRE2 + Sh::SUF2) L.zero[lane] = make_double2(0.0, 0.0);
            if (lane < 4) L.zsum[lane] = 0;
        }
        __syncthreads();
    }
    int key_f = -1, key_b = -1;   // key each lane-owned program was recorded for

    for (;;) {
        const bool active = live_stage && pos < len;
        const uint64_t act_mask = ballot(active);
        if (act_mask == 0) break;
        const int nf_left = shr1(nf), nb_right = shl1(nb);   // slot-start counters
        bool bwd = false, ready = false;
        int k = 0;
        if (active) {
            // forward-only / GPipe / synchronous 1F1B position -> (direction, microbatch)
            if (!train) {
                k = pos;
            } else if (M.schedule == DSIM_SCHED_GPIPE) {
                bwd = pos >= K;
                k = bwd ? pos - K : pos;
            } else {
                const int wu = (P - 1 - s) < K ? (P - 1 - s) : K;
                if (pos < wu) {
                    k = pos;
                } else if (pos < wu + 2 * (K - wu)) {
                    const int j = pos - wu;
                    bwd = (j & 1) != 0;
                    k = bwd ? (j - 1) / 2 : wu + j / 2;
                } else {
                    bwd = true;
                    k = pos - wu - (K - wu);
                }
            }
            ready = !bwd ? (s == 0 || nf_left > k) : (s == P - 1 ? nf > k : nb_right > k);
        }
        const uint64_t rdy_mask = ballot(ready);
        const uint64_t segmask = W == 64 ? ~0ull : (((1ull << W) - 1) << (lane & ~(W - 1)));
        if ((act_mask & segmask) != 0 && (rdy_mask & segmask) == 0) {
            // no stage can proceed: impossible for 1F1B, stops the candidate
            status |= DSIM_ST_BAD_STRATEGY;
            live_stage = false;
        }
        const bool all_fwd = ballot(ready && bwd) == 0;

        // long unit runs take the binade-wise path (uniform per wavefront)
        const bool fast = kBinadeSums && ballot(ready && (bwd ? n_b : n_f) >= kFastUnits) != 0;
        // under recomputation a wave with backward blocks walks the pre ops
        // and the replay first (forward lanes: their pre ops, no units), then
        // every lane's units and suf
        const bool replay = rc && !all_fwd;
        const bool fast_r = kBinadeSums && replay && ballot(ready && bwd && n_r >= kFastUnits) != 0;
        const int d = bwd ? 1 : 0;
        const int mc = k < mr ? 1 : 0;
        const uint64_t m = mq + (uint64_t)mc;
        if (ready) {
            const bool acc = bwd && k >= 1;
            const int key = bwd ? 2 + mc + (acc ? 2 : 0) : mc;
            const int n = bwd ? n_b : n_f;
            const int nr = bwd ? n_r : 0, np = bwd ? n_part : 0;
            int64_t delta = 0, top = 0;
            bool lane_done = false;
            if constexpr (OV) {
                if (ov_c && bwd && k == K - 1) {
                    // the last backward block under overlap hands each
                    // finished gradient to the communication stream: walked
                    // op by op with both clocks, memory as it goes
                    Ctx x = {};
                    make_ctx(kernel_args<ParArgs>()->m, kernel_args<ParArgs>()->c, st, x);
                    x.mlp = !TF;
                    Walk w{x, clk, live, live, 0, 0, nullptr};
                    w.tm = clkm;
                    block_bwd(x, w, s, k);
                    clk = w.clk;
                    clkm = w.tm;
                    delta = w.live - live;
                    top = w.peak - live;
                    lane_done = true;
                }
            }
            if constexpr (!WIDE) {
                if (!shared && !lane_done) {
                    double2 *pp = &L.a.prog[d][0][lane];
                    if ((bwd ? key_b : key_f) != key || (replay && bwd && key_f != mc)) {
                        Ctx x = {};
                        make_ctx(kernel_args<ParArgs>()->m, kernel_args<ParArgs>()->c, st, x);
                        x.mlp = !TF;
                        if ((bwd ? key_b : key_f) != key) {
                            record_lane<TF, Sh>(x, s, bwd, m, acc, n, n_r, pp, L.a.sum[d][0][lane], L.a.sum[d][1][lane]);
                            if (bwd) key_b = key;
                            else key_f = key;
                        }
                        if (replay && bwd && key_f != mc) {   // the replay walks the forward unit of this size
                            record_lane<TF, Sh>(x, s, false, m, false, n_f, n_r, &L.a.prog[0][0][lane], L.a.sum[0][0][lane],
                                            L.a.sum[0][1][lane]);
                            key_f = mc;
                        }
                    }
                    const double2 *up = pp + Sh::PRE2 * kLanes, *sp = pp + (Sh::PRE2 + Sh::U2) * kLanes;
                    if (replay) {
                        const double2 *fu = &L.a.prog[0][Sh::PRE2][lane];
                        clk = walk3<Sh::PRE2, Sh::F_U2, 0, kLanes, kLanes>(pp, fu, nullptr, clk, nr, fast_r);
                        clk = walk_prefix<kLanes>(fu, np, clk);
                        clk = walk3<0, Sh::U2, Sh::SUF2, kLanes, kLanes>(nullptr, up, sp, clk, n, fast);
                    } else if (all_fwd) {
                        clk = walk3<Sh::F_PRE2, Sh::F_U2, Sh::F_SUF2, kLanes, kLanes>(pp, up, sp, clk, n, fast);
                    } else {
                        clk = walk3<Sh::PRE2, Sh::U2, Sh::SUF2, kLanes, kLanes>(pp, up, sp, clk, n, fast);
                    }
                    delta = L.a.sum[d][0][lane];
                    top = L.a.sum[d][1][lane];
                    lane_done = true;
                }
            }
            if (!lane_done) {
                // edge program and summary of this lane and direction
                const bool has_edges = !TF || s == 0 || s == P - 1;
                double2 *ep;
                int64_t *es;
                int es_stride;
                if constexpr (WIDE) {
                    const int slot = s == 0 ? 0 : 1;
                    ep = has_edges ? &L.edge[seg][slot][d][0] : &L.zero[0];
                    es = has_edges ? &L.esum[seg][slot][d][0] : &L.zsum[0];
                    es_stride = 1;
                } else {
                    ep = &L.b.edge[d][0][lane];
                    es = &L.b.esum[d][0][lane];
                    es_stride = kLanes;
                }
                // transformer edges sit on stages 0 and P-1 only; every MLP
                // stage ends its backward with its first unit
                if (has_edges && (bwd ? key_b : key_f) != key) {
                    Ctx x = {};
                    make_ctx(kernel_args<ParArgs>()->m, kernel_args<ParArgs>()->c, st, x);
                    x.mlp = !TF;
                    double *base = reinterpret_cast<double *>(ep);
                    Record rp{x, base, 2 * PST, 0, 0, 0};
                    Record rs{x, base + Sh::PRE2 * 2 * PST, 2 * PST, 0, 0, 0};
                    record_edges<TF>(x, s, bwd, m, acc, rp, rs);
                    rp.pad(Sh::PRE2);
                    rs.pad(Sh::SUF2);
                    es[0 * es_stride] = rp.cur;
                    es[1 * es_stride] = rp.top;
                    es[2 * es_stride] = rs.cur;
                    es[3 * es_stride] = rs.top;
                    if (bwd) key_b = key;
                    else key_f = key;
                }
                const double2 *up, *fu, *sp = ep + Sh::PRE2 * PST;
                const int64_t *us, *xs;
                if constexpr (WIDE) {
                    up = &L.unit[seg][key][0];
                    us = &L.usum[seg][key][0];
                    fu = &L.unit[seg][mc][0];
                    xs = &L.xsum[seg][mc][0];
                } else {
                    up = &L.b.unit[seg][key][0];
                    us = &L.b.usum[seg][key][0];
                    fu = &L.b.unit[seg][mc][0];
                    xs = &L.b.xsum[seg][mc][0];
                }
                if (replay) {
                    clk = walk3<Sh::PRE2, Sh::F_U2, 0, PST, 1>(ep, fu, nullptr, clk, nr, fast_r);
                    clk = walk_prefix<1>(fu, np, clk);
                    clk = walk3<0, Sh::U2, Sh::SUF2, PST, 1>(nullptr, up, sp, clk, n, fast);
                } else if (all_fwd) {
                    clk = walk3<Sh::F_PRE2, Sh::F_U2, Sh::F_SUF2, PST, 1>(ep, up, sp, clk, n, fast);
                } else {
                    clk = walk3<Sh::PRE2, Sh::U2, Sh::SUF2, PST, 1>(ep, up, sp, clk, n, fast);
                }
                const int64_t pd = es[0], pt = es[1 * es_stride], sd = es[2 * es_stride], st2 = es[3 * es_stride];
                if (!rc) {
                    compose(pd, pt, us[0], us[1], n, sd, st2, delta, top);
                } else if (!bwd) {
                    compose_first(pd, pt, xs[0], xs[1], us[0], us[1], n, sd, st2, delta, top);
                } else {
                    compose(pd, pt, xs[2], xs[3], n_r, xs[4], xs[5], delta, top);
                    int64_t d2, t2;
                    compose(0, 0, us[0], us[1], n, sd, st2, d2, t2);
                    chain(delta, top, d2, t2);
                }
            }
            if constexpr (ZR) {
                // the net bytes do not depend on ownership; the highest point does
                if (zero_c) top = s_ztop[key][lane];
            }
            const int64_t hi = live + top;
            peak = hi > peak ? hi : peak;
            live += delta;
            ++pos;
            if (bwd) ++nb;
            else ++nf;
        }

        // the slot's sends, ascending by source stage
        int sdir = 0;
        double scost = 0.0;
        uint64_t ssz = 0, sfre = 0;
        if (ready && ((!bwd && s < P - 1) || (bwd && s > 0))) {
            sdir = bwd ? -1 : 1;
            ssz = m * (bwd ? rb_b : rb_f);
            sfre = (TF || bwd || !train) ? ssz : 0;
            const bool net = send_spans(g.c.node, st.D, st.H, s, bwd ? s - 1 : s + 1);
            scost = (net ? g.c.net_lat : g.c.lat) + (double)ssz * (net ? g.c.net_inv_l : g.c.inv_l);
        }
        const int l_dir = shr1(sdir), r_dir = shl1(sdir);
        const double l_cost = shr1(scost), r_cost = shl1(scost);
        const uint64_t l_sz = shr1(ssz), r_sz = shl1(ssz);
        const bool from_left = live_stage && s >= 1 && l_dir == 1;
        const bool from_right = live_stage && s + 1 < P && r_dir == -1;
        // Send s depends on send s-1 only if s-1 went forward (it moved clock
        // s) or s goes backward (it reads clock s-1); elsewhere the chain
        // splits into runs that touch disjoint clocks and proceed in parallel.
        // rpos = position of the stage in its run.
        const bool linked = s >= 1 && s < P && (l_dir == 1 || sdir == -1);
        const uint64_t starts = ballot(!linked);
        const uint64_t upto = starts & (lane == 63 ? ~0ull : ((2ull << lane) - 1));
        const int rpos = lane - (63 - __builtin_clzll(upto));
        // the last run position of the wave (a position without a Send
        // changes nothing: its receivers need a sender there)
        int last = 0;
        for (int b = 32; b >= 1; b >>= 1)
            if (ballot(rpos >= last + b) != 0) last += b;
        // long runs (pipeline fill and drain) take the scans, short ones the steps
        if (last < kScanMinRun || !send_scan(clk, sdir, scost, from_left, from_right, lane, 32 - __clz(last))) {
        for (int r = 0; r <= last; ++r) {
            const bool src = rpos == r && sdir != 0;
            const double cl = shr1(clk), cr = shl1(clk);
            const bool tl = rpos == r + 1 && from_left;
            const bool tr = rpos == r - 1 && from_right;
            const double a = ((src && sdir < 0) || tl) ? cl : cr;
            // clocks are sums of costs >= 0 from +0.0: never NaN or -0.0,
            // so the bare maximum instruction gives the larger value (fmax
            // would first canonicalize both operands)
            const double e = max_nn(a, clk) + (src ? scost : (tl ? l_cost : r_cost));
            if (src || tl || tr) clk = e;
        }
        }
        if (live_stage) {
            if (from_left) {
                live += (int64_t)l_sz;
                peak = live > peak ? live : peak;
            }
            if (sdir != 0) live -= (int64_t)sfre;
            if (from_right) {
                live += (int64_t)r_sz;
                peak = live > peak ? live : peak;
            }
        }
    }
    if (live_stage && status == 0) {
        Ctx x = {};
        // (the narrow kernels and the wide ZeRO one keep these values live
        // across the loop instead: reading the argument block again here
        // makes the register allocator reserve a private frame in them that
        // no instruction uses)
        if constexpr (WIDE && !(ZR && !RC))
            make_ctx(kernel_args<ParArgs>()->m, kernel_args<ParArgs>()->c, st, x);
        else
            make_ctx(M, g.c, st, x);
        x.mlp = !TF;
        ZStage zs;
        if (ZR && x.zero) z_stage(x, s, zs);
        Walk w{x, clk, live, peak, walked, nops, &zs};
        w.tm = clkm;
        if (train) weight_update(x, w, s);
        // the stage's latest device (under overlap the computation stream
        // ends last: its final op is an optimizer step after a hand-back)
        clk = w.clk > w.tm ? w.clk : w.tm;
        live = w.live;
        peak = w.peak;
        walked = w.walked;
        nops = w.nops;
        count_blocks(x, s, walked, nops);
    }

    // per-candidate results: reductions over the segment
    const bool contributes = s < P && status == 0;
    const double mk = seg_reduce(contributes ? clk : 0.0, W, [](double a, double b) { return a > b ? a : b; });
    const uint64_t cp = seg_reduce(contributes ? (uint64_t)peak : 0ull, W,
                                   [](uint64_t a, uint64_t b) { return a > b ? a : b; });
    const uint64_t tops = seg_reduce(contributes ? nops : 0ull, W, [](uint64_t a, uint64_t b) { return a + b; });
    const uint64_t twalk = seg_reduce(contributes ? walked : 0ull, W, [](uint64_t a, uint64_t b) { return a + b; });
    status = seg_reduce(status, W, [](int32_t a, int32_t b) { return a | b; });
    if (c < 0) return;
    const bool valid = status == 0;
    if (s == 0) {
        int32_t stt = status;
        if (valid && g.c.cap != 0 && cp > g.c.cap) stt |= DSIM_ST_OVER_CAP;
        g.makespan[c] = valid ? mk : 0.0;
        g.cand_peak[c] = valid ? cp : 0;
        g.status[c] = stt;
        if (g.n_ops) g.n_ops[c] = valid ? tops : 0;
        if (g.walked) g.walked[c] = valid ? twalk : 0;
    }
    const bool mine = valid && s < P;
    if (g.finish) {
        double *row = g.finish + (size_t)c * g.row_width;
        for (int j = s; j < g.row_width; j += W) row[j] = (mine && j == s) ? clk : 0.0;
    }
    if (g.peak) {
        uint64_t *row = g.peak + (size_t)c * g.row_width;
        for (int j = s; j < g.row_width; j += W) row[j] = (mine && j == s) ? (uint64_t)peak : 0;
    }
}

template <bool TF, bool RC, bool ZR, bool OV>
__global__ __launch_bounds__(kLanes) void k_parametric(const ParArgs g)
{
    parametric_body<TF, false, RC, ZR, OV>(g);
}

// wide segments of a transformer: two wavefronts per SIMD
template <bool RC, bool ZR, bool OV>
__global__ __launch_bounds__(kLanes) __attribute__((amdgpu_waves_per_eu(2))) void k_parametric_wide(const ParArgs g)
{
    parametric_body<true, true, RC, ZR, OV>(g);
}

// the kernel of a launch, by family, width class and model options
template <bool RC, bool ZR, bool OV>
void launch_variant(bool tf, bool wide, dim3 grid, dim3 block, hipStream_t s, const ParArgs &g)
{
    if (!tf) hipLaunchKernelGGL((k_parametric<false, RC, ZR, OV>), grid, block, 0, s, g);
    else if (!wide) hipLaunchKernelGGL((k_parametric<true, RC, ZR, OV>), grid, block, 0, s, g);
    else hipLaunchKernelGGL((k_parametric_wide<RC, ZR, OV>), grid, block, 0, s, g);
}

// (ZeRO and overlap exclude one another)
void launch_kernel(bool rc, bool zr, bool ov, bool tf, bool wide, dim3 grid, dim3 block, hipStream_t s,
                   const ParArgs &g)
{
    if (rc) {
        if (zr) launch_variant<true, true, false>(tf, wide, grid, block, s, g);
        else if (ov) launch_variant<true, false, true>(tf, wide, grid, block, s, g);
        else launch_variant<true, false, false>(tf, wide, grid, block, s, g);
    } else {
        if (zr) launch_variant<false, true, false>(tf, wide, grid, block, s, g);
        else if (ov) launch_variant<false, false, true>(tf, wide, grid, block, s, g);
        else launch_variant<false, false, false>(tf, wide, grid, block, s, g);
    }
}

// ---------------------------------------------------------------------------
// Pre-pass: stable counting sort of the candidates by segment class, and the
// order in which the wide launch's wavefronts start
// ---------------------------------------------------------------------------
// A slot's fixed work (schedule, Sends, memory updates) costs about as much
// as walking this many layers of a transformer stage.
constexpr uint32_t kSlotLayers = 8;

// Relative length of the wavefront that simulates a candidate: slots (the
// stage's blocks plus the pipeline's fill and drain) times the work of a
// slot (a fixed part and the stage's share of the layers), in half layers.
// Only orders the wide launch's wavefronts.
__device__ __forceinline__ uint32_t wave_length(const dsim_strategy &st, int n_layers, bool train)
{
    const uint32_t P = (uint32_t)(st.P < 1 ? 1 : (st.P > kMaxStages ? kMaxStages : st.P));
    const uint32_t K = (uint32_t)(st.K < 1 ? 1 : (st.K > kMaxK ? kMaxK : st.K));
    const uint32_t L = (uint32_t)(n_layers < 1 ? 1 : (n_layers > 65536 ? 65536 : n_layers));
    const uint32_t slots = (train ? 2u : 1u) * K + 2u * P;      // <= 32,894
    const uint32_t work = 2u * kSlotLayers + (2u * L + P - 1) / P;   // <= 131,088
    const uint64_t len = (uint64_t)slots * work;
    return len > 0xffffffffu ? 0xffffffffu : (uint32_t)len;
}

// (wave_len, when given: n + 8 words cleared for k_class_scatter)
__global__ __launch_bounds__(kScanBlock) void k_class_count(const dsim_strategy *cand, int64_t n, int p_bound,
                                                           uint32_t *counts, uint32_t *wave_len)
{
    __shared__ uint32_t s_cnt[8];
    if (threadIdx.x < 8) s_cnt[threadIdx.x] = 0;
    __syncthreads();
    const int64_t c = (int64_t)blockIdx.x * kScanBlock + threadIdx.x;
    if (wave_len) {
        if (c < n) wave_len[c] = 0;
        if (c < 8) wave_len[n + c] = 0;
    }
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

// wave_length quantized: 16 steps per doubling
constexpr int kLenBuckets = 512;
constexpr int kOrderBlock = 1024;
__device__ __forceinline__ int len_bucket(uint32_t len)
{
    if (len == 0) return 0;
    const int e = 31 - __clz(len);
    const uint32_t f = e >= 4 ? (len >> (e - 4)) & 15u : (len << (4 - e)) & 15u;
    return e * 16 + (int)f;
}

// The wide launch's wavefronts longest first: a counting sort of
// wave_len (each wavefront's longest candidate, from k_class_scatter) over
// len_bucket, wavefronts of one bucket in any order.  One block.
__global__ __launch_bounds__(kOrderBlock) void k_wave_order(const uint32_t *meta, int narrow_end,
                                                           const uint32_t *wave_len, uint32_t *order)
{
    __shared__ uint32_t s_cnt[kLenBuckets];
    const int t = threadIdx.x;
    const uint32_t w_lo = meta[16 + narrow_end] / (uint32_t)kLanes, w_hi = meta[16 + kClasses] / (uint32_t)kLanes;
    const uint32_t n_w = w_hi - w_lo;
    for (int i = t; i < kLenBuckets; i += kOrderBlock) s_cnt[i] = 0;
    __syncthreads();
    for (uint32_t i = t; i < n_w; i += kOrderBlock) atomicAdd(&s_cnt[len_bucket(wave_len[i])], 1u);
    __syncthreads();
    if (t == 0) {   // bucket starts, longest bucket first
        uint32_t pos = 0;
        for (int i = kLenBuckets - 1; i >= 0; --i) {
            const uint32_t k = s_cnt[i];
            s_cnt[i] = pos;
            pos += k;
        }
    }
    __syncthreads();
    for (uint32_t i = t; i < n_w; i += kOrderBlock) order[atomicAdd(&s_cnt[len_bucket(wave_len[i])], 1u)] = w_lo + i;
}

// (wave_len, when given: each wide wavefront's longest wave_length, the
// wavefronts counted from the first wide one, class narrow_end)
__global__ __launch_bounds__(kScanBlock) void k_class_scatter(const dsim_strategy *cand, int64_t n, int p_bound,
                                                             const uint32_t *offsets, const uint32_t *meta,
                                                             uint32_t *perm, int narrow_end, int n_layers,
                                                             bool train, uint32_t *wave_len)
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
        const uint32_t slot = offsets[(size_t)blockIdx.x * 8 + j] + rank;
        perm[meta[8 + j] + slot] = (uint32_t)c;
        if (wave_len && j >= narrow_end) {
            const uint32_t w = (meta[16 + j] + (slot << j)) / (uint32_t)kLanes - meta[16 + narrow_end] / (uint32_t)kLanes;
            atomicMax(&wave_len[w], wave_length(cand[c], n_layers, train));
        }
    }
}

}  // namespace

// Scratch of dsim_simulate_parametric_static: the grouping workspace of at
// most kStaticMaxCand candidates, one copy per GPU for the whole process.
// Host code never uses this name as an address; it takes the device address
// once per GPU (static_scratch).
constexpr int64_t kStaticMaxCand = (int64_t)1 << 20;
constexpr int64_t kStaticWords = (kStaticMaxCand / kScanBlock) * 8 + 32 + 3 * kStaticMaxCand + 16;
static __device__ __align__(256) uint32_t scratch[kStaticWords];

dsim_status static_scratch(void **out)
{
    static std::mutex mu;
    static void *addr[kMaxGpus] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "parametric (static): current device");
    if (dev < 0 || dev >= kMaxGpus) return fail(DSIM_ERANGE, "parametric (static): device %d beyond %d", dev, kMaxGpus);
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) return hip_fail(e, "parametric (static): scratch address");
        addr[dev] = p;
    }
    *out = addr[dev];
    return DSIM_OK;
}

int64_t static_max_cand() { return kStaticMaxCand; }

size_t parametric_workspace(int64_t n_cand)
{
    const int64_t nb = (n_cand + kScanBlock - 1) / kScanBlock;
    // per-block class counts, the class table (32 words), the permutation,
    // the wide launch's wavefront order and lengths (at most n_cand +
    // kClasses wavefronts each)
    return (size_t)(nb * 8 + 32 + 3 * n_cand + 16) * sizeof(uint32_t);
}

dsim_status launch_parametric(const dsim_model &m, const dsim_strategy *cand, int64_t n_cand, const CostConsts &c,
                              const dsim_results &r, void *ws, hipStream_t s, hipStream_t side)
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
    // one dispatch covers every class at the widest segment: its work-item
    // count (a 32-bit field) bounds the call
    if ((n_cand * wmax + kLanes - 1) / kLanes + kClasses > (int64_t)(0xffffffffu / kLanes))
        return fail(DSIM_ERANGE, "parametric: n_cand * %d lanes (the widest segment for row_width %d) exceed one "
                                 "dispatch; split the call", wmax, pb);
    g.makespan = r.makespan;
    g.finish = r.finish;
    g.peak = r.peak;
    g.cand_peak = r.cand_peak;
    g.n_ops = r.n_ops;
    g.walked = r.walked_ops;
    g.status = r.status;
    g.c = ParConsts{c.inv_f, c.inv_b, c.inv_l, c.lat, c.launch, c.cap, c.mm, c.mm_c0, c.mm_c1, c.mm_c2,
                    c.mm_c3, c.mm_floor, c.node, c.net_lat, c.net_inv_l, c.streams, c.st_lat, c.st_inv_l};

    // workspace: per-block class counts, class table, permutation, wide
    // wavefront order and lengths (every word is written before it is read:
    // the caller clears nothing)
    const int64_t nb = (n_cand + kScanBlock - 1) / kScanBlock;
    uint32_t *counts = static_cast<uint32_t *>(ws);
    uint32_t *meta = counts + (size_t)nb * 8;
    uint32_t *perm = meta + 32;
    uint32_t *order = perm + n_cand;
    uint32_t *wave_len = order + n_cand + 8;
    g.perm = perm;
    g.order = order;
    g.meta = meta;

    // A large transformer grid splits: the narrow classes run beside the
    // wide ones (whose smaller LDS footprint lets two wavefronts share a
    // SIMD) when the caller gives a second stream, else after them on the
    // one stream.  Small grids and MLPs take one launch for every class.
    const bool split = m.family == DSIM_TRANSFORMER && n_cand >= kSplitMinCand;
    const bool zr_only = m.mode != DSIM_INFER && m.zero != 0 && m.recompute == 0;
    g.narrow_end = split ? first_wide_class(m.mode != DSIM_INFER && m.overlap != 0, zr_only) : kClasses;

    hipLaunchKernelGGL(k_class_count, dim3((unsigned)nb), dim3(kScanBlock), 0, s, cand, n_cand, pb, counts,
                       split ? wave_len : nullptr);
    hipLaunchKernelGGL(k_class_scan, dim3(1), dim3(kScanBlock), 0, s, counts, nb, meta);
    hipLaunchKernelGGL(k_class_scatter, dim3((unsigned)nb), dim3(kScanBlock), 0, s, cand, n_cand, pb,
                       (const uint32_t *)counts, (const uint32_t *)meta, perm, g.narrow_end, m.n_layers,
                       m.mode != DSIM_INFER, split ? wave_len : nullptr);
    if (split)
        hipLaunchKernelGGL(k_wave_order, dim3(1), dim3(kOrderBlock), 0, s, (const uint32_t *)meta, g.narrow_end,
                           (const uint32_t *)wave_len, order);
    // every class's lanes round up to whole wavefronts: at most one partial
    // wavefront per class beyond n * wmax lanes
    const int64_t waves = (n_cand * wmax + kLanes - 1) / kLanes + kClasses;
    const bool rc = m.mode != DSIM_INFER && m.recompute != 0;
    const bool zr = m.mode != DSIM_INFER && m.zero != 0;
    const bool ov = m.mode != DSIM_INFER && m.overlap != 0;
    const bool tf = m.family == DSIM_TRANSFORMER;
    const dim3 grid((unsigned)waves), block(kLanes);
    hipError_t e = hipSuccess;
    if (!split) {
        launch_kernel(rc, zr, ov, tf, false, grid, block, s, g);
        e = hipGetLastError();
        return e == hipSuccess ? DSIM_OK : hip_fail(e, "parametric launch");
    }
    // the narrow classes (1 to 8 lanes per candidate) come first in the
    // class layout: a grid over their lanes is enough
    const int64_t narrow_waves = (n_cand * (1 << (g.narrow_end - 1)) + kLanes - 1) / kLanes + kClasses;
    const dim3 grid_n((unsigned)(narrow_waves < waves ? narrow_waves : waves));
    if (!side || side == s) {
        launch_kernel(rc, zr, ov, true, true, grid, block, s, g);
        launch_kernel(rc, zr, ov, true, false, grid_n, block, s, g);
        e = hipGetLastError();
        return e == hipSuccess ? DSIM_OK : hip_fail(e, "parametric launch");
    }
    // narrow segments on the caller's stream, right after the pre-pass, and
    // wide ones on the side stream, which waits for the pre-pass; the
    // caller's stream then waits for both.  The narrow wavefronts (36 KB of
    // LDS each) find room only on CUs that wide ones have not filled: started
    // first, they no longer finish last (GPT-3-shaped grid 3.06 -> 2.78 ms,
    // recomputation 4.60 -> 3.80)
    hipEvent_t fork = nullptr, join = nullptr;
    e = hipEventCreateWithFlags(&fork, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&join, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventRecord(fork, s);
    if (e == hipSuccess) e = hipStreamWaitEvent(side, fork, 0);
    if (e == hipSuccess) {
        launch_kernel(rc, zr, ov, true, false, grid_n, block, s, g);
        e = hipGetLastError();
    }
    if (e == hipSuccess) {
        launch_kernel(rc, zr, ov, true, true, grid, block, side, g);
        e = hipGetLastError();
    }
    if (e == hipSuccess) e = hipEventRecord(join, side);
    if (e == hipSuccess) e = hipStreamWaitEvent(s, join, 0);
    if (fork) (void)hipEventDestroy(fork);
    if (join) (void)hipEventDestroy(join);
    return e == hipSuccess ? DSIM_OK : hip_fail(e, "parametric launch");
}

}  // namespace dsim
