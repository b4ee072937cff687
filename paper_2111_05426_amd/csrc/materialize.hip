// materialize.hip -- write the whole distributed program of a strategy as an
// explicit op table.
//
// One lane per candidate expands the transform of Sec. 4 for every device
// (device p*(D*H) + d*H + h runs stage p of data replica d, tensor rank h)
// in a program order whose per-device projections are those of the
// transform (Sec. 2.1 semantics depend on nothing else): the splits, then
// slot by slot every ready stage's block (each compute op once per replica
// device, each tensor-parallel all-reduce once per data replica over its H
// ranks) followed by the slot's Sends in ascending source order (one per
// replica), then every stage's weight update (each gradient all-reduce once
// per tensor rank over the D replicas, each optimizer op once per device).
// With ZeRO (Fig. 9) a weight read is preceded by a broadcast record from
// its owner per tensor rank, the reading op also frees the copy on the other
// replicas, and each gradient all-reduce becomes a reduce record onto the
// owner followed by the owner's optimizer op.  With overlap every GPU g is
// two devices, 2g computing and 2g + 1 communicating: the last backward
// block hands each finished gradient over (a Send of zero alloc and free
// per replica, then an all-reduce over the communication streams per tensor
// rank), and the weight update hands each one back before its optimizer op.
// The records go to the op-major, candidate-fastest table layout that
// dsim_simulate_tables reads.
#include "model.h"

namespace dsim {
namespace {

constexpr int kLanes = 64;
constexpr uint16_t kNoBlock = 0xffffu;

struct MatArgs {
    dsim_model m;
    const dsim_strategy *cand;
    int64_t n_cand;
    int32_t max_ops;
    int32_t n_dev;
    uint32_t *code;
    float *flops;
    float *bytes;
    uint32_t *alloc;
    uint32_t *freeb;
    uint32_t *mm_k;     // may be NULL
    uint32_t *n_ops;
    uint64_t *init_live;
    int32_t *status;
};

// Appends records for one stage's ops on every replica device.
struct Emit {
    const Ctx &x;
    const MatArgs &g;
    int64_t c;
    int64_t j;          // records emitted so far (may pass max_ops: counted, not written)
    bool inexact;       // a value does not fit the record format exactly
    int base;           // first GPU of the stage
    uint64_t pend;      // ZeRO: bytes of the broadcast copy the next op frees on non-owners
    int pend_owner;     // ZeRO: the replica that owns it
    int S;              // devices per GPU: 1, or 2 with overlap

    // the computation device of GPU gpu (its communication stream is the next one)
    __device__ __forceinline__ uint32_t dv(int gpu) const { return (uint32_t)(S * gpu); }

    __device__ __forceinline__ void put(uint32_t code, uint64_t fl, uint64_t by, uint64_t al, uint64_t fr,
                                        uint64_t k = 0)
    {
        // flops and bytes must be exact in fp32, alloc, free and the
        // reduction length in u32
        const float ff = (float)fl, fb = (float)by;
        inexact |= fl >= (1ull << 62) || by >= (1ull << 62) || (uint64_t)ff != fl || (uint64_t)fb != by ||
                   al > 0xffffffffull || fr > 0xffffffffull || k > 0xffffffffull;
        if (j < (int64_t)g.max_ops) {
            const size_t o = (size_t)j * (size_t)g.n_cand + (size_t)c;
            g.code[o] = code;
            g.flops[o] = ff;
            g.bytes[o] = fb;
            g.alloc[o] = (uint32_t)al;
            g.freeb[o] = (uint32_t)fr;
            if (g.mm_k) g.mm_k[o] = (uint32_t)k;
        }
        ++j;
    }
    __device__ void compute(uint32_t cls, uint64_t fl, uint64_t by, uint64_t al, uint64_t fr, uint64_t k)
    {
        for (int r = 0; r < x.D * x.H; ++r) {
            const uint64_t copy = (pend != 0 && r / x.H != pend_owner) ? pend : 0;
            put((dv(base + r) << 8) | (cls << 24), fl, by, al, fr + copy, k);
        }
        pend = 0;
    }
    __device__ void local(uint64_t fl, uint64_t by, uint64_t al, uint64_t fr) { compute(0u, fl, by, al, fr, 0); }
    // a matrix multiplication of reduction length k: cost class 1 of the
    // table format
    __device__ void mm(uint64_t fl, uint64_t by, uint64_t al, uint64_t fr, uint64_t k)
    {
        compute(1u, fl, by, al, fr, k);
    }
    // ZeRO: the owner's broadcast over the D replicas of each tensor rank
    // (kind 3, root = the owner: the others allocate their copy)
    __device__ void bcast(uint64_t by, int grp)
    {
        if (!x.zero) return;
        const int o = grp % x.D;
        for (int h = 0; h < x.H; ++h)
            put(3u | (dv(base + o * x.H + h) << 8) | (dp_mask(h) << 16), 0, by, by, 0);
        pend = by;
        pend_owner = o;
    }
    // ZeRO: reduce onto the owner (kind 4: the owner allocates the reduced
    // gradient, every member frees its own)
    __device__ void reduce(uint64_t by, int grp)
    {
        const int o = grp % x.D;
        for (int h = 0; h < x.H; ++h)
            put(4u | (dv(base + o * x.H + h) << 8) | (dp_mask(h) << 16), 0, by, by, by);
    }
    __device__ void owner_local(uint64_t fl, uint64_t by, uint64_t al, uint64_t fr, int grp)
    {
        const int o = grp % x.D;
        for (int h = 0; h < x.H; ++h) put(dv(base + o * x.H + h) << 8, fl, by, al, fr);
    }
    // the D replicas of tensor rank h on this stage (stream 0: computation,
    // 1: communication)
    __device__ uint32_t dp_mask(int h, int stream = 0) const
    {
        uint32_t mask = 0;
        for (int d = 0; d < x.D; ++d) mask |= 1u << (dv(base + d * x.H + h) + (uint32_t)stream);
        return mask;
    }
    __device__ void ar_tp(uint64_t by)
    {
        if (x.H <= 1) return;
        for (int d = 0; d < x.D; ++d) {
            uint32_t mask = 0;
            for (int h = 0; h < x.H; ++h) mask |= 1u << dv(base + d * x.H + h);
            put(2u | (mask << 16), 0, by, 0, 0);
        }
    }
    __device__ void ar_dp(uint64_t by)
    {
        if (x.D <= 1) return;
        for (int h = 0; h < x.H; ++h) put(2u | (dp_mask(h) << 16), 0, by, 0, 0);
    }
    __device__ void send(int t, uint64_t sz, uint64_t fre)
    {
        const int tbase = t * x.D * x.H;
        for (int r = 0; r < x.D * x.H; ++r)
            put(1u | (dv(base + r) << 8) | (dv(tbase + r) << 16), 0, sz, sz, fre);
    }
    // overlap: each replica hands the finished gradient to its communication
    // stream (nothing allocated or freed), whose D replicas all-reduce it
    __device__ void handover(uint64_t by)
    {
        for (int r = 0; r < x.D * x.H; ++r) put(1u | (dv(base + r) << 8) | ((dv(base + r) + 1u) << 16), 0, by, 0, 0);
        for (int h = 0; h < x.H; ++h) put(2u | (dp_mask(h, 1) << 16), 0, by, 0, 0);
    }
    // overlap: the reduced gradient comes back to the computation stream
    __device__ void handback(uint64_t by)
    {
        for (int r = 0; r < x.D * x.H; ++r) put(1u | ((dv(base + r) + 1u) << 8) | (dv(base + r) << 16), 0, by, 0, 0);
    }
};

__global__ __launch_bounds__(kLanes) void k_materialize(const MatArgs g)
{
    __shared__ uint16_t s_pos[kMaxTableDev][kLanes], s_nf[kMaxTableDev][kLanes], s_nb[kMaxTableDev][kLanes],
        s_em[kMaxTableDev][kLanes];
    const int lane = threadIdx.x;
    const int64_t c = (int64_t)blockIdx.x * kLanes + lane;
    if (c >= g.n_cand) return;
    const dsim_strategy st = g.cand[c];
    for (int dev = 0; dev < g.n_dev; ++dev) g.init_live[c * g.n_dev + dev] = 0;
    const int S = g.m.overlap ? 2 : 1;
    const bool ok = strategy_ok(g.m, st.D, st.H, st.P, st.K) && st.K <= kMaxK &&
                    (int64_t)S * st.D * st.H * st.P <= (int64_t)g.n_dev;
    if (!ok) {
        g.n_ops[c] = 0;
        g.status[c] = DSIM_ST_BAD_STRATEGY;
        return;
    }
    CostConsts none = {};
    Ctx x = {};
    make_ctx(g.m, none, st, x);
    const int DH = x.D * x.H;
    Emit e{x, g, c, 0, false, 0, 0, 0, S};
    for (int s = 0; s < x.P; ++s) {
        if (x.zero) {
            // each data replica holds the groups it owns
            ZStage zs;
            z_stage(x, s, zs);
            const uint64_t in = resident_inputs(x, s);
            for (int r = 0; r < DH; ++r) g.init_live[c * g.n_dev + s * DH + r] = in + z_owned(x, zs, r / x.H);
        } else {
            // (a communication stream holds nothing)
            const uint64_t r0 = resident(x, s);
            for (int r = 0; r < DH; ++r) g.init_live[c * g.n_dev + e.dv(s * DH + r)] = r0;
        }
        s_pos[s][lane] = 0;
        s_nf[s][lane] = 0;
        s_nb[s][lane] = 0;
    }
    // microbatch splits before the pipeline
    if (x.K > 1) {
        e.base = 0;
        split(x, e);
        if (x.train) {
            e.base = (x.P - 1) * DH;
            split(x, e);
        }
    }
    const int len = x.train ? 2 * x.K : x.K;
    for (;;) {
        bool left = false, any = false;
        int prev_nf0 = 0;
        for (int s = 0; s < x.P; ++s) {
            int pos = s_pos[s][lane], nf = s_nf[s][lane], nb = s_nb[s][lane];
            const int nf0 = nf;
            uint16_t em = kNoBlock;
            if (pos < len) {
                left = true;
                bool bwd;
                int k;
                block_at(x, s, pos, bwd, k);
                const bool ready = !bwd ? (s == 0 || prev_nf0 > k) : (s == x.P - 1 ? nf0 > k : s_nb[s + 1][lane] > k);
                if (ready) {
                    e.base = s * DH;
                    if (bwd) block_bwd(x, e, s, k);
                    else block_fwd(x, e, s, k);
                    ++pos;
                    if (bwd) ++nb;
                    else ++nf;
                    em = (uint16_t)((k << 1) | (bwd ? 1 : 0));
                    any = true;
                }
            }
            s_pos[s][lane] = (uint16_t)pos;
            s_nf[s][lane] = (uint16_t)nf;
            s_nb[s][lane] = (uint16_t)nb;
            s_em[s][lane] = em;
            prev_nf0 = nf0;
        }
        if (!left) break;
        if (!any) {   // no stage can proceed: impossible for 1F1B
            g.n_ops[c] = 0;
            g.status[c] = DSIM_ST_BAD_STRATEGY;
            return;
        }
        for (int s = 0; s < x.P; ++s) {
            const uint16_t em = s_em[s][lane];
            if (em == kNoBlock) continue;
            const bool bwd = em & 1;
            const int k = em >> 1;
            if ((!bwd && s == x.P - 1) || (bwd && s == 0)) continue;
            uint64_t sz, fre;
            send_size(x, s, mb_rows(x, k), bwd, sz, fre);
            e.base = s * DH;
            e.send(bwd ? s - 1 : s + 1, sz, fre);
        }
    }
    if (x.train) {
        for (int s = 0; s < x.P; ++s) {
            e.base = s * DH;
            weight_update(x, e, s);
        }
    }
    const bool fits = e.j <= (int64_t)g.max_ops && !e.inexact;
    g.n_ops[c] = fits ? (uint32_t)e.j : 0u;
    g.status[c] = fits ? 0 : DSIM_ST_NOT_TABLE;
}

}  // namespace

dsim_status launch_materialize(const dsim_model &m, const dsim_strategy *cand, int64_t n_cand, int32_t max_ops,
                               int32_t n_dev, uint32_t *code, float *flops, float *bytes, uint32_t *alloc,
                               uint32_t *freeb, uint32_t *mm_k, uint32_t *n_ops, uint64_t *init_live,
                               int32_t *status, hipStream_t s)
{
    MatArgs g;
    g.m = m;
    g.cand = cand;
    g.n_cand = n_cand;
    g.max_ops = max_ops;
    g.n_dev = n_dev;
    g.code = code;
    g.flops = flops;
    g.bytes = bytes;
    g.alloc = alloc;
    g.freeb = freeb;
    g.mm_k = mm_k;
    g.n_ops = n_ops;
    g.init_live = init_live;
    g.status = status;
    const int64_t blocks = (n_cand + kLanes - 1) / kLanes;
    hipLaunchKernelGGL(k_materialize, dim3((unsigned)blocks), dim3(kLanes), 0, s, g);
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? DSIM_OK : hip_fail(e, "materialize launch");
}

}  // namespace dsim
