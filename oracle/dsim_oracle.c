/*
 * dsim_oracle.c -- reference CPU simulator for DistIR programs.
 *
 * TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
 * cpu_baseline leg of bench.py may load or call this library.  It shares no
 * code, header, table or constant with the HIP library under
 * paper_2111_05426_amd/; each side is written separately from the paper.
 *
 * What it computes (Santhanam et al., "DistIR: An Intermediate Representation
 * and Simulator for Efficient Neural Network Distribution", MLSys 2022):
 *
 *  - Distributed semantics (Sec. 2.1): a fixed set of single-threaded devices;
 *    an op runs synchronously on its device set, so it starts when every
 *    device in the set is free and all of them finish together; ops run in
 *    program order.  The drawing macros of the trace figure (Fig. 3) encode
 *    the same clock rule: a local event adds its duration to its device's
 *    clock, a communication event starts at the max of the two clocks and
 *    sets both to the end.
 *  - Simulator (Sec. 3.3, Algorithm 1 with calls inlined): op cost from its
 *    input shapes, then clock advance with synchronisation; live memory per
 *    device, a tensor being live from its creation until its last use.
 *  - Cost functions (Sec. 3.3 and Sec. 4): compute ops use a roofline
 *    launch + max(flops/F, bytes/B_mem) (with launch 0 and bytes 0 this is the
 *    paper's Add cost N/f); Send uses latency + bytes/B_link; AllReduce uses
 *    the ring form 2(n-1)*latency + 2(n-1)/n * bytes/B_link.  Every division
 *    by a device constant is taken once as a reciprocal rounded to fp64.
 *  - The D/T/P(/K) transform (Sec. 4; Fig. 2 gives the P=2, K=2 instance):
 *    data parallel replicas with gradient all-reduce, Megatron-style tensor
 *    parallel layers, uniform contiguous pipeline stages with synchronous
 *    1F1B scheduling, K microbatches and gradient accumulation.
 *  - Grid search (Sec. 5.1, Sec. 5.2): power-of-two D, T, P up to a device
 *    budget, microbatch counts, a per-device memory filter and the top-k by
 *    predicted time.
 *
 * Where the paper is silent, the reading taken is stated at the code that
 * implements it.  The transformer's per-op FLOP/byte formulas and the slot
 * order for P >= 3 are this project's definitions (the paper prints neither);
 * they are pinned by a GPT rank's program written out by hand (bytes, matmul
 * flops and one-stage peaks) and by a hand trace of P = 3, K = 4 with unequal
 * per-type costs.  Parity unpinned: which random draw of the table generator
 * feeds which field (its PRNG and its log-uniform transform are pinned).  The
 * pins are exercised by tests/test_oracle_pins.py.
 *
 * Floating point: IEEE fp64, compiled with -ffp-contract=off and no fast-math;
 * expressions are evaluated exactly in the order written.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>
#include <pthread.h>

/* ------------------------------------------------------------------------ */
/* Public enums (mirrored by value, not by code, in the Python wrapper).     */
/* ------------------------------------------------------------------------ */
enum { OR_COMPUTE = 0, OR_SEND = 1, OR_ALLREDUCE = 2, OR_BCAST = 3, OR_REDUCE = 4 };

enum {
    ST_BAD_OP = 1, ST_BAD_DEVICE = 2, ST_SELF_SEND = 4, ST_MEM_UNDERFLOW = 8,
    ST_BAD_STRATEGY = 16, ST_OVER_CAP = 32
};

enum { FAM_MLP = 0, FAM_TRANSFORMER = 1 };
enum { MODE_INFER = 0, MODE_SGD = 1, MODE_ADAM = 2, MODE_ADAM_MIXED = 3 };

/* Op type tags: only used for per-type cost injection in tests and for
 * per-type FLOP totals. */
enum {
    T_SPLIT = 0, T_GEMM, T_RELU, T_AR_TP, T_LOSSGRAD, T_RELUGRAD, T_GEMMDW,
    T_ADDGRAD, T_GEMMDX, T_SEND_F, T_SEND_B, T_AR_DP, T_OPT,
    /* transformer */
    T_LN, T_QKV, T_SCORES, T_SOFTMAX, T_AV, T_OUTPROJ, T_RESADD, T_FC1,
    T_GELU, T_FC2, T_EMBED, T_LMHEAD, T_XENT_STATS, T_XENT_GRAD, T_LN_B,
    T_RESADD_B, T_GELU_B, T_AV_B, T_SOFTMAX_B, T_SCORES_B, T_EMBED_DW,
    /* ZeRO */
    T_BCAST, T_REDUCE,
    /* overlap: a gradient handed between the two streams of one GPU */
    T_STREAM,
    T_GENERIC, T_NTYPES
};

typedef struct {
    double flops_per_s, mem_bytes_per_s, link_bytes_per_s, link_latency_s, launch_s;
    uint64_t mem_cap_bytes;
    /* Empirical MatMul cost (Sec. 4: MatMul gets a linear regression in its
     * input sizes, fitted on single-op microbenchmarks): when mm_enabled,
     * a matrix multiplication of `flops` flops touching `bytes` bytes with
     * reduction length k costs
     *   max(mm_floor, ((mm_c0 + mm_c1 * flops) + mm_c2 * bytes) + mm_c3 * k)
     * instead of the roofline (mm_c3 and mm_floor at the end of the struct;
     * both 0 give the paper's linear form). */
    int32_t mm_enabled;
    double mm_c0, mm_c1, mm_c2;
    /* Two-tier interconnect (hardware topologies, Sec. 1; the paper models
     * communication by network bandwidth coefficients, Sec. 4): with
     * node_size > 0, device d lies in node d / node_size, and a send or
     * collective whose devices lie in more than one node crosses the
     * network (net_bytes_per_s, net_latency_s) instead of the node's links
     * (link_bytes_per_s, link_latency_s).  node_size = 0: one uniform
     * interconnect. */
    int32_t node_size;
    double net_bytes_per_s, net_latency_s;
    /* Streams (Sec. 2.2, Limitations: communication that overlaps
     * computation is modelled with one device per stream, the streams of a
     * GPU communicating at low or zero cost): with streams_per_gpu = S > 1,
     * device d is a stream of GPU d / S, nodes hold node_size GPUs, and a
     * send or collective whose devices all lie on one GPU costs
     * stream_latency_s and stream_bytes_per_s (+inf: no byte term) in
     * place of the links.  S = 0 or 1: every device is its own GPU. */
    int32_t streams_per_gpu;
    double stream_bytes_per_s, stream_latency_s;
    /* the MatMul cost's reduction-length term and floor (see mm_enabled) */
    double mm_c3, mm_floor;
} or_device_model;

typedef struct {
    int32_t family, mode, n_layers, n_heads;
    int64_t d_model, d_ff, seq_len, vocab, global_batch;
    int32_t elem_bytes;
    int32_t schedule;   /* 0: synchronous 1F1B (Sec. 4); 1: GPipe (all forwards, then all backwards) */
    int32_t recompute;  /* 1: activation recomputation (gradient checkpointing, Fig. 8), training only */
    int32_t zero;       /* 1: ZeRO parameter and gradient partitioning (Fig. 9), training only */
    int32_t overlap;    /* 1: data-parallel gradient all-reduce on a second stream per GPU (Sec. 2.2,
                           Limitations), overlapping the last backward pass; training, not with ZeRO */
} or_model;

/* ------------------------------------------------------------------------ */
/* Cost functions (Sec. 3.3, Sec. 4).                                        */
/* ------------------------------------------------------------------------ */
static double cost_compute(const or_device_model *m, double flops, double bytes)
{
    double inv_f = 1.0 / m->flops_per_s;
    double inv_b = 1.0 / m->mem_bytes_per_s;
    double tf = flops * inv_f;
    double tb = bytes * inv_b;
    return m->launch_s + (tf > tb ? tf : tb);
}

/* The tier a communication op crosses (`spans`): 0 the links inside a node,
 * 1 the network (its devices lie in more than one node), 2 the streams of
 * one GPU (all its devices lie on one GPU). */
enum { TIER_LINK = 0, TIER_NET = 1, TIER_STREAM = 2 };

static double link_lat(const or_device_model *m, int spans)
{
    if (spans == TIER_STREAM && m->streams_per_gpu > 1) return m->stream_latency_s;
    return spans == TIER_NET && m->node_size > 0 ? m->net_latency_s : m->link_latency_s;
}
static double link_bw(const or_device_model *m, int spans)
{
    if (spans == TIER_STREAM && m->streams_per_gpu > 1) return m->stream_bytes_per_s;
    return spans == TIER_NET && m->node_size > 0 ? m->net_bytes_per_s : m->link_bytes_per_s;
}

static double cost_send(const or_device_model *m, double bytes, int spans)
{
    double inv_l = 1.0 / link_bw(m, spans);
    return link_lat(m, spans) + bytes * inv_l;
}

static double cost_allreduce(const or_device_model *m, double bytes, int n, int spans)
{
    double inv_l, a, two_a;
    if (n <= 1) return 0.0;
    inv_l = 1.0 / link_bw(m, spans);
    a = (double)(n - 1);
    two_a = 2.0 * a;
    return two_a * link_lat(m, spans) + (two_a / (double)n) * (bytes * inv_l);
}

/* Broadcast from one member of a group to the others, and reduce of the
 * members' tensors onto one member (the weight distribution and gradient
 * reduction of Fig. 9): a pipelined chain, (n-1) link latencies plus the
 * bytes crossing one link once.  With two devices this is the Send of
 * Sec. 2.1 / Fig. 9; one device costs nothing. */
static double cost_chain(const or_device_model *m, double bytes, int n, int spans)
{
    double inv_l;
    if (n <= 1) return 0.0;
    inv_l = 1.0 / link_bw(m, spans);
    return (double)(n - 1) * link_lat(m, spans) + bytes * inv_l;
}

/* the tier of an op over the given devices: the streams of one GPU when
 * every device lies on the same GPU (streams_per_gpu > 1), else the network
 * when their GPUs lie in more than one node, else the links */
static int spans_nodes(const or_device_model *m, const int32_t *devs, int64_t n)
{
    int64_t q;
    int S = m->streams_per_gpu > 1 ? m->streams_per_gpu : 1;
    if (n < 1) return TIER_LINK;
    if (S > 1) {
        int one_gpu = 1;
        for (q = 1; q < n; q++)
            if (devs[q] / S != devs[0] / S) one_gpu = 0;
        if (one_gpu) return TIER_STREAM;
    }
    if (m->node_size <= 0 || n < 2) return TIER_LINK;
    for (q = 1; q < n; q++)
        if (devs[q] / S / m->node_size != devs[0] / S / m->node_size) return TIER_NET;
    return TIER_LINK;
}
static int mask_spans_nodes(const or_device_model *m, uint32_t mask)
{
    int32_t devs[32];
    int n = 0, d;
    for (d = 0; d < 32; d++)
        if (mask & (1u << d)) devs[n++] = d;
    return spans_nodes(m, devs, n);
}

/* The op types that multiply two matrices: the dense layer's Gemm and its
 * two gradients, the transformer's projections, MLP and LM-head products,
 * the attention scores and P.V products, and their gradients. */
static int is_matmul(int type)
{
    switch (type) {
    case T_GEMM: case T_GEMMDW: case T_GEMMDX: case T_QKV: case T_SCORES: case T_AV: case T_OUTPROJ:
    case T_FC1: case T_FC2: case T_LMHEAD: case T_AV_B: case T_SCORES_B:
        return 1;
    default:
        return 0;
    }
}

/* Regression cost of a matrix multiplication (Sec. 4): linear in the input
 * sizes, plus a term in the reduction length k (the serial part of a
 * product: few output tiles with a long k take time that neither the flops
 * nor the bytes show), at least mm_floor (the per-product dispatch that an
 * eagerly issued product never finishes sooner than). */
static double cost_matmul(const or_device_model *m, double flops, double bytes, double k)
{
    double c = ((m->mm_c0 + m->mm_c1 * flops) + m->mm_c2 * bytes) + m->mm_c3 * k;
    return m->mm_floor > c ? m->mm_floor : c;
}

/* cost of an op; spans: its devices lie in more than one node */
double or_cost_spans(const or_device_model *m, int kind, double flops, double bytes, int n, int spans)
{
    if (kind == OR_COMPUTE) return cost_compute(m, flops, bytes);
    if (kind == OR_SEND) return cost_send(m, bytes, spans);
    if (kind == OR_BCAST || kind == OR_REDUCE) return cost_chain(m, bytes, n, spans);
    return cost_allreduce(m, bytes, n, spans);
}

double or_cost(const or_device_model *m, int kind, double flops, double bytes, int n)
{
    return or_cost_spans(m, kind, flops, bytes, n, 0);
}

/* cost of an op of a given type: matrix multiplications (reduction length k)
 * take the empirical regression when the device model carries one */
double or_cost_typed(const or_device_model *m, int kind, int type, double flops, double bytes, double k, int n,
                     int spans)
{
    if (kind == OR_COMPUTE && m->mm_enabled && is_matmul(type)) return cost_matmul(m, flops, bytes, k);
    return or_cost_spans(m, kind, flops, bytes, n, spans);
}

/* ------------------------------------------------------------------------ */
/* Explicit op tables (at most 8 devices): one candidate, per-op amounts.    */
/* code = kind | a << 8 | b_or_mask << 16 | cost class << 24; flops and     */
/* bytes must be finite and >= 0 (costs are then never negative).  Cost     */
/* class 0 is the model's own cost; class 1, on a compute op only, marks a  */
/* matrix multiplication, which takes the empirical MatMul regression when  */
/* the device model carries one (the roofline otherwise).  Any other class  */
/* is invalid.                                                               */
/* compute: runs on a, allocates and frees on a.                             */
/* send a->b: runs on {a,b}, allocates on b, frees on a.                     */
/* allreduce: runs on the devices of the mask; alloc/free fields ignored.    */
/* broadcast (ZeRO's weight distribution, Fig. 9): root a sends to the other */
/* devices of the mask (a must be in it); each of them allocates `alloc`     */
/* bytes (its copy), then a frees `free` bytes.                              */
/* reduce (ZeRO's gradient reduction onto the owner, Fig. 9): the devices of */
/* the mask send to root a (a in the mask), which allocates `alloc` bytes    */
/* (the reduced tensor); then every member frees `free` bytes (its own      */
/* contribution dies there).  Both cost the pipelined chain over the mask.  */
/* Every touched device samples its peak after the allocation and before    */
/* the free.                                                                 */
/* An invalid op is skipped and flagged in the status word.                  */
/* ------------------------------------------------------------------------ */
int or_sim_table(int64_t n_ops, int n_dev,
                 const uint32_t *code, const float *flops, const float *bytes,
                 const uint32_t *alloc, const uint32_t *freeb, const uint32_t *mm_k, int64_t stride,
                 const uint64_t *init_live, const or_device_model *m,
                 double *makespan, double *finish, uint64_t *peak,
                 uint64_t *cand_peak, int32_t *status)
{
    double clk[8];
    uint64_t live[8], pk[8];
    int32_t st = 0;
    int64_t j;
    int d;
    if (n_dev < 1 || n_dev > 8) return -1;
    for (d = 0; d < n_dev; d++) {
        clk[d] = 0.0;
        live[d] = init_live ? init_live[d] : 0;
        pk[d] = live[d];
    }
    for (j = 0; j < n_ops; j++) {
        int64_t o = j * stride;
        uint32_t c = code[o];
        int kind = (int)(c & 0xffu), a = (int)((c >> 8) & 0xffu), b = (int)((c >> 16) & 0xffu);
        int cls = (int)(c >> 24);
        uint32_t mask;
        double start, end, cost;
        {
            uint32_t fb, bb;
            memcpy(&fb, &flops[o], 4);
            memcpy(&bb, &bytes[o], 4);
            if (cls > 1 || (cls == 1 && kind != OR_COMPUTE) || kind > 4 || fb >= 0x7f800000u || bb >= 0x7f800000u) {
                st |= ST_BAD_OP;
                continue;
            }
        }
        if (kind == OR_COMPUTE) {
            if (a >= n_dev) { st |= ST_BAD_DEVICE; continue; }
            mask = 1u << a;
            if (cls == 1 && m->mm_enabled)
                cost = cost_matmul(m, (double)flops[o], (double)bytes[o], mm_k ? (double)mm_k[o] : 0.0);
            else cost = cost_compute(m, (double)flops[o], (double)bytes[o]);
        } else if (kind == OR_SEND) {
            if (a >= n_dev || b >= n_dev) { st |= ST_BAD_DEVICE; continue; }
            if (a == b) { st |= ST_SELF_SEND; continue; }
            mask = (1u << a) | (1u << b);
            cost = cost_send(m, (double)bytes[o], mask_spans_nodes(m, mask));
        } else if (kind == OR_ALLREDUCE) {
            int n = 0;
            mask = (uint32_t)b;
            if (mask == 0 || (mask >> n_dev) != 0) { st |= ST_BAD_DEVICE; continue; }
            for (d = 0; d < n_dev; d++) if (mask & (1u << d)) n++;
            cost = cost_allreduce(m, (double)bytes[o], n, mask_spans_nodes(m, mask));
        } else {
            int n = 0;
            mask = (uint32_t)b;
            if (a >= n_dev || (mask >> n_dev) != 0 || !(mask & (1u << a))) { st |= ST_BAD_DEVICE; continue; }
            for (d = 0; d < n_dev; d++) if (mask & (1u << d)) n++;
            cost = cost_chain(m, (double)bytes[o], n, mask_spans_nodes(m, mask));
        }
        start = 0.0;
        for (d = 0; d < n_dev; d++)
            if ((mask & (1u << d)) && clk[d] > start) start = clk[d];
        end = start + cost;
        for (d = 0; d < n_dev; d++)
            if (mask & (1u << d)) clk[d] = end;
        if (kind == OR_COMPUTE || kind == OR_SEND) {
            int tgt = (kind == OR_SEND) ? b : a;
            live[tgt] += (uint64_t)alloc[o];
            if (live[tgt] > pk[tgt]) pk[tgt] = live[tgt];
            if ((uint64_t)freeb[o] > live[a]) { st |= ST_MEM_UNDERFLOW; live[a] = 0; }
            else live[a] -= (uint64_t)freeb[o];
        } else if (kind == OR_BCAST || kind == OR_REDUCE) {
            /* allocate on the receivers (broadcast) or the root (reduce),
             * sample every member, then free on the root (broadcast) or on
             * every member (reduce) */
            for (d = 0; d < n_dev; d++) {
                if (!(mask & (1u << d))) continue;
                if (kind == OR_BCAST ? d != a : d == a) live[d] += (uint64_t)alloc[o];
                if (live[d] > pk[d]) pk[d] = live[d];
            }
            for (d = 0; d < n_dev; d++) {
                if (!(mask & (1u << d)) || (kind == OR_BCAST && d != a)) continue;
                if ((uint64_t)freeb[o] > live[d]) { st |= ST_MEM_UNDERFLOW; live[d] = 0; }
                else live[d] -= (uint64_t)freeb[o];
            }
        }
    }
    {
        double mk = 0.0;
        uint64_t cp = 0;
        for (d = 0; d < n_dev; d++) {
            if (clk[d] > mk) mk = clk[d];
            if (pk[d] > cp) cp = pk[d];
            if (finish) finish[d] = clk[d];
            if (peak) peak[d] = pk[d];
        }
        if (m->mem_cap_bytes != 0 && cp > m->mem_cap_bytes) st |= ST_OVER_CAP;
        *makespan = mk;
        *cand_peak = cp;
        *status = st;
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Random explicit op tables (the synthetic workload of random programs).    */
/*                                                                          */
/* Draws: r(c, j, f) is output number c*2^32 + j*2^5 + f + 1 of SplitMix64   */
/* (Steele, Lea & Flood 2014) started from `seed`, i.e.                     */
/* mix(seed + n * 0x9E3779B97F4A7C15).  range(r, n) = floor(hi32(r) * n /   */
/* 2^32).  A log-uniform float in [lo, hi] is 2^t rounded to fp32, with    */
/* t = L(lo) + u (L(hi) - L(lo)), u = the top 53 bits of the draw / 2^53   */
/* and L(b) the base-2 logarithm of the bound to double precision; 2^t =   */
/* 2^floor(t) * e^(f ln 2), f = t - floor(t), with the exponential summed   */
/* as its Taylor series up to the 13th power in Horner form (truncation     */
/* below 1e-13 relative), all in fp64 without contraction.                  */
/* ------------------------------------------------------------------------ */
#define GEN_SLOTS 16
static uint64_t sm64_at(uint64_t seed, uint64_t n)
{
    uint64_t z = seed + n * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* output n (n >= 1) of SplitMix64 started from seed (tests) */
uint64_t or_splitmix64(uint64_t seed, uint64_t n) { return sm64_at(seed, n); }

static uint64_t draw(uint64_t seed, uint64_t c, uint64_t j, uint64_t f)
{
    return sm64_at(seed, (c << 32) + (j << 5) + f + 1);
}

static uint32_t urange(uint64_t r, uint32_t n)
{
    return (uint32_t)(((r >> 32) * (uint64_t)n) >> 32);
}


/* base-2 logarithms of the bounds 1e3, 1e6, 1e9, 1e12 (nearest doubles) */
#define LOG2_1E3 0x1.3ee7b471b3a95p+3
#define LOG2_1E6 0x1.3ee7b471b3a95p+4
#define LOG2_1E9 0x1.de5b8eaa8d7e0p+4
#define LOG2_1E12 0x1.3ee7b471b3a95p+5

/* e^y for 0 <= y < ln 2: sum of y^k / k!, k = 0..13, Horner form */
static double exp_series(double y)
{
    static const double inv_fact[14] = {
        1.0, 1.0, 0.5, 0x1.5555555555555p-3, 0x1.5555555555555p-5, 0x1.1111111111111p-7,
        0x1.6c16c16c16c17p-10, 0x1.a01a01a01a01ap-13, 0x1.a01a01a01a01ap-16, 0x1.71de3a556c734p-19,
        0x1.27e4fb7789f5cp-22, 0x1.ae64567f544e4p-26, 0x1.1eed8eff8d898p-29, 0x1.6124613a86d09p-33};
    double s = inv_fact[13];
    int k;
    for (k = 12; k >= 0; k--) s = s * y + inv_fact[k];
    return s;
}

static float log_uniform(uint64_t r, double log2_lo, double log2_hi)
{
    const double ln2 = 0x1.62e42fefa39efp-1;
    double u = (double)(r >> 11) * 0x1p-53;
    double t = log2_lo + u * (log2_hi - log2_lo);
    double n = floor(t);
    return (float)ldexp(exp_series((t - n) * ln2), (int)n);
}

/* the i-th (ascending) n_dev-bit mask with at least two bits set */
static uint32_t nth_group_mask(int n_dev, uint32_t i)
{
    uint32_t mask, seen = 0;
    for (mask = 0; mask < (1u << n_dev); mask++) {
        int pc = 0, d;
        for (d = 0; d < n_dev; d++) if (mask & (1u << d)) pc++;
        if (pc >= 2) {
            if (seen == i) return mask;
            seen++;
        }
    }
    return 0;
}

int or_gen_table(uint64_t seed, int64_t cand, int32_t n_ops, int32_t n_dev,
                 uint32_t *code, float *flops, float *bytes,
                 uint32_t *alloc, uint32_t *freeb, int64_t stride)
{
    uint32_t slot[8][GEN_SLOTS];
    int cnt[8];
    int32_t j;
    uint32_t n_masks;
    uint64_t c = (uint64_t)cand;
    if (n_dev < 2 || n_dev > 8 || n_ops < 0 || cand < 0) return -1;
    n_masks = (1u << n_dev) - (uint32_t)n_dev - 1u;
    memset(cnt, 0, sizeof cnt);
    for (j = 0; j < n_ops; j++) {
        int64_t o = (int64_t)j * stride;
        uint64_t r0 = draw(seed, c, (uint64_t)j, 0);
        uint32_t kd = urange(r0, 10);
        uint32_t a = urange(draw(seed, c, (uint64_t)j, 1), (uint32_t)n_dev);
        uint32_t al = 0, fr = 0;
        if (kd < 9) {
            /* compute or send: free a uniformly chosen live buffer of a */
            uint64_t r5 = draw(seed, c, (uint64_t)j, 5);
            if ((r5 >> 63) && cnt[a] > 0) {
                uint32_t i = (uint32_t)(((r5 & 0xffffffffull) * (uint64_t)cnt[a]) >> 32);
                fr = slot[a][i];
                slot[a][i] = slot[a][cnt[a] - 1];
                cnt[a]--;
            }
        }
        if (kd < 7) {
            uint64_t r6 = draw(seed, c, (uint64_t)j, 6);
            code[o] = 0u | (a << 8);
            flops[o] = log_uniform(draw(seed, c, (uint64_t)j, 3), LOG2_1E6, LOG2_1E12);
            bytes[o] = log_uniform(draw(seed, c, (uint64_t)j, 4), LOG2_1E3, LOG2_1E9);
            if ((r6 >> 63) && cnt[a] < GEN_SLOTS) {
                al = (uint32_t)log_uniform(draw(seed, c, (uint64_t)j, 7), LOG2_1E3, LOG2_1E9);
                slot[a][cnt[a]++] = al;
            }
        } else if (kd < 9) {
            uint32_t b = (a + 1u + urange(draw(seed, c, (uint64_t)j, 2), (uint32_t)(n_dev - 1))) % (uint32_t)n_dev;
            uint32_t msg = (uint32_t)log_uniform(draw(seed, c, (uint64_t)j, 7), LOG2_1E3, LOG2_1E9);
            code[o] = 1u | (a << 8) | (b << 16);
            flops[o] = 0.0f;
            bytes[o] = (float)msg;
            if (cnt[b] < GEN_SLOTS) {
                al = msg;
                slot[b][cnt[b]++] = msg;
            }
        } else {
            uint32_t mask = nth_group_mask(n_dev, urange(draw(seed, c, (uint64_t)j, 2), n_masks));
            code[o] = 2u | (mask << 16);
            flops[o] = 0.0f;
            bytes[o] = log_uniform(draw(seed, c, (uint64_t)j, 4), LOG2_1E3, LOG2_1E9);
        }
        alloc[o] = al;
        freeb[o] = fr;
    }
    return 0;
}


/* ------------------------------------------------------------------------ */
/* Programs over tensors (def/use), as produced by the transforms below and  */
/* as handed over directly by the figure pins.                               */
/* ------------------------------------------------------------------------ */
enum { TF_RESIDENT = 1, TF_KEEP = 2 };

typedef struct {
    int64_t n_ops, cap_ops;
    uint8_t *kind, *type;
    int32_t *nsz;          /* group size used by the all-reduce cost */
    int32_t *gfirst, *glast;  /* device range of the whole group of a collective
                                 (a projection materialises part of it); -1: its
                                 devices as listed */
    double *flops, *bytes;
    double *kred;          /* reduction length of a matrix multiplication, 0 otherwise */
    double *ocost;         /* per-op duration override (< 0: cost model) */
    int64_t *dev_beg, *in_beg, *out_beg;
    int32_t *devs, *ins, *outs;
    int64_t n_devs, cap_devs, n_ins, cap_ins, n_outs, cap_outs;
    int64_t n_t, cap_t;
    int32_t *t_dev;
    uint64_t *t_size;
    uint8_t *t_flags;
    int64_t program_ops;   /* ops of the whole program (a projection counts skipped ones) */
    int failed;
} or_prog;

static void *grow(void *p, int64_t cap_now, int64_t need, size_t elem, int64_t *cap_out, int *failed)
{
    int64_t nc;
    void *q;
    if (need <= cap_now) { *cap_out = cap_now; return p; }
    nc = cap_now ? cap_now : 256;
    while (nc < need) nc *= 2;
    q = realloc(p, (size_t)nc * elem);
    if (!q) { *failed = 1; *cap_out = cap_now; return p; }
    *cap_out = nc;
    return q;
}

static void prog_init(or_prog *g) { memset(g, 0, sizeof *g); }

static void prog_free(or_prog *g)
{
    free(g->kind); free(g->type); free(g->nsz); free(g->gfirst); free(g->glast);
    free(g->flops); free(g->bytes); free(g->kred); free(g->ocost);
    free(g->dev_beg); free(g->in_beg); free(g->out_beg);
    free(g->devs); free(g->ins); free(g->outs);
    free(g->t_dev); free(g->t_size); free(g->t_flags);
    memset(g, 0, sizeof *g);
}

static int32_t prog_tensor(or_prog *g, int dev, uint64_t size, int flags)
{
    int64_t n = g->n_t, c;
    if (g->failed) return -1;
    if (n + 1 > g->cap_t) {
        g->t_dev = grow(g->t_dev, g->cap_t, n + 1, sizeof(int32_t), &c, &g->failed);
        g->t_size = grow(g->t_size, g->cap_t, n + 1, sizeof(uint64_t), &c, &g->failed);
        g->t_flags = grow(g->t_flags, g->cap_t, n + 1, sizeof(uint8_t), &c, &g->failed);
        if (g->failed) return -1;
        g->cap_t = c;
    }
    g->t_dev[n] = dev;
    g->t_size[n] = size;
    g->t_flags[n] = (uint8_t)flags;
    g->n_t = n + 1;
    return (int32_t)n;
}

static void op_begin(or_prog *g, int kind, int type, double flops, double bytes)
{
    int64_t i = g->n_ops, c;
    if (g->failed) return;
    if (i + 2 > g->cap_ops) {
        g->kind = grow(g->kind, g->cap_ops, i + 2, 1, &c, &g->failed);
        g->type = grow(g->type, g->cap_ops, i + 2, 1, &c, &g->failed);
        g->nsz = grow(g->nsz, g->cap_ops, i + 2, sizeof(int32_t), &c, &g->failed);
        g->gfirst = grow(g->gfirst, g->cap_ops, i + 2, sizeof(int32_t), &c, &g->failed);
        g->glast = grow(g->glast, g->cap_ops, i + 2, sizeof(int32_t), &c, &g->failed);
        g->flops = grow(g->flops, g->cap_ops, i + 2, sizeof(double), &c, &g->failed);
        g->bytes = grow(g->bytes, g->cap_ops, i + 2, sizeof(double), &c, &g->failed);
        g->kred = grow(g->kred, g->cap_ops, i + 2, sizeof(double), &c, &g->failed);
        g->ocost = grow(g->ocost, g->cap_ops, i + 2, sizeof(double), &c, &g->failed);
        g->dev_beg = grow(g->dev_beg, g->cap_ops, i + 2, sizeof(int64_t), &c, &g->failed);
        g->in_beg = grow(g->in_beg, g->cap_ops, i + 2, sizeof(int64_t), &c, &g->failed);
        g->out_beg = grow(g->out_beg, g->cap_ops, i + 2, sizeof(int64_t), &c, &g->failed);
        if (g->failed) return;
        g->cap_ops = c;
    }
    g->kind[i] = (uint8_t)kind;
    g->type[i] = (uint8_t)type;
    g->nsz[i] = 0;
    g->gfirst[i] = -1;
    g->glast[i] = -1;
    g->flops[i] = flops;
    g->bytes[i] = bytes;
    g->kred[i] = 0.0;
    g->ocost[i] = -1.0;
    g->dev_beg[i] = g->n_devs;
    g->in_beg[i] = g->n_ins;
    g->out_beg[i] = g->n_outs;
}

/* the whole group of the op being built spans devices first..last */
static void op_group(or_prog *g, int first, int last)
{
    if (g->failed) return;
    g->gfirst[g->n_ops] = first;
    g->glast[g->n_ops] = last;
}

static void op_dev(or_prog *g, int d)
{
    if (g->failed) return;
    g->devs = grow(g->devs, g->cap_devs, g->n_devs + 1, sizeof(int32_t), &g->cap_devs, &g->failed);
    if (!g->failed) g->devs[g->n_devs++] = d;
}

static void op_in(or_prog *g, int32_t t)
{
    if (g->failed) return;
    g->ins = grow(g->ins, g->cap_ins, g->n_ins + 1, sizeof(int32_t), &g->cap_ins, &g->failed);
    if (!g->failed) g->ins[g->n_ins++] = t;
}

static void op_out(or_prog *g, int32_t t)
{
    if (g->failed) return;
    g->outs = grow(g->outs, g->cap_outs, g->n_outs + 1, sizeof(int32_t), &g->cap_outs, &g->failed);
    if (!g->failed) g->outs[g->n_outs++] = t;
}

/* close the op; nsz > 0 overrides the group size of an all-reduce; mult is
 * how many ops of the whole program this emitted op stands for */
static void op_end(or_prog *g, int nsz, int64_t mult)
{
    int64_t i = g->n_ops;
    if (g->failed) return;
    g->nsz[i] = nsz > 0 ? nsz : (int32_t)(g->n_devs - g->dev_beg[i]);
    g->n_ops = i + 1;
    g->dev_beg[i + 1] = g->n_devs;
    g->in_beg[i + 1] = g->n_ins;
    g->out_beg[i + 1] = g->n_outs;
    g->program_ops += mult;
}

/*
 * Simulate a program (Sec. 2.1 semantics; Sec. 3.3 trace and live memory).
 *  - start = max of the participants' clocks, end = start + cost, every
 *    participant's clock := end;
 *  - a tensor is live from its defining op (t = 0 for resident tensors)
 *    until the last op that reads it; a defined tensor nothing reads is freed
 *    right after its defining op; KEEP tensors (weights and optimizer state,
 *    updated in place) are never freed; resident tensors nothing reads stay;
 *  - every device the op touches samples its peak after the op's outputs
 *    are allocated and before its dead tensors are freed.
 * type_cost (optional, T_NTYPES entries, < 0 = no override) replaces the
 * duration of every op of a type; ocost[i] >= 0 replaces one op's duration.
 */
static int prog_simulate(const or_prog *g, int n_dev, const or_device_model *m,
                         const double *type_cost, double *finish, uint64_t *peak,
                         uint64_t *resident, double *tstart, double *tend)
{
    int64_t *last = NULL;
    uint8_t *freed = NULL;
    double *clk = NULL;
    uint64_t *live = NULL, *pk = NULL;
    int64_t i, t, q;
    int d, rc = 0;
    size_t nt = (size_t)(g->n_t > 0 ? g->n_t : 1);
    last = malloc(sizeof(int64_t) * nt);
    freed = calloc(nt, 1);
    clk = calloc((size_t)n_dev, sizeof(double));
    live = calloc((size_t)n_dev, sizeof(uint64_t));
    pk = calloc((size_t)n_dev, sizeof(uint64_t));
    if (!last || !freed || !clk || !live || !pk) { rc = -3; goto out; }
    for (t = 0; t < g->n_t; t++) last[t] = -1;
    for (i = 0; i < g->n_ops; i++)
        for (q = g->in_beg[i]; q < g->in_beg[i + 1]; q++) last[g->ins[q]] = i;
    for (i = 0; i < g->n_ops; i++)
        for (q = g->out_beg[i]; q < g->out_beg[i + 1]; q++)
            if (last[g->outs[q]] < i) last[g->outs[q]] = i;
    for (t = 0; t < g->n_t; t++) {
        if (g->t_dev[t] < 0 || g->t_dev[t] >= n_dev) { rc = -2; goto out; }
        if (g->t_flags[t] & TF_RESIDENT) live[g->t_dev[t]] += g->t_size[t];
    }
    for (d = 0; d < n_dev; d++) {
        pk[d] = live[d];
        if (resident) resident[d] = live[d];
    }
    for (i = 0; i < g->n_ops; i++) {
        double start = 0.0, end, cost;
        if (type_cost && type_cost[g->type[i]] >= 0.0) cost = type_cost[g->type[i]];
        else if (g->ocost[i] >= 0.0) cost = g->ocost[i];
        else {
            int spans;
            if (g->gfirst[i] >= 0) {
                int32_t ends[2];
                ends[0] = g->gfirst[i];
                ends[1] = g->glast[i];
                spans = spans_nodes(m, ends, 2);
            } else {
                spans = spans_nodes(m, g->devs + g->dev_beg[i], g->dev_beg[i + 1] - g->dev_beg[i]);
            }
            cost = or_cost_typed(m, g->kind[i], g->type[i], g->flops[i], g->bytes[i], g->kred[i], g->nsz[i],
                                 spans);
        }
        for (q = g->dev_beg[i]; q < g->dev_beg[i + 1]; q++) {
            d = g->devs[q];
            if (d < 0 || d >= n_dev) { rc = -2; goto out; }
            if (clk[d] > start) start = clk[d];
        }
        end = start + cost;
        for (q = g->dev_beg[i]; q < g->dev_beg[i + 1]; q++) clk[g->devs[q]] = end;
        if (tstart) tstart[i] = start;
        if (tend) tend[i] = end;
        for (q = g->out_beg[i]; q < g->out_beg[i + 1]; q++) {
            t = g->outs[q];
            live[g->t_dev[t]] += g->t_size[t];
        }
        for (q = g->dev_beg[i]; q < g->dev_beg[i + 1]; q++) {
            d = g->devs[q];
            if (live[d] > pk[d]) pk[d] = live[d];
        }
        for (q = g->out_beg[i]; q < g->out_beg[i + 1]; q++) {
            d = g->t_dev[g->outs[q]];
            if (live[d] > pk[d]) pk[d] = live[d];
        }
        for (q = g->in_beg[i]; q < g->in_beg[i + 1]; q++) {
            t = g->ins[q];
            if (last[t] == i && !(g->t_flags[t] & TF_KEEP) && !freed[t]) {
                live[g->t_dev[t]] -= g->t_size[t];
                freed[t] = 1;
            }
        }
        for (q = g->out_beg[i]; q < g->out_beg[i + 1]; q++) {
            t = g->outs[q];
            if (last[t] == i && !(g->t_flags[t] & TF_KEEP) && !freed[t]) {
                live[g->t_dev[t]] -= g->t_size[t];
                freed[t] = 1;
            }
        }
    }
    for (d = 0; d < n_dev; d++) {
        if (finish) finish[d] = clk[d];
        if (peak) peak[d] = pk[d];
    }
out:
    free(last); free(freed); free(clk); free(live); free(pk);
    return rc;
}

/*
 * Simulate an explicit program handed over as flat arrays (figure pins,
 * brute-force cross-checks).  cost[i] >= 0 gives an op's duration directly;
 * otherwise the cost model applies to (kind, flops, bytes, #participants).
 */
int or_sim_program(int64_t n_ops, const int32_t *kind, const double *cost,
                   const double *flops, const double *bytes,
                   const int64_t *dev_beg, const int32_t *devs,
                   const int64_t *in_beg, const int32_t *ins,
                   const int64_t *out_beg, const int32_t *outs,
                   int64_t n_t, const int32_t *t_dev, const uint64_t *t_size,
                   const int32_t *t_flags, int n_dev, const or_device_model *m,
                   double *finish, uint64_t *peak, double *tstart, double *tend,
                   const int32_t *is_matmul, const double *mm_k)
{
    or_prog g;
    int64_t i, q;
    int rc;
    prog_init(&g);
    for (q = 0; q < n_t; q++) prog_tensor(&g, t_dev[q], t_size[q], t_flags[q]);
    for (i = 0; i < n_ops; i++) {
        /* is_matmul (optional): the op multiplies two matrices (Sec. 4's
         * empirical MatMul cost applies when the device model has one) */
        op_begin(&g, kind[i], is_matmul && is_matmul[i] ? T_GEMM : T_GENERIC,
                 flops ? flops[i] : 0.0, bytes ? bytes[i] : 0.0);
        for (q = dev_beg[i]; q < dev_beg[i + 1]; q++) op_dev(&g, devs[q]);
        for (q = in_beg[i]; q < in_beg[i + 1]; q++) op_in(&g, ins[q]);
        for (q = out_beg[i]; q < out_beg[i + 1]; q++) op_out(&g, outs[q]);
        if (!g.failed && cost) g.ocost[i] = cost[i];
        /* mm_k (optional): a matrix multiplication's reduction length */
        if (!g.failed && mm_k) g.kred[i] = mm_k[i];
        op_end(&g, 0, 1);
    }
    if (g.failed) { prog_free(&g); return -3; }
    rc = prog_simulate(&g, n_dev, m, NULL, finish, peak, NULL, tstart, tend);
    prog_free(&g);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* The D/T/P(/K) transform (Sec. 4; Fig. 2 is its P = 2, K = 2 instance).    */
/*                                                                          */
/* Devices: dev = s*(D*H) + d*H + h  (stage s, data replica d, tensor rank  */
/* h).  Stage s holds the contiguous layer range [l0(s), l0(s+1)); with     */
/* L = q*P + r the first r stages get q+1 layers.  Replica d gets B/D rows  */
/* (sequences); microbatch k gets (B/D)/K rows plus one for k < (B/D)%K.    */
/* Each stage runs synchronous 1F1B: w = min(P-1-s, K) warm-up forwards,    */
/* then F/B pairs, then w backwards (or, with the GPipe schedule, all K     */
/* forwards then all K backwards); inference runs the K forwards.           */
/* The global op order follows slots: in slot t every stage, ascending,     */
/* emits its next block if the block's input was produced in an earlier     */
/* slot; then the Sends of the slot's results are emitted, ascending by     */
/* source stage; after the last slot every stage emits its weight update.  */
/* Within a block every template op is emitted for all replicas of the      */
/* stage before the next one (collectives once per group).                  */
/*                                                                          */
/* Activation recomputation (gradient checkpointing, Fig. 8): the forward   */
/* block is unchanged, but the backward no longer reads the activations it  */
/* produced inside the stage's layers, so def/use liveness frees them at    */
/* their last forward use; the block input (the checkpoint) and the block   */
/* output (read by the loss / the last stage's final LN) stay live.  The    */
/* backward block first runs what precedes the layers' backward (the loss   */
/* gradient; the transformer's head gradients), then replays from the       */
/* checkpoint, in forward order, every forward op of the stage's layers     */
/* whose result the layers' backward reads directly or through another     */
/* replayed op, and then runs the layers' backward on the replayed tensors. */
/* Ops whose results nothing would read are not replayed: the MLP's last    */
/* layer (its output is still live) and, in the transformer's last layer,  */
/* fc2, its all-reduce and the residual add.  For one stage of the 2-layer  */
/* MLP this is exactly the program of Fig. 8.                               */
/*                                                                          */
/* ZeRO partitioning (Fig. 9, training): every parameter group -- in model  */
/* order the embedding, each layer (an MLP column/row pair when H > 1) and  */
/* the LM head -- belongs to data replica (group index mod D), which alone  */
/* holds its weights and optimizer state.  Right before every op that reads */
/* a weight, its owner broadcasts it to the other replicas of the stage's   */
/* data-parallel group (one collective per tensor rank; for D = 2 the Send  */
/* of Fig. 9), and the copies die after that op.  Gradients accumulate on   */
/* every replica as before; at the weight update each is reduced onto its   */
/* owner (replacing the all-reduce), whose optimizer step consumes it.      */
/* Fig. 9's listing computes the owner's first layer before sending the     */
/* weight; the transform broadcasts before the op on every replica.         */
/*                                                                          */
/* In projection mode only the devices of replica (0,0) of every stage are  */
/* materialised (Sec. 3.2 projects a program onto devices by dropping the   */
/* ops that do not touch them); collectives keep their full group size for  */
/* the cost, and every skipped op is still counted in program_ops.          */
/* ------------------------------------------------------------------------ */
#define F_IN 0
#define F_XK 1
#define F_YK 2
#define F_RECVA 3
#define F_RECVG 4
#define F_OUTA 5
#define F_OUTG 6
#define F_XL 7
#define F_YF 8
#define F_LOGITS 9
#define F_LAYER0 16
#define NLF 9     /* saved fields per layer */
/* transformer per-layer saved fields */
#define L_X 0
#define L_Y1 1
#define L_QKV 2
#define L_PM 3
#define L_O 4
#define L_X2 5
#define L_Y2 6
#define L_U 7
#define L_GE 8
/* MLP per-layer saved field: the layer output */
#define L_A 0

typedef struct {
    const or_model *M;
    or_prog *g;
    int D, H, P, K, slice, train, fam, mode, rc, zero;
    int ov;               /* gradient all-reduce on the communication stream */
    int S;                /* devices (streams) per GPU: 1, or 2 with ov */
    int R;                /* replicas materialised per stage */
    int64_t e, rows;      /* element bytes, rows (sequences) per replica */
    int *l0;              /* P+1 stage boundaries */
    int nl_max, nslot, nps;
    int32_t *sv;          /* per (s, r, k) saved tensor ids */
    int32_t *W, *OS, *G;  /* per (s, r, param slot) */
    int32_t *GC;          /* per (s, r, param slot): the gradient's alias on the communication stream */
    int32_t *X, *Y;       /* per (s, r) resident inputs */
    int32_t *cur;         /* per r scratch */
    int32_t *tmp;         /* per r scratch */
    double mmk;           /* reduction length of the product emit_mm is emitting */
} mat;

/* Materialised replicas r of a stage: every (d, h) as r = d*H + h; in
 * projection mode replica (0,0) alone, or with ZeRO (whose replicas differ
 * in what they own) every data replica d of tensor rank 0 as r = d. */
static int rep_of(const mat *x, int d, int h)
{
    if (!x->slice) return d * x->H + h;
    return x->zero ? d : 0;
}

/* GPU of replica r of stage s: stage-major, then data replica, then tensor
 * rank */
static int gpu_of(const mat *x, int s, int r)
{
    if (x->slice && x->zero) return s * x->D * x->H + r * x->H;
    return s * x->D * x->H + r;
}

/* device of the replica's computation: its GPU, or with overlap the GPU's
 * first stream (device 2g); the GPU's second stream (2g + 1) carries the
 * data-parallel gradient all-reduce */
static int dev_of(const mat *x, int s, int r) { return x->S * gpu_of(x, s, r); }
static int comm_of(const mat *x, int s, int r) { return x->S * gpu_of(x, s, r) + 1; }

static int data_rep(const mat *x, int r)
{
    if (!x->slice) return r / x->H;
    return x->zero ? r : 0;
}

static int32_t *SV(mat *x, int s, int r, int k, int f)
{
    return &x->sv[(((int64_t)s * x->R + r) * x->K + k) * x->nslot + f];
}

static int32_t *PW(int32_t *a, const mat *x, int s, int r, int p)
{
    return &a[((int64_t)s * x->R + r) * x->nps + p];
}

static int64_t mb_rows(const mat *x, int k)
{
    return x->rows / x->K + (k < (int)(x->rows % x->K) ? 1 : 0);
}

/* multiplicities of one emitted op in projection mode */
static int64_t mult_dev(const mat *x) { return x->slice ? (int64_t)(x->zero ? 1 : x->D) * x->H : 1; }
static int64_t mult_tp(const mat *x) { return x->slice && !x->zero ? (int64_t)x->D : 1; }
static int64_t mult_dp(const mat *x) { return x->slice ? (int64_t)x->H : 1; }

/* one local compute op on every materialised replica: in1/in2/in3 arrays of
 * tensor ids per replica (NULL = absent), output sizes (0 = no output) */
static void emit_local(mat *x, int s, int type, double flops, double bytes,
                       const int32_t *in1, const int32_t *in2, const int32_t *in3,
                       uint64_t out_size, int32_t *out_ids,
                       uint64_t out2_size, int32_t *out2_ids)
{
    int r;
    for (r = 0; r < x->R; r++) {
        int dv = dev_of(x, s, r);
        int32_t o1 = -1, o2 = -1;
        if (out_size) o1 = prog_tensor(x->g, dv, out_size, 0);
        if (out2_size) o2 = prog_tensor(x->g, dv, out2_size, 0);
        op_begin(x->g, OR_COMPUTE, type, flops, bytes);
        if (!x->g->failed) x->g->kred[x->g->n_ops] = x->mmk;
        op_dev(x->g, dv);
        if (in1) op_in(x->g, in1[r]);
        if (in2) op_in(x->g, in2[r]);
        if (in3) op_in(x->g, in3[r]);
        if (out_size) op_out(x->g, o1);
        if (out2_size) op_out(x->g, o2);
        op_end(x->g, 0, mult_dev(x));
        if (out_ids) out_ids[r] = o1;
        if (out2_ids) out2_ids[r] = o2;
    }
}

/* a matrix multiplication whose products reduce over k (the sum of the
 * reduction lengths when one op stands for several products) */
static void emit_mm(mat *x, int s, int type, int64_t k, double flops, double bytes,
                    const int32_t *in1, const int32_t *in2, const int32_t *in3,
                    uint64_t out_size, int32_t *out_ids, uint64_t out2_size, int32_t *out2_ids)
{
    x->mmk = (double)k;
    emit_local(x, s, type, flops, bytes, in1, in2, in3, out_size, out_ids, out2_size, out2_ids);
    x->mmk = 0.0;
}

/* all-reduce over the tensor-parallel group of every data replica */
static void emit_ar_tp(mat *x, int s, int type, double bytes, const int32_t *t)
{
    int d, h, nd = x->slice && !x->zero ? 1 : x->D, nh = x->slice ? 1 : x->H;
    if (x->H <= 1) return;
    for (d = 0; d < nd; d++) {
        int first = s * x->D * x->H + d * x->H;
        op_begin(x->g, OR_ALLREDUCE, type, 0.0, bytes);
        op_group(x->g, x->S * first, x->S * (first + x->H - 1));
        for (h = 0; h < nh; h++) {
            int r = rep_of(x, d, h);
            op_dev(x->g, dev_of(x, s, r));
            op_in(x->g, t[r]);
        }
        op_end(x->g, x->H, mult_tp(x));
    }
}

/* the op being built runs over the D data replicas of tensor rank h (on
 * stream `stream` of their GPUs) */
static void dp_group_on(mat *x, int s, int h, int stream)
{
    int base = s * x->D * x->H;
    op_group(x->g, x->S * (base + h) + stream, x->S * (base + (x->D - 1) * x->H + h) + stream);
}
static void dp_group(mat *x, int s, int h) { dp_group_on(x, s, h, 0); }

/* all-reduce over the data-parallel group of every tensor rank */
static void emit_ar_dp(mat *x, int s, double bytes, int p)
{
    int d, h, nd = x->slice ? 1 : x->D, nh = x->slice ? 1 : x->H;
    if (x->D <= 1) return;
    for (h = 0; h < nh; h++) {
        op_begin(x->g, OR_ALLREDUCE, T_AR_DP, 0.0, bytes);
        dp_group(x, s, h);
        for (d = 0; d < nd; d++) {
            int r = d * x->H + h;
            op_dev(x->g, dev_of(x, s, r));
            op_in(x->g, *PW(x->G, x, s, r, p));
        }
        op_end(x->g, x->D, mult_dp(x));
    }
}

/* Overlap (Sec. 2.2, Limitations: one device per stream, the streams of a
 * GPU exchanging tensors at low or zero cost).  Once the last microbatch
 * has finished a weight gradient, every replica hands it to its GPU's
 * communication stream (a Send between the GPU's two streams; the copy
 * aliases the gradient's memory, so it allocates nothing), and the
 * communication streams of the D data replicas all-reduce it there while
 * the computation stream goes on with the backward pass.  One data replica
 * has nothing to reduce. */
static void grad_final(mat *x, int s, int k, int p, uint64_t nparam)
{
    int r, d, h, nd, nh;
    double by = (double)((uint64_t)x->e * nparam);
    if (!x->ov || x->D <= 1 || k != x->K - 1) return;
    for (r = 0; r < x->R; r++) {
        int32_t c = prog_tensor(x->g, comm_of(x, s, r), 0, 0);
        op_begin(x->g, OR_SEND, T_STREAM, 0.0, by);
        op_dev(x->g, dev_of(x, s, r));
        op_dev(x->g, comm_of(x, s, r));
        op_in(x->g, *PW(x->G, x, s, r, p));
        op_out(x->g, c);
        op_end(x->g, 0, mult_dev(x));
        *PW(x->GC, x, s, r, p) = c;
    }
    nd = x->slice ? 1 : x->D;
    nh = x->slice ? 1 : x->H;
    for (h = 0; h < nh; h++) {
        op_begin(x->g, OR_ALLREDUCE, T_AR_DP, 0.0, by);
        dp_group_on(x, s, h, 1);
        for (d = 0; d < nd; d++) {
            r = d * x->H + h;
            op_dev(x->g, comm_of(x, s, r));
            op_in(x->g, *PW(x->GC, x, s, r, p));
        }
        op_end(x->g, x->D, mult_dp(x));
    }
}

/* gradient accumulation: microbatch 0's weight gradient becomes the
 * accumulator, later ones are added into it in place; after microbatch k
 * the gradient may be final (overlap) */
static void accumulate(mat *x, int s, int k, int p, uint64_t nparam, const int32_t *gw)
{
    int r;
    if (*PW(x->G, x, s, 0, p) < 0) {
        for (r = 0; r < x->R; r++) *PW(x->G, x, s, r, p) = gw[r];
        grad_final(x, s, k, p, nparam);
        return;
    }
    for (r = 0; r < x->R; r++) {
        int dv = dev_of(x, s, r);
        op_begin(x->g, OR_COMPUTE, T_ADDGRAD, (double)nparam, (double)(3 * x->e * nparam));
        op_dev(x->g, dv);
        op_in(x->g, *PW(x->G, x, s, r, p));
        op_in(x->g, gw[r]);
        op_end(x->g, 0, mult_dev(x));
    }
    grad_final(x, s, k, p, nparam);
}

static void gather_sv(mat *x, int s, int k, int f, int32_t *dst)
{
    int r;
    for (r = 0; r < x->R; r++) dst[r] = *SV(x, s, r, k, f);
}

static void store_sv(mat *x, int s, int k, int f, const int32_t *src)
{
    int r;
    for (r = 0; r < x->R; r++) *SV(x, s, r, k, f) = src[r];
}

static void gather_pw(mat *x, int32_t *a, int s, int p, int32_t *dst)
{
    int r;
    for (r = 0; r < x->R; r++) dst[r] = *PW(a, x, s, r, p);
}

static void use_weight(mat *x, int s, int p, int32_t *dst);

/* ---- MLP: square d x d layers, @dense = Gemm + Relu (Fig. 2) ----------- */
/* With H > 1 even layers are column-parallel (W: d x d/H, local Relu) and  */
/* odd layers row-parallel (W: d/H x d, AllReduce of the output over the H  */
/* group before Relu); backward all-reduces dX of column-parallel layers.   */
static void mlp_dims(const mat *x, int i, int64_t *din, int64_t *dout, int *row)
{
    int64_t d = x->M->d_model;
    int col = x->H > 1 && (i % 2) == 0;
    *row = x->H > 1 && (i % 2) == 1;
    *din = *row ? d / x->H : d;
    *dout = col ? d / x->H : d;
}

/* layer i forward on microbatch k: cur (layer input ids) -> cur (output) */
static void mlp_layer(mat *x, int s, int k, int i, int32_t *cur, int32_t *tmp)
{
    int64_t m = mb_rows(x, k), e = x->e, din, dout;
    int32_t w[1024];
    int row;
    mlp_dims(x, i, &din, &dout, &row);
    use_weight(x, s, i - x->l0[s], w);
    emit_mm(x, s, T_GEMM, din, (double)(2 * m * din * dout), (double)(e * (m * din + din * dout + m * dout)),
               cur, w, NULL, (uint64_t)(e * m * dout), tmp, 0, NULL);
    if (row) emit_ar_tp(x, s, T_AR_TP, (double)(e * m * dout), tmp);
    emit_local(x, s, T_RELU, (double)(m * dout), (double)(2 * e * m * dout),
               tmp, NULL, NULL, (uint64_t)(e * m * dout), cur, 0, NULL);
    store_sv(x, s, k, F_LAYER0 + (i - x->l0[s]) * NLF + L_A, cur);
}

static void mlp_fwd(mat *x, int s, int k)
{
    int32_t *cur = x->cur, *tmp = x->tmp;
    int i, r;
    if (s == 0) {
        if (x->K > 1) gather_sv(x, s, k, F_XK, cur);
        else for (r = 0; r < x->R; r++) cur[r] = x->X[s * x->R + r];
    } else {
        gather_sv(x, s, k, F_RECVA, cur);
    }
    store_sv(x, s, k, F_IN, cur);
    for (i = x->l0[s]; i < x->l0[s + 1]; i++) mlp_layer(x, s, k, i, cur, tmp);
    store_sv(x, s, k, F_OUTA, cur);
}

static void mlp_bwd(mat *x, int s, int k)
{
    int64_t m = mb_rows(x, k), e = x->e, d = x->M->d_model, din, dout;
    int32_t *cur = x->cur, *tmp = x->tmp;
    int32_t a[1024], xin[1024], w[1024], gw[1024];
    int i, row;
    if (s == x->P - 1) {
        int32_t y[1024];
        gather_sv(x, s, k, F_LAYER0 + (x->l0[s + 1] - 1 - x->l0[s]) * NLF + L_A, a);
        if (x->K > 1) gather_sv(x, s, k, F_YK, y);
        else { int r; for (r = 0; r < x->R; r++) y[r] = x->Y[s * x->R + r]; }
        emit_local(x, s, T_LOSSGRAD, (double)(3 * m * d), (double)(3 * e * m * d),
                   a, y, NULL, (uint64_t)(e * m * d), cur, 0, NULL);
    } else {
        gather_sv(x, s, k, F_RECVG, cur);
    }
    if (x->rc) {
        /* replay every layer but the last from the checkpoint; the replayed
         * outputs replace the saved ones the layers' backward reads */
        int32_t ra[1024], rt[1024];
        gather_sv(x, s, k, F_IN, ra);
        for (i = x->l0[s]; i < x->l0[s + 1] - 1; i++) mlp_layer(x, s, k, i, ra, rt);
    }
    for (i = x->l0[s + 1] - 1; i >= x->l0[s]; i--) {
        int li = i - x->l0[s];
        mlp_dims(x, i, &din, &dout, &row);
        gather_sv(x, s, k, F_LAYER0 + li * NLF + L_A, a);
        emit_local(x, s, T_RELUGRAD, (double)(m * dout), (double)(3 * e * m * dout),
                   cur, a, NULL, (uint64_t)(e * m * dout), tmp, 0, NULL);
        if (i == x->l0[s]) gather_sv(x, s, k, F_IN, xin);
        else gather_sv(x, s, k, F_LAYER0 + (li - 1) * NLF + L_A, xin);
        emit_mm(x, s, T_GEMMDW, m, (double)(2 * m * din * dout), (double)(e * (m * din + m * dout + din * dout)),
                   xin, tmp, NULL, (uint64_t)(e * din * dout), gw, 0, NULL);
        accumulate(x, s, k, li, (uint64_t)(din * dout), gw);
        use_weight(x, s, li, w);
        emit_mm(x, s, T_GEMMDX, dout, (double)(2 * m * din * dout), (double)(e * (m * dout + din * dout + m * din)),
                   tmp, w, NULL, (uint64_t)(e * m * din), cur, 0, NULL);
        if (!row && x->H > 1 && i != 0) emit_ar_tp(x, s, T_AR_TP, (double)(e * m * din), cur);
    }
    if (s > 0) store_sv(x, s, k, F_OUTG, cur);
}

static uint64_t mlp_param(const mat *x, int s, int p)
{
    int64_t din, dout;
    int row;
    mlp_dims(x, x->l0[s] + p, &din, &dout, &row);
    return (uint64_t)(din * dout);
}

/* ---- Transformer (GPT-2 shaped decoder, Megatron tensor parallelism) --- */
typedef struct {
    int64_t m, T, s, d, dH, aH, hd, FH, Vh, e;
    int64_t ACT, QKV, OH, S2, FF, LOG, ST, IDS;
} tfdims;

static void tf_dims(const mat *x, int k, tfdims *t)
{
    const or_model *M = x->M;
    t->e = x->e;
    t->m = mb_rows(x, k);
    t->s = M->seq_len;
    t->T = t->m * t->s;
    t->d = M->d_model;
    t->dH = M->d_model / x->H;
    t->aH = M->n_heads / x->H;
    t->hd = M->d_model / M->n_heads;   /* one head's width */
    t->FH = M->d_ff / x->H;
    t->Vh = (M->vocab + x->H - 1) / x->H;
    t->ACT = t->e * t->T * t->d;
    t->QKV = t->e * t->T * 3 * t->dH;
    t->OH = t->e * t->T * t->dH;
    t->S2 = t->e * t->m * t->aH * t->s * t->s;
    t->FF = t->e * t->T * t->FH;
    t->LOG = t->e * t->T * t->Vh;
    t->ST = 12 * t->T;
    t->IDS = 4 * t->T;
}

/* parameter slot p of stage s: 4 per layer (qkv, out, fc1, fc2), then the
 * embedding (stage 0) and the LM head (last stage) */
static uint64_t tf_param(const mat *x, int s, int p)
{
    const or_model *M = x->M;
    int64_t d = M->d_model, dH = d / x->H, FH = M->d_ff / x->H;
    int64_t Vh = (M->vocab + x->H - 1) / x->H;
    int nl = x->l0[s + 1] - x->l0[s];
    (void)s;
    if (p < 4 * nl) {
        switch (p % 4) {
        case 0: return (uint64_t)(d * 3 * dH);
        case 1: return (uint64_t)(dH * d);
        case 2: return (uint64_t)(d * FH);
        default: return (uint64_t)(FH * d);
        }
    }
    return (uint64_t)(Vh * d);
}

static int tf_slot_emb(const mat *x) { return 4 * x->nl_max; }
static int tf_slot_head(const mat *x) { return 4 * x->nl_max + 1; }

/* ZeRO (Fig. 9 gives each weight and its gradient to one device): the
 * model's parameters form groups in model order -- the transformer's
 * embedding, every layer (with H > 1 an MLP column/row pair), the LM head --
 * and group g belongs to data replica g mod D of every stage replica set. */
static int owner_of(const mat *x, int s, int p)
{
    int g;
    if (x->fam == FAM_MLP) {
        int i = x->l0[s] + p;
        g = x->H > 1 ? i / 2 : i;
    } else if (p == tf_slot_emb(x)) {
        g = 0;
    } else if (p == tf_slot_head(x)) {
        g = x->M->n_layers + 1;
    } else {
        g = x->l0[s] + p / 4 + 1;
    }
    return g % x->D;
}

/* The weight of slot p as every materialised replica reads it: its own
 * tensor, or with ZeRO on a non-owner a copy that the owner broadcasts to
 * the other replicas of its data-parallel group right before the use (the
 * Sends of Fig. 9 for D = 2); the copy dies after that use. */
static void use_weight(mat *x, int s, int p, int32_t *dst)
{
    int d, h, o, nh;
    if (!x->zero || x->D == 1) { gather_pw(x, x->W, s, p, dst); return; }
    o = owner_of(x, s, p);
    nh = x->slice ? 1 : x->H;
    for (h = 0; h < nh; h++) {
        int32_t src = *PW(x->W, x, s, rep_of(x, o, h), p);
        uint64_t sz = x->g->failed ? 0 : x->g->t_size[src];
        for (d = 0; d < x->D; d++) {
            int r = rep_of(x, d, h);
            dst[r] = d == o ? src : prog_tensor(x->g, dev_of(x, s, r), sz, 0);
        }
        op_begin(x->g, OR_BCAST, T_BCAST, 0.0, (double)sz);
        dp_group(x, s, h);
        for (d = 0; d < x->D; d++) op_dev(x->g, dev_of(x, s, rep_of(x, d, h)));
        op_in(x->g, src);
        for (d = 0; d < x->D; d++)
            if (d != o) op_out(x->g, dst[rep_of(x, d, h)]);
        op_end(x->g, 0, mult_dp(x));
    }
}

/* layer li of stage s on microbatch k: cur (layer input ids) -> cur
 * (output), storing the activations the layer's backward reads.  full == 0
 * stops after GeLU: fc2, its all-reduce and the residual add only produce
 * the layer output. */
static void tf_layer(mat *x, int s, int k, int li, const tfdims *tp, int32_t *cur, int full)
{
    const tfdims t = *tp;
    int32_t w[1024], y1[1024], qkv[1024], S[1024], pm[1024], o[1024], z[1024], x2[1024],
            y2[1024], u[1024], ge[1024], v[1024];
    int base = F_LAYER0 + li * NLF;
    store_sv(x, s, k, base + L_X, cur);
    emit_local(x, s, T_LN, (double)(8 * t.T * t.d), (double)(2 * t.ACT), cur, NULL, NULL, (uint64_t)t.ACT, y1, 0, NULL);
    use_weight(x, s, 4 * li + 0, w);
    emit_mm(x, s, T_QKV, t.d, (double)(2 * t.T * t.d * 3 * t.dH),
               (double)(t.e * (t.T * t.d + t.d * 3 * t.dH + t.T * 3 * t.dH)),
               y1, w, NULL, (uint64_t)t.QKV, qkv, 0, NULL);
    emit_mm(x, s, T_SCORES, t.hd, (double)(2 * t.T * t.s * t.dH), (double)(2 * t.OH + t.S2),
               qkv, NULL, NULL, (uint64_t)t.S2, S, 0, NULL);
    emit_local(x, s, T_SOFTMAX, (double)(5 * t.m * t.aH * t.s * t.s), (double)(2 * t.S2),
               S, NULL, NULL, (uint64_t)t.S2, pm, 0, NULL);
    emit_mm(x, s, T_AV, t.s, (double)(2 * t.T * t.s * t.dH), (double)(t.S2 + 2 * t.OH),
               pm, qkv, NULL, (uint64_t)t.OH, o, 0, NULL);
    use_weight(x, s, 4 * li + 1, w);
    emit_mm(x, s, T_OUTPROJ, t.dH, (double)(2 * t.T * t.dH * t.d),
               (double)(t.e * (t.T * t.dH + t.dH * t.d + t.T * t.d)),
               o, w, NULL, (uint64_t)t.ACT, z, 0, NULL);
    emit_ar_tp(x, s, T_AR_TP, (double)t.ACT, z);
    emit_local(x, s, T_RESADD, (double)(t.T * t.d), (double)(3 * t.ACT), cur, z, NULL, (uint64_t)t.ACT, x2, 0, NULL);
    emit_local(x, s, T_LN, (double)(8 * t.T * t.d), (double)(2 * t.ACT), x2, NULL, NULL, (uint64_t)t.ACT, y2, 0, NULL);
    use_weight(x, s, 4 * li + 2, w);
    emit_mm(x, s, T_FC1, t.d, (double)(2 * t.T * t.d * t.FH),
               (double)(t.e * (t.T * t.d + t.d * t.FH + t.T * t.FH)),
               y2, w, NULL, (uint64_t)t.FF, u, 0, NULL);
    emit_local(x, s, T_GELU, (double)(8 * t.T * t.FH), (double)(2 * t.FF), u, NULL, NULL, (uint64_t)t.FF, ge, 0, NULL);
    store_sv(x, s, k, base + L_Y1, y1);
    store_sv(x, s, k, base + L_QKV, qkv);
    store_sv(x, s, k, base + L_PM, pm);
    store_sv(x, s, k, base + L_O, o);
    store_sv(x, s, k, base + L_X2, x2);
    store_sv(x, s, k, base + L_Y2, y2);
    store_sv(x, s, k, base + L_U, u);
    store_sv(x, s, k, base + L_GE, ge);
    if (!full) return;
    use_weight(x, s, 4 * li + 3, w);
    emit_mm(x, s, T_FC2, t.FH, (double)(2 * t.T * t.FH * t.d),
               (double)(t.e * (t.T * t.FH + t.FH * t.d + t.T * t.d)),
               ge, w, NULL, (uint64_t)t.ACT, v, 0, NULL);
    emit_ar_tp(x, s, T_AR_TP, (double)t.ACT, v);
    emit_local(x, s, T_RESADD, (double)(t.T * t.d), (double)(3 * t.ACT), x2, v, NULL, (uint64_t)t.ACT, cur, 0, NULL);
}

static void tf_fwd(mat *x, int s, int k)
{
    tfdims t;
    int32_t *cur = x->cur;
    int32_t w[1024];
    int i, r;
    tf_dims(x, k, &t);
    if (s == 0) {
        int32_t tok[1024];
        if (x->K > 1) gather_sv(x, s, k, F_XK, tok);
        else for (r = 0; r < x->R; r++) tok[r] = x->X[s * x->R + r];
        use_weight(x, s, tf_slot_emb(x), w);
        emit_local(x, s, T_EMBED, (double)(t.T * t.d), (double)(2 * t.ACT + t.IDS),
                   tok, w, NULL, (uint64_t)t.ACT, cur, 0, NULL);
        emit_ar_tp(x, s, T_AR_TP, (double)t.ACT, cur);
    } else {
        gather_sv(x, s, k, F_RECVA, cur);
    }
    store_sv(x, s, k, F_IN, cur);
    for (i = x->l0[s]; i < x->l0[s + 1]; i++) tf_layer(x, s, k, i - x->l0[s], &t, cur, 1);
    if (s == x->P - 1) {
        int32_t yf[1024], lg[1024];
        store_sv(x, s, k, F_XL, cur);
        emit_local(x, s, T_LN, (double)(8 * t.T * t.d), (double)(2 * t.ACT), cur, NULL, NULL, (uint64_t)t.ACT, yf, 0, NULL);
        use_weight(x, s, tf_slot_head(x), w);
        emit_mm(x, s, T_LMHEAD, t.d, (double)(2 * t.T * t.d * t.Vh),
                   (double)(t.e * (t.T * t.d + t.d * t.Vh + t.T * t.Vh)),
                   yf, w, NULL, (uint64_t)t.LOG, lg, 0, NULL);
        store_sv(x, s, k, F_YF, yf);
        store_sv(x, s, k, F_LOGITS, lg);
    } else {
        store_sv(x, s, k, F_OUTA, cur);
    }
}

static void tf_bwd(mat *x, int s, int k)
{
    tfdims t;
    int32_t *cur = x->cur;
    int32_t w[1024], a1[1024], a2[1024], gw[1024], dg[1024], du[1024], dy[1024], dxa[1024],
            dx2[1024], dO[1024], dP[1024], dq[1024], dS[1024];
    int i, r;
    tf_dims(x, k, &t);
    if (s == x->P - 1) {
        int32_t lg[1024], st[1024], lab[1024], dl[1024], yf[1024], xl[1024];
        gather_sv(x, s, k, F_LOGITS, lg);
        emit_local(x, s, T_XENT_STATS, (double)(3 * t.T * t.Vh), (double)(t.LOG + t.ST),
                   lg, NULL, NULL, (uint64_t)t.ST, st, 0, NULL);
        emit_ar_tp(x, s, T_AR_TP, (double)t.ST, st);
        if (x->K > 1) gather_sv(x, s, k, F_YK, lab);
        else for (r = 0; r < x->R; r++) lab[r] = x->Y[s * x->R + r];
        emit_local(x, s, T_XENT_GRAD, (double)(2 * t.T * t.Vh), (double)(2 * t.LOG + t.ST + t.IDS),
                   lg, st, lab, (uint64_t)t.LOG, dl, 0, NULL);
        use_weight(x, s, tf_slot_head(x), w);
        emit_mm(x, s, T_GEMMDX, t.Vh, (double)(2 * t.T * t.d * t.Vh),
                   (double)(t.e * (t.T * t.Vh + t.d * t.Vh + t.T * t.d)),
                   dl, w, NULL, (uint64_t)t.ACT, dy, 0, NULL);
        emit_ar_tp(x, s, T_AR_TP, (double)t.ACT, dy);
        gather_sv(x, s, k, F_YF, yf);
        emit_mm(x, s, T_GEMMDW, t.T, (double)(2 * t.T * t.d * t.Vh),
                   (double)(t.e * (t.T * t.d + t.T * t.Vh + t.d * t.Vh)),
                   yf, dl, NULL, (uint64_t)(t.e * t.d * t.Vh), gw, 0, NULL);
        accumulate(x, s, k, tf_slot_head(x), (uint64_t)(t.d * t.Vh), gw);
        gather_sv(x, s, k, F_XL, xl);
        emit_local(x, s, T_LN_B, (double)(8 * t.T * t.d), (double)(3 * t.ACT),
                   dy, xl, NULL, (uint64_t)t.ACT, cur, 0, NULL);
    } else {
        gather_sv(x, s, k, F_RECVG, cur);
    }
    if (x->rc) {
        /* replay the stage's layers from the checkpoint; the last one stops
         * after GeLU (nothing reads the rest) */
        int32_t ra[1024];
        int nl = x->l0[s + 1] - x->l0[s];
        gather_sv(x, s, k, F_IN, ra);
        for (i = 0; i < nl; i++) tf_layer(x, s, k, i, &t, ra, i < nl - 1);
    }
    for (i = x->l0[s + 1] - 1; i >= x->l0[s]; i--) {
        int li = i - x->l0[s], base = F_LAYER0 + li * NLF;
        use_weight(x, s, 4 * li + 3, w);
        emit_mm(x, s, T_GEMMDX, t.d, (double)(2 * t.T * t.FH * t.d),
                   (double)(t.e * (t.T * t.d + t.FH * t.d + t.T * t.FH)),
                   cur, w, NULL, (uint64_t)t.FF, dg, 0, NULL);
        gather_sv(x, s, k, base + L_GE, a1);
        emit_mm(x, s, T_GEMMDW, t.T, (double)(2 * t.T * t.FH * t.d),
                   (double)(t.e * (t.T * t.FH + t.T * t.d + t.FH * t.d)),
                   a1, cur, NULL, (uint64_t)(t.e * t.FH * t.d), gw, 0, NULL);
        accumulate(x, s, k, 4 * li + 3, (uint64_t)(t.FH * t.d), gw);
        gather_sv(x, s, k, base + L_U, a1);
        emit_local(x, s, T_GELU_B, (double)(8 * t.T * t.FH), (double)(3 * t.FF),
                   dg, a1, NULL, (uint64_t)t.FF, du, 0, NULL);
        use_weight(x, s, 4 * li + 2, w);
        emit_mm(x, s, T_GEMMDX, t.FH, (double)(2 * t.T * t.d * t.FH),
                   (double)(t.e * (t.T * t.FH + t.d * t.FH + t.T * t.d)),
                   du, w, NULL, (uint64_t)t.ACT, dy, 0, NULL);
        emit_ar_tp(x, s, T_AR_TP, (double)t.ACT, dy);
        gather_sv(x, s, k, base + L_Y2, a1);
        emit_mm(x, s, T_GEMMDW, t.T, (double)(2 * t.T * t.d * t.FH),
                   (double)(t.e * (t.T * t.d + t.T * t.FH + t.d * t.FH)),
                   a1, du, NULL, (uint64_t)(t.e * t.d * t.FH), gw, 0, NULL);
        accumulate(x, s, k, 4 * li + 2, (uint64_t)(t.d * t.FH), gw);
        gather_sv(x, s, k, base + L_X2, a1);
        emit_local(x, s, T_LN_B, (double)(8 * t.T * t.d), (double)(3 * t.ACT),
                   dy, a1, NULL, (uint64_t)t.ACT, dxa, 0, NULL);
        emit_local(x, s, T_RESADD_B, (double)(t.T * t.d), (double)(3 * t.ACT),
                   cur, dxa, NULL, (uint64_t)t.ACT, dx2, 0, NULL);
        use_weight(x, s, 4 * li + 1, w);
        emit_mm(x, s, T_GEMMDX, t.d, (double)(2 * t.T * t.dH * t.d),
                   (double)(t.e * (t.T * t.d + t.dH * t.d + t.T * t.dH)),
                   dx2, w, NULL, (uint64_t)t.OH, dO, 0, NULL);
        gather_sv(x, s, k, base + L_O, a1);
        emit_mm(x, s, T_GEMMDW, t.T, (double)(2 * t.T * t.dH * t.d),
                   (double)(t.e * (t.T * t.dH + t.T * t.d + t.dH * t.d)),
                   a1, dx2, NULL, (uint64_t)(t.e * t.dH * t.d), gw, 0, NULL);
        accumulate(x, s, k, 4 * li + 1, (uint64_t)(t.dH * t.d), gw);
        gather_sv(x, s, k, base + L_PM, a1);
        gather_sv(x, s, k, base + L_QKV, a2);
        emit_mm(x, s, T_AV_B, t.hd + t.s, (double)(4 * t.T * t.s * t.dH), (double)(2 * t.S2 + 3 * t.OH),
                   dO, a1, a2, (uint64_t)t.S2, dP, (uint64_t)t.QKV, dq);
        emit_local(x, s, T_SOFTMAX_B, (double)(5 * t.m * t.aH * t.s * t.s), (double)(3 * t.S2),
                   dP, a1, NULL, (uint64_t)t.S2, dS, 0, NULL);
        emit_mm(x, s, T_SCORES_B, 2 * t.s, (double)(4 * t.T * t.s * t.dH), (double)(t.S2 + 4 * t.OH),
                   dS, a2, dq, 0, NULL, 0, NULL);
        use_weight(x, s, 4 * li + 0, w);
        emit_mm(x, s, T_GEMMDX, 3 * t.dH, (double)(2 * t.T * 3 * t.dH * t.d),
                   (double)(t.e * (t.T * 3 * t.dH + 3 * t.dH * t.d + t.T * t.d)),
                   dq, w, NULL, (uint64_t)t.ACT, dy, 0, NULL);
        emit_ar_tp(x, s, T_AR_TP, (double)t.ACT, dy);
        gather_sv(x, s, k, base + L_Y1, a1);
        emit_mm(x, s, T_GEMMDW, t.T, (double)(2 * t.T * t.d * 3 * t.dH),
                   (double)(t.e * (t.T * t.d + t.T * 3 * t.dH + t.d * 3 * t.dH)),
                   a1, dq, NULL, (uint64_t)(t.e * t.d * 3 * t.dH), gw, 0, NULL);
        accumulate(x, s, k, 4 * li + 0, (uint64_t)(t.d * 3 * t.dH), gw);
        gather_sv(x, s, k, base + L_X, a1);
        emit_local(x, s, T_LN_B, (double)(8 * t.T * t.d), (double)(3 * t.ACT),
                   dy, a1, NULL, (uint64_t)t.ACT, dxa, 0, NULL);
        emit_local(x, s, T_RESADD_B, (double)(t.T * t.d), (double)(3 * t.ACT),
                   dx2, dxa, NULL, (uint64_t)t.ACT, cur, 0, NULL);
    }
    if (s == 0) {
        int32_t tok[1024];
        if (x->K > 1) gather_sv(x, s, k, F_XK, tok);
        else for (r = 0; r < x->R; r++) tok[r] = x->X[s * x->R + r];
        emit_local(x, s, T_EMBED_DW, (double)(t.T * t.d), (double)(t.ACT + t.IDS + t.e * t.Vh * t.d),
                   cur, tok, NULL, (uint64_t)(t.e * t.Vh * t.d), gw, 0, NULL);
        accumulate(x, s, k, tf_slot_emb(x), (uint64_t)(t.Vh * t.d), gw);
    } else {
        store_sv(x, s, k, F_OUTG, cur);
    }
}

/* ---- shared pieces: splits, sends, weight update ----------------------- */
static uint64_t input_row_bytes(const mat *x)
{
    /* one row of the stage-0 input / last-stage target */
    if (x->fam == FAM_MLP) return (uint64_t)(x->e * x->M->d_model);
    return (uint64_t)(4 * x->M->seq_len);
}

static void emit_split(mat *x, int s, int which)
{
    int r, k;
    uint64_t rb = input_row_bytes(x), whole = rb * (uint64_t)x->rows;
    int32_t *ids = malloc(sizeof(int32_t) * (size_t)x->K);
    if (!ids) { x->g->failed = 1; return; }
    for (r = 0; r < x->R; r++) {
        int dv = dev_of(x, s, r);
        int32_t src = which == 0 ? x->X[s * x->R + r] : x->Y[s * x->R + r];
        for (k = 0; k < x->K; k++) ids[k] = prog_tensor(x->g, dv, rb * (uint64_t)mb_rows(x, k), 0);
        op_begin(x->g, OR_COMPUTE, T_SPLIT, 0.0, (double)(2 * whole));
        op_dev(x->g, dv);
        op_in(x->g, src);
        for (k = 0; k < x->K; k++) op_out(x->g, ids[k]);
        op_end(x->g, 0, mult_dev(x));
        for (k = 0; k < x->K; k++) *SV(x, s, r, k, which == 0 ? F_XK : F_YK) = ids[k];
    }
    free(ids);
}

static void emit_send(mat *x, int s, int k, int fwd)
{
    int r, s2 = fwd ? s + 1 : s - 1;
    for (r = 0; r < x->R; r++) {
        int32_t src = *SV(x, s, r, k, fwd ? F_OUTA : F_OUTG);
        uint64_t sz = x->g->t_size[src];
        int32_t dst = prog_tensor(x->g, dev_of(x, s2, r), sz, 0);
        op_begin(x->g, OR_SEND, fwd ? T_SEND_F : T_SEND_B, 0.0, (double)sz);
        op_dev(x->g, dev_of(x, s, r));
        op_dev(x->g, dev_of(x, s2, r));
        op_in(x->g, src);
        op_out(x->g, dst);
        op_end(x->g, 0, mult_dev(x));
        *SV(x, s2, r, k, fwd ? F_RECVA : F_RECVG) = dst;
    }
}

static void opt_cost(const mat *x, uint64_t n, double *flops, double *bytes)
{
    if (x->mode == MODE_SGD) { *flops = (double)(2 * n); *bytes = (double)(3 * (uint64_t)x->e * n); }
    else if (x->mode == MODE_ADAM) { *flops = (double)(12 * n); *bytes = (double)(7 * (uint64_t)x->e * n); }
    else { *flops = (double)(12 * n); *bytes = (double)(28 * n); }
}

static uint64_t opt_state_bytes(const mat *x, uint64_t n)
{
    if (x->mode == MODE_ADAM) return 2 * (uint64_t)x->e * n;
    if (x->mode == MODE_ADAM_MIXED) return 12 * n;
    return 0;
}

static void emit_wu_slot(mat *x, int s, int p, uint64_t n)
{
    double fl, by;
    int r;
    opt_cost(x, n, &fl, &by);
    if (x->zero && x->D > 1) {
        /* ZeRO (Fig. 9): reduce the gradient onto its owner (every
         * replica's accumulated gradient dies there), then the owner's
         * optimizer step consumes the reduced gradient */
        int d, h, o = owner_of(x, s, p), nh = x->slice ? 1 : x->H;
        for (h = 0; h < nh; h++) {
            int ro = rep_of(x, o, h);
            int32_t red = prog_tensor(x->g, dev_of(x, s, ro), (uint64_t)x->e * n, 0);
            op_begin(x->g, OR_REDUCE, T_REDUCE, 0.0, (double)((uint64_t)x->e * n));
            dp_group(x, s, h);
            for (d = 0; d < x->D; d++) op_dev(x->g, dev_of(x, s, rep_of(x, d, h)));
            for (d = 0; d < x->D; d++) op_in(x->g, *PW(x->G, x, s, rep_of(x, d, h), p));
            op_out(x->g, red);
            op_end(x->g, 0, mult_dp(x));
            op_begin(x->g, OR_COMPUTE, T_OPT, fl, by);
            op_dev(x->g, dev_of(x, s, ro));
            op_in(x->g, *PW(x->W, x, s, ro, p));
            op_in(x->g, red);
            if (*PW(x->OS, x, s, ro, p) >= 0) op_in(x->g, *PW(x->OS, x, s, ro, p));
            op_end(x->g, 0, mult_dp(x));
        }
        return;
    }
    if (x->ov && x->D > 1) {
        /* overlap: the reduced gradient comes back from the communication
         * stream (into the gradient's own memory) before the optimizer */
        for (r = 0; r < x->R; r++) {
            op_begin(x->g, OR_SEND, T_STREAM, 0.0, (double)((uint64_t)x->e * n));
            op_dev(x->g, comm_of(x, s, r));
            op_dev(x->g, dev_of(x, s, r));
            op_in(x->g, *PW(x->GC, x, s, r, p));
            op_in(x->g, *PW(x->G, x, s, r, p));
            op_end(x->g, 0, mult_dev(x));
        }
    } else {
        emit_ar_dp(x, s, (double)((uint64_t)x->e * n), p);
    }
    for (r = 0; r < x->R; r++) {
        op_begin(x->g, OR_COMPUTE, T_OPT, fl, by);
        op_dev(x->g, dev_of(x, s, r));
        op_in(x->g, *PW(x->W, x, s, r, p));
        op_in(x->g, *PW(x->G, x, s, r, p));
        if (*PW(x->OS, x, s, r, p) >= 0) op_in(x->g, *PW(x->OS, x, s, r, p));
        op_end(x->g, 0, mult_dev(x));
    }
}

static void emit_wu(mat *x, int s)
{
    int p, nl = x->l0[s + 1] - x->l0[s];
    if (x->fam == FAM_MLP) {
        for (p = 0; p < nl; p++) emit_wu_slot(x, s, p, mlp_param(x, s, p));
        return;
    }
    if (s == 0) emit_wu_slot(x, s, tf_slot_emb(x), tf_param(x, s, tf_slot_emb(x)));
    for (p = 0; p < 4 * nl; p++) emit_wu_slot(x, s, p, tf_param(x, s, p));
    if (s == x->P - 1) emit_wu_slot(x, s, tf_slot_head(x), tf_param(x, s, tf_slot_head(x)));
}

/* ------------------------------------------------------------------------ */
/* Size rule of the transform's integer arithmetic.  Every op's flops,       */
/* bytes, allocation and free, and every live-byte count, must stay below    */
/* 2^62 (64-bit integers with room to spare), and op counts below 2^62 too:  */
/* at most 65,536 layers, at most 2^24 devices per strategy (below).  With   */
/* B rows, e bytes per element, L layers, width d (MLP), and for the         */
/* transformer s tokens per sequence, T = B * s, F = d_ff, V = vocab, a      */
/* heads, N1 = 3d^2 + dF + Vd and Kx = min(B, 16383) microbatches:           */
/*   MLP  Q = 2Bd^2 + e(3Bd + d^2) + 64d^2                                   */
/*        Z = L(16eBd + 8eKx d^2) + 32Ld^2 + 8eBd                            */
/*   TF   Q = 2Td(3d + F + V + 2s) + (5 + 3e)Ba s^2 + (8 + 8e)T(d + F + V)   */
/*            + (68 + 8e)N1 + 64T                                            */
/*        Z = L(eT(64d + 16F + 16as) + 8eKx(4d^2 + 2dF)) + eT(8V + 16d)      */
/*            + 48T + 16eKx Vd + 32(L(4d^2 + 2dF) + 2Vd)                      */
/* Q bounds each op's quantities at any tensor degree H >= 1 and microbatch  */
/* of at most B rows (each term is one of the op formulas, summed); Z bounds */
/* the resident bytes plus every allocation of a stage's whole program (the */
/* row-sized ones scale with the microbatch rows, which sum to at most B;    */
/* the parameter-sized ones -- gradients, broadcast copies, the reduced      */
/* gradient -- come at most four times per layer and microbatch plus once).  */
/* Both are evaluated in fp64 and must be below 2^62.  Returns 1 when the    */
/* model is within the rule, 0 otherwise. */
int or_model_size_ok(const or_model *M)
{
    const double lim = 4611686018427387904.0;   /* 2^62 */
    double B = (double)M->global_batch, e = (double)M->elem_bytes, L = (double)M->n_layers;
    double d = (double)M->d_model, Kx, Q, Z;
    if (M->n_layers > 65536) return 0;
    Kx = B < 16383.0 ? B : 16383.0;
    if (M->family == FAM_MLP) {
        Q = 2.0 * B * d * d + e * (3.0 * B * d + d * d) + 64.0 * d * d;
        Z = L * (16.0 * e * B * d + 8.0 * e * Kx * d * d) + 32.0 * L * d * d + 8.0 * e * B * d;
    } else {
        double s = (double)M->seq_len, F = (double)M->d_ff, V = (double)M->vocab, a = (double)M->n_heads;
        double T = B * s, N1 = 3.0 * d * d + d * F + V * d;
        Q = 2.0 * T * d * (3.0 * d + F + V + 2.0 * s) + (5.0 + 3.0 * e) * B * a * s * s +
            (8.0 + 8.0 * e) * T * (d + F + V) + (68.0 + 8.0 * e) * N1 + 64.0 * T;
        Z = L * (e * T * (64.0 * d + 16.0 * F + 16.0 * a * s) + 8.0 * e * Kx * (4.0 * d * d + 2.0 * d * F)) +
            e * T * (8.0 * V + 16.0 * d) + 48.0 * T + 16.0 * e * Kx * V * d +
            32.0 * (L * (4.0 * d * d + 2.0 * d * F) + 2.0 * V * d);
    }
    return Q < lim && Z < lim;
}

/* filters of a strategy (the grid's validity rules and the transform's
 * preconditions); returns 0 when valid */
static int strategy_invalid(const or_model *M, int D, int H, int P, int K)
{
    int64_t B = M->global_batch, L = M->n_layers;
    if (D < 1 || H < 1 || P < 1 || K < 1) return 1;
    /* at most 2^24 devices: with at most 65,536 layers and 16,383
     * microbatches every op count of the program stays below 2^62 */
    if ((int64_t)D * H * P > ((int64_t)1 << 24)) return 1;
    if (M->elem_bytes < 1 || M->d_model < 1 || L < 1 || B < 1) return 1;
    if (B % D != 0) return 1;
    if ((int64_t)K > B / D) return 1;
    if ((int64_t)P > L) return 1;
    if (M->mode < MODE_INFER || M->mode > MODE_ADAM_MIXED) return 1;
    if (M->family == FAM_MLP) {
        if (M->d_model % H != 0) return 1;
        if (H > 1) {
            int s;
            int64_t q = L / P, rr = L % P;
            for (s = 0; s < P; s++) {
                int64_t n = q + (s < rr ? 1 : 0);
                if (n % 2 != 0) return 1;
            }
        }
        return 0;
    }
    if (M->family == FAM_TRANSFORMER) {
        if (M->n_heads < 1 || M->seq_len < 1 || M->vocab < 1 || M->d_ff < 1) return 1;
        if (M->d_model % M->n_heads != 0) return 1;
        if (M->n_heads % H != 0 || M->d_model % H != 0 || M->d_ff % H != 0) return 1;
        return 0;
    }
    return 1;
}

typedef struct {
    double makespan;
    uint64_t cand_peak, n_ops;
    int32_t status;
} or_result;

/*
 * Materialise (D, H, P, K) applied to the model and simulate it.
 * slice != 0: projection onto replica (0,0) of every stage.
 * Outputs per stage s (replica (0,0)): stage_finish[s], stage_peak[s];
 * optional per-device arrays (size D*H*P) for the full program.
 */
static int sim_strategy(const or_model *M, int D, int H, int P, int K,
                        const or_device_model *dm, int slice, const double *type_cost,
                        double *stage_finish, uint64_t *stage_peak,
                        double *dev_finish, uint64_t *dev_peak, uint64_t *dev_resident,
                        double *by_type, or_result *res)
{
    mat x;
    or_prog g;
    int s, r, n_dev, rc = 0, p;
    int *seq_t = NULL, *seq_k = NULL, *len = NULL, *pos = NULL, *nf = NULL, *nb = NULL,
        *nf0 = NULL, *nb0 = NULL, *em = NULL, *emk = NULL;
    double *fin = NULL;
    uint64_t *pk = NULL;
    memset(res, 0, sizeof *res);
    if (!or_model_size_ok(M)) return -5;
    if (strategy_invalid(M, D, H, P, K)) { res->status = ST_BAD_STRATEGY; return 0; }
    if (dm->node_size > 0) {
        /* nodes must cut every tensor-parallel group, data-parallel group
         * and stage alike: node_size and D*H, and node_size and H, divide
         * one another (always so for powers of two) */
        int G = dm->node_size, DH = D * H;
        if (!(G % DH == 0 || DH % G == 0) || !(G % H == 0 || H % G == 0)) {
            res->status = ST_BAD_STRATEGY;
            return 0;
        }
    }
    if ((int64_t)D * H > 1024 || K > 16383) return -1;
    /* overlap: two streams per GPU (and no ZeRO); otherwise one device per GPU */
    if (M->overlap ? (M->zero || dm->streams_per_gpu != 2) : dm->streams_per_gpu > 1) return -1;
    memset(&x, 0, sizeof x);
    prog_init(&g);
    x.M = M; x.g = &g; x.D = D; x.H = H; x.P = P; x.K = K; x.slice = slice;
    x.fam = M->family; x.mode = M->mode; x.train = M->mode != MODE_INFER;
    x.rc = x.train && M->recompute;
    x.zero = x.train && M->zero;
    x.S = M->overlap ? 2 : 1;
    x.ov = x.train && M->overlap;
    x.R = slice ? (x.zero ? D : 1) : D * H;
    x.e = M->elem_bytes;
    x.rows = M->global_batch / D;
    n_dev = x.S * D * H * P;
    x.l0 = malloc(sizeof(int) * (size_t)(P + 1));
    if (!x.l0) return -3;
    {
        int q = M->n_layers / P, rr = M->n_layers % P;
        x.l0[0] = 0;
        x.nl_max = 0;
        for (s = 0; s < P; s++) {
            int n = q + (s < rr ? 1 : 0);
            x.l0[s + 1] = x.l0[s] + n;
            if (n > x.nl_max) x.nl_max = n;
        }
    }
    x.nslot = F_LAYER0 + x.nl_max * NLF;
    x.nps = x.fam == FAM_MLP ? x.nl_max : 4 * x.nl_max + 2;
    x.sv = malloc(sizeof(int32_t) * (size_t)P * x.R * K * x.nslot);
    x.W = malloc(sizeof(int32_t) * (size_t)P * x.R * x.nps);
    x.OS = malloc(sizeof(int32_t) * (size_t)P * x.R * x.nps);
    x.G = malloc(sizeof(int32_t) * (size_t)P * x.R * x.nps);
    x.GC = malloc(sizeof(int32_t) * (size_t)P * x.R * x.nps);
    x.X = malloc(sizeof(int32_t) * (size_t)P * x.R);
    x.Y = malloc(sizeof(int32_t) * (size_t)P * x.R);
    x.cur = malloc(sizeof(int32_t) * (size_t)x.R);
    x.tmp = malloc(sizeof(int32_t) * (size_t)x.R);
    seq_t = malloc(sizeof(int) * (size_t)P * 2 * K);
    seq_k = malloc(sizeof(int) * (size_t)P * 2 * K);
    len = calloc((size_t)P, sizeof(int));
    pos = calloc((size_t)P, sizeof(int));
    nf = calloc((size_t)P, sizeof(int));
    nb = calloc((size_t)P, sizeof(int));
    nf0 = calloc((size_t)P, sizeof(int));
    nb0 = calloc((size_t)P, sizeof(int));
    em = calloc((size_t)P, sizeof(int));
    emk = calloc((size_t)P, sizeof(int));
    fin = calloc((size_t)n_dev, sizeof(double));
    pk = calloc((size_t)n_dev, sizeof(uint64_t));
    if (!x.sv || !x.W || !x.OS || !x.G || !x.GC || !x.X || !x.Y || !x.cur || !x.tmp || !seq_t || !seq_k ||
        !len || !pos || !nf || !nb || !nf0 || !nb0 || !em || !emk || !fin || !pk) { rc = -3; goto out; }
    memset(x.sv, 0xff, sizeof(int32_t) * (size_t)P * x.R * K * x.nslot);
    memset(x.G, 0xff, sizeof(int32_t) * (size_t)P * x.R * x.nps);
    memset(x.GC, 0xff, sizeof(int32_t) * (size_t)P * x.R * x.nps);
    memset(x.OS, 0xff, sizeof(int32_t) * (size_t)P * x.R * x.nps);
    memset(x.W, 0xff, sizeof(int32_t) * (size_t)P * x.R * x.nps);
    /* resident tensors */
    for (s = 0; s < P; s++) {
        int nl = x.l0[s + 1] - x.l0[s];
        for (r = 0; r < x.R; r++) {
            int dv = dev_of(&x, s, r);
            int np = x.fam == FAM_MLP ? nl : 4 * nl;
            for (p = 0; p < x.nps; p++) {
                uint64_t n;
                if (p >= np) {
                    if (x.fam == FAM_MLP) continue;
                    if (p == tf_slot_emb(&x) && s != 0) continue;
                    if (p == tf_slot_head(&x) && s != P - 1) continue;
                    if (p != tf_slot_emb(&x) && p != tf_slot_head(&x)) continue;
                }
                n = x.fam == FAM_MLP ? mlp_param(&x, s, p) : tf_param(&x, s, p);
                if (x.zero && owner_of(&x, s, p) != data_rep(&x, r)) continue;   /* held by its owner only */
                *PW(x.W, &x, s, r, p) = prog_tensor(&g, dv, (uint64_t)x.e * n, TF_RESIDENT | TF_KEEP);
                if (x.train && opt_state_bytes(&x, n) > 0)
                    *PW(x.OS, &x, s, r, p) = prog_tensor(&g, dv, opt_state_bytes(&x, n), TF_RESIDENT | TF_KEEP);
            }
            x.X[s * x.R + r] = -1;
            x.Y[s * x.R + r] = -1;
            if (s == 0) x.X[s * x.R + r] = prog_tensor(&g, dv, input_row_bytes(&x) * (uint64_t)x.rows, TF_RESIDENT);
            if (s == P - 1 && x.train)
                x.Y[s * x.R + r] = prog_tensor(&g, dv, input_row_bytes(&x) * (uint64_t)x.rows, TF_RESIDENT);
        }
    }
    /* per-stage block sequences */
    for (s = 0; s < P; s++) {
        int *tt = seq_t + (size_t)s * 2 * K, *kk = seq_k + (size_t)s * 2 * K, n = 0, i;
        if (!x.train) {
            for (i = 0; i < K; i++) { tt[n] = 0; kk[n++] = i; }
        } else if (M->schedule == 1) {
            /* GPipe: every forward, then every backward, in microbatch order */
            for (i = 0; i < K; i++) { tt[n] = 0; kk[n++] = i; }
            for (i = 0; i < K; i++) { tt[n] = 1; kk[n++] = i; }
        } else {
            int w = P - 1 - s < K ? P - 1 - s : K;
            for (i = 0; i < w; i++) { tt[n] = 0; kk[n++] = i; }
            for (i = 0; i < K - w; i++) {
                tt[n] = 0; kk[n++] = w + i;
                tt[n] = 1; kk[n++] = i;
            }
            for (i = K - w; i < K; i++) { tt[n] = 1; kk[n++] = i; }
        }
        len[s] = n;
    }
    /* microbatch splits before the pipeline */
    if (K > 1) {
        emit_split(&x, 0, 0);
        if (x.train) emit_split(&x, P - 1, 1);
    }
    /* slots */
    for (;;) {
        int any_left = 0, any = 0;
        for (s = 0; s < P; s++) {
            if (pos[s] < len[s]) any_left = 1;
            nf0[s] = nf[s];
            nb0[s] = nb[s];
            em[s] = -1;
        }
        if (!any_left) break;
        for (s = 0; s < P; s++) {
            int typ, kk, ready;
            if (pos[s] >= len[s]) continue;
            typ = seq_t[(size_t)s * 2 * K + pos[s]];
            kk = seq_k[(size_t)s * 2 * K + pos[s]];
            if (typ == 0) ready = (s == 0) || nf0[s - 1] > kk;
            else ready = (s == P - 1) ? nf0[s] > kk : nb0[s + 1] > kk;
            if (!ready) continue;
            if (typ == 0) { if (x.fam == FAM_MLP) mlp_fwd(&x, s, kk); else tf_fwd(&x, s, kk); }
            else { if (x.fam == FAM_MLP) mlp_bwd(&x, s, kk); else tf_bwd(&x, s, kk); }
            pos[s]++;
            em[s] = typ;
            emk[s] = kk;
            any = 1;
        }
        if (!any) { rc = -4; goto out; }   /* cannot happen for 1F1B */
        for (s = 0; s < P; s++) {
            if (em[s] == 0) nf[s]++;
            if (em[s] == 1) nb[s]++;
        }
        for (s = 0; s < P; s++) {
            if (em[s] == 0 && s < P - 1) emit_send(&x, s, emk[s], 1);
            if (em[s] == 1 && s > 0) emit_send(&x, s, emk[s], 0);
        }
    }
    if (x.train) for (s = 0; s < P; s++) emit_wu(&x, s);
    if (g.failed) { rc = -3; goto out; }
    if (by_type) {
        /* per-type totals of the materialised ops: flops at [type], bytes
         * at [T_NTYPES + type], reduction lengths at [2 T_NTYPES + type] */
        int64_t i;
        for (i = 0; i < 3 * T_NTYPES; i++) by_type[i] = 0.0;
        for (i = 0; i < g.n_ops; i++) {
            by_type[g.type[i]] += g.flops[i];
            by_type[T_NTYPES + g.type[i]] += g.bytes[i];
            by_type[2 * T_NTYPES + g.type[i]] += g.kred[i];
        }
    }
    rc = prog_simulate(&g, n_dev, dm, type_cost, fin, pk, dev_resident, NULL, NULL);
    if (rc) goto out;
    /* devices a projection does not materialise stay at 0; per stage, the
     * latest finish and the highest peak of its devices */
    res->makespan = 0.0;
    res->cand_peak = 0;
    for (s = 0; s < n_dev; s++) {
        if (fin[s] > res->makespan) res->makespan = fin[s];
        if (pk[s] > res->cand_peak) res->cand_peak = pk[s];
    }
    for (s = 0; s < P; s++) {
        double f = 0.0;
        uint64_t q = 0;
        for (r = 0; r < x.S * D * H; r++) {
            if (fin[s * x.S * D * H + r] > f) f = fin[s * x.S * D * H + r];
            if (pk[s * x.S * D * H + r] > q) q = pk[s * x.S * D * H + r];
        }
        if (stage_finish) stage_finish[s] = f;
        if (stage_peak) stage_peak[s] = q;
    }
    if (dev_finish) memcpy(dev_finish, fin, sizeof(double) * (size_t)n_dev);
    if (dev_peak) memcpy(dev_peak, pk, sizeof(uint64_t) * (size_t)n_dev);
    res->n_ops = (uint64_t)g.program_ops;
    if (dm->mem_cap_bytes != 0 && res->cand_peak > dm->mem_cap_bytes) res->status |= ST_OVER_CAP;
out:
    free(x.l0); free(x.sv); free(x.W); free(x.OS); free(x.G); free(x.GC); free(x.X); free(x.Y);
    free(x.cur); free(x.tmp);
    free(seq_t); free(seq_k); free(len); free(pos); free(nf); free(nb); free(nf0); free(nb0);
    free(em); free(emk); free(fin); free(pk);
    prog_free(&g);
    return rc;
}

/* Single strategy with every diagnostic output (tests).  by_type (optional):
 * 3 * T_NTYPES per-type totals -- flops, bytes, reduction lengths. */
int or_sim_strategy(const or_model *M, int D, int H, int P, int K,
                    const or_device_model *dm, int slice, const double *type_cost,
                    double *stage_finish, uint64_t *stage_peak,
                    double *dev_finish, uint64_t *dev_peak, uint64_t *dev_resident,
                    double *by_type,
                    double *makespan, uint64_t *cand_peak, uint64_t *n_ops, int32_t *status)
{
    or_result res;
    int rc = sim_strategy(M, D, H, P, K, dm, slice, type_cost, stage_finish, stage_peak,
                          dev_finish, dev_peak, dev_resident, by_type, &res);
    *makespan = res.makespan;
    *cand_peak = res.cand_peak;
    *n_ops = res.n_ops;
    *status = res.status;
    return rc;
}

/* ------------------------------------------------------------------------ */
/* Grid enumeration (Sec. 5.1): power-of-two D, H, P; K per k_mode.          */
/* Order: P outermost, then K, then H, then D innermost, each ascending.     */
/* k_mode 0: K in powers of two <= k_max; 1: every integer 1..k_max;         */
/* 2 (the paper's rule): K = 1 when P = 1, else powers of two 2..k_max.     */
/* ------------------------------------------------------------------------ */
int or_create_grid(const or_model *M, int max_devices, int exact_devices, int k_mode,
                   int k_max, int require_k_divides, int32_t *out, int64_t cap, int64_t *n_out)
{
    int64_t n = 0;
    int P, K, H, D;
    if (max_devices < 1 || k_max < 1 || k_mode < 0 || k_mode > 2) return -1;
    if (!or_model_size_ok(M)) return -5;
    for (P = 1; P <= max_devices; P *= 2) {
        for (K = 1; K <= k_max; K++) {
            if (k_mode == 0 && (K & (K - 1)) != 0) continue;
            if (k_mode == 2) {
                if (P == 1 && K != 1) continue;
                if (P > 1 && (K < 2 || (K & (K - 1)) != 0)) continue;
            }
            for (H = 1; H * P <= max_devices; H *= 2) {
                for (D = 1; D * H * P <= max_devices; D *= 2) {
                    if (exact_devices && D * H * P != max_devices) continue;
                    if (strategy_invalid(M, D, H, P, K)) continue;
                    if (require_k_divides && (M->global_batch / D) % K != 0) continue;
                    if (out && n < cap) {
                        out[4 * n + 0] = D;
                        out[4 * n + 1] = H;
                        out[4 * n + 2] = P;
                        out[4 * n + 3] = K;
                    }
                    n++;
                }
            }
        }
    }
    *n_out = n;
    return (out && n > cap) ? -2 : 0;
}

/* ------------------------------------------------------------------------ */
/* Selection (Sec. 5.2): drop candidates with an error status or a peak      */
/* above the cap (cap 0 = none), rank the rest by predicted time (makespan   */
/* ascending; ties to the lower index), return the first k.                  */
/* ------------------------------------------------------------------------ */
typedef struct { double mk; int64_t idx; } or_pair;

static int pair_cmp(const void *a, const void *b)
{
    const or_pair *x = a, *y = b;
    if (x->mk < y->mk) return -1;
    if (x->mk > y->mk) return 1;
    return (x->idx > y->idx) - (x->idx < y->idx);
}

int or_topk(const double *mk, const uint64_t *pk, const int32_t *st, int64_t n,
            uint64_t cap, int k, int64_t *idx_out, double *mk_out, int32_t *found)
{
    or_pair *v;
    int64_t i, m = 0;
    int j;
    if (k < 1) return -1;
    v = malloc(sizeof(or_pair) * (size_t)(n > 0 ? n : 1));
    if (!v) return -3;
    for (i = 0; i < n; i++) {
        if (st[i] != 0) continue;
        if (cap != 0 && pk[i] > cap) continue;
        v[m].mk = mk[i];
        v[m].idx = i;
        m++;
    }
    qsort(v, (size_t)m, sizeof(or_pair), pair_cmp);
    for (j = 0; j < k; j++) {
        idx_out[j] = j < m ? v[j].idx : -1;
        mk_out[j] = j < m ? v[j].mk : HUGE_VAL;
    }
    *found = (int32_t)(m < k ? m : k);
    free(v);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Batch drivers: the same single-candidate code, run over a list of          */
/* candidates by a few threads (used for timing and for parity sampling).    */
/* ------------------------------------------------------------------------ */
typedef struct {
    int kind;                 /* 0 random tables, 1 strategies */
    uint64_t seed;
    int32_t n_ops, n_dev;
    const int64_t *cands;
    const or_model *M;
    const int32_t *strat;
    int slice, row_width;
    const or_device_model *dm;
    int64_t lo, hi;
    double *makespan, *finish;
    uint64_t *peak, *cand_peak, *nops;
    int32_t *status;
    int rc;
} job;

static void *job_run(void *arg)
{
    job *J = arg;
    int64_t i;
    if (J->kind == 0) {
        uint32_t *code = malloc(sizeof(uint32_t) * (size_t)J->n_ops);
        float *fl = malloc(sizeof(float) * (size_t)J->n_ops);
        float *by = malloc(sizeof(float) * (size_t)J->n_ops);
        uint32_t *al = malloc(sizeof(uint32_t) * (size_t)J->n_ops);
        uint32_t *fr = malloc(sizeof(uint32_t) * (size_t)J->n_ops);
        if (!code || !fl || !by || !al || !fr) { J->rc = -3; goto done0; }
        for (i = J->lo; i < J->hi; i++) {
            int rc = or_gen_table(J->seed, J->cands[i], J->n_ops, J->n_dev, code, fl, by, al, fr, 1);
            if (rc) { J->rc = rc; break; }
            or_sim_table(J->n_ops, J->n_dev, code, fl, by, al, fr, NULL, 1, NULL, J->dm,
                         &J->makespan[i], J->finish ? &J->finish[i * J->n_dev] : NULL,
                         J->peak ? &J->peak[i * J->n_dev] : NULL, &J->cand_peak[i], &J->status[i]);
            if (J->nops) J->nops[i] = (uint64_t)J->n_ops;
        }
    done0:
        free(code); free(fl); free(by); free(al); free(fr);
        return NULL;
    }
    for (i = J->lo; i < J->hi; i++) {
        or_result res;
        const int32_t *q = J->strat + 4 * i;
        double *sf = J->finish ? &J->finish[i * J->row_width] : NULL;
        uint64_t *sp = J->peak ? &J->peak[i * J->row_width] : NULL;
        int rc, s;
        if (sf) for (s = 0; s < J->row_width; s++) sf[s] = 0.0;
        if (sp) for (s = 0; s < J->row_width; s++) sp[s] = 0;
        if (q[2] > J->row_width) { J->rc = -1; break; }
        rc = sim_strategy(J->M, q[0], q[1], q[2], q[3], J->dm, J->slice, NULL, sf, sp,
                          NULL, NULL, NULL, NULL, &res);
        if (rc) { J->rc = rc; break; }
        J->makespan[i] = res.makespan;
        J->cand_peak[i] = res.cand_peak;
        if (J->nops) J->nops[i] = res.n_ops;
        J->status[i] = res.status;
    }
    return NULL;
}

static int run_jobs(job *proto, int64_t n, int threads)
{
    pthread_t th[256];
    job jb[256];
    int t, rc = 0;
    if (threads < 1) threads = 1;
    if (threads > 256) threads = 256;
    if (threads > n) threads = (int)(n > 0 ? n : 1);
    for (t = 0; t < threads; t++) {
        jb[t] = *proto;
        jb[t].lo = n * t / threads;
        jb[t].hi = n * (t + 1) / threads;
        jb[t].rc = 0;
    }
    if (threads == 1) job_run(&jb[0]);
    else {
        for (t = 0; t < threads; t++) pthread_create(&th[t], NULL, job_run, &jb[t]);
        for (t = 0; t < threads; t++) pthread_join(th[t], NULL);
    }
    for (t = 0; t < threads; t++) if (jb[t].rc) rc = jb[t].rc;
    return rc;
}

/* generate and simulate the random tables of the listed candidates */
int or_run_random_tables(uint64_t seed, int32_t n_ops, int32_t n_dev, const int64_t *cands,
                         int64_t n, const or_device_model *dm, int threads,
                         double *makespan, double *finish, uint64_t *peak,
                         uint64_t *cand_peak, uint64_t *nops, int32_t *status)
{
    job J;
    memset(&J, 0, sizeof J);
    J.kind = 0; J.seed = seed; J.n_ops = n_ops; J.n_dev = n_dev; J.cands = cands; J.dm = dm;
    J.makespan = makespan; J.finish = finish; J.peak = peak; J.cand_peak = cand_peak;
    J.nops = nops; J.status = status;
    return run_jobs(&J, n, threads);
}

/* materialise and simulate a list of strategies (int32 D,H,P,K each) */
int or_run_strategies(const or_model *M, const int32_t *strat, int64_t n,
                      const or_device_model *dm, int slice, int row_width, int threads,
                      double *makespan, double *finish, uint64_t *peak,
                      uint64_t *cand_peak, uint64_t *nops, int32_t *status)
{
    job J;
    memset(&J, 0, sizeof J);
    J.kind = 1; J.M = M; J.strat = strat; J.slice = slice; J.row_width = row_width; J.dm = dm;
    J.makespan = makespan; J.finish = finish; J.peak = peak; J.cand_peak = cand_peak;
    J.nops = nops; J.status = status;
    return run_jobs(&J, n, threads);
}
