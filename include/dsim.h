/*
 * dsim.h -- C ABI of the MI355X batched DistIR strategy simulator.
 *
 * The operation (Santhanam et al., "DistIR", MLSys 2022):
 *   A distributed program is a straight-line list of ops over a fixed set of
 *   single-threaded devices (Sec. 2.1).  An op runs synchronously on its device
 *   set: it starts when all of them are free and they all finish together; ops
 *   run in program order.  The simulator (Sec. 3.3) advances each device's
 *   clock by the op's cost and tracks every device's live memory, a tensor
 *   being live from its creation until its last use.  Costs (Sec. 3.3, Sec. 4)
 *   are, with F, B_mem, B_link, lat, launch from dsim_device_model:
 *     compute      launch + max(flops * (1/F), bytes * (1/B_mem))
 *     send         lat + bytes * (1/B_link)
 *     all-reduce   (2(n-1)) * lat + ((2(n-1)) / n) * (bytes * (1/B_link)),
 *                  0 for n = 1 (ring over the n participants)
 *   every reciprocal rounded once to fp64; fp64 throughout, no FMA contraction.
 *   Candidates are a D/T/P/K transform (Sec. 4) of an MLP or GPT-style model
 *   (T is called H here), or explicit op tables; the grid search (Sec. 5.1,
 *   5.2) simulates all of them, drops those over the memory cap and ranks
 *   the rest by predicted time.
 *
 * Conventions for every call:
 *   - Returns a dsim_status: 0 on success, < 0 on an argument or HIP error;
 *     never throws, never exits.  dsim_last_error() describes the last
 *     failure of the calling thread.
 *   - Pointers documented as "device" are HIP device pointers; "host" ones
 *     are host memory.  The caller owns every buffer, workspaces included;
 *     the library allocates no device memory and keeps nothing between
 *     calls.
 *   - Kernels are enqueued on `hip_stream` (a hipStream_t, NULL = the null
 *     stream); results are valid once that stream has been synchronised.
 *   - Arguments are validated on the host before any launch.  Errors inside
 *     one candidate (an invalid op, a free of more bytes than are live, an
 *     invalid strategy) never abort: they set bits of that candidate's status
 *     word, and dsim_argmin skips every candidate whose status is non-zero.
 *   - Results are deterministic: the same inputs give bit-identical outputs.
 */
#ifndef DSIM_H
#define DSIM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DSIM_API __attribute__((visibility("default")))

typedef enum {
    DSIM_OK = 0,
    DSIM_EINVAL = -1,   /* invalid argument (null pointer, bad size, bad constant) */
    DSIM_ERANGE = -2,   /* a size beyond what a format or kernel supports           */
    DSIM_ENOSPC = -3,   /* an output or workspace buffer is too small               */
    DSIM_EHIP = -4      /* a HIP runtime call or kernel launch failed               */
} dsim_status;

/* per-candidate status bits */
#define DSIM_ST_BAD_OP 1          /* op kind unknown, reserved code bits set, or flops /
                                     bytes not finite and >= 0                          */
#define DSIM_ST_BAD_DEVICE 2      /* a device id >= n_dev, or an empty device mask      */
#define DSIM_ST_SELF_SEND 4       /* send with source == destination                    */
#define DSIM_ST_MEM_UNDERFLOW 8   /* an op frees more bytes than its device holds       */
#define DSIM_ST_BAD_STRATEGY 16   /* (D,H,P,K) violates the transform's preconditions   */
#define DSIM_ST_OVER_CAP 32       /* peak above dsim_device_model.mem_cap_bytes (> 0)   */
#define DSIM_ST_NOT_TABLE 64      /* dsim_materialize_tables: the program does not fit  */
                                  /* the table format (see there)                       */

/* Model families and modes. */
#define DSIM_MLP 0
#define DSIM_TRANSFORMER 1
#define DSIM_INFER 0
#define DSIM_TRAIN_SGD 1
#define DSIM_TRAIN_ADAM 2
#define DSIM_TRAIN_ADAM_MIXED 3   /* fp16 weights and gradients, fp32 master, m, v */
#define DSIM_SCHED_1F1B 0
#define DSIM_SCHED_GPIPE 1

DSIM_API const char *dsim_last_error(void);

/* Device constants of the simulated cluster (Sec. 4: the cost functions'
 * coefficients are device DRAM bandwidth, kernel launch overhead, network
 * bandwidth; F is the device's flop rate, Sec. 3.3).  All five doubles must
 * be finite and > 0 (latency and launch may be 0), and each rate's
 * reciprocal finite too (costs multiply by 1/rate, so a rate below about
 * 5.6e-309 is rejected).  Costs may still overflow to +inf; an all-reduce
 * over a single device costs 0 whatever its bytes.  mem_cap_bytes = 0 means
 * no cap; otherwise candidates whose peak exceeds it get DSIM_ST_OVER_CAP.
 * mm_enabled = 1 gives matrix multiplications the empirical cost of Sec. 4
 * (a regression in the input sizes, fitted on single-op microbenchmarks):
 *   max(mm_floor, ((mm_c0 + mm_c1 * flops) + mm_c2 * bytes) + mm_c3 * k)
 * with k the product's reduction length (the operands' inner dimension;
 * an op standing for two products, the attention gradients, has the sum of
 * theirs) and every coefficient finite and >= 0.  mm_c3 = mm_floor = 0 is
 * the paper's linear form.  The transform's matrix multiplications are the
 * dense layer's Gemm and its two gradients, the transformer's QKV, output,
 * fc1, fc2 and LM-head products, the attention score and P.V products, and
 * their gradients; in explicit tables, compute records of cost class 1,
 * whose k comes from dsim_tables.mm_k.  mm_enabled = 0: every compute op
 * takes the roofline (mm_* ignored).
 * node_size > 0 makes the interconnect two-tier: device d lies in node
 * d / node_size, and a send or collective whose devices lie in more than one
 * node crosses the network (net_bytes_per_s > 0 with a finite reciprocal,
 * net_latency_s >= 0, both finite) instead of the node's links (link_bytes_per_s, link_latency_s).
 * node_size = 0: one uniform interconnect, net_* ignored.
 * streams_per_gpu = S > 1 models communication that overlaps computation the
 * way Sec. 2.2 (Limitations) describes, one device per stream: device d is
 * a stream of GPU d / S (nodes then hold node_size GPUs), and a send or
 * collective whose devices are all streams of one GPU costs
 * stream_latency_s (finite, >= 0) and stream_bytes_per_s (> 0 with a finite
 * reciprocal, +inf for no byte term) in place of the links.  S = 0 or 1: every device is its own
 * GPU, stream_* ignored.  The transform's devices follow model.overlap:
 * S must be 2 with it and at most 1 without (else DSIM_EINVAL). */
typedef struct {
    double flops_per_s, mem_bytes_per_s, link_bytes_per_s, link_latency_s, launch_s;
    uint64_t mem_cap_bytes;
    int32_t mm_enabled;
    double mm_c0, mm_c1, mm_c2;
    int32_t node_size;
    double net_bytes_per_s, net_latency_s;
    int32_t streams_per_gpu;
    double stream_bytes_per_s, stream_latency_s;
    double mm_c3, mm_floor;   /* the MatMul cost's reduction-length term and floor */
} dsim_device_model;

/* The sequential program the transform distributes (Sec. 4, Sec. 5):
 *   MLP: n_layers square d_model x d_model dense layers (Gemm + Relu, Fig. 2),
 *        global_batch rows; n_heads, d_ff, seq_len, vocab are ignored.
 *   TRANSFORMER: GPT-2-shaped decoder; global_batch sequences of seq_len
 *        tokens, n_heads heads, MLP width d_ff, vocabulary vocab.
 *   elem_bytes: bytes per weight/activation element (2 or 4).
 *   schedule: pipeline schedule of each stage's microbatch blocks in
 *        training: DSIM_SCHED_1F1B (the paper's synchronous 1F1B,
 *        w = min(P-1-s, K) warm-up forwards, then forward/backward pairs,
 *        then w backwards) or DSIM_SCHED_GPIPE (all K forwards, then all K
 *        backwards, both in microbatch order).  Inference runs the K
 *        forwards either way.
 *   recompute: 0 or 1.  1 = activation recomputation (gradient
 *        checkpointing, the appendix's Fig. 8), training only: a forward
 *        block keeps its input (the checkpoint) and its output live, and the
 *        activations produced inside the stage's layers die at their last
 *        forward use; a backward block runs the loss / LM-head gradients,
 *        then replays from the checkpoint the forward ops of the stage's
 *        layers whose results the layers' backward reads (all but the last
 *        MLP layer; every transformer layer, the last one up to its GeLU),
 *        then the layers' backward.
 *   zero: 0 or 1.  1 = ZeRO partitioning of weights, gradients and
 *        optimizer state over the D data-parallel replicas (the appendix's
 *        Fig. 9), training only, D > 1: the parameter groups in model order
 *        (the transformer's embedding, each layer -- for the MLP with H > 1
 *        each column/row layer pair -- and the LM head) belong to replica
 *        (group index mod D), which alone holds their weights and optimizer
 *        state from t = 0.  Right before every op that reads a weight, its
 *        owner broadcasts it over the stage's D replicas of that tensor rank
 *        (one collective per tensor rank); each other replica's copy dies
 *        after that op.  Gradients accumulate on every replica; at the
 *        weight update each one is reduced onto its owner (replacing the
 *        all-reduce; every replica's gradient dies there) and only the owner
 *        runs the optimizer op, which consumes the reduced gradient.
 *        Broadcast and reduce over n devices cost (n-1) * lat +
 *        bytes * (1/B_link) (a pipelined chain; a Send for n = 2).
 *   overlap: 0 or 1 (not with zero).  1 = every GPU is two devices (Sec. 2.2,
 *        Limitations: a device per stream), 2g computing and 2g + 1
 *        communicating, and in training with D > 1 the data-parallel
 *        gradient all-reduce runs on the communication streams, overlapping
 *        the last backward block: once the last microbatch has finished a
 *        weight gradient (its weight-gradient op, or its accumulation), each
 *        replica hands it to its communication stream (a Send between the
 *        GPU's two streams that allocates nothing: the streams share the
 *        gradient's memory), and the communication streams of the D
 *        replicas all-reduce it there; at the weight update each reduced
 *        gradient is handed back (a Send, again allocating nothing) right
 *        before its optimizer op.  Sends are blocking (Sec. 2.1), so a
 *        hand-over waits for the communication stream's previous
 *        all-reduce.  Requires device.streams_per_gpu == 2. */
/* Size rule (every call taking a model returns DSIM_ERANGE beyond it): the
 * transform computes every op's flops, bytes, allocation and free, and every
 * live-byte count, in 64-bit integers.  A model must have n_layers <= 65536,
 * each of d_model, d_ff, seq_len, vocab, global_batch <= 1e15, and, with
 * B = global_batch, e = elem_bytes, L = n_layers, d = d_model, and for the
 * transformer s = seq_len, F = d_ff, V = vocab, a = n_heads, T = B*s,
 * N1 = 3d^2 + dF + Vd, Kx = min(B, 16383), both of
 *   MLP  Q = 2Bd^2 + e(3Bd + d^2) + 64d^2
 *        Z = L(16eBd + 8eKx d^2) + 32Ld^2 + 8eBd
 *   TF   Q = 2Td(3d + F + V + 2s) + (5 + 3e)Ba s^2 + (8 + 8e)T(d + F + V)
 *            + (68 + 8e)N1 + 64T
 *        Z = L(eT(64d + 16F + 16as) + 8eKx(4d^2 + 2dF)) + eT(8V + 16d) + 48T
 *            + 16eKx Vd + 32(L(4d^2 + 2dF) + 2Vd)
 * evaluated in fp64, below 2^62.  Q bounds any single op quantity for every
 * tensor degree and microbatch, Z the resident bytes plus all allocations
 * of a stage's program.  A strategy with D*H*P > 2^24 devices is invalid
 * (status DSIM_ST_BAD_STRATEGY), which with the layer and microbatch bounds
 * keeps every op count below 2^62. */
typedef struct {
    int32_t family, mode, n_layers, n_heads;
    int64_t d_model, d_ff, seq_len, vocab, global_batch;
    int32_t elem_bytes;
    int32_t schedule;
    int32_t recompute;
    int32_t zero;
    int32_t overlap;
} dsim_model;

/* A candidate: data-parallel D, tensor-parallel H (the paper's T), pipeline
 * P, microbatches K (Sec. 4). */
typedef struct {
    int32_t D, H, P, K;
} dsim_strategy;

/* Grid rule (Sec. 5.1): power-of-two D, H, P with D*H*P <= max_devices
 * (== if exact_devices); k_mode 0: K in powers of two <= k_max; 1: every
 * K in 1..k_max; 2 (the paper's rule): K = 1 if P = 1, else powers of two
 * 2..k_max.  require_k_divides: keep only K | global_batch/D. */
typedef struct {
    int32_t max_devices, exact_devices, k_mode, k_max, require_k_divides;
} dsim_grid_spec;

/*
 * dsim_create_grid -- enumerate the valid strategies (Sec. 5.1).
 * Host call.  Writes at most `cap` strategies to the host array `out`
 * (NULL: count only) and the total count to *n_out.  Order: P outermost,
 * then K, then H, then D innermost, each ascending.  A strategy is valid
 * when D*H*P <= 2^24, D | global_batch, K <= global_batch/D, P <= n_layers and H divides
 * the sharded widths (MLP: d_model; transformer: n_heads, d_model, d_ff),
 * and, for the MLP with H > 1, every stage holds an even number of layers
 * (column/row-parallel pairs).  Returns DSIM_ENOSPC if out != NULL and the
 * count exceeds cap (the first cap entries are still written).
 */
DSIM_API dsim_status dsim_create_grid(const dsim_model *model, const dsim_grid_spec *grid,
                             dsim_strategy *out, int64_t cap, int64_t *n_out);

/*
 * Explicit op tables (device memory).  Structure of arrays, op-major,
 * candidate-fastest: the record of op j of candidate c is at j*n_cand + c.
 *   code:  kind | a << 8 | b_or_mask << 16 | cost_class << 24.  Cost class
 *          0: the op's own cost; 1 (compute records only): a matrix
 *          multiplication, costed by the device model's MatMul regression
 *          when it has one (the roofline otherwise); any other class, or
 *          class 1 on another kind, makes the op invalid.
 *          kind 0 compute on device a; 1 send a -> b; 2 all-reduce over the
 *          devices set in the 8-bit mask; 3 broadcast from root a to the
 *          other devices of the mask; 4 reduce over the mask onto root a
 *          (3 and 4: a must be in the mask; ZeRO's collectives, Fig. 9).
 *          Broadcast and reduce over n devices cost
 *          (n-1) * lat + bytes * (1/B_link), 0 for n = 1.
 *   flops, bytes: fp32 values, promoted exactly to fp64 (flops ignored by
 *          every kind but compute); both must be finite and >= 0 (-0.0,
 *          NaN, infinities and negative values make the op invalid), so
 *          that no cost is negative or NaN.
 *   alloc_bytes, free_bytes: compute allocates and frees on a; send
 *          allocates on b and frees on a; all-reduce ignores both;
 *          broadcast allocates on every member but a and frees on a;
 *          reduce allocates on a and frees on every member.  Every touched
 *          device samples its peak after the allocation and before the
 *          free.
 *   n_ops: per candidate op count; NULL = max_ops for all.  A count above
 *          max_ops sets DSIM_ST_BAD_OP and max_ops ops are simulated.
 *   init_live: [n_cand * n_dev] bytes live at t = 0; NULL = zero.  A
 *          device's live bytes (init_live plus its allocations) must stay
 *          below 2^64; candidates starting at 2^62 or more on some device
 *          take a slower exact path (same results).
 *   n_dev: 1..8.
 *   mm_k:  per record, the reduction length of a class-1 record (ignored
 *          on every other record); NULL = 0 for all.
 * An invalid op is skipped (no time, no memory) and flagged in status.
 */
typedef struct {
    const uint32_t *code;
    const float *flops, *bytes;
    const uint32_t *alloc_bytes, *free_bytes;
    const uint32_t *n_ops;
    const uint64_t *init_live;
    int32_t max_ops, n_dev;
    const uint32_t *mm_k;
} dsim_tables;

/*
 * Per-candidate outputs (device memory, caller-allocated, n_cand entries or
 * n_cand * row_width for the per-device rows; row-major per candidate).
 *   makespan:  max over devices of the final clock (seconds)
 *   finish:    per-device final clocks (tables: device d at column d;
 *              parametric: pipeline stage s at column s, the latest of its
 *              devices -- every replica of a stage finishes at the same
 *              time unless ZeRO leaves the last optimizer op to one owner);
 *              unused columns are 0.  May be NULL.
 *   peak:      per-device (per-stage: the highest of the stage's devices)
 *              peak live bytes; may be NULL.
 *   cand_peak: max over devices of the peak.
 *   n_ops:     ops of the whole distributed program (each collective and
 *              each send counted once); may be NULL.
 *   walked_ops: tables: the ops simulated (n_ops); parametric: the ops of
 *              the per-stage projection the result stands for (every op of
 *              one replica per stage, each collective and send once) -- not
 *              arithmetic steps: repeated layers are summed in closed form;
 *              may be NULL.
 *   status:    DSIM_ST_* bits, 0 = valid.
 *   row_width: columns of finish/peak (>= n_dev, or >= max P).
 */
typedef struct {
    double *makespan;
    double *finish;
    uint64_t *peak;
    uint64_t *cand_peak;
    uint64_t *n_ops;
    uint64_t *walked_ops;
    int32_t *status;
    int32_t row_width;
} dsim_results;

/*
 * dsim_simulate_tables -- simulate n_cand explicit programs (Sec. 2.1, 3.3).
 * One GPU lane per candidate walks its ops in order.  n_cand <= 2^32 - 256
 * (DSIM_ERANGE beyond); above 2^28 - 1 candidates every op takes the
 * op-by-op path (same results, slower).
 */
DSIM_API dsim_status dsim_simulate_tables(const dsim_tables *tables, int64_t n_cand,
                                 const dsim_device_model *device,
                                 const dsim_results *results, void *hip_stream);

/*
 * dsim_simulate_parametric -- simulate the D/H/P/K transform (Sec. 4) of
 * `model` for n_cand strategies (device array `cand`) without building op
 * lists: the per-stage 1F1B schedule, layers and ops are expanded on the fly.
 * Every replica (d, h) of a pipeline stage runs the same ops at the same
 * times, so one replica per stage is walked; collectives keep their full
 * group size in the cost.  With device.node_size > 0, nodes must cut every
 * tensor-parallel group, data-parallel group and stage alike: node_size and
 * D*H, and node_size and H, divide one another (always so for powers of
 * two), otherwise DSIM_ST_BAD_STRATEGY.  With model.zero the replicas own different
 * parameter groups: the stage's memory is the maximum over its replicas,
 * taken in closed form per block, and its finish time is that of the owner
 * of its last parameter.  results.row_width must be >= every candidate's P;
 * a candidate with P > min(row_width, 64, n_layers) or K > 16383 gets
 * DSIM_ST_BAD_STRATEGY.  With model.overlap a stage's finish time and peak
 * cover both streams of its GPUs.  The transform: GPU p*(D*H) + d*H + h
 * runs stage p of data replica d, tensor rank h (one device per GPU, or
 * two with model.overlap); contiguous stages (the first L mod P
 * get one extra layer); synchronous 1F1B (forward only in inference) with
 * uneven microbatches (the first rows mod K get one extra row); Megatron
 * column/row tensor parallelism; each gradient is all-reduced over the D
 * replicas before its optimizer op; memory by def/use liveness (outputs
 * allocated, peak sampled, inputs at their last use freed; weights,
 * optimizer state and the replica's inputs resident from t = 0).
 * Candidates are simulated one pipeline stage per GPU lane, grouped by P
 * through a permutation held in `workspace`: a device buffer of at least
 * dsim_parametric_workspace(n_cand) bytes (about 12 bytes per candidate,
 * DSIM_ENOSPC if shorter), owned by the caller, in use until hip_stream has
 * passed the call; no word of it needs clearing.  Transformer grids of
 * 8,192 or more candidates are simulated by two kernels, one for the
 * candidates of 1 to 8 stages (1 to 4 with the overlapped all-reduce, or with
 * ZeRO and no recomputation) and
 * one for the others; they run side by side
 * when side_stream is a second stream (hip_stream's earlier work is awaited
 * on it and the call's work on side_stream is awaited on hip_stream before
 * anything later, through two events the call creates and destroys), and
 * one after the other on hip_stream when side_stream is NULL or equal to
 * it; the results are the same.  n_cand < 2^31, and n_cand * W below
 * 2^32 - 2^9 lanes, W = min(row_width, 64, n_layers) rounded up to a power
 * of two (DSIM_ERANGE otherwise: split the call).
 */
DSIM_API size_t dsim_parametric_workspace(int64_t n_cand);
DSIM_API dsim_status dsim_simulate_parametric(const dsim_model *model, const dsim_strategy *cand,
                                     int64_t n_cand, const dsim_device_model *device,
                                     const dsim_results *results, void *workspace, size_t ws_bytes,
                                     void *side_stream, void *hip_stream);

/*
 * dsim_simulate_parametric_static -- dsim_simulate_parametric for callers
 * that cannot allocate (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the same simulation, results and
 * argument checks, with the grouping workspace in a fixed buffer the
 * library holds on each GPU it runs on (12.7 MB, kept until the process
 * ends; its address is taken on the first call on a GPU), and every kernel
 * on hip_stream (no second stream, no events).  The call allocates
 * nothing.  n_cand <= 2^20 (DSIM_ERANGE beyond).  All calls on one GPU
 * share that buffer: calls whose work overlaps on one GPU (different
 * streams, or host threads, without ordering between them) race and give
 * wrong results; calls ordered on one stream are safe.
 */
DSIM_API dsim_status dsim_simulate_parametric_static(const dsim_model *model, const dsim_strategy *cand,
                                            int64_t n_cand, const dsim_device_model *device,
                                            const dsim_results *results, void *hip_stream);

/*
 * dsim_materialize_tables -- write the whole distributed program of each of
 * n_cand strategies (device array `cand`) of `model` -- every op of every
 * device, the transform of Sec. 4 executed with the semantics of Sec. 2.1 --
 * as explicit op tables in the dsim_tables layout (op j of candidate c at
 * j * n_cand + c), so that dsim_simulate_tables simulates it.  GPU
 * g = p*(D*H) + d*H + h runs stage p of data replica d, tensor rank h, as
 * device g, or with model.overlap as devices 2g (computation) and 2g + 1
 * (communication), whose hand-overs are Sends of zero alloc and free.  The
 * program order interleaves devices, but each device's own op sequence is
 * the transform's: splits, then slot by slot the ready stages' blocks (a
 * compute op once per replica device, a tensor-parallel all-reduce once per
 * data replica over its H ranks) and the slot's Sends in ascending source
 * stage (one per replica), then the weight update (a gradient all-reduce
 * once per tensor rank over the D replicas, an optimizer op per device).
 * The record fields are those of dsim_tables: compute on a, send a -> b
 * (alloc on b, free on a), all-reduce over a device mask.
 *   code, flops, bytes, alloc_bytes, free_bytes: device arrays of
 *     max_ops * n_cand records, written for j < n_ops[c];
 *   mm_k:      device array of max_ops * n_cand entries or NULL: each
 *     record's reduction length (that of its matrix multiplication, 0 on
 *     other records), for dsim_tables.mm_k;
 *   n_ops:     device array [n_cand], the program's op count (0 on error);
 *   init_live: device array [n_cand * n_dev], bytes resident on each device
 *     at t = 0 (0 for devices the candidate does not use);
 *   status:    device array [n_cand]: 0, DSIM_ST_BAD_STRATEGY (the
 *     transform's preconditions fail, more devices than n_dev (D*H*P, twice that with overlap) or K > 16383), or
 *     DSIM_ST_NOT_TABLE (more than max_ops ops, a FLOP or byte count not
 *     exact in fp32, or an alloc / free size or a reduction length above
 *     2^32 - 1).
 * 1 <= n_dev <= 8, max_ops >= 0, n_cand <= 2^32 - 256.  One GPU lane per
 * candidate.
 */
DSIM_API dsim_status dsim_materialize_tables(const dsim_model *model, const dsim_strategy *cand, int64_t n_cand,
                                    int32_t max_ops, int32_t n_dev, uint32_t *code, float *flops,
                                    float *bytes, uint32_t *alloc_bytes, uint32_t *free_bytes,
                                    uint32_t *mm_k, uint32_t *n_ops, uint64_t *init_live, int32_t *status,
                                    void *hip_stream);

/*
 * dsim_argmin -- selection of Sec. 5.2 over device arrays of n entries:
 * feasible = status == 0 and (mem_cap == 0 or cand_peak <= mem_cap); the
 * feasible entries ranked by (makespan, index) ascending; the first k
 * (1 <= k <= 64) go to out_idx / out_makespan (device arrays of k entries),
 * padded with -1 / +inf; *out_found (device) = number written (<= k).
 * workspace: device buffer of at least dsim_argmin_workspace(n, k) bytes.
 * makespan values must not be NaN.
 */
DSIM_API size_t dsim_argmin_workspace(int64_t n, int32_t k);
DSIM_API dsim_status dsim_argmin(const double *makespan, const uint64_t *cand_peak, const int32_t *status,
                        int64_t n, uint64_t mem_cap, int32_t k, void *workspace, size_t ws_bytes,
                        int64_t *out_idx, double *out_makespan, int32_t *out_found,
                        void *hip_stream);

/*
 * dsim_generate_random_tables -- the random-program workload, written in the
 * dsim_tables layout (device buffers of n_ops * n_cand entries each, plus
 * n_ops_out[n_cand], which may be NULL).  Bit-reproducible from
 * (seed, candidate, op): draw f of op j of candidate c is output number
 * c*2^32 + j*32 + f + 1 of SplitMix64 seeded with `seed`.  Per op: kind 70%
 * compute / 20% send / 10% all-reduce; compute FLOPs log-uniform in
 * [1e6, 1e12], bytes log-uniform in [1e3, 1e9]; send to a uniform other
 * device; all-reduce over a uniform mask of >= 2 devices; every device
 * keeps up to 16 live buffers of log-uniform sizes in [1e3, 1e9] bytes,
 * freed in a valid order: a compute op or send first frees a uniformly
 * chosen live buffer of its (source) device with probability 1/2; a compute
 * op then allocates a new buffer with probability 1/2, and a send's message
 * (its bytes) becomes a live buffer of the destination, each only while the
 * device holds fewer than 16.
 * Log-uniform in [lo, hi]: 2^t rounded to fp32, t = log2 lo + u (log2 hi -
 * log2 lo), u = the top 53 bits of the draw / 2^53 (2^t from a fixed fp64
 * Taylor series, reproducible bit for bit).
 * Constraints: 2 <= n_dev <= 8, 0 <= n_ops < 2^27, 0 <= n_cand <= 2^32 - 256.
 */
DSIM_API dsim_status dsim_generate_random_tables(uint64_t seed, int64_t n_cand, int32_t n_ops,
                                        int32_t n_dev, uint32_t *code, float *flops,
                                        float *bytes, uint32_t *alloc_bytes,
                                        uint32_t *free_bytes, uint32_t *n_ops_out,
                                        void *hip_stream);

/*
 * Program front end (host only: no HIP call, no device memory; several
 * threads may call it at once).
 *
 * Program text, one statement per line, `#` starting a comment:
 *   func NAME(%p: TYPE [keep], ...)        -- first non-empty line
 *   %out, ... = OpType[key = VALUE, ...](%in, ...)
 *   return %v, ...                         -- ignored
 * TYPE is Tensor[DTYPE, (d0, d1, ...), DEVICE], Tensor[DTYPE, ??, DEVICE]
 * (shape unknown), DTYPE or DTYPE[DEVICE] (an abstract scalar); DTYPE one of
 * Float64 Float32 Float16 BFloat16 Int64 Int32 Int8 Bool.  VALUE is a number,
 * a quoted string or a (nested) list.  A parameter marked keep (weights)
 * stays resident for the whole program.  Op types: Constant Shape Gather
 * Unsqueeze Squeeze Concat Reshape Add Sub Mul Div Pow Relu Neg Sqrt Exp Tanh
 * Erf Gelu Identity Cast Softmax LayerNormalization Transpose Flatten Split
 * MatMul Gemm Send AllReduce, with ONNX's attributes (axis, axes, perm,
 * split, transA, transB, to, value; Send's device).
 *
 * Inputs text (NULL or empty: none): one binding per line, `%name = VALUE`
 * (a concrete value: a number or a rectangular nested list; int64 unless an
 * entry is a float) or `%name: TYPE` (an abstract value); each name must be
 * a parameter, and its binding replaces the declared type.
 *
 * Interpretation (Sec. 3, Algorithm 1; Sec. 3.3 and Fig. 4): the ops are
 * stepped through in order over a state mapping each variable to a value,
 * concrete (an int64 or fp64 array) or abstract (a tensor: element type,
 * shape or unknown, device; or a scalar), each op evaluated by its most
 * precise implementation for the kinds of its arguments (an op whose
 * arguments are all concrete is evaluated; Shape of a tensor of known shape
 * is concrete; Reshape of a tensor by a concrete target has a known shape).
 * mixed = 0 gives the abstract-only interpretation: every concrete value is
 * replaced by its type (shape arithmetic Int32, fp64 values Float64) as soon
 * as it appears.
 */

/*
 * dsim_interpret_program -- the final state of one interpretation as text:
 * one line `%name = VALUE` per variable (parameters first, then each op's
 * results in program order); VALUE is a concrete value as a number or a
 * nested list (fp64 values with a '.', an exponent, inf or nan), a tensor
 * as Tensor[DTYPE, (d0, ...), DEVICE] (?? for an unknown shape, None for no
 * device), a scalar as its DTYPE.  out: host buffer of cap bytes, written
 * NUL-terminated; *out_len (if out_len != NULL) = the bytes needed,
 * terminator included.  DSIM_ENOSPC if cap is smaller (out == NULL with
 * cap == 0 asks for the size); DSIM_EINVAL for a program that cannot be
 * read or interpreted (the message names the line); DSIM_ERANGE for a size
 * beyond 64 bits or a concrete value of more than 2^20 entries.
 */
DSIM_API dsim_status dsim_interpret_program(const char *program, const char *inputs, int32_t mixed,
                                            char *out, size_t cap, size_t *out_len);

/*
 * dsim_lower_programs -- n_prog programs interpreted (mixed) and lowered to
 * op tables in the dsim_tables layout, ready to be copied to the device for
 * dsim_simulate_tables (Sec. 3.3).  Lowering: an op that yields no abstract
 * tensor runs here and emits nothing; Reshape, Unsqueeze, Squeeze, Flatten
 * and Identity are views sharing their input's memory and emit nothing;
 * every other op on abstract tensors is one record: compute on the one
 * device of its tensors (MatMul and Gemm cost class 1), Send (alloc on the
 * receiver), AllReduce over the devices of its inputs (in place).  Compute
 * bytes: every abstract input and output tensor; flops: 1 per output element
 * for elementwise ops (Gelu 8, Softmax 5, LayerNormalization 8, Cast 0),
 * 2 * (output elements) * k for MatMul and Gemm (+1 per element with a
 * bias), 0 for Transpose, Concat, Split, Gather; Send and AllReduce: their
 * input's bytes.  Memory per storage: allocated by the record that creates
 * it, freed by its last reader (or its creator if unread); parameters are
 * resident at t = 0 (init_live), keep ones never freed; a storage last read
 * by an AllReduce stays live.
 *   programs, inputs: host arrays of n_prog strings; inputs may be NULL and
 *     its entries NULL (no inputs).
 *   n_dev: 1..8, the width of init_live's rows; every device a program uses
 *     must be below it (DSIM_ERANGE otherwise).
 *   max_ops: rows of the output arrays.
 *   code, flops, bytes, alloc_bytes, free_bytes: host arrays of
 *     max_ops * n_prog records, op-major and program-fastest (record j of
 *     program c at j * n_prog + c); rows from n_ops[c] on are zero.
 *   mm_k: host array of max_ops * n_prog entries, or NULL: each record's
 *     reduction length (MatMul: its left operand's last dimension; Gemm:
 *     the shared dimension; 0 on other records), for dsim_tables.mm_k;
 *     a length of 2^32 or more is DSIM_ERANGE.
 *   n_ops: host array [n_prog]; init_live: host array [n_prog * n_dev].
 *     All seven arrays (and mm_k) NULL: nothing is written and max_ops is
 *     not checked (a sizing pass).
 *   max_ops_used, n_dev_used (may be NULL): the largest record count of any
 *     program, and 1 + the highest device any program uses.
 *   n_threads: host threads to use (<= 1: the calling thread only).
 * Returns DSIM_EINVAL for a program that cannot be read, interpreted or
 * simulated (an unknown shape, an op on tensors of several devices, a
 * received tensor nothing reads), with the program's index and line in the
 * message; DSIM_ERANGE for a value that does not fit the record format
 * exactly (flops or bytes not exact in fp32, alloc or free >= 2^32) or a
 * device >= n_dev; DSIM_ENOSPC if some program needs more than max_ops
 * records (its n_ops entry is 0 and its column unwritten; *max_ops_used
 * says how many are needed).  On any error but DSIM_ENOSPC the outputs are
 * unspecified.
 */
DSIM_API dsim_status dsim_lower_programs(const char *const *programs, const char *const *inputs, int64_t n_prog,
                                         int32_t n_dev, int32_t max_ops, uint32_t *code, float *flops,
                                         float *bytes, uint32_t *alloc_bytes, uint32_t *free_bytes,
                                         uint32_t *mm_k, uint32_t *n_ops, uint64_t *init_live,
                                         int32_t *max_ops_used, int32_t *n_dev_used, int32_t n_threads);

#ifdef __cplusplus
}
#endif
#endif /* DSIM_H */
