// sim_tables.hip -- batched simulation of explicit op tables on CDNA4.
//
// One lane per candidate walks the candidate's ops in program order (DistIR
// semantics, Sec. 2.1: an op starts when all its devices are free, all of
// them finish together; Sec. 3.3: clock advance by the op's cost, live-memory
// tracking with the peak sampled after allocation and before the free).
//
// Layout: the tables are op-major and candidate-fastest, so at every step the
// 64 lanes of a wavefront read 64 consecutive records of each field (five
// coalesced 256-byte loads per op).  The record stream is read once with
// non-temporal raw buffer loads: one descriptor per field and group of ops,
// based at the workgroup's first record, so the per-lane address is a 32-bit
// byte offset and no lane does 64-bit address arithmetic.  Two register sets
// of kUnroll ops alternate: one is processed while the other is in flight.
//
// Per-lane state: the device clocks live in VGPRs (n_dev <= 8 fp64) and take
// the op's device mask as their sign bits (set outside the op) while the
// start is taken, so an op touching any subset of devices runs the same
// branch-free sequence; the per-device (live,
// peak) byte counters are indexed by a per-lane device id and live in LDS as
// 16-byte pairs laid out [device][lane], so the 64 lanes of a wavefront
// always hit 64 distinct pairs.  An op's cost is base + coef * x with
// x = max(flops * g, bytes * w): (base, coef) and (w, g) come from small LDS
// tables indexed by the op class (compute: launch, 1, 1/B, 1/F; send:
// latency, 1, 1/L, 0; all-reduce over n devices: the ring terms for n, 1/L,
// 0), so every lane runs one straight sequence.  The tables hold one copy per
// lane of a 16-lane group, so that lanes reading different classes spread
// over the banks (a 64-lane b128 read still takes several LDS cycles).
//
// The kernel runs close to the rate at which HBM returns its op records
// (about 82 vector instructions per op keep the vector units partly busy
// beside that); it has a fast path for the ops every lane of a wavefront
// has, which assumes valid compute, send and all-reduce ops of cost class 0
// (indices clamped, so even an invalid op stays in bounds) and only tests
// whether each op is one; a lane that meets an op it cannot vouch for (a
// free that would underflow, a broadcast or reduce record, a matrix
// multiplication record), and every lane's ops past the wavefront's common
// count, go through the exact per-op path below it.
#include "internal.h"

namespace dsim {
namespace {

constexpr int kBlock = 256;       // 4 wavefronts; 32 KB of LDS counters
constexpr int kWavesPerSimd = 4;
constexpr int kUnroll = 4;   // ops per register set; two sets in flight
constexpr int kCopies = 16;  // copies of the per-class cost rows (one per lane of an LDS phase)

struct TabArgs {
    const uint32_t *code;
    const float *flops;
    const float *bytes;
    const uint32_t *alloc;
    const uint32_t *freeb;
    const uint32_t *n_ops;
    const uint64_t *init_live;
    const uint32_t *mm_k;   // reduction lengths of class-1 records (NULL: 0)
    int64_t n_cand;
    int32_t max_ops;
    int32_t row_width;
    double *makespan;
    double *finish;
    uint64_t *peak;
    uint64_t *cand_peak;
    uint64_t *n_ops_out;
    uint64_t *walked;
    int32_t *status;
    CostConsts c;
};

// Buffer resource covering one workgroup's 64 consecutive 4-byte records of
// one op row (raw buffer, gfx9 descriptor word 3); the base is wave-uniform,
// so the per-lane address is just a 32-bit byte offset.
constexpr int kRsrcWord3 = 0x00020000;
constexpr int kNonTemporal = 2;   // streamed once: do not keep in the caches
// the fast path's loads reach kUnroll op rows (kUnroll * n_cand * 4 bytes)
// from one descriptor with 32-bit offsets
constexpr int64_t kMaxFastCand = (int64_t)(0xffffffffu / (4u * kUnroll));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t group_rsrc(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, kRsrcWord3);
}

// max of two doubles that are never NaN.  The compiler's fmax first
// canonicalizes an operand it cannot prove canonical (a loop-carried clock),
// one extra instruction per device and op; the bare instruction gives the
// same value (of +0.0 and -0.0 it may return either).
__device__ __forceinline__ double max_nn(double a, double b)
{
    double r;
    asm("v_max_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}

// max(|a|, b), the absolute value taken by the instruction's input modifier
__device__ __forceinline__ double max_abs(double a, double b)
{
    double r;
    asm("v_max_f64 %0, |%1|, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}

// x with its sign bit replaced by bit 31 of s (one bit-field insert on the
// high word; the low word is untouched)
__device__ __forceinline__ double with_sign(double x, uint32_t s)
{
    const uint64_t b = (uint64_t)__double_as_longlong(x);
    const uint32_t hi = (s & 0x80000000u) | ((uint32_t)(b >> 32) & 0x7fffffffu);
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | (b & 0xffffffffull)));
}

// max of two byte counts below 2^63 as one fp64 max of their bit patterns:
// those are non-negative doubles (denormal below 2^52; fp64 denormals are
// preserved in this kernel's float mode), which order like the integers
__device__ __forceinline__ uint64_t max_bits(uint64_t a, uint64_t b)
{
    return (uint64_t)__double_as_longlong(max_nn(__longlong_as_double((long long)a), __longlong_as_double((long long)b)));
}

__device__ __forceinline__ double bits_double(uint32_t lo, uint32_t hi)
{
    return __hiloint2double((int)hi, (int)lo);
}

// Status bits of one op, exactly as the table format defines validity.
template <int ND>
__device__ __forceinline__ uint32_t op_flags(uint32_t code, uint32_t flops_bits, uint32_t bytes_bits)
{
    const uint32_t kind = code & 0xffu, ia = (code >> 8) & 0xffu, ib = (code >> 16) & 0xffu, cls = code >> 24;
    // kind, cost class (1 only on compute records), and flops/bytes finite
    // and >= 0 (bit patterns below +inf)
    if (cls > 1u || (cls == 1u && kind != 0u) || kind > 4u || flops_bits >= 0x7f800000u || bytes_bits >= 0x7f800000u)
        return DSIM_ST_BAD_OP;
    if (kind == 0u) return ia < (uint32_t)ND ? 0u : (uint32_t)DSIM_ST_BAD_DEVICE;
    if (kind == 1u) {
        if (ia >= (uint32_t)ND || ib >= (uint32_t)ND) return DSIM_ST_BAD_DEVICE;
        return ia == ib ? (uint32_t)DSIM_ST_SELF_SEND : 0u;
    }
    if (kind == 2u) return (ib == 0u || (ib >> ND) != 0u) ? (uint32_t)DSIM_ST_BAD_DEVICE : 0u;
    // broadcast / reduce: the root is a member of the mask
    return (ia >= (uint32_t)ND || (ib >> ND) != 0u || ((ib >> ia) & 1u) == 0u) ? (uint32_t)DSIM_ST_BAD_DEVICE : 0u;
}

template <int ND>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(kWavesPerSimd))) void k_sim_tables(
    const TabArgs a)
{
    __shared__ ulonglong2 s_mem[ND][kBlock];   // (live, peak) bytes
    // per op class -- all-reduce over n = 0..ND devices, then compute, then
    // send -- the cost terms (base, coef) and (1/bandwidth, 1/flop rate or 0)
    // (one array: the second pair sits at a fixed offset from the first, so
    // one address serves both loads)
    __shared__ double2 s_ct[2][ND + 3][kCopies];
    __shared__ double2 s_cost[ND + 3];   // (base, coef) for the exact path

    const int tid = threadIdx.x;
    if (tid <= ND) s_cost[tid] = make_double2(a.c.ar_lat[tid], a.c.ar_coef[tid]);
    if (tid == ND + 1) s_cost[tid] = make_double2(a.c.launch, 1.0);
    if (tid == ND + 2) s_cost[tid] = make_double2(a.c.lat, 1.0);
    for (int i = tid; i < (ND + 3) * kCopies; i += kBlock) {
        const int e = i / kCopies, k = i % kCopies;
        const bool cmp = e == ND + 1;
        s_ct[0][e][k] = make_double2(e <= ND ? a.c.ar_lat[e] : (cmp ? a.c.launch : a.c.lat), e <= ND ? a.c.ar_coef[e] : 1.0);
        // an all-reduce over one device costs nothing, whatever its bytes
        // (zero weights keep an overflowing byte term out: 0 * inf is NaN)
        s_ct[1][e][k] = make_double2(e <= 1 ? 0.0 : (cmp ? a.c.inv_b : a.c.inv_l), cmp ? a.c.inv_f : 0.0);
    }

    const int64_t c = (int64_t)blockIdx.x * kBlock + tid;
    const bool active = c < a.n_cand;
    // the fast path compares live bytes as fp64 bit patterns, which order
    // like the integers below 2^63 - 2^52: a lane starting at 2^62 or more
    // live bytes on a device (its ops add less than 2^43) takes the exact path
    bool big_init = false;
#pragma unroll
    for (int d = 0; d < ND; ++d) {
        const uint64_t init = (active && a.init_live) ? a.init_live[c * ND + d] : 0;
        big_init |= init >= (1ull << 62);
        s_mem[d][tid] = make_ulonglong2(init, init);
    }
    __syncthreads();

    uint32_t nops = active ? (a.n_ops ? a.n_ops[c] : (uint32_t)a.max_ops) : 0xffffffffu;
    // a lane whose op count exceeds max_ops is flagged and simulates max_ops
    // ops; the flag survives the exact path's restart (st0)
    const int32_t st0 = (active && nops > (uint32_t)a.max_ops) ? DSIM_ST_BAD_OP : 0;
    int32_t st = st0;
    if (st0) nops = (uint32_t)a.max_ops;
    // ops every lane of the wavefront has (inactive lanes do not constrain it)
    uint32_t wave_min = nops;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) wave_min = min(wave_min, (uint32_t)__shfl_xor((int)wave_min, off));
    if (!active) return;
    double clk[ND];
#pragma unroll
    for (int d = 0; d < ND; ++d) clk[d] = 0.0;

    const double inv_f = a.c.inv_f, inv_b = a.c.inv_b, inv_l = a.c.inv_l;
    const double lat = a.c.lat, launch = a.c.launch;
    const size_t N = (size_t)a.n_cand;

    // ---- fast path: the ops every lane of the wavefront has ------------------
    // Ops are assumed valid; a cheap test marks any lane that meets an op it
    // cannot vouch for, and that lane is re-simulated by the exact path below.
    // Indices are clamped so that even an invalid op stays inside the arrays.
    // (with nodes or streams, communication costs depend on which devices an
    // op spans: every op takes the exact path; so do tables of more than
    // kMaxFastCand candidates, whose op rows are too far apart for the 32-bit
    // offsets of the fast path's loads)
    const int32_t fast_end = (a.c.node || a.c.streams || a.n_cand > kMaxFastCand)
                                 ? 0
                                 : (int32_t)(__builtin_amdgcn_readfirstlane(wave_min) / kUnroll) * kUnroll;

    const size_t blk = (size_t)blockIdx.x * kBlock;
    const uint32_t lane_b = (uint32_t)tid * 4u;
    bool suspect = big_init;
    uint32_t fb_max = 0;   // largest flops or bytes bit pattern met on the fast path

    // two register sets of kUnroll op records: one is processed while the
    // other is in flight
    uint32_t cdA[kUnroll], flA[kUnroll], byA[kUnroll], alA[kUnroll], frA[kUnroll];
    uint32_t cdB[kUnroll], flB[kUnroll], byB[kUnroll], alB[kUnroll], frB[kUnroll];
    // One buffer descriptor per field and group of kUnroll op rows (based at
    // this workgroup's first record); op u of the group is u*N records
    // further, a scalar offset.
    const uint32_t row_bytes = (uint32_t)(N * 4u);
    const uint32_t grp_bytes = (uint32_t)min((size_t)0xffffffffu, (size_t)kUnroll * N * 4u);
    auto load_group = [&](int32_t j0, uint32_t(&cd)[kUnroll], uint32_t(&fl)[kUnroll], uint32_t(&by)[kUnroll],
                          uint32_t(&al)[kUnroll], uint32_t(&fr)[kUnroll]) {
        const size_t base = (size_t)j0 * N + blk;
        const __amdgpu_buffer_rsrc_t rc = group_rsrc(a.code + base, grp_bytes);
        const __amdgpu_buffer_rsrc_t rf = group_rsrc(a.flops + base, grp_bytes);
        const __amdgpu_buffer_rsrc_t rb = group_rsrc(a.bytes + base, grp_bytes);
        const __amdgpu_buffer_rsrc_t ra = group_rsrc(a.alloc + base, grp_bytes);
        const __amdgpu_buffer_rsrc_t rr = group_rsrc(a.freeb + base, grp_bytes);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int so = (int)(u * row_bytes);
            cd[u] = __builtin_amdgcn_raw_buffer_load_b32(rc, (int)lane_b, so, kNonTemporal);
            fl[u] = __builtin_amdgcn_raw_buffer_load_b32(rf, (int)lane_b, so, kNonTemporal);
            by[u] = __builtin_amdgcn_raw_buffer_load_b32(rb, (int)lane_b, so, kNonTemporal);
            al[u] = __builtin_amdgcn_raw_buffer_load_b32(ra, (int)lane_b, so, kNonTemporal);
            fr[u] = __builtin_amdgcn_raw_buffer_load_b32(rr, (int)lane_b, so, kNonTemporal);
        }
    };
    auto run_group = [&](const uint32_t(&cd)[kUnroll], const uint32_t(&fl)[kUnroll],
                         const uint32_t(&by)[kUnroll], const uint32_t(&al)[kUnroll],
                         const uint32_t(&fr)[kUnroll]) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            // Everything below is computed for every lane and combined with
            // selects, so the wavefront runs one straight sequence whatever
            // the op kinds of its lanes.
            const uint32_t code = cd[u];
            const uint32_t ia = (code >> 8) & 0xffu, ib = (code >> 16) & 0xffu;
            bool is_c, is_s, is_a;
            if constexpr ((ND & (ND - 1)) == 0) {
                // one masked compare per kind tests the reserved byte, the
                // kind and the device fields that must be < ND at once; an
                // op that passes none is invalid, and the selects below
                // treat it as an all-reduce over its (clamped) fields
                constexpr uint32_t hi = ~(uint32_t)(ND - 1) & 0xffu;
                constexpr uint32_t m0 = 0xff0000ffu | (hi << 8), m1 = m0 | (hi << 16), m2 = 0xff0000ffu;
                is_c = (code & m0) == 0u;
                is_s = (code & m1) == 1u;
                is_a = (code & m2) == 2u;
                const uint32_t ma = ib & ((1u << ND) - 1u);
                suspect |= !(is_c | (is_s & (ia != ib)) | (is_a & (ma != 0u) & (ib == ma)));
            } else {
                const uint32_t kind = code & 0xffu;
                is_c = kind == 0u;
                is_s = kind == 1u;
                is_a = kind == 2u;
                suspect |= (code >= (1u << 24)) | (kind > 2u) | ((ia >= (uint32_t)ND) & !is_a) |
                           (is_s & ((ib >= (uint32_t)ND) | (ia == ib))) | (is_a & ((ib == 0u) | (ib >= (1u << ND))));
            }
            // flops and bytes must be finite and >= 0: as integers, below
            // the bits of +inf (negative values have the sign bit set)
            fb_max = max(fb_max, max(fl[u], by[u]));
            const uint32_t ias = min(ia, (uint32_t)ND - 1u), ibs = min(ib, (uint32_t)ND - 1u);
            const uint32_t mc = 1u << ias, ms = mc | (1u << ibs), ma = ib & ((1u << ND) - 1u);
            const uint32_t m = is_c ? mc : (is_s ? ms : ma);

            // op cost (Sec. 3.3 / Sec. 4 cost functions) as base + coef * x:
            // compute (launch, 1, max(flops/F, bytes/B)), send (lat, 1,
            // bytes/L), all-reduce over n devices (ar_lat[n], ar_coef[n],
            // bytes/L); multiplying by 1.0 is exact
            const uint32_t idx = is_c ? (uint32_t)ND + 1u : (is_s ? (uint32_t)ND + 2u : (uint32_t)__popc(m));
            const double2 bc = s_ct[0][idx][tid & (kCopies - 1)], rw = s_ct[1][idx][tid & (kCopies - 1)];
            // a non-compute class carries 0 as its flop reciprocal: a valid
            // op's flops are finite, so that term is +0 and the max is the
            // bandwidth term, as in the per-kind formulas
            const double f = (double)__uint_as_float(fl[u]), b = (double)__uint_as_float(by[u]);
            const double cost = bc.x + bc.y * max_nn(f * rw.y, b * rw.x);

            // synchronous start on the device set, common end.  Bit 31 of
            // xs[d] is set for a device outside the op; the clocks take it
            // as their sign, so the max over all of them is the max over the
            // participants (clocks are >= 0: outside clocks become <= -0.0,
            // below every participant's).  The update takes max(|clk|, e)
            // with e = end for a participant and -end outside: participants
            // (clk <= start <= end) get end, the others keep their clock,
            // bit-exact.  A clock may come out as -0.0 (max of +0.0 and
            // -0.0), which compares equal to 0.0; the epilogue adds +0.0
            // to every stored clock.
            const uint32_t nm = ~m;
            uint32_t xs[ND];
#pragma unroll
            for (int d = 0; d < ND; ++d) xs[d] = nm << (31 - d);
#pragma unroll
            for (int d = 0; d < ND; ++d) clk[d] = with_sign(clk[d], xs[d]);
            // pairwise max tree (max is exact, so the order does not matter)
            double v[ND];
#pragma unroll
            for (int d = 0; d < ND; ++d) v[d] = clk[d];
#pragma unroll
            for (int w = 1; w < ND; w *= 2)
#pragma unroll
                for (int d = 0; d + w < ND; d += 2 * w) v[d] = max_nn(v[d], v[d + w]);
            const double end = v[0] + cost;
#pragma unroll
            for (int d = 0; d < ND; ++d) clk[d] = max_abs(clk[d], with_sign(end, xs[d]));

            // live memory: allocate on the target, sample, free on the
            // source (an all-reduce moves no memory).  A free that would
            // underflow marks the lane for the exact path.
            const uint32_t alloc = is_a ? 0u : al[u];
            const uint32_t fre = is_a ? 0u : fr[u];
            const uint32_t tdev = is_s ? ibs : ias;
            const uint32_t fdev = ias;
            const ulonglong2 tm = s_mem[tdev][tid];
            const uint64_t lt = tm.x + (uint64_t)alloc;
            s_mem[tdev][tid] = make_ulonglong2(lt, max_bits(lt, tm.y));
            // read after that write: a compute op frees on the device it
            // allocated on, and sees its own allocation
            const uint64_t lf = s_mem[fdev][tid].x;
            suspect |= (uint64_t)fre > lf;
            s_mem[fdev][tid].x = lf - (uint64_t)fre;
        }
    };
    if (fast_end > 0) load_group(0, cdA, flA, byA, alA, frA);
    for (int32_t j0 = 0; j0 < fast_end; j0 += 2 * kUnroll) {
        if (j0 + kUnroll < fast_end) load_group(j0 + kUnroll, cdB, flB, byB, alB, frB);
        run_group(cdA, flA, byA, alA, frA);
        if (j0 + kUnroll >= fast_end) break;
        if (j0 + 2 * kUnroll < fast_end) load_group(j0 + 2 * kUnroll, cdA, flA, byA, alA, frA);
        run_group(cdB, flB, byB, alB, frB);
    }

    suspect |= fb_max >= 0x7f800000u;

    // ---- exact path: this lane's remaining ops, or all of them again if the
    // fast path met an op it could not vouch for -------------------------------
    int32_t j = fast_end;
    if (suspect) {
        j = 0;
        st = st0;
#pragma unroll
        for (int d = 0; d < ND; ++d) {
            clk[d] = 0.0;
            // read again rather than kept in registers across the fast path
            const uint64_t init = a.init_live ? a.init_live[c * ND + d] : 0;
            s_mem[d][tid] = make_ulonglong2(init, init);
        }
    }
    for (; j < (int32_t)nops; ++j) {
        const size_t o = (size_t)j * N + (size_t)c;
        const uint32_t code = a.code[o];
        const float flf = a.flops[o], byf = a.bytes[o];
        const uint32_t flag = op_flags<ND>(code, __float_as_uint(flf), __float_as_uint(byf));
        st |= (int32_t)flag;
        if (flag) continue;   // an invalid op is skipped: no time, no memory
        const uint32_t kind = code & 0xffu, ia = (code >> 8) & 0xffu, ib = (code >> 16) & 0xffu;
        const uint32_t m = kind == 0u ? (1u << ia) : (kind == 1u ? ((1u << ia) | (1u << ib)) : ib);
        const double f = (double)flf, b = (double)byf;
        // the tier a communication op crosses: the streams of one GPU when
        // all its devices lie on one GPU (GPUs hold consecutive devices, so
        // its lowest and highest device decide), the network when its GPUs
        // lie in more than one node, the node's links otherwise
        int tier = 0;
        if ((a.c.node || a.c.streams) && kind != 0u) {
            const int lo = __ffs(m) - 1, hi = 31 - __clz(m);
            const int S = a.c.streams ? a.c.streams : 1;
            const int glo = lo / S, ghi = hi / S;
            if (a.c.streams && glo == ghi) tier = 2;
            else if (a.c.node && glo / a.c.node != ghi / a.c.node) tier = 1;
        }
        const double c_lat = tier == 2 ? a.c.st_lat : (tier == 1 ? a.c.net_lat : lat);
        const double c_inv_l = tier == 2 ? a.c.st_inv_l : (tier == 1 ? a.c.net_inv_l : inv_l);
        double cost;
        if (kind == 0u && (code >> 24) == 1u && a.c.mm) {
            // a matrix multiplication: the empirical regression of Sec. 4,
            // with its reduction-length term and floor
            const double k = a.mm_k ? (double)a.mm_k[o] : 0.0;
            const double lin = ((a.c.mm_c0 + a.c.mm_c1 * f) + a.c.mm_c2 * b) + a.c.mm_c3 * k;
            cost = a.c.mm_floor > lin ? a.c.mm_floor : lin;
        } else if (kind == 0u) {
            const double tf = f * inv_f, tb = b * inv_b;
            cost = launch + (tf > tb ? tf : tb);
        } else if (kind == 1u) {
            cost = c_lat + b * c_inv_l;
        } else if (kind == 2u) {
            // over one device it costs nothing (its byte term may overflow)
            const double2 ar = s_cost[__popc(m)];
            const int n = __popc(m);
            cost = n > 1 ? (tier == 2 ? a.c.ar_lat_st[n] : (tier == 1 ? a.c.ar_lat_net[n] : ar.x)) + ar.y * (b * c_inv_l)
                         : 0.0;
        } else {
            // broadcast / reduce: a chain of n - 1 hops (Fig. 9's Send for n = 2)
            const int n = __popc(m);
            cost = n > 1 ? (double)(n - 1) * c_lat + b * c_inv_l : 0.0;
        }
        double start = 0.0;
#pragma unroll
        for (int d = 0; d < ND; ++d)
            if (((m >> d) & 1u) && clk[d] > start) start = clk[d];
        const double end = start + cost;
#pragma unroll
        for (int d = 0; d < ND; ++d)
            if ((m >> d) & 1u) clk[d] = end;
        if (kind >= 3u) {
            // the receivers (broadcast) or the root (reduce) allocate, every
            // member samples its peak, then the root (broadcast) or every
            // member (reduce) frees
            const uint64_t al = a.alloc[o], fr = a.freeb[o];
#pragma unroll
            for (int d = 0; d < ND; ++d) {
                if (((m >> d) & 1u) == 0u) continue;
                const bool gets = kind == 3u ? (uint32_t)d != ia : (uint32_t)d == ia;
                const uint64_t lt = s_mem[d][tid].x + (gets ? al : 0u);
                s_mem[d][tid].x = lt;
                if (lt > s_mem[d][tid].y) s_mem[d][tid].y = lt;
            }
#pragma unroll
            for (int d = 0; d < ND; ++d) {
                if (((m >> d) & 1u) == 0u || (kind == 3u && (uint32_t)d != ia)) continue;
                const uint64_t lf = s_mem[d][tid].x;
                if (fr > lf) {
                    st |= DSIM_ST_MEM_UNDERFLOW;
                    s_mem[d][tid].x = 0;
                } else {
                    s_mem[d][tid].x = lf - fr;
                }
            }
        } else if (kind != 2u) {
            const uint32_t tdev = kind == 1u ? ib : ia;
            const uint64_t lt = s_mem[tdev][tid].x + (uint64_t)a.alloc[o];
            s_mem[tdev][tid].x = lt;
            if (lt > s_mem[tdev][tid].y) s_mem[tdev][tid].y = lt;
            const uint64_t lf = s_mem[ia][tid].x, fre = (uint64_t)a.freeb[o];
            if (fre > lf) {
                st |= DSIM_ST_MEM_UNDERFLOW;
                s_mem[ia][tid].x = 0;
            } else {
                s_mem[ia][tid].x = lf - fre;
            }
        }
    }

    double mk = 0.0;
    uint64_t cp = 0;
#pragma unroll
    for (int d = 0; d < ND; ++d) {
        mk = clk[d] > mk ? clk[d] : mk;
        const uint64_t p = s_mem[d][tid].y;
        cp = p > cp ? p : cp;
    }
    if (a.c.cap != 0 && cp > a.c.cap) st |= DSIM_ST_OVER_CAP;
    a.makespan[c] = mk;
    a.cand_peak[c] = cp;
    a.status[c] = st;
    if (a.n_ops_out) a.n_ops_out[c] = nops;
    if (a.walked) a.walked[c] = nops;
    if (a.finish) {
        double *row = a.finish + (size_t)c * a.row_width;
#pragma unroll
        for (int d = 0; d < ND; ++d) row[d] = clk[d] + 0.0;   // -0.0 -> +0.0
        for (int d = ND; d < a.row_width; ++d) row[d] = 0.0;
    }
    if (a.peak) {
        uint64_t *row = a.peak + (size_t)c * a.row_width;
#pragma unroll
        for (int d = 0; d < ND; ++d) row[d] = s_mem[d][tid].y;
        for (int d = ND; d < a.row_width; ++d) row[d] = 0;
    }
}

template <int ND>
hipError_t launch_nd(const TabArgs &a, hipStream_t s)
{
    const int64_t blocks = (a.n_cand + kBlock - 1) / kBlock;
    hipLaunchKernelGGL(k_sim_tables<ND>, dim3((unsigned)blocks), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

}  // namespace

dsim_status launch_sim_tables(const dsim_tables &t, int64_t n_cand, const CostConsts &c,
                              const dsim_results &r, hipStream_t s)
{
    if (n_cand == 0) return DSIM_OK;
    TabArgs a;
    a.code = t.code;
    a.flops = t.flops;
    a.bytes = t.bytes;
    a.alloc = t.alloc_bytes;
    a.freeb = t.free_bytes;
    a.n_ops = t.n_ops;
    a.init_live = t.init_live;
    a.mm_k = t.mm_k;
    a.n_cand = n_cand;
    a.max_ops = t.max_ops;
    a.row_width = r.row_width;
    a.makespan = r.makespan;
    a.finish = r.finish;
    a.peak = r.peak;
    a.cand_peak = r.cand_peak;
    a.n_ops_out = r.n_ops;
    a.walked = r.walked_ops;
    a.status = r.status;
    a.c = c;
    hipError_t e;
    switch (t.n_dev) {
    case 1: e = launch_nd<1>(a, s); break;
    case 2: e = launch_nd<2>(a, s); break;
    case 3: e = launch_nd<3>(a, s); break;
    case 4: e = launch_nd<4>(a, s); break;
    case 5: e = launch_nd<5>(a, s); break;
    case 6: e = launch_nd<6>(a, s); break;
    case 7: e = launch_nd<7>(a, s); break;
    default: e = launch_nd<8>(a, s); break;
    }
    return e == hipSuccess ? DSIM_OK : hip_fail(e, "sim_tables launch");
}

}  // namespace dsim
