// sim_tables.hip -- batched simulation of explicit op tables on CDNA4.
//
// One lane per candidate walks the candidate's ops in program order (DistIR
// semantics, Sec. 2.1: an op starts when all its devices are free, all of
// them finish together; Sec. 3.3: clock advance by the op's cost, live-memory
// tracking with the peak sampled after allocation and before the free).
//
// Layout: the tables are op-major and candidate-fastest, so at every step the
// 64 lanes of a wavefront read 64 consecutive records of each field (five
// coalesced 256-byte loads per op).  The record stream is read once, with
// non-temporal loads, `kUnroll` ops ahead of the arithmetic.
//
// Per-lane state: the device clocks live in VGPRs (n_dev <= 8 fp64) and are
// selected with the op's device mask, so an op touching any subset of devices
// costs the same branch-free instruction sequence; the per-device live and
// peak byte counters are indexed by a per-lane device id and live in LDS,
// laid out [device][lane] so that the 64 lanes of a wavefront always hit 64
// distinct 8-byte words.
#include "internal.h"

namespace dsim {
namespace {

constexpr int kBlock = 256;
constexpr int kUnroll = 4;

struct TabArgs {
    const uint32_t *code;
    const float *flops;
    const float *bytes;
    const uint32_t *alloc;
    const uint32_t *freeb;
    const uint32_t *n_ops;
    const uint64_t *init_live;
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

template <typename T>
__device__ __forceinline__ T stream_load(const T *p)
{
    return __builtin_nontemporal_load(p);
}

template <int ND>
__global__ __launch_bounds__(kBlock) void k_sim_tables(const TabArgs a)
{
    __shared__ uint64_t s_live[ND][kBlock];
    __shared__ uint64_t s_peak[ND][kBlock];
    __shared__ double s_arl[ND + 1];
    __shared__ double s_arc[ND + 1];

    const int tid = threadIdx.x;
    if (tid <= ND) {
        s_arl[tid] = a.c.ar_lat[tid];
        s_arc[tid] = a.c.ar_coef[tid];
    }
    const int64_t c = (int64_t)blockIdx.x * kBlock + tid;
    const bool active = c < a.n_cand;
#pragma unroll
    for (int d = 0; d < ND; ++d) {
        const uint64_t v = (active && a.init_live) ? a.init_live[c * ND + d] : 0;
        s_live[d][tid] = v;
        s_peak[d][tid] = v;
    }
    __syncthreads();
    if (!active) return;

    uint32_t nops = a.n_ops ? a.n_ops[c] : (uint32_t)a.max_ops;
    int32_t st = 0;
    if (nops > (uint32_t)a.max_ops) {
        st |= DSIM_ST_BAD_OP;
        nops = (uint32_t)a.max_ops;
    }
    double clk[ND];
#pragma unroll
    for (int d = 0; d < ND; ++d) clk[d] = 0.0;

    const double inv_f = a.c.inv_f, inv_b = a.c.inv_b, inv_l = a.c.inv_l;
    const double lat = a.c.lat, launch = a.c.launch;
    const size_t N = (size_t)a.n_cand;

    for (int32_t j0 = 0; j0 < a.max_ops; j0 += kUnroll) {
        uint32_t cd[kUnroll], al[kUnroll], fr[kUnroll];
        float fl[kUnroll], by[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int32_t j = j0 + u;
            if (j < a.max_ops) {
                const size_t o = (size_t)j * N + (size_t)c;
                cd[u] = stream_load(a.code + o);
                fl[u] = stream_load(a.flops + o);
                by[u] = stream_load(a.bytes + o);
                al[u] = stream_load(a.alloc + o);
                fr[u] = stream_load(a.freeb + o);
            } else {
                cd[u] = 0; fl[u] = 0.f; by[u] = 0.f; al[u] = 0; fr[u] = 0;
            }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            if ((uint32_t)(j0 + u) >= nops) break;
            const uint32_t code = cd[u];
            const uint32_t kind = code & 0xffu;
            const uint32_t ia = (code >> 8) & 0xffu;
            const uint32_t ib = (code >> 16) & 0xffu;
            const bool a_ok = ia < (uint32_t)ND, b_ok = ib < (uint32_t)ND;
            const uint32_t bit_a = a_ok ? (1u << ia) : 0u;
            const uint32_t bit_b = b_ok ? (1u << ib) : 0u;

            // validity, in the order the format defines it
            uint32_t flag, m;
            if ((code >> 24) != 0u || kind > 2u) {
                flag = DSIM_ST_BAD_OP;
                m = 0u;
            } else if (kind == 0u) {
                flag = a_ok ? 0u : (uint32_t)DSIM_ST_BAD_DEVICE;
                m = bit_a;
            } else if (kind == 1u) {
                flag = (!a_ok || !b_ok) ? (uint32_t)DSIM_ST_BAD_DEVICE
                                        : (ia == ib ? (uint32_t)DSIM_ST_SELF_SEND : 0u);
                m = bit_a | bit_b;
            } else {
                flag = (ib == 0u || (ib >> ND) != 0u) ? (uint32_t)DSIM_ST_BAD_DEVICE : 0u;
                m = ib;
            }
            if (flag) m = 0u;
            st |= (int32_t)flag;

            // op cost (Sec. 3.3 / Sec. 4 cost functions)
            const double f = (double)fl[u], b = (double)by[u];
            const double tf = f * inv_f, tb = b * inv_b;
            const double t_comp = launch + (tf > tb ? tf : tb);
            const double tl = b * inv_l;
            const double t_send = lat + tl;
            const int n = __popc(m);
            const double t_ar = s_arl[n] + s_arc[n] * tl;
            const double cost = kind == 0u ? t_comp : (kind == 1u ? t_send : t_ar);

            // synchronous start on the device set, common end
            double start = 0.0;
#pragma unroll
            for (int d = 0; d < ND; ++d) {
                const double v = ((m >> d) & 1u) ? clk[d] : 0.0;
                start = v > start ? v : start;
            }
            const double end = start + cost;
#pragma unroll
            for (int d = 0; d < ND; ++d) clk[d] = ((m >> d) & 1u) ? end : clk[d];

            // live memory: allocate on the target, sample, free on the source
            const bool memop = flag == 0u && kind != 2u;
            const uint32_t alloc = memop ? al[u] : 0u;
            const uint32_t fre = memop ? fr[u] : 0u;
            const uint32_t tdev = memop ? (kind == 1u ? ib : ia) : 0u;
            const uint32_t fdev = memop ? ia : 0u;
            const uint64_t lv = s_live[tdev][tid] + (uint64_t)alloc;
            s_live[tdev][tid] = lv;
            const uint64_t pk = s_peak[tdev][tid];
            s_peak[tdev][tid] = lv > pk ? lv : pk;
            const uint64_t lf = s_live[fdev][tid];
            const bool under = (uint64_t)fre > lf;
            st |= under ? DSIM_ST_MEM_UNDERFLOW : 0;
            s_live[fdev][tid] = under ? 0ull : lf - (uint64_t)fre;
        }
    }

    double mk = 0.0;
    uint64_t cp = 0;
#pragma unroll
    for (int d = 0; d < ND; ++d) {
        mk = clk[d] > mk ? clk[d] : mk;
        const uint64_t p = s_peak[d][tid];
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
        for (int d = 0; d < ND; ++d) row[d] = clk[d];
        for (int d = ND; d < a.row_width; ++d) row[d] = 0.0;
    }
    if (a.peak) {
        uint64_t *row = a.peak + (size_t)c * a.row_width;
#pragma unroll
        for (int d = 0; d < ND; ++d) row[d] = s_peak[d][tid];
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
