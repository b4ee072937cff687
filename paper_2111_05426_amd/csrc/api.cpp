// api.cpp -- the extern "C" entry points of libdsim (include/dsim.h).
//
// Host side only: argument validation, the grid enumeration of Sec. 5.1,
// the device-model constants, and the kernel launches on the caller's stream.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "internal.h"

namespace dsim {

static thread_local char g_err[512] = "";

dsim_status fail(dsim_status st, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return st;
}

dsim_status hip_fail(hipError_t e, const char *what)
{
    return fail(DSIM_EHIP, "%s: %s", what, hipGetErrorString(e));
}

CostConsts make_consts(const dsim_device_model &m)
{
    CostConsts c;
    std::memset(&c, 0, sizeof c);
    c.inv_f = 1.0 / m.flops_per_s;
    c.inv_b = 1.0 / m.mem_bytes_per_s;
    c.inv_l = 1.0 / m.link_bytes_per_s;
    c.lat = m.link_latency_s;
    c.launch = m.launch_s;
    c.cap = m.mem_cap_bytes;
    c.mm = m.mm_enabled;
    c.mm_c0 = m.mm_enabled ? m.mm_c0 : 0.0;
    c.mm_c1 = m.mm_enabled ? m.mm_c1 : 0.0;
    c.mm_c2 = m.mm_enabled ? m.mm_c2 : 0.0;
    c.mm_c3 = m.mm_enabled ? m.mm_c3 : 0.0;
    c.mm_floor = m.mm_enabled ? m.mm_floor : 0.0;
    c.node = m.node_size > 0 ? m.node_size : 0;
    c.net_lat = c.node ? m.net_latency_s : 0.0;
    c.net_inv_l = c.node ? 1.0 / m.net_bytes_per_s : 0.0;
    c.streams = m.streams_per_gpu > 1 ? m.streams_per_gpu : 0;
    c.st_lat = c.streams ? m.stream_latency_s : 0.0;
    c.st_inv_l = c.streams ? 1.0 / m.stream_bytes_per_s : 0.0;   // +inf bandwidth: no byte term
    c.ar_lat[0] = 0.0;
    c.ar_coef[0] = 0.0;
    for (int n = 1; n <= kMaxTableDev; ++n) {
        const double two_a = 2.0 * (double)(n - 1);
        c.ar_lat[n] = two_a * m.link_latency_s;
        c.ar_coef[n] = two_a / (double)n;
        c.ar_lat_net[n] = two_a * c.net_lat;
        c.ar_lat_st[n] = two_a * c.st_lat;
    }
    return c;
}

static bool finite_pos(double v) { return std::isfinite(v) && v > 0.0; }
// a rate whose reciprocal is finite too: every cost multiplies by 1/rate,
// and an infinite 1/rate times a zero byte or flop count would be NaN
static bool rate_ok(double v) { return finite_pos(v) && std::isfinite(1.0 / v); }
static bool finite_nonneg(double v) { return std::isfinite(v) && v >= 0.0; }

static dsim_status check_device(const dsim_device_model *m)
{
    if (!m) return fail(DSIM_EINVAL, "device model is NULL");
    if (!rate_ok(m->flops_per_s) || !rate_ok(m->mem_bytes_per_s) || !rate_ok(m->link_bytes_per_s))
        return fail(DSIM_EINVAL, "device rates must be finite and > 0, with finite reciprocals");
    if (!finite_nonneg(m->link_latency_s) || !finite_nonneg(m->launch_s))
        return fail(DSIM_EINVAL, "latency and launch must be finite and >= 0");
    if (m->mm_enabled != 0 && m->mm_enabled != 1) return fail(DSIM_EINVAL, "mm_enabled must be 0 or 1");
    if (m->mm_enabled && (!finite_nonneg(m->mm_c0) || !finite_nonneg(m->mm_c1) || !finite_nonneg(m->mm_c2) ||
                          !finite_nonneg(m->mm_c3) || !finite_nonneg(m->mm_floor)))
        return fail(DSIM_EINVAL, "MatMul regression coefficients must be finite and >= 0");
    if (m->node_size < 0) return fail(DSIM_EINVAL, "node_size must be >= 0");
    if (m->node_size > 0 && (!rate_ok(m->net_bytes_per_s) || !finite_nonneg(m->net_latency_s)))
        return fail(DSIM_EINVAL, "network bandwidth must be finite and > 0 (finite reciprocal), latency finite and >= 0");
    if (m->streams_per_gpu < 0 || m->streams_per_gpu > (1 << 20))
        return fail(DSIM_EINVAL, "streams_per_gpu must be in 0..2^20");
    if (m->streams_per_gpu > 1 && (!(m->stream_bytes_per_s > 0.0) || !std::isfinite(1.0 / m->stream_bytes_per_s) ||
                                   !finite_nonneg(m->stream_latency_s)))
        return fail(DSIM_EINVAL, "stream bandwidth must be > 0 (inf allowed) with a finite reciprocal, latency finite "
                                 "and >= 0");
    return DSIM_OK;
}

static dsim_status check_model(const dsim_model *m)
{
    if (!m) return fail(DSIM_EINVAL, "model is NULL");
    if (m->family != DSIM_MLP && m->family != DSIM_TRANSFORMER)
        return fail(DSIM_EINVAL, "unknown model family %d", m->family);
    if (m->mode < DSIM_INFER || m->mode > DSIM_TRAIN_ADAM_MIXED)
        return fail(DSIM_EINVAL, "unknown mode %d", m->mode);
    if (m->n_layers < 1 || m->d_model < 1 || m->global_batch < 1)
        return fail(DSIM_EINVAL, "n_layers, d_model and global_batch must be >= 1");
    if (m->elem_bytes < 1 || m->elem_bytes > 8) return fail(DSIM_EINVAL, "elem_bytes must be 1..8");
    if (m->schedule != DSIM_SCHED_1F1B && m->schedule != DSIM_SCHED_GPIPE)
        return fail(DSIM_EINVAL, "unknown schedule %d", m->schedule);
    if (m->recompute != 0 && m->recompute != 1) return fail(DSIM_EINVAL, "recompute must be 0 or 1");
    if (m->zero != 0 && m->zero != 1) return fail(DSIM_EINVAL, "zero must be 0 or 1");
    if (m->overlap != 0 && m->overlap != 1) return fail(DSIM_EINVAL, "overlap must be 0 or 1");
    if (m->overlap && m->zero) return fail(DSIM_EINVAL, "overlap and zero cannot be combined");
    if (m->family == DSIM_TRANSFORMER) {
        if (m->n_heads < 1 || m->d_ff < 1 || m->seq_len < 1 || m->vocab < 1)
            return fail(DSIM_EINVAL, "transformer needs n_heads, d_ff, seq_len, vocab >= 1");
        if (m->d_model % m->n_heads != 0) return fail(DSIM_EINVAL, "d_model must be a multiple of n_heads");
    }
    const double big = 1e15;
    if ((double)m->d_model > big || (double)m->global_batch > big || (double)m->d_ff > big ||
        (double)m->seq_len > big || (double)m->vocab > big)
        return fail(DSIM_ERANGE, "model dimensions too large");
    if (m->n_layers > kMaxLayers) return fail(DSIM_ERANGE, "at most %d layers", kMaxLayers);
    // the size rule (dsim.h): every op quantity below 2^62 (q) and every
    // live-byte count below 2^62 (z), bounded in fp64 over any tensor degree
    // and microbatch split
    const double rows = (double)m->global_batch, eb = (double)m->elem_bytes, nl = (double)m->n_layers;
    const double w = (double)m->d_model, kx = std::fmin(rows, (double)kMaxK);
    double q, z;
    if (m->family == DSIM_MLP) {
        const double ww = w * w;
        q = 2.0 * rows * ww + eb * (3.0 * rows * w + ww) + 64.0 * ww;
        z = nl * (16.0 * eb * rows * w + 8.0 * eb * kx * ww) + 32.0 * nl * ww + 8.0 * eb * rows * w;
    } else {
        const double sq = (double)m->seq_len, ff = (double)m->d_ff, voc = (double)m->vocab;
        const double hd = (double)m->n_heads, tok = rows * sq;
        const double lay = 4.0 * w * w + 2.0 * w * ff;          // one layer's parameters
        const double n1 = 3.0 * w * w + w * ff + voc * w;       // largest parameter slots
        q = 2.0 * tok * w * (3.0 * w + ff + voc + 2.0 * sq) + (5.0 + 3.0 * eb) * rows * hd * sq * sq +
            (8.0 + 8.0 * eb) * tok * (w + ff + voc) + (68.0 + 8.0 * eb) * n1 + 64.0 * tok;
        z = nl * (eb * tok * (64.0 * w + 16.0 * ff + 16.0 * hd * sq) + 8.0 * eb * kx * lay) +
            eb * tok * (8.0 * voc + 16.0 * w) + 48.0 * tok + 16.0 * eb * kx * voc * w +
            32.0 * (nl * lay + 2.0 * voc * w);
    }
    const double lim = 0x1p62;
    if (!(q < lim) || !(z < lim))
        return fail(DSIM_ERANGE, "model beyond the size rule: op quantities up to %.3g, live bytes up to %.3g "
                                 "(both must stay below 2^62)", q, z);
    return DSIM_OK;
}

// Preconditions of the transform for one strategy (true = usable).
static bool strategy_ok(const dsim_model &m, int D, int H, int P, int K)
{
    if (D < 1 || H < 1 || P < 1 || K < 1) return false;
    if ((int64_t)D * H * P > kMaxDevices) return false;
    const int64_t B = m.global_batch;
    if (B % D != 0 || (int64_t)K > B / D || P > m.n_layers) return false;
    if (m.family == DSIM_MLP) {
        if (m.d_model % H != 0) return false;
        if (H > 1) {
            const int q = m.n_layers / P, r = m.n_layers % P;
            for (int s = 0; s < P; ++s)
                if (((q + (s < r ? 1 : 0)) & 1) != 0) return false;
        }
        return true;
    }
    return m.n_heads % H == 0 && m.d_model % H == 0 && m.d_ff % H == 0;
}

// arguments of the transform's simulation (both entry points)
static dsim_status check_parametric(const dsim_model *model, const dsim_strategy *cand, int64_t n_cand,
                                    const dsim_device_model *device, const dsim_results *results)
{
    dsim_status st = check_model(model);
    if (st) return st;
    st = check_device(device);
    if (st) return st;
    if (model->overlap ? device->streams_per_gpu != 2 : device->streams_per_gpu > 1)
        return fail(DSIM_EINVAL, "the transform places %s; the device model has streams_per_gpu = %d",
                    model->overlap ? "two streams on every GPU (overlap)" : "one device on every GPU",
                    device->streams_per_gpu);
    if (!results) return fail(DSIM_EINVAL, "results must not be NULL");
    if (n_cand < 0 || n_cand > ((int64_t)1 << 40)) return fail(DSIM_EINVAL, "bad n_cand");
    if (n_cand == 0) return DSIM_OK;
    if (!cand) return fail(DSIM_EINVAL, "candidate array must not be NULL");
    if (!results->makespan || !results->cand_peak || !results->status)
        return fail(DSIM_EINVAL, "makespan, cand_peak and status must not be NULL");
    if ((results->finish || results->peak) && results->row_width < 1)
        return fail(DSIM_ENOSPC, "row_width must be >= 1");
    return DSIM_OK;
}

}  // namespace dsim

using namespace dsim;

extern "C" {

const char *dsim_last_error(void) { return g_err; }

dsim_status dsim_create_grid(const dsim_model *model, const dsim_grid_spec *grid, dsim_strategy *out,
                             int64_t cap, int64_t *n_out)
{
    dsim_status st = check_model(model);
    if (st) return st;
    if (!grid || !n_out) return fail(DSIM_EINVAL, "grid spec and n_out must not be NULL");
    if (grid->max_devices < 1 || grid->max_devices > (1 << 20) || grid->k_max < 1 ||
        grid->k_max > (1 << 20) || grid->k_mode < 0 || grid->k_mode > 2)
        return fail(DSIM_EINVAL, "bad grid spec");
    if (out && cap < 0) return fail(DSIM_EINVAL, "cap must be >= 0");
    const int64_t maxd = grid->max_devices;
    int64_t n = 0;
    for (int64_t P = 1; P <= maxd; P *= 2) {
        for (int64_t K = 1; K <= grid->k_max; ++K) {
            const bool pow2 = (K & (K - 1)) == 0;
            if (grid->k_mode == 0 && !pow2) continue;
            if (grid->k_mode == 2 && (P == 1 ? K != 1 : (K < 2 || !pow2))) continue;
            for (int64_t H = 1; H * P <= maxd; H *= 2) {
                for (int64_t D = 1; D * H * P <= maxd; D *= 2) {
                    if (grid->exact_devices && D * H * P != maxd) continue;
                    if (!strategy_ok(*model, (int)D, (int)H, (int)P, (int)K)) continue;
                    if (grid->require_k_divides && (model->global_batch / D) % K != 0) continue;
                    if (out && n < cap) out[n] = dsim_strategy{(int32_t)D, (int32_t)H, (int32_t)P, (int32_t)K};
                    ++n;
                }
            }
        }
    }
    *n_out = n;
    if (out && n > cap) return fail(DSIM_ENOSPC, "grid has %lld strategies, cap %lld", (long long)n, (long long)cap);
    return DSIM_OK;
}

dsim_status dsim_simulate_tables(const dsim_tables *tables, int64_t n_cand, const dsim_device_model *device,
                                 const dsim_results *results, void *hip_stream)
{
    dsim_status st = check_device(device);
    if (st) return st;
    if (!tables || !results) return fail(DSIM_EINVAL, "tables and results must not be NULL");
    if (n_cand < 0) return fail(DSIM_EINVAL, "bad n_cand");
    if (n_cand > kMaxLaneCand) return fail(DSIM_ERANGE, "n_cand must be <= 2^32 - 256 for the table format");
    if (tables->n_dev < 1 || tables->n_dev > kMaxTableDev)
        return fail(DSIM_ERANGE, "n_dev must be 1..%d for the table format", kMaxTableDev);
    if (tables->max_ops < 0) return fail(DSIM_EINVAL, "max_ops must be >= 0");
    if (n_cand == 0) return DSIM_OK;
    if (tables->max_ops > 0 && (!tables->code || !tables->flops || !tables->bytes || !tables->alloc_bytes ||
                                !tables->free_bytes))
        return fail(DSIM_EINVAL, "table arrays must not be NULL");
    if (!results->makespan || !results->cand_peak || !results->status)
        return fail(DSIM_EINVAL, "makespan, cand_peak and status must not be NULL");
    if ((results->finish || results->peak) && results->row_width < tables->n_dev)
        return fail(DSIM_ENOSPC, "row_width %d < n_dev %d", results->row_width, tables->n_dev);
    return launch_sim_tables(*tables, n_cand, make_consts(*device), *results, (hipStream_t)hip_stream);
}

size_t dsim_parametric_workspace(int64_t n_cand)
{
    if (n_cand < 0 || n_cand > ((int64_t)1 << 40)) return 0;
    return parametric_workspace(n_cand);
}

dsim_status dsim_simulate_parametric_static(const dsim_model *model, const dsim_strategy *cand, int64_t n_cand,
                                            const dsim_device_model *device, const dsim_results *results,
                                            void *hip_stream)
{
    dsim_status st = check_parametric(model, cand, n_cand, device, results);
    if (st || n_cand == 0) return st;
    if (n_cand > static_max_cand())
        return fail(DSIM_ERANGE, "parametric (static): at most %lld candidates per call",
                    (long long)static_max_cand());
    void *ws = nullptr;
    st = static_scratch(&ws);
    if (st) return st;
    return launch_parametric(*model, cand, n_cand, make_consts(*device), *results, ws, (hipStream_t)hip_stream,
                             nullptr);
}

dsim_status dsim_simulate_parametric(const dsim_model *model, const dsim_strategy *cand, int64_t n_cand,
                                     const dsim_device_model *device, const dsim_results *results,
                                     void *workspace, size_t ws_bytes, void *side_stream, void *hip_stream)
{
    dsim_status st = check_parametric(model, cand, n_cand, device, results);
    if (st || n_cand == 0) return st;
    if (!workspace || ws_bytes < parametric_workspace(n_cand))
        return fail(DSIM_ENOSPC, "workspace needs %zu bytes", parametric_workspace(n_cand));
    return launch_parametric(*model, cand, n_cand, make_consts(*device), *results, workspace,
                             (hipStream_t)hip_stream, (hipStream_t)side_stream);
}

size_t dsim_argmin_workspace(int64_t n, int32_t k)
{
    if (n < 0 || k < 1 || k > 64) return 0;
    return argmin_workspace(n, k);
}

dsim_status dsim_argmin(const double *makespan, const uint64_t *cand_peak, const int32_t *status, int64_t n,
                        uint64_t mem_cap, int32_t k, void *workspace, size_t ws_bytes, int64_t *out_idx,
                        double *out_makespan, int32_t *out_found, void *hip_stream)
{
    if (k < 1 || k > 64) return fail(DSIM_ERANGE, "k must be 1..64");
    if (n < 0 || n > ((int64_t)1 << 40)) return fail(DSIM_EINVAL, "bad n");
    if (!out_idx || !out_makespan || !out_found) return fail(DSIM_EINVAL, "outputs must not be NULL");
    if (n > 0 && (!makespan || !cand_peak || !status)) return fail(DSIM_EINVAL, "inputs must not be NULL");
    if (!workspace || ws_bytes < argmin_workspace(n, k))
        return fail(DSIM_ENOSPC, "workspace needs %zu bytes", argmin_workspace(n, k));
    return launch_argmin(makespan, cand_peak, status, n, mem_cap, k, workspace, out_idx, out_makespan, out_found,
                         (hipStream_t)hip_stream);
}

dsim_status dsim_materialize_tables(const dsim_model *model, const dsim_strategy *cand, int64_t n_cand,
                                    int32_t max_ops, int32_t n_dev, uint32_t *code, float *flops, float *bytes,
                                    uint32_t *alloc_bytes, uint32_t *free_bytes, uint32_t *mm_k, uint32_t *n_ops,
                                    uint64_t *init_live, int32_t *status, void *hip_stream)
{
    dsim_status st = check_model(model);
    if (st) return st;
    if (n_dev < 1 || n_dev > kMaxTableDev) return fail(DSIM_ERANGE, "n_dev must be 1..%d", kMaxTableDev);
    if (max_ops < 0) return fail(DSIM_ERANGE, "max_ops must be >= 0");
    if (n_cand < 0) return fail(DSIM_EINVAL, "bad n_cand");
    if (n_cand > kMaxLaneCand) return fail(DSIM_ERANGE, "n_cand must be <= 2^32 - 256 for the table format");
    if (n_cand == 0) return DSIM_OK;
    if (!cand || !n_ops || !init_live || !status) return fail(DSIM_EINVAL, "cand, n_ops, init_live and status must not be NULL");
    if (max_ops > 0 && (!code || !flops || !bytes || !alloc_bytes || !free_bytes))
        return fail(DSIM_EINVAL, "table buffers must not be NULL");
    return launch_materialize(*model, cand, n_cand, max_ops, n_dev, code, flops, bytes, alloc_bytes, free_bytes,
                              max_ops > 0 ? mm_k : nullptr, n_ops, init_live, status, (hipStream_t)hip_stream);
}

dsim_status dsim_generate_random_tables(uint64_t seed, int64_t n_cand, int32_t n_ops, int32_t n_dev,
                                        uint32_t *code, float *flops, float *bytes, uint32_t *alloc_bytes,
                                        uint32_t *free_bytes, uint32_t *n_ops_out, void *hip_stream)
{
    if (n_dev < 2 || n_dev > kMaxTableDev) return fail(DSIM_ERANGE, "n_dev must be 2..%d", kMaxTableDev);
    if (n_ops < 0 || n_ops >= (1 << 27)) return fail(DSIM_ERANGE, "n_ops must be in [0, 2^27)");
    if (n_cand < 0 || n_cand > kMaxLaneCand) return fail(DSIM_ERANGE, "n_cand must be in [0, 2^32 - 256]");
    if (n_cand == 0) return DSIM_OK;
    if (n_ops > 0 && (!code || !flops || !bytes || !alloc_bytes || !free_bytes))
        return fail(DSIM_EINVAL, "table buffers must not be NULL");
    return launch_gen_tables(seed, n_cand, n_ops, n_dev, code, flops, bytes, alloc_bytes, free_bytes, n_ops_out,
                             (hipStream_t)hip_stream);
}

}  // extern "C"
