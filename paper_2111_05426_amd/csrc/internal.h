// internal.h -- declarations shared by the HIP translation units of libdsim.
//
// Not part of the ABI.  The public contract is include/dsim.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/dsim.h"

namespace dsim {

// Largest device group of the explicit-table format.
constexpr int kMaxTableDev = 8;
// Microbatches per strategy; layers per model and devices per strategy (the
// size rule): with at most kMaxLayers layers, kMaxK microbatches and
// kMaxDevices devices every op count of a program stays below 2^62.
constexpr int kMaxK = 16383;
constexpr int kMaxLayers = 65536;
constexpr int64_t kMaxDevices = (int64_t)1 << 24;
// one GPU lane per candidate in a single dispatch, whose work-item count is
// a 32-bit field
constexpr int64_t kMaxLaneCand = ((int64_t)1 << 32) - 256;

// Device-model constants as the kernels consume them.  Every reciprocal is
// rounded once on the host.  For the table format (groups of at most 8) the
// ring all-reduce terms are tabulated on the host as well:
//   ar_lat[n]  = (2(n-1)) * lat
//   ar_coef[n] = (2(n-1)) / n
// so cost(n, bytes) = ar_lat[n] + ar_coef[n] * (bytes * inv_l).
struct CostConsts {
    double inv_f;      // 1 / flops_per_s
    double inv_b;      // 1 / mem_bytes_per_s
    double inv_l;      // 1 / link_bytes_per_s
    double lat;        // link latency
    double launch;     // per compute op
    uint64_t cap;      // memory cap, 0 = none
    int32_t mm;        // matrix multiplications take the regression below
    double mm_c0, mm_c1, mm_c2;
    double mm_c3, mm_floor;   // reduction-length term, floor
    int32_t node;      // devices per node, 0 = one uniform interconnect
    double net_lat;    // network latency (ops spanning nodes)
    double net_inv_l;  // 1 / network bytes per second
    int32_t streams;   // devices (streams) per GPU, 0 = one device per GPU
    double st_lat;     // latency between the streams of one GPU
    double st_inv_l;   // 1 / their bytes per second (0: no byte term)
    double ar_lat[kMaxTableDev + 1];
    double ar_coef[kMaxTableDev + 1];
    double ar_lat_net[kMaxTableDev + 1];   // (2(n-1)) * net_lat
    double ar_lat_st[kMaxTableDev + 1];    // (2(n-1)) * st_lat
};

CostConsts make_consts(const dsim_device_model &m);

// Error reporting (thread-local message).
dsim_status fail(dsim_status st, const char *fmt, ...);
dsim_status hip_fail(hipError_t e, const char *what);

// Kernel launchers (each returns DSIM_OK or DSIM_EHIP).
dsim_status launch_sim_tables(const dsim_tables &t, int64_t n_cand, const CostConsts &c,
                              const dsim_results &r, hipStream_t s);
dsim_status launch_gen_tables(uint64_t seed, int64_t n_cand, int32_t n_ops, int32_t n_dev,
                              uint32_t *code, float *flops, float *bytes, uint32_t *alloc,
                              uint32_t *freeb, uint32_t *n_ops_out, hipStream_t s);
size_t argmin_workspace(int64_t n, int32_t k);
dsim_status launch_argmin(const double *mk, const uint64_t *pk, const int32_t *st, int64_t n,
                          uint64_t cap, int32_t k, void *ws, int64_t *out_idx, double *out_mk,
                          int32_t *out_found, hipStream_t s);
size_t parametric_workspace(int64_t n_cand);
// the fixed scratch of dsim_simulate_parametric_static on the current GPU
// (its address taken once per GPU) and the candidates it holds
constexpr int kMaxGpus = 64;
dsim_status static_scratch(void **out);
int64_t static_max_cand();
dsim_status launch_parametric(const dsim_model &m, const dsim_strategy *cand, int64_t n_cand,
                              const CostConsts &c, const dsim_results &r, void *ws, hipStream_t s,
                              hipStream_t side);
dsim_status launch_materialize(const dsim_model &m, const dsim_strategy *cand, int64_t n_cand, int32_t max_ops,
                               int32_t n_dev, uint32_t *code, float *flops, float *bytes, uint32_t *alloc,
                               uint32_t *freeb, uint32_t *mm_k, uint32_t *n_ops, uint64_t *init_live,
                               int32_t *status, hipStream_t s);

}  // namespace dsim
