// Calls every host entry point of include/dsim.h with a spread of bad and
// good arguments -- NULL pointers, negative and huge sizes, non-finite and
// tiny rates, models at and beyond the size rule, every grid rule -- built
// with AddressSanitizer and UndefinedBehaviorSanitizer against launch
// stand-ins, so any out-of-bounds access or undefined arithmetic in the
// validation is reported.  Test code only.
#include <cmath>
#include <cstdio>
#include <cstring>
#include <limits>
#include <vector>

#include "dsim.h"

namespace dsim { extern int g_launches; }

static dsim_device_model dev()
{
    dsim_device_model m;
    std::memset(&m, 0, sizeof m);
    m.flops_per_s = 14e12; m.mem_bytes_per_s = 900e9; m.link_bytes_per_s = 25e9;
    m.link_latency_s = 5e-6; m.launch_s = 5e-6;
    return m;
}

static dsim_model model(int fam)
{
    dsim_model m;
    std::memset(&m, 0, sizeof m);
    m.family = fam; m.mode = DSIM_TRAIN_ADAM; m.n_layers = 12; m.n_heads = 12; m.d_model = 768; m.d_ff = 3072;
    m.seq_len = 1024; m.vocab = 50257; m.global_batch = 512; m.elem_bytes = 2;
    return m;
}

int main()
{
    const double inf = std::numeric_limits<double>::infinity(), nan = std::numeric_limits<double>::quiet_NaN();
    const double rates[] = {14e12, 0.0, -1.0, 1e-310, 5e-309, 1e-290, inf, nan, 1e308};
    int calls = 0;
    std::vector<char> buf(1 << 16);
    void *p = buf.data();
    dsim_results res;
    std::memset(&res, 0, sizeof res);
    res.makespan = (double *)p; res.cand_peak = (uint64_t *)p; res.status = (int32_t *)p; res.row_width = 8;
    // device models
    for (double f : rates)
        for (double b : rates) {
            dsim_device_model m = dev();
            m.flops_per_s = f; m.link_bytes_per_s = b; m.link_latency_s = b == inf ? nan : 1e-6;
            m.mm_enabled = f == 0.0 ? 2 : 1; m.mm_c0 = f; m.mm_c1 = b; m.mm_c2 = 1e-12;
            m.mm_c3 = b; m.mm_floor = f;
            m.node_size = b < 0 ? -1 : 4; m.net_bytes_per_s = f; m.net_latency_s = 1e-5;
            m.streams_per_gpu = f > 1e300 ? (1 << 21) : 2; m.stream_bytes_per_s = b; m.stream_latency_s = 0.0;
            dsim_tables t;
            std::memset(&t, 0, sizeof t);
            t.code = (const uint32_t *)p; t.flops = t.bytes = (const float *)p;
            t.alloc_bytes = t.free_bytes = (const uint32_t *)p; t.max_ops = 4; t.n_dev = 8;
            for (int64_t n : {(int64_t)-1, (int64_t)0, (int64_t)1, ((int64_t)1 << 32) - 256, ((int64_t)1 << 32)}) {
                dsim_simulate_tables(&t, n, &m, &res, nullptr);
                ++calls;
            }
        }
    // models: every field at its edges, the size rule on both sides
    const int64_t dims[] = {-1, 0, 1, 7, 768, (int64_t)1 << 20, (int64_t)1 << 40, (int64_t)1e15, (int64_t)1e15 + 1,
                            INT64_MAX};
    dsim_grid_spec g = {64, 0, 1, 128, 0};
    std::vector<dsim_strategy> out(1 << 16);
    for (int fam : {DSIM_MLP, DSIM_TRANSFORMER, 5})
        for (int64_t d : dims)
            for (int64_t B : dims)
                for (int L : {-1, 0, 1, 96, 65536, 65537, INT32_MAX}) {
                    dsim_model m = model(fam);
                    m.d_model = d; m.d_ff = d; m.global_batch = B; m.n_layers = L;
                    m.seq_len = d > 4096 ? 2048 : d; m.vocab = B;
                    int64_t n = 0;
                    dsim_create_grid(&m, &g, out.data(), (int64_t)out.size(), &n);
                    dsim_model m2 = m;
                    dsim_device_model dv = dev();
                    dsim_simulate_parametric(&m2, (const dsim_strategy *)p, 10, &dv, &res, p, buf.size(), nullptr,
                                             nullptr);
                    dsim_simulate_parametric_static(&m2, (const dsim_strategy *)p, 10, &dv, &res, nullptr);
                    dsim_materialize_tables(&m2, (const dsim_strategy *)p, 10, 100, 8, (uint32_t *)p, (float *)p,
                                            (float *)p, (uint32_t *)p, (uint32_t *)p, (uint32_t *)p, (uint32_t *)p,
                                            (uint64_t *)p, (int32_t *)p, nullptr);
                    calls += 4;
                }
    // grid rules
    for (int md : {-1, 1, 16, 1024, 1 << 20, (1 << 20) + 1, INT32_MAX})
        for (int km : {-1, 0, 1, 2, 3})
            for (int kx : {-5, 1, 128, 1 << 20, INT32_MAX}) {
                dsim_grid_spec gs = {md, md & 1, km, kx, kx & 1};
                dsim_model m = model(DSIM_TRANSFORMER);
                int64_t n = 0;
                dsim_create_grid(&m, &gs, nullptr, 0, &n);
                dsim_create_grid(&m, &gs, out.data(), 3, &n);
                calls += 2;
            }
    // selection and the generator
    for (int64_t n : {(int64_t)-1, (int64_t)0, (int64_t)5, (int64_t)1 << 40, ((int64_t)1 << 40) + 1})
        for (int k : {-1, 0, 1, 64, 65}) {
            int64_t idx[64];
            double mk[64];
            int32_t found;
            dsim_argmin((double *)p, (uint64_t *)p, (int32_t *)p, n, 0, k, p, dsim_argmin_workspace(n, k), idx, mk,
                        &found, nullptr);
            dsim_generate_random_tables(1, n, k * 1000, k, (uint32_t *)p, (float *)p, (float *)p, (uint32_t *)p,
                                        (uint32_t *)p, nullptr, nullptr);
            dsim_parametric_workspace(n);
            calls += 3;
        }
    std::printf("api driver: %d calls, %d reached a launch; last error: %s\n", calls, dsim::g_launches,
                dsim_last_error());
    return 0;
}
