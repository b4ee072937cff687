// Stand-ins for the library's kernel launchers, so that the host-side
// entry points (argument validation, the size rule, grid enumeration, the
// device-model constants) can be built for the CPU alone with sanitizers.
// Test code only: every stand-in records the call and launches nothing.
#include "../../paper_2111_05426_amd/csrc/internal.h"

namespace dsim {

int g_launches = 0;

dsim_status launch_sim_tables(const dsim_tables &, int64_t, const CostConsts &, const dsim_results &, hipStream_t)
{
    ++g_launches;
    return DSIM_OK;
}
dsim_status launch_gen_tables(uint64_t, int64_t, int32_t, int32_t, uint32_t *, float *, float *, uint32_t *,
                              uint32_t *, uint32_t *, hipStream_t)
{
    ++g_launches;
    return DSIM_OK;
}
size_t argmin_workspace(int64_t n, int32_t k) { return (size_t)(n + 1) * 16 + (size_t)k * 16; }
dsim_status launch_argmin(const double *, const uint64_t *, const int32_t *, int64_t, uint64_t, int32_t, void *,
                          int64_t *, double *, int32_t *, hipStream_t)
{
    ++g_launches;
    return DSIM_OK;
}
size_t parametric_workspace(int64_t n) { return (size_t)(((n + 255) / 256) * 8 + 32 + n) * 4; }
dsim_status launch_parametric(const dsim_model &, const dsim_strategy *, int64_t, const CostConsts &,
                              const dsim_results &, void *, hipStream_t, hipStream_t)
{
    ++g_launches;
    return DSIM_OK;
}
static uint32_t g_scratch[64];
dsim_status static_scratch(void **out)
{
    *out = g_scratch;
    return DSIM_OK;
}
int64_t static_max_cand() { return (int64_t)1 << 20; }
dsim_status launch_materialize(const dsim_model &, const dsim_strategy *, int64_t, int32_t, int32_t, uint32_t *,
                               float *, float *, uint32_t *, uint32_t *, uint32_t *, uint32_t *, uint64_t *,
                               int32_t *, hipStream_t)
{
    ++g_launches;
    return DSIM_OK;
}

}  // namespace dsim
