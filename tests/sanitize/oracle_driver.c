/* Runs the oracle's entry points over a spread of inputs -- random and
 * invalid tables, every model family, mode and schedule variant, valid,
 * invalid and uneven strategies in full and projection mode, grids, top-k,
 * the size rule at extreme sizes -- so that a build with AddressSanitizer
 * and UndefinedBehaviorSanitizer reports any out-of-bounds access, use of
 * freed memory or undefined arithmetic on these paths.  Test code only:
 * the oracle source is compiled into this translation unit. */
#include <stdio.h>

#include "../../oracle/dsim_oracle.c"

static or_device_model dev(int net, int streams)
{
    or_device_model m;
    memset(&m, 0, sizeof m);
    m.flops_per_s = 14e12; m.mem_bytes_per_s = 900e9; m.link_bytes_per_s = 25e9;
    m.link_latency_s = 5e-6; m.launch_s = 5e-6; m.mem_cap_bytes = 1000000;
    if (net) { m.node_size = 2; m.net_bytes_per_s = 4.7e9; m.net_latency_s = 2e-5; }
    if (streams) { m.streams_per_gpu = 2; m.stream_bytes_per_s = 5e11; m.stream_latency_s = 1e-6; }
    return m;
}

static or_model model(int fam, int mode, int L, int sched, int rc, int zero, int ov)
{
    or_model M;
    memset(&M, 0, sizeof M);
    M.family = fam; M.mode = mode; M.n_layers = L; M.n_heads = 4; M.d_model = 32; M.d_ff = 64;
    M.seq_len = 8; M.vocab = 101; M.global_batch = 24; M.elem_bytes = 2;
    M.schedule = sched; M.recompute = rc; M.zero = zero; M.overlap = ov;
    return M;
}

int main(void)
{
    int i, fails = 0;
    /* random tables and their simulation, every device count */
    for (i = 2; i <= 8; i++) {
        const int n = 300;
        uint32_t code[300], al[300], fr[300];
        float fl[300], by[300];
        double mk, fin[8];
        uint64_t pk[8], cp, init[8] = {0};
        int32_t st;
        or_device_model m = dev(i > 4, 0);
        if (or_gen_table(7, i, n, i, code, fl, by, al, fr, 1)) fails++;
        or_sim_table(n, i, code, fl, by, al, fr, NULL, 1, init, &m, &mk, fin, pk, &cp, &st);
        /* the same table with garbage records and frees too large */
        {
            int j;
            for (j = 0; j < n; j += 7) code[j] = (uint32_t)or_splitmix64(9, (uint64_t)j);
            for (j = 3; j < n; j += 11) fr[j] = 0xffffffffu;
            for (j = 5; j < n; j += 13) by[j] = -1.0f;
            or_sim_table(n, i, code, fl, by, al, fr, NULL, 1, init, &m, &mk, fin, pk, &cp, &st);
        }
    }
    /* every family, mode and variant over valid, invalid and uneven strategies */
    {
        static const int S[][4] = {{1, 1, 1, 1}, {2, 2, 2, 3}, {3, 1, 3, 5}, {2, 4, 1, 2}, {4, 2, 2, 1},
                                   {1, 2, 4, 7}, {5, 1, 1, 1}, {1, 3, 1, 1}, {0, 1, 1, 1}, {2, 1, 9, 1}};
        int fam, mode, v, s, sl;
        for (fam = 0; fam <= 1; fam++)
            for (mode = 0; mode <= 3; mode++)
                for (v = 0; v < 6; v++) {
                    or_model M = model(fam, mode, fam ? 4 : 8, v == 1, v == 2 || v == 5, v == 3, v == 4);
                    or_device_model m = dev(v == 5, v == 4);
                    for (s = 0; s < (int)(sizeof S / sizeof S[0]); s++)
                        for (sl = 0; sl <= 1; sl++) {
                            double sf[16], dfin[256];
                            uint64_t sp[16], dpk[256], dres[256], cp, no;
                            double by_type[3 * T_NTYPES], mk;
                            int32_t st;
                            int rc = or_sim_strategy(&M, S[s][0], S[s][1], S[s][2], S[s][3], &m, sl, NULL, sf, sp,
                                                     dfin, dpk, dres, by_type, &mk, &cp, &no, &st);
                            if (rc < -1) fails++;
                        }
                }
    }
    /* grids and selection */
    {
        or_model M = model(1, 0, 12, 0, 0, 0, 0);
        int32_t out[4 * 4096];
        int64_t n;
        double mk[1000];
        uint64_t pk[1000];
        int32_t st[1000];
        int64_t idx[64];
        double mo[64];
        int32_t found;
        M.global_batch = 512;
        if (or_create_grid(&M, 64, 0, 0, 128, 0, out, 4096, &n)) fails++;
        for (i = 0; i < 1000; i++) { mk[i] = (double)(or_splitmix64(3, (uint64_t)i) % 50); pk[i] = (uint64_t)i; st[i] = i % 7 == 0; }
        if (or_topk(mk, pk, st, 1000, 500, 64, idx, mo, &found)) fails++;
    }
    /* the size rule at extreme sizes (no arithmetic may overflow deciding it) */
    {
        or_model M = model(1, 3, 65536, 0, 0, 0, 0);
        M.d_model = M.d_ff = M.seq_len = M.vocab = M.global_batch = (int64_t)1 << 50;
        or_model_size_ok(&M);
        M.family = 0;
        or_model_size_ok(&M);
    }
    printf("oracle driver done, %d failures\n", fails);
    return fails != 0;
}
