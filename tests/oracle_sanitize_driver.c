/*
 * Test driver: runs every entry point of the CPU oracle (oracle/mx_oracle.c,
 * included as one translation unit) on small, odd-shaped inputs that
 * include bf16 subnormals, signed zeros, NaN and infinities, zero and
 * constant rows.  Built by tests/test_oracle_sanitize.py with
 * -fsanitize=address,undefined and no recovery, so any out-of-bounds
 * access, use of uninitialised heap, integer overflow or invalid shift in
 * the oracle ends the run with an error.  Every output buffer is allocated
 * to its exact size, so a write one past the end is caught.
 */
#include "../oracle/mx_oracle.c"

#include <stdio.h>

static uint32_t rng_state = 12345u;

static uint32_t next_u32(void)
{
    /* xorshift32 (Marsaglia 2003) */
    uint32_t x = rng_state;
    x ^= x << 13;
    x ^= x >> 17;
    x ^= x << 5;
    rng_state = x;
    return x;
}

/* bf16 bit patterns: mostly moderate normals, with the special values mixed in */
static void fill_bf16(uint16_t *x, int64_t n, int specials)
{
    static const uint16_t special[] = {0x0000, 0x8000, 0x0001, 0x8001, 0x007F, 0x0080,
                                       0x7F7F, 0xFF7F, 0x7F80, 0xFF80, 0x7FC0, 0x3F80};
    int64_t i;
    for (i = 0; i < n; i++) {
        const uint32_t r = next_u32();
        uint16_t v = (uint16_t)(((r >> 16) & 0x8000u) | ((118u + (r % 20u)) << 7) | (r & 0x7Fu));
        if (specials && (r >> 8) % 17u == 0)
            v = special[(r >> 4) % (sizeof special / sizeof special[0])];
        x[i] = v;
    }
}

static void *xalloc(size_t n)
{
    void *p = malloc(n ? n : 1);
    if (!p) {
        fprintf(stderr, "out of memory\n");
        exit(2);
    }
    return p;
}

static void run_norms(int64_t T, int64_t d, int specials)
{
    uint16_t *x = xalloc((size_t)(T * d) * 2), *g = xalloc((size_t)d * 2);
    float *r32 = xalloc((size_t)T * 4);
    double *r64 = xalloc((size_t)T * 8);
    int B, elem, mode, p;
    fill_bf16(x, T * d, specials);
    fill_bf16(g, d, 0);
    if (T > 2) { /* a zero row and a constant row */
        memset(x, 0, (size_t)d * 2);
        for (int64_t j = 0; j < d; j++)
            x[d + j] = 0x3FC0;
    }
    for (B = 16; B <= 64; B *= 2) {
        if (d % B)
            continue;
        for (elem = 0; elem < 2; elem++) {
            const int64_t cb = elem == MXO_ELEM_E4M3 ? T * d : T * d / 2;
            uint8_t *c = xalloc((size_t)cb), *s = xalloc((size_t)(T * d / B));
            for (mode = 0; mode < 2; mode++) {
                for (p = 1; p <= 2; p++)
                    mxo_mxnorm_mx(x, T, d, B, elem, p, 0.0f, 1e-6f, mode, c, s, r32, r64);
                mxo_mxnorm_mx(x, T, d, B, elem, 2, 0.0f, 0.0f, mode, c, s, r32, r64);
                mxo_rmsnorm_mx(x, g, T, d, B, elem, 1e-6f, mode, c, s, r32, r64);
                mxo_rmsnorm_mx(x, NULL, T, d, B, elem, 0.0f, mode, c, s, r32, r64);
                mxo_mxnorm_postround_mx(x, T, d, B, elem, 1e-6f, mode, c, s, r32, r64);
            }
            free(c);
            free(s);
        }
    }
    if (d % 32 == 0) {
        uint8_t *c = xalloc((size_t)(T * d)), *s = xalloc((size_t)(T * d / 32));
        mxo_mxnorm_mxfp8(x, T, d, 2, 0.0f, 1e-6f, MXO_SCALE_RCEIL, c, s, r32, r64);
        mxo_rmsnorm_mxfp8(x, g, T, d, 1e-6f, MXO_SCALE_FLOOR, c, s, r32, r64);
        free(c);
        free(s);
    }
    if (d % 16 == 0) {
        uint8_t *c = xalloc((size_t)(T * d / 2)), *s = xalloc((size_t)(T * d / 16));
        const float sg = (float)mxo_mxnorm_default_global_scale(d, 16, 2, 0.0f);
        mxo_mxnorm_nvfp4(x, T, d, 2, 0.0f, 1e-6f, sg, c, s, r32, r64);
        mxo_mxnorm_nvfp4(x, T, d, 1, 0.0f, 0.0f, 1e-3f, c, s, r32, r64);
        mxo_rmsnorm_nvfp4(x, g, T, d, 1e-6f, (float)mxo_rmsnorm_default_global_scale(d, 2.0f),
                          c, s, r32, r64);
        mxo_rmsnorm_nvfp4(x, NULL, T, d, 0.0f, 3e-38f, c, s, r32, r64);
        free(c);
        free(s);
    }
    free(x);
    free(g);
    free(r32);
    free(r64);
}

static void run_linear(int64_t M, int64_t N, int64_t K)
{
    uint16_t *a = xalloc((size_t)(M * K) * 2), *w = xalloc((size_t)(N * K) * 2);
    uint16_t *gam = xalloc((size_t)K * 2), *gz = xalloc((size_t)(M * K) * 2);
    float *rho = xalloc((size_t)M * 4), *af = xalloc((size_t)(M * K) * 4);
    double *gx = xalloc((size_t)(M * K) * 8), *gg = xalloc((size_t)K * 8);
    int elem;
    int64_t i;
    fill_bf16(a, M * K, 1);
    fill_bf16(w, N * K, 0);
    fill_bf16(gam, K, 0);
    fill_bf16(gz, M * K, 1);
    for (i = 0; i < M; i++)
        rho[i] = 0.5f + (float)(i % 5) * 0.25f;
    for (i = 0; i < M * K; i++)
        af[i] = mxo_bf16_to_float(a[i]);
    for (elem = 0; elem < 2; elem++) {
        const int64_t ab = elem == MXO_ELEM_E4M3 ? K : K / 2;
        uint8_t *ac = xalloc((size_t)(M * ab)), *as = xalloc((size_t)(M * K / 32));
        uint8_t *bc = xalloc((size_t)(N * ab)), *bs = xalloc((size_t)(N * K / 32));
        double *h = xalloc((size_t)(M * N) * 8);
        const int64_t tb = elem == MXO_ELEM_E4M3 ? M : M / 2;
        uint8_t *tc = xalloc((size_t)(K * tb)), *ts = xalloc((size_t)(K * M / 32));
        mxo_mxcast(af, M, K, 32, elem, MXO_SCALE_RCEIL, ac, as);
        mxo_mxcast_gain(w, gam, N, K, 32, elem, MXO_SCALE_FLOOR, bc, bs);
        mxo_mxcast_gain(w, NULL, N, K, 32, elem, MXO_SCALE_RCEIL, bc, bs);
        if (mxo_mx_matmul(ac, as, bc, bs, M, N, K, 32, elem, h) != 0) {
            fprintf(stderr, "matmul rejected its arguments\n");
            exit(3);
        }
        if (mxo_mxcast_t(a, rho, M, K, 32, elem, MXO_SCALE_RCEIL, tc, ts) != 0 ||
            mxo_mxcast_t(a, NULL, M, K, 32, elem, MXO_SCALE_FLOOR, tc, ts) != 0) {
            fprintf(stderr, "column cast rejected its arguments\n");
            exit(3);
        }
        free(ac);
        free(as);
        free(bc);
        free(bs);
        free(h);
        free(tc);
        free(ts);
    }
    mxo_ste_bwd(a, gz, gam, rho, M, K, gx, gg);
    mxo_ste_bwd(a, gz, NULL, rho, M, K, gx, gg);
    free(a);
    free(w);
    free(gam);
    free(gz);
    free(rho);
    free(af);
    free(gx);
    free(gg);
}

int main(void)
{
    static const int64_t shapes[][2] = {{1, 32}, {3, 64}, {5, 96}, {2, 768}, {4, 1024},
                                        {3, 1280}, {2, 4096}, {1, 16384}};
    size_t i;
    for (i = 0; i < sizeof shapes / sizeof shapes[0]; i++) {
        run_norms(shapes[i][0], shapes[i][1], 1);
        run_norms(shapes[i][0], shapes[i][1], 0);
    }
    run_norms(0, 64, 1); /* no rows */
    run_linear(64, 48, 128);
    run_linear(96, 16, 256);
    {
        /* the codec array forms over every bf16 pattern */
        float *v = xalloc(65536 * 4);
        uint8_t *o = xalloc(65536);
        int32_t *e = xalloc(65536 * 4);
        int j;
        for (j = 0; j < 65536; j++)
            v[j] = mxo_bf16_to_float((uint16_t)j);
        mxo_e4m3_encode_array(v, 65536, o);
        mxo_e2m1_encode_array(v, 65536, o);
        mxo_scale_exponent_array(v, 65536, MXO_SCALE_RCEIL, e);
        mxo_scale_exponent_fmt_array(v, 65536, MXO_SCALE_FLOOR, MXO_ELEM_E2M1, e);
        free(v);
        free(o);
        free(e);
    }
    puts("oracle sanitizer run: ok");
    return 0;
}
