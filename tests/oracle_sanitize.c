/* Test infrastructure: drives every entry point of the CPU oracle
 * (oracle/niti_oracle.c) over small and edge-case shapes, to be built with
 * gcc's AddressSanitizer and UndefinedBehaviorSanitizer, so that any
 * out-of-bounds access, overflow of a signed type or other undefined
 * behaviour in the oracle aborts the run.  Inputs come from a tiny local
 * linear congruential generator (test data only, no method arithmetic).
 * Exit status 0 and no sanitizer report = clean. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

typedef struct { uint64_t max_abs; int32_t b, bp, flags, s_out; } orc_stats;
typedef struct { int64_t n, c, h, w, k, r, s, sh, sw, ph, pw; } orc_conv;

int orc_bitlen(uint64_t m);
int64_t orc_psr(int64_t v, int bp);
int64_t orc_rtn(int64_t v, int bp);
int64_t orc_sr(int64_t v, int bp, uint64_t r);
uint64_t orc_sr_draw(uint64_t seed, uint32_t call, uint64_t index);
int orc_shift_round_i64(const int64_t *v, int64_t n, int target, int mode, int8_t *out, orc_stats *st,
                        uint64_t seed, uint32_t call, const int64_t *idx);
int orc_shift_round_i32(const int32_t *v, int64_t n, int target, int mode, int8_t *out, orc_stats *st,
                        uint64_t seed, uint32_t call, const int64_t *idx);
void orc_round_fixed_i32(const int32_t *v, int64_t n, int bp, int mode, int8_t *out, uint64_t seed,
                         uint32_t call);
int orc_out_exponent(int s_a, int s_w, int bp, int32_t *flags);
void orc_gemm_nt_raw(const int8_t *A, const int8_t *B, int64_t M, int64_t N, int64_t K, int64_t *S);
void orc_gemm_nt_pick(const int8_t *A, const int8_t *B, int64_t K, const int64_t *rows, const int64_t *cols,
                      int64_t cnt, int64_t *S);
void orc_conv_fwd_raw(const orc_conv *d, const int8_t *x, const int8_t *w, int64_t *y);
void orc_conv_bwd_data_raw(const orc_conv *d, const int8_t *dy, const int8_t *w, int64_t *dx);
void orc_conv_bwd_weight_raw(const orc_conv *d, const int8_t *x, const int8_t *dy, int64_t *g);
int64_t orc_conv_fwd_one(const orc_conv *d, const int8_t *x, const int8_t *w, int64_t n, int64_t k, int64_t p,
                         int64_t q);
void orc_finish_i64(const int64_t *S, int64_t n, int relu, int target, int mode, int8_t *out, int32_t *acc32,
                    orc_stats *st, int64_t red_len, uint64_t seed, uint32_t call, const int64_t *idx);
void orc_sgd_update(int8_t *w, const int32_t *g32, int64_t n, int mu, int mode, orc_stats *st, uint64_t seed,
                    uint32_t call);
void orc_int_ce_loss_grad(const int8_t *logits, int s_a, const int32_t *labels, int64_t B, int64_t N, int mode,
                          int8_t *err, int64_t *e_hi, uint64_t *e_lo, orc_stats *st, uint64_t seed,
                          uint32_t call);
void orc_relu_mask(int8_t *e, const int8_t *a, int64_t n);
void orc_maxpool2_fwd(const int8_t *x, int64_t n, int64_t c, int64_t h, int64_t w, int8_t *y, uint8_t *idx);
void orc_maxpool2_bwd(const int8_t *dy, const uint8_t *idx, int64_t n, int64_t c, int64_t h, int64_t w,
                      int8_t *dx);
void orc_quantize_u8(const uint8_t *px, int64_t n, int8_t *q);
void orc_dropout_fwd(const int8_t *x, const int64_t *idx, int64_t n, uint64_t seed, uint32_t call, int drop256,
                     int8_t *y, uint8_t *keep);
void orc_dropout_bwd(const int8_t *dy, const uint8_t *keep, int64_t n, int8_t *dx);

static uint64_t lcg = 88172645463325252ull;
static uint32_t next_u32(void) { lcg = lcg * 6364136223846793005ull + 1442695040888963407ull; return (uint32_t)(lcg >> 33); }
static void fill_i8(int8_t *p, int64_t n, int lo, int hi) {
    for (int64_t i = 0; i < n; i++) p[i] = (int8_t)(lo + (int)(next_u32() % (uint32_t)(hi - lo + 1)));
}
static void *xalloc(int64_t n) { void *p = malloc((size_t)(n > 0 ? n : 1)); if (!p) exit(3); return p; }

static int64_t od(int64_t in, int64_t pad, int64_t k, int64_t st) { return (in + 2 * pad - k) / st + 1; }

static void conv_case(int64_t n, int64_t c, int64_t h, int64_t w, int64_t k, int64_t r, int64_t s, int64_t st,
                      int64_t pd) {
    orc_conv d = {n, c, h, w, k, r, s, st, st, pd, pd};
    const int64_t P = od(h, pd, r, st), Q = od(w, pd, s, st);
    int8_t *x = xalloc(n * c * h * w), *wt = xalloc(k * c * r * s), *dy = xalloc(n * k * P * Q);
    int64_t *y = xalloc(8 * n * k * P * Q), *dx = xalloc(8 * n * c * h * w), *g = xalloc(8 * k * c * r * s);
    fill_i8(x, n * c * h * w, -127, 127);
    fill_i8(wt, k * c * r * s, -127, 127);
    fill_i8(dy, n * k * P * Q, -127, 127);
    orc_conv_fwd_raw(&d, x, wt, y);
    orc_conv_bwd_data_raw(&d, dy, wt, dx);
    orc_conv_bwd_weight_raw(&d, x, dy, g);
    (void)orc_conv_fwd_one(&d, x, wt, n - 1, k - 1, P - 1, Q - 1);
    /* finishing passes over the three sums, every rounding mode */
    for (int mode = 0; mode < 3; mode++) {
        int8_t *o = xalloc(n * k * P * Q);
        int32_t *a32 = xalloc(4 * n * k * P * Q);
        orc_stats st = {0, 0, 0, 0, 0};
        orc_finish_i64(y, n * k * P * Q, mode != 1, 7, mode, o, a32, &st, c * r * s, 5, 3, NULL);
        int8_t *o2 = xalloc(n * c * h * w);
        orc_finish_i64(dx, n * c * h * w, 0, 7, mode, o2, NULL, &st, k * r * s, 5, 3, NULL);
        int32_t *g32 = xalloc(4 * k * c * r * s);
        int8_t *o3 = xalloc(k * c * r * s);
        orc_finish_i64(g, k * c * r * s, 0, 5, mode, o3, g32, &st, n * P * Q, 5, 3, NULL);
        int8_t *wc = xalloc(k * c * r * s);
        for (int64_t i = 0; i < k * c * r * s; i++) wc[i] = wt[i];
        for (int mu = 1; mu <= 8; mu += 3) orc_sgd_update(wc, g32, k * c * r * s, mu, mode, &st, 9, 1);
        free(o); free(a32); free(o2); free(g32); free(o3); free(wc);
    }
    free(x); free(wt); free(dy); free(y); free(dx); free(g);
}

int main(void) {
    /* scalar rounding at every binary point and at the int64 / int32 edges */
    const int64_t vals[] = {0, 1, -1, 127, -127, 128, -128, 255, 1000003, -1000003, 2147483647LL,
                            -2147483647LL - 1, (int64_t)1 << 40, -((int64_t)1 << 40) + 7};
    for (int bp = 0; bp <= 62; bp++)
        for (unsigned i = 0; i < sizeof vals / sizeof vals[0]; i++) {
            (void)orc_psr(vals[i], bp);
            (void)orc_rtn(vals[i], bp);
            (void)orc_sr(vals[i], bp, orc_sr_draw(7, (uint32_t)bp, i));
        }
    for (int s = 0; s < 64; s++) (void)orc_bitlen((uint64_t)1 << s);
    (void)orc_bitlen(0);
    (void)orc_bitlen(~0ull);
    /* tensor rounding, every mode, with and without offsets; n = 0 and 1 */
    {
        const int64_t n = 1000;
        int64_t *v = xalloc(8 * n), *idx = xalloc(8 * n);
        int32_t *v32 = xalloc(4 * n);
        int8_t *out = xalloc(n);
        for (int64_t i = 0; i < n; i++) {
            v[i] = (int64_t)(next_u32() % 2000003u) - 1000001;
            v32[i] = (int32_t)v[i];
            idx[i] = n - 1 - i;
        }
        v32[0] = INT32_MIN;
        for (int mode = 0; mode < 3; mode++)
            for (int64_t m = 0; m <= n; m += (m < 2 ? 1 : 499)) {
                orc_stats st = {0, 0, 0, 0, 0};
                (void)orc_shift_round_i64(v, m, 7, mode, out, &st, 1, 2, (mode == 2 && m) ? idx : NULL);
                (void)orc_shift_round_i32(v32, m, 5, mode, out, &st, 1, 2, NULL);
                for (int bp = 0; bp <= 31; bp += 5) orc_round_fixed_i32(v32, m, bp, mode, out, 3, 4);
            }
        free(v); free(idx); free(v32); free(out);
    }
    for (int sa = -128; sa <= 127; sa += 17) {
        int32_t fl = 0;
        (void)orc_out_exponent(sa, -sa, 30, &fl);
        (void)orc_out_exponent(127, 127, 31, &fl);
        (void)orc_out_exponent(-128, -128, 0, &fl);
    }
    /* products */
    {
        const int64_t M = 37, N = 19, K = 70;
        int8_t *A = xalloc(M * K), *B = xalloc(N * K);
        int64_t *S = xalloc(8 * M * N), rows[3] = {0, 5, M - 1}, cols[3] = {N - 1, 0, 3}, pick[3];
        fill_i8(A, M * K, -128, 127);
        fill_i8(B, N * K, -128, 127);
        orc_gemm_nt_raw(A, B, M, N, K, S);
        orc_gemm_nt_raw(A, B, M, N, 0, S);
        orc_gemm_nt_pick(A, B, K, rows, cols, 3, pick);
        free(A); free(B); free(S);
    }
    conv_case(2, 4, 7, 6, 8, 3, 3, 1, 1);
    conv_case(1, 5, 9, 9, 3, 3, 3, 2, 1);
    conv_case(2, 3, 11, 13, 4, 7, 7, 2, 3);
    conv_case(1, 2, 5, 5, 2, 1, 1, 2, 0);
    conv_case(1, 4, 3, 3, 2, 1, 1, 2, 1);
    conv_case(1, 2, 17, 15, 3, 11, 11, 4, 2);
    conv_case(2, 6, 6, 6, 5, 5, 5, 1, 2);
    conv_case(1, 1, 1, 1, 1, 1, 1, 1, 0);
    /* the loss at every exponent regime, both branches, one and many classes */
    {
        const int64_t Bs = 3, Ns = 1025;
        int8_t *lg = xalloc(Bs * Ns), *err = xalloc(Bs * Ns);
        int32_t lab[3] = {0, 7, (int32_t)Ns - 1};
        int64_t *eh = xalloc(8 * Bs * Ns);
        uint64_t *el = xalloc(8 * Bs * Ns);
        fill_i8(lg, Bs * Ns, -128, 127);
        for (int sa = -128; sa <= 127; sa += 3)
            for (int mode = 0; mode < 3; mode++) {
                orc_stats st = {0, 0, 0, 0, 0};
                orc_int_ce_loss_grad(lg, sa, lab, Bs, Ns, mode, err, eh, el, &st, 11, 3);
                orc_int_ce_loss_grad(lg, sa, lab, 1, 1, mode, err, eh, el, &st, 11, 3);
            }
        for (int64_t i = 0; i < Bs * Ns; i++) lg[i] = (i & 1) ? 127 : -128;
        for (int sa = -60; sa <= 20; sa += 7) {
            orc_stats st = {0, 0, 0, 0, 0};
            orc_int_ce_loss_grad(lg, sa, lab, Bs, Ns, 0, err, eh, el, &st, 0, 0);
        }
        free(lg); free(err); free(eh); free(el);
    }
    /* glue */
    {
        const int64_t n = 2, c = 3, h = 6, w = 8, e = n * c * h * w;
        int8_t *x = xalloc(e), *y = xalloc(e / 4), *dx = xalloc(e), *q = xalloc(e), *yd = xalloc(e), *dd = xalloc(e);
        uint8_t *idx = xalloc(e / 4), *px = xalloc(e), *keep = xalloc(e);
        int64_t *off = xalloc(8 * e);
        fill_i8(x, e, -128, 127);
        for (int64_t i = 0; i < e; i++) { px[i] = (uint8_t)(next_u32() & 255); off[i] = e - 1 - i; }
        orc_maxpool2_fwd(x, n, c, h, w, y, idx);
        orc_maxpool2_bwd(y, idx, n, c, h, w, dx);
        orc_relu_mask(dx, x, e);
        orc_quantize_u8(px, e, q);
        for (int drop = 0; drop <= 256; drop += 64) {
            orc_dropout_fwd(x, off, e, 5, 2, drop, yd, keep);
            orc_dropout_fwd(x, NULL, e, 5, 2, drop, yd, keep);
            orc_dropout_bwd(yd, keep, e, dd);
        }
        free(x); free(y); free(dx); free(q); free(yd); free(dd); free(idx); free(px); free(keep); free(off);
    }
    printf("oracle sanitize run: clean\n");
    return 0;
}
