/*
 * CPU oracle for the integer-only low-bit convolution of AQD
 * (Chen et al., "AQD: Towards Accurate Fully-Quantized Object Detection",
 * arXiv 2007.06919).
 *
 * TEST INFRASTRUCTURE. Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark load this file's library. It shares no code
 * with the GPU path. It is written to be read against the paper: plain
 * nested loops, exact integer arithmetic, no blocking or reordering.
 *
 * Definitions (integer, exact):
 *   RSM(a, c, d) = floor((a*c + 2^(d-1)) / 2^d) for d >= 1, and a*c for d = 0:
 *   the product a*c/2^d rounded to nearest, ties toward +infinity.
 *
 * Per output element (n, oh, ow, co) of a k x k convolution with stride s and
 * zero padding p:
 *   acc = sum_{r,q,ci} x[n][oh*s-p+r][ow*s-p+q][ci] * w[co][r][q][ci]
 *         (taps outside the image contribute nothing: code 0 is real zero)
 *                                                      -- Sec. 3.2.1, Eq. 4
 *   v   = acc + bias[co]      (bias = round(s) of BN)  -- Sec. 3.2.2, Eq. 6
 *   skip (optional), k = skip[n][oh>>u][ow>>u][co], u = 1 for a nearest 2x
 *   upsampled skip (Sec. 3.2.4), else 0:
 *       side 0 (skip scale >= conv scale): u_ = v + RSM(k, c, d)
 *       side 1 (otherwise):                u_ = RSM(v, c, d) + k
 *                                                      -- Sec. 3.2.3, Eq. 7-8
 *   requantisation to the next layer's b-bit codes (Eq. 2 carried out on
 *   integers with the dyadic scale M / 2^(31+sh)):
 *       out = clamp(RSM(u_, M[co], 31 + sh[co]), 0, 2^b - 1)
 *   or, in int32-output mode, out = v.
 *
 * Every intermediate (acc, v, u_) must fit a signed 32-bit integer, the
 * representation the paper assumes for the integer values (Sec. 3.2.3);
 * a violation is reported as an error, never wrapped.
 */
#include <stdint.h>
#include <stdlib.h>

typedef __int128 i128;

enum {
    ORACLE_OK = 0,
    ORACLE_ERR_ACC_RANGE = 1,
    ORACLE_ERR_V_RANGE = 2,
    ORACLE_ERR_U_RANGE = 3,
    ORACLE_ERR_ARGS = 4,
};

static const int64_t I32_LIM = (int64_t)1 << 31;

/* floor(num / 2^d), written as a division with an explicit floor step */
static i128 floor_div_pow2(i128 num, int d)
{
    i128 den = (i128)1 << d;
    i128 q = num / den; /* C division truncates toward zero */
    if (num % den != 0 && num < 0)
        q -= 1;
    return q;
}

/* nearest integer to a*c/2^d, ties toward +infinity */
static i128 rsm(int64_t a, int64_t c, int d)
{
    i128 prod = (i128)a * (i128)c;
    if (d == 0)
        return prod;
    return floor_div_pow2(prod + ((i128)1 << (d - 1)), d);
}

static int in_i32(i128 v) { return v > -(i128)I32_LIM && v < (i128)I32_LIM; }

/* Eq. 7 alignment of one element: returns u_ (see header) */
static i128 align_add(i128 v, int64_t k, int32_t c, int32_t d, int32_t side)
{
    if (side == 0)
        return v + rsm(k, c, d);
    return rsm((int64_t)v, c, d) + k;
}

static int64_t requant_clamp(i128 u, int32_t mult, int32_t sh, int64_t qmax)
{
    i128 y = rsm((int64_t)u, mult, 31 + sh);
    if (y < 0)
        return 0;
    if (y > qmax)
        return qmax;
    return (int64_t)y;
}

/*
 * x     : [n][h][w][cin] activation codes
 * wt    : [cout][kh][kw][cin] decoded signed weight values
 * bias  : [cout]
 * mult, shift : [cout] (ignored when out_int32)
 * skip  : [n][hs][ws][cout] skip values (codes or int32), or NULL
 * skip_c, skip_d, skip_side : [cout]
 * out   : [n][ho][wo][cout]
 */
int oracle_qconv(int n, int h, int w, int cin, const int32_t *x,
                 int cout, int kh, int kw, int stride, int pad, const int32_t *wt,
                 const int32_t *bias, int out_int32,
                 const int32_t *mult, const int32_t *shift, int qmax_out,
                 const int64_t *skip, int skip_up2, int hs, int ws,
                 const int32_t *skip_c, const int32_t *skip_d, const int32_t *skip_side,
                 int ho, int wo, int64_t *out)
{
    if (n < 0 || h < 1 || w < 1 || cin < 1 || cout < 1 || kh < 1 || kw < 1 || stride < 1 ||
        pad < 0 || ho != (h + 2 * pad - kh) / stride + 1 || wo != (w + 2 * pad - kw) / stride + 1)
        return ORACLE_ERR_ARGS;
    if (skip && out_int32)
        return ORACLE_ERR_ARGS;
    int err = ORACLE_OK;
#pragma omp parallel for collapse(2) schedule(dynamic, 1) reduction(max : err)
    for (int in = 0; in < n; ++in) {
        for (int oh = 0; oh < ho; ++oh) {
            for (int ow = 0; ow < wo; ++ow) {
                for (int co = 0; co < cout; ++co) {
                    int64_t acc = 0;
                    for (int r = 0; r < kh; ++r) {
                        int ih = oh * stride - pad + r;
                        if (ih < 0 || ih >= h)
                            continue;
                        for (int q = 0; q < kw; ++q) {
                            int iw = ow * stride - pad + q;
                            if (iw < 0 || iw >= w)
                                continue;
                            const int32_t *xp = x + (((int64_t)in * h + ih) * w + iw) * cin;
                            const int32_t *wp = wt + (((int64_t)co * kh + r) * kw + q) * cin;
                            /* one tap: |sum| <= cin * 255 * 128 < 2^31 for cin < 65793 */
                            int32_t part = 0;
                            for (int ci = 0; ci < cin; ++ci)
                                part += xp[ci] * wp[ci];
                            acc += part;
                        }
                    }
                    int64_t *o = out + (((int64_t)in * ho + oh) * wo + ow) * cout + co;
                    if (!in_i32(acc)) {
                        err = err > ORACLE_ERR_ACC_RANGE ? err : ORACLE_ERR_ACC_RANGE;
                        *o = 0;
                        continue;
                    }
                    i128 v = (i128)acc + bias[co];
                    if (!in_i32(v)) {
                        err = err > ORACLE_ERR_V_RANGE ? err : ORACLE_ERR_V_RANGE;
                        *o = 0;
                        continue;
                    }
                    if (out_int32) {
                        *o = (int64_t)v;
                        continue;
                    }
                    i128 u = v;
                    if (skip) {
                        int sh_ = skip_up2 ? oh / 2 : oh;
                        int sw_ = skip_up2 ? ow / 2 : ow;
                        int64_t kv = skip[(((int64_t)in * hs + sh_) * ws + sw_) * cout + co];
                        u = align_add(v, kv, skip_c[co], skip_d[co], skip_side[co]);
                    }
                    if (!in_i32(u)) {
                        err = err > ORACLE_ERR_U_RANGE ? err : ORACLE_ERR_U_RANGE;
                        *o = 0;
                        continue;
                    }
                    *o = requant_clamp(u, mult[co], shift[co], qmax_out);
                }
            }
        }
    }
    return err;
}

/*
 * Standalone integer skip connection (Eq. 7) followed by requantisation:
 *   out[n][y][x][c] = clamp(RSM(align(a[n][y][x][c], b[n][y>>u][x>>u][c]), M, 31+sh), 0, qmax)
 * with u = 1 when b is the coarser map of a nearest 2x upsample (Sec. 3.2.4).
 */
int oracle_qadd(int n, int h, int w, int c, const int64_t *a,
                int up2, int hb, int wb, const int64_t *b,
                const int32_t *skip_c, const int32_t *skip_d, const int32_t *skip_side,
                const int32_t *mult, const int32_t *shift, int qmax_out, int64_t *out)
{
    if (n < 0 || h < 1 || w < 1 || c < 1)
        return ORACLE_ERR_ARGS;
    if (up2 ? ((h - 1) / 2 >= hb || (w - 1) / 2 >= wb) : (hb != h || wb != w))
        return ORACLE_ERR_ARGS;
    int err = ORACLE_OK;
#pragma omp parallel for collapse(2) schedule(static) reduction(max : err)
    for (int in = 0; in < n; ++in) {
        for (int y = 0; y < h; ++y) {
            for (int x = 0; x < w; ++x) {
                for (int ch = 0; ch < c; ++ch) {
                    int by = up2 ? y / 2 : y, bx = up2 ? x / 2 : x;
                    int64_t av = a[(((int64_t)in * h + y) * w + x) * c + ch];
                    int64_t bv = b[(((int64_t)in * hb + by) * wb + bx) * c + ch];
                    i128 u = align_add(av, bv, skip_c[ch], skip_d[ch], skip_side[ch]);
                    int64_t *o = out + (((int64_t)in * h + y) * w + x) * c + ch;
                    if (!in_i32(u)) {
                        err = err > ORACLE_ERR_U_RANGE ? err : ORACLE_ERR_U_RANGE;
                        *o = 0;
                        continue;
                    }
                    *o = requant_clamp(u, mult[ch], shift[ch], qmax_out);
                }
            }
        }
    }
    return err;
}

/* Element-wise RSM over arrays (exposed so that tests can pin it directly). */
void oracle_rsm_array(int64_t count, const int64_t *a, const int64_t *c, const int32_t *d,
                      int64_t *out_hi, uint64_t *out_lo)
{
    for (int64_t i = 0; i < count; ++i) {
        i128 r = rsm(a[i], c[i], d[i]);
        out_hi[i] = (int64_t)(r >> 64);
        out_lo[i] = (uint64_t)r;
    }
}

int oracle_num_threads(void)
{
    int t = 1;
#pragma omp parallel
    {
#pragma omp single
        {
#ifdef _OPENMP
            extern int omp_get_num_threads(void);
            t = omp_get_num_threads();
#endif
        }
    }
    return t;
}
