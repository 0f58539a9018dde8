/*
 * aqd.h - C ABI of the MI355X (gfx950) integer low-bit convolution library.
 *
 * The library runs the integer-only inference path of AQD (Chen et al.,
 * "AQD: Towards Accurate Fully-Quantized Object Detection", CVPR 2021,
 * arXiv 2007.06919): convolutions on b-bit activation codes and b-bit weight
 * codes with int32 accumulation (Sec. 3.2.1, Eq. 4), the folded batch norm as
 * an integer bias (Sec. 3.2.2, Eq. 5-6), the integer skip connection with a
 * power-of-two-denominator scale ratio (Sec. 3.2.3, Eq. 7-8), and the
 * requantisation back to b-bit codes (Eq. 2 carried out on integers).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Tensors are NHWC. A code tensor of bitwidth b in {2, 4, 8} stores each
 * pixel's C codes packed along the channel axis in C*b/8 bytes: channel c
 * occupies bits (c*b) mod 8 .. (c*b) mod 8 + b - 1 of byte (c*b) div 8
 * (little-endian within a byte). Activation codes are unsigned, in
 * [0, 2^b - 1] (Eq. 2: the zero point is 0, so code 0 is the real 0 and zero
 * padding is code 0). Bitwidth 3 (the paper's 3-bit networks, Tables 2 and 4)
 * is stored like bitwidth 4, one code per 4-bit container (C/2 bytes per
 * pixel, codes in [0, 7]); every width field below accepts 3 with that
 * layout, and an output of width 3 is clamped to [0, 7]. Weight fields of
 * width 3 sit in 4-bit containers too. An int32 tensor ("bits" = 32) stores
 * one int32 per element.
 *
 * Integer rounding: RSM(a, c, d) = floor((a*c + 2^(d-1)) / 2^d) for d >= 1
 * and a*c for d = 0, i.e. a*c/2^d rounded to nearest with ties toward
 * +infinity, computed exactly in 64-bit.
 *
 * Per output element of a convolution (n, oh, ow, co):
 *   acc = sum over taps (r, q) inside the image and input channels ci of
 *         x[n][oh*s - p + r][ow*s - p + q][ci] * w[co][r][q][ci]     (Eq. 4)
 *   v   = acc + bias[co]                                             (Eq. 6)
 *   with a skip value k = skip[n][oh >> u][ow >> u][co] (u = 1 for a nearest
 *   2x upsampled skip, Sec. 3.2.4):
 *         side 0: u_ = v + RSM(k, c[co], d[co])      (skip has the larger scale)
 *         side 1: u_ = RSM(v, c[co], d[co]) + k                      (Eq. 7-8)
 *   codes out: y = clamp(RSM(u_, mult[co], 31 + shift[co]), 0, 2^b_out - 1)
 *   int32 out: y = v
 * acc, v and u_ must fit in a signed 32-bit integer (the paper's integer
 * width); inputs that break this give unspecified outputs (never a fault).
 *
 * Ownership: a qconv handle owns device copies of its weights and epilogue
 * tables; qconv_destroy frees them. The caller owns every activation, skip
 * and output buffer and the qadd parameter arrays. Run calls never allocate.
 *
 * Streams: run calls enqueue on the caller's HIP stream (aqd_stream_t is a
 * hipStream_t; NULL is the null stream) and return after the enqueue. Device
 * faults surface at the caller's next synchronisation.
 *
 * Errors: every entry point validates its arguments before touching the
 * device. A bad argument returns AQD_ERR_INVALID with no launch; a valid but
 * unimplemented combination returns AQD_ERR_UNSUPPORTED; aqd_last_error()
 * returns a message for the calling thread's last failure.
 *
 * Device pointers must be 16-byte aligned. An output buffer must not overlap
 * any input buffer of the same call.
 *
 * Thread safety: handles are immutable after creation; concurrent run calls
 * on different streams are safe. aqd_last_error is per thread.
 */
#ifndef AQD_H
#define AQD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    AQD_OK = 0,
    AQD_ERR_INVALID = 1,
    AQD_ERR_UNSUPPORTED = 2,
    AQD_ERR_NOMEM = 3,
    AQD_ERR_DEVICE = 4
} aqd_status_t;

typedef void *aqd_stream_t; /* a hipStream_t */

/* Weight grids.
 * AQD_WENC_TWOS:      a b-bit field f is the two's-complement value
 *                     (f >= 2^(b-1) ? f - 2^b : f).
 * AQD_WENC_PAPER_ODD: a b-bit field eta_w is the value 2*eta_w - (2^b - 1),
 *                     the factor multiplying eta_x in Eq. 4 (Sec. 3.1.2, Eq. 3). */
enum { AQD_WENC_TWOS = 0, AQD_WENC_PAPER_ODD = 1 };

/* Output modes: requantised b-bit codes, or v = acc + bias as int32 (the
 * prediction layers, and a normalised branch that feeds a skip add). */
enum { AQD_OUT_CODES = 0, AQD_OUT_INT32 = 1 };

/* Description of one convolution layer (shared weights, one epilogue table
 * per level: multi-level BN, Sec. 3.2.2, Fig. 3). */
typedef struct {
    int cin, cout;     /* >= 1; cin*bits_in and cin*bits_w multiples of 8 (stored widths) */
    int kh, kw;        /* 1..7 */
    int stride;        /* 1..4 */
    int pad;           /* 0..kh-1 (same for both axes) */
    int bits_in;       /* activation code width: 2, 3, 4 or 8 */
    int bits_w;        /* weight field width: 2, 3, 4 or 8 */
    int wenc;          /* AQD_WENC_* */
    int out_mode;      /* AQD_OUT_* */
    int bits_out;      /* 2, 3, 4 or 8 for AQD_OUT_CODES (cout*bits_out multiple of 8) */
    int skip_bits;     /* 0: no skip; 2/3/4/8: code skip; 32: int32 skip (codes out only) */
    int skip_up2;      /* 1: skip is the coarser map of a nearest 2x upsample */
    int num_levels;    /* number of epilogue tables, 1..64 */
    /* Step sizes alpha of the uniform quantizers (Sec. 3.1.1, Eq. 1): real
     * input = step_in * code, real weight = step_w * decoded weight value
     * (for the odd grid of Eq. 3 that is nu_w / (2^b - 1)), real output =
     * step_out * code. Metadata for the host-side derivation of the integer
     * parameters (qconv_scales); stored on the handle, never used on the
     * device. 0 means "not given"; otherwise finite and > 0. */
    double step_in, step_w, step_out;
} qconv_desc_t;

/* One epilogue table; host arrays of length cout, copied at create.
 * mult/shift are ignored (may be NULL) for AQD_OUT_INT32; skip_* are ignored
 * (may be NULL) without a skip. Ranges: shift in [-31, 31]; skip_c any
 * int32 (negative when the two scales of Eq. 7 have opposite signs, see
 * aqd_skip_params); skip_d in [0, 31]; skip_side in {0, 1}. */
typedef struct {
    const int32_t *bias;      /* round(s) of the folded BN, Eq. 6 */
    const int32_t *mult;      /* requantisation multiplier M */
    const int32_t *shift;     /* requantisation exponent: scale M / 2^(31+shift) */
    const int32_t *skip_c;    /* Eq. 8 numerator c */
    const int32_t *skip_d;    /* Eq. 8 exponent d */
    const int32_t *skip_side; /* 0: scale the skip operand, 1: scale the conv operand (Eq. 7) */
} qconv_epilogue_t;

typedef struct qconv_s *qconv_t;

/* Create a convolution handle (Sec. 3.2.1-3.2.3).
 * w_packed: host, [cout][kh][kw][cin] b-bit weight fields packed along cin
 *           (the code tensor layout above with bits_w).
 * levels:   host array of desc->num_levels epilogue tables.
 * The arithmetic is fixed here (qconv_path): the matrix cores take 2/3/4-bit
 * codes with cin a multiple of 64 and weights that fit int8 (code outputs of
 * the input's width, or 8-bit code outputs of 4-bit layers with cin a
 * multiple of 256 and cout >= 256); 2-bit codes with 2-bit weights and cin,
 * cout multiples of 256 take the FP4 matrix cores; 8-bit codes with cin a
 * multiple of 128 and int32 outputs, and the 7x7 stride-2 pad-3 stem on 3
 * channels of 8-bit codes (4-bit or int32 outputs), take the int8 matrix
 * cores on codes re-centred by -128, the handle's bias carrying
 * 128 * sum(w); every other description runs on the direct kernel.
 * On success *out receives the handle. Errors: INVALID (bad description,
 * NULL pointers, parameter out of range), UNSUPPORTED (accumulator bound
 * K * (2^bits_in - 1) * max|w| >= 2^31, 8-bit odd-grid weights, or a
 * re-centred bias outside int32), NOMEM / DEVICE (device allocation or copy
 * failed; nothing is leaked). */
aqd_status_t qconv_create(const qconv_desc_t *desc, const uint8_t *w_packed,
                          const qconv_epilogue_t *levels, qconv_t *out);

/* Output spatial size for an h x w input: floor((h + 2p - kh)/s) + 1. */
aqd_status_t qconv_out_shape(qconv_t conv, int h, int w, int *ho, int *wo);

/* Scales of a handle's integer tensors, from its step sizes (Sec. 3.2.1,
 * Eq. 4: the accumulator acc = sum eta_x * w_value has the scale
 * alpha_conv = step_in * step_w). *alpha_conv receives step_in * step_w and
 * *step_out the output step (0 if not given; either pointer may be NULL).
 * INVALID if the handle was created without step_in or step_w. */
aqd_status_t qconv_scales(qconv_t conv, double *alpha_conv, double *step_out);

/* Run the convolution with epilogue table `level` on n images of h x w.
 * x:    device, [n][h][w][cin] codes (bits_in).
 * skip: device, [n][hs][ws][cout] (skip_bits) or NULL when the handle has no
 *       skip; hs == ho and ws == wo, or with skip_up2 (ho-1)/2 < hs and
 *       (wo-1)/2 < ws.
 * y:    device, [n][ho][wo][cout] codes (bits_out) or int32.
 * n == 0 is a no-op. Asynchronous on `stream`. */
aqd_status_t qconv_run(qconv_t conv, int level, int n, int h, int w, const void *x,
                       const void *skip, int hs, int ws, void *y, aqd_stream_t stream);

/* One segment of a grouped launch. */
typedef struct {
    qconv_t conv;
    int level;
    int n, h, w;
    const void *x;
    const void *skip;
    int hs, ws;
    void *y;
} qconv_seg_t;

/* Run up to AQD_MAX_SEGS segments in one kernel launch. All handles must
 * have the same description apart from num_levels (same shapes, bitwidths
 * and modes); each segment has its own weights (its handle), epilogue table
 * (level) and tensors. This is how the detection heads run every pyramid
 * level of a tower layer, and both towers, at once (Sec. 3.2.2: per-level
 * BN tables over shared convolution weights). Same argument rules as
 * qconv_run for each segment; no output may overlap another segment's
 * inputs or outputs. */
#define AQD_MAX_SEGS 16
aqd_status_t qconv_run_group(int count, const qconv_seg_t *segs, aqd_stream_t stream);

/* Split reduction over K (Sec. 3.2.1, Eq. 4: acc is an integer sum over the
 * taps and input channels, so summing it in parts, in any order, gives the
 * same int32 value).
 *
 * qconv_group_workspace: *bytes receives the device workspace size with
 * which qconv_run_group_ws may split this group's reduction over several
 * workgroups; 0 when the group is not worth splitting (its launch already
 * fills the GPU). The size depends on the handles' shapes and on n, h, w of
 * every segment, not on the tensor pointers. Errors as qconv_run_group.
 *
 * qconv_run_group_ws: as qconv_run_group. With workspace non-NULL and
 * ws_bytes at least the queried size (and the size non-zero), the K range of
 * every output tile is cut into parts whose int32 partial sums go to the
 * workspace, and a second kernel adds the parts and applies the epilogue;
 * the outputs are identical to qconv_run_group's. Otherwise the call is
 * exactly qconv_run_group. The workspace is scratch (device memory owned by
 * the caller, 256-byte aligned, contents irrelevant on entry and undefined
 * on return); calls that share a workspace must not overlap in time (use one
 * stream, or one workspace per stream). */
aqd_status_t qconv_group_workspace(int count, const qconv_seg_t *segs, size_t *bytes);
aqd_status_t qconv_run_group_ws(int count, const qconv_seg_t *segs, void *workspace,
                                size_t ws_bytes, aqd_stream_t stream);

/* qconv_run_group_ws without a caller workspace, for callers that cannot
 * allocate device memory (code recorded under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc). The split K reduction
 * uses a scratch array of AQD_STATIC_SCRATCH_BYTES (64 MiB) that the library
 * holds on each GPU it runs on, until the process ends; the call allocates
 * nothing. Outputs are identical to qconv_run_group_ws's with a workspace of
 * the queried size. A group whose split would need more scratch than that
 * returns AQD_ERR_UNSUPPORTED (the message names the size) with no launch;
 * run it with qconv_run_group_ws instead. Every call on one GPU shares that
 * GPU's scratch and leaves its contents behind: calls that overlap in time on
 * one GPU (on two streams, or from two threads) race; serialise them on one
 * stream. Other errors as qconv_run_group. */
#define AQD_STATIC_SCRATCH_BYTES (64u << 20)
aqd_status_t qconv_run_group_static(int count, const qconv_seg_t *segs, aqd_stream_t stream);

/* Tail of a residual block with a projection shortcut, in one launch
 * (Sec. 3.2.3, Eq. 7-8: the skip operand is the shortcut convolution's int32
 * output v_p = acc_p + bias_p, one of the paper's 32-bit integer operands;
 * here it stays in registers instead of making a round trip through memory).
 * The outputs are exactly those of
 *     qconv_run(proj, level, n, hp, wp, xp, NULL, 0, 0, t)    (t: int32)
 *     qconv_run(conv, level, n, h, w, x, t, ho, wo, y)
 * without the tensor t.
 * x:  device, [n][h][w][conv cin] codes; xp: device, [n][hp][wp][proj cin]
 *     codes; y: device, [n][ho][wo][cout] codes (bits_out of conv).
 * Requirements, else AQD_ERR_UNSUPPORTED (nothing launched; run the two
 * calls above instead): conv has AQD_OUT_CODES, skip_bits 32 and no
 * upsample; proj has AQD_OUT_INT32, no skip, a 1x1 kernel and pad 0; both
 * take 4-bit activations, have the same cout, a multiple of 256, and cin a
 * multiple of 64; proj's output size for hp x wp equals conv's for h x w.
 * level must be valid for both handles. Other errors as qconv_run. */
aqd_status_t qconv_run_proj(qconv_t conv, qconv_t proj, int level, int n, int h, int w,
                            const void *x, int hp, int wp, const void *xp, void *y,
                            aqd_stream_t stream);

void qconv_destroy(qconv_t conv);

/* The arithmetic a handle's launches run on, fixed at create: "fp4-mfma"
 * (2-bit codes and 2-bit weights with cin and cout multiples of 256, exact
 * while K * 3 * max|w| < 2^24: the scaled FP4 MFMA with e2m1 operands and
 * fp32 sums of integers), "i8-mfma" (codes widened to int8 on the int8
 * MFMA), "direct" (every other shape: one thread per output). A static
 * string; "invalid" for a null handle. With the environment variable
 * AQD_NO_FP4=1 at create, 2-bit layers take the int8 MFMA path instead (the
 * same results; for comparing the two). */
const char *qconv_path(qconv_t conv);

/* Standalone integer skip connection (Sec. 3.2.3, Eq. 7) with
 * requantisation, for a top-down add that is not fused into a conv:
 *   y[n][i][j][c] = clamp(RSM(u_, mult[c], 31 + shift[c]), 0, 2^bits_out - 1)
 *   u_ = side 0: a + RSM(b, c_[c], d[c]);  side 1: RSM(a, c_[c], d[c]) + b
 *   with b read at (i >> 1, j >> 1) when up2 (nearest 2x upsample, Sec. 3.2.4).
 * a: device [n][h][w][c] (bits_a in {2, 3, 4, 8, 32}); b: device
 * [n][hb][wb][c] (bits_b in {2, 3, 4, 8, 32}); y: device [n][h][w][c] codes.
 * Without up2, hb == h and wb == w; with up2, (h-1)/2 < hb, (w-1)/2 < wb. */
typedef struct {
    int n, h, w, c;
    int bits_a, bits_b, bits_out;
    int up2, hb, wb;
} qadd_desc_t;

/* Device arrays of length c (int32 each). */
typedef struct {
    const int32_t *skip_c, *skip_d, *skip_side, *mult, *shift;
} qadd_params_t;

aqd_status_t qadd_run(const qadd_desc_t *desc, const void *a, const void *b, void *y,
                      const qadd_params_t *dev_params, aqd_stream_t stream);

/* Max-pooling of a code tensor (Sec. 3.2.4: the layer leaves its input's
 * scale factor unchanged, so the codes are pooled directly):
 *   y[n][i][j][c] = max of x[n][i*stride - pad + dy][j*stride - pad + dx][c]
 *   over 0 <= dy, dx < k, skipping positions outside the input,
 * ho = (h + 2*pad - k) / stride + 1, wo likewise (both >= 1; pad < k, so
 * every window holds an input position). x: device [n][h][w][c] codes of
 * `bits` in {2, 3, 4, 8}; y: device [n][ho][wo][c], same width; c * bits a
 * multiple of 8; y must not overlap x. 1 <= k <= 7, 1 <= stride <= 4. */
typedef struct {
    int n, h, w, c, bits, k, stride, pad;
} aqd_maxpool_desc_t;

aqd_status_t aqd_maxpool_run(const aqd_maxpool_desc_t *desc, const void *x, void *y,
                             aqd_stream_t stream);

/* Diagnostic for measurements (the benchmark's measured ceiling next to the
 * dense int8 peak figure): launches `workgroups` workgroups of 4 waves,
 * each wave issuing iters x 16 independent 16x16x64 int8 MFMAs on register
 * operands of 4-bit magnitudes, nothing else in its loop; every workgroup
 * writes 256 int32 checksums to out (device, workgroups x 256 entries,
 * caller-owned). Integer operations per launch: workgroups x 4 x iters x 16
 * x 32768. Time it with events on `stream`. INVALID for workgroups outside
 * 1..2^20, iters < 1 or a null out. */
aqd_status_t aqd_mfma_probe(int workgroups, int iters, int32_t *out, aqd_stream_t stream);

/* Exact per-channel sums of an int32 tensor [rows][c] on the device:
 * sums[ch] += sum_r v[r][ch], sums[c + ch] += sum_r v[r][ch]^2 (int64,
 * accumulated into the caller's zeroed array). These are the statistics a
 * BN layer keeps (Sec. 3.2.2), computed on an int32 conv output; the caller
 * guarantees rows * max v^2 < 2^63. */
aqd_status_t aqd_channel_sums(const int32_t *v, int64_t rows, int c, int64_t *sums,
                              aqd_stream_t stream);

/* Whole-network capture: the launches a network pass enqueues on one stream
 * (each a grouped convolution of Sec. 3.2.2's multi-level tables, a fused
 * shortcut or a split K range) are recorded once into a HIP graph and
 * replayed as one launch.
 * aqd_graph_begin: starts capturing `stream` (not the null stream, not a
 *   stream already capturing), in thread-local mode: until aqd_graph_end,
 *   calls of this library from the calling thread on that stream are
 *   recorded, not run. qconv_run, qconv_run_group(_ws), qconv_run_proj,
 *   qadd_run and aqd_channel_sums allocate nothing and may be recorded.
 * aqd_graph_end: ends the capture and instantiates the graph; *graph_exec
 *   receives the executable graph (owned by the caller, freed by
 *   aqd_graph_destroy), or NULL with AQD_ERR_DEVICE if the capture failed.
 * aqd_graph_launch: enqueues one replay on `stream`; the device pointers and
 *   argument values recorded at capture are used again, so the tensors must
 *   still be allocated (their contents may change between replays).
 * aqd_graph_destroy: frees an executable graph (NULL is ignored); no replay
 *   of it may be pending. */
aqd_status_t aqd_graph_begin(aqd_stream_t stream);
aqd_status_t aqd_graph_end(aqd_stream_t stream, void **graph_exec);
aqd_status_t aqd_graph_launch(void *graph_exec, aqd_stream_t stream);
void aqd_graph_destroy(void *graph_exec);

/* Message of the calling thread's last failed call ("" if none). */
const char *aqd_last_error(void);

/* ---- host helpers: offline derivation of the integer parameters ---------
 * Floating point is used only here, before inference, as the paper allows
 * (the scale factors are "passed to the next layer", Sec. 3.2.1-3.2.3).
 * All are deterministic IEEE double computations (no contraction), in the
 * order written. */

/* Pack `rows` x c codes (one byte each, values < 2^bits) into the code tensor
 * layout; out has rows * c * bits / 8 bytes (rows * c / 2 for bits 3). */
aqd_status_t aqd_pack_codes(const uint8_t *codes, int64_t rows, int c, int bits, uint8_t *out);
/* Inverse of aqd_pack_codes. */
aqd_status_t aqd_unpack_codes(const uint8_t *packed, int64_t rows, int c, int bits, uint8_t *out);

/* Eq. 8: F(m, n) = c / 2^d minimising |r - c/2^d| for r = m/n >= 1, over
 * d in [1, 31] and 0 <= c < 2^31; among equally good pairs the smallest d.
 * INVALID unless 1 <= r < 2^30. */
aqd_status_t aqd_approx_ratio(double r, int32_t *c, int32_t *d);

/* Dyadic form of a scale r != 0: mult / 2^(31 + shift) with
 * |mult| in [2^30, 2^31), sign of r, shift in [-31, 31];
 * mult = round(|r| * 2^(31 + shift)). INVALID if out of range. */
aqd_status_t aqd_normalize_multiplier(double r, int32_t *mult, int32_t *shift);

/* BN running statistics from exact accumulator sums (aqd_channel_sums):
 * m = s1/count, mean = alpha_conv * m, var = alpha_conv^2 * (s2/count - m*m). */
aqd_status_t aqd_bn_stats_from_sums(int cout, const int64_t *s1, const int64_t *s2,
                                    int64_t count, double alpha_conv, double *mean,
                                    double *var);

/* Eq. 5-6: sd = sqrt(var + eps); s = (beta * sd / gamma - mean) / alpha_conv;
 * bias = round(s) (half up); alpha_z = alpha_conv * gamma / sd.
 * INVALID for gamma == 0, var + eps <= 0 or a bias outside int32. */
aqd_status_t aqd_fold_bn(int cout, const double *gamma, const double *beta, const double *mean,
                         const double *var, double eps, double alpha_conv, int32_t *bias,
                         double *alpha_z);

/* Eq. 7-8 per channel: the operand with the larger scale is rescaled to the
 * smaller one, and the sum carries the smaller scale:
 *   |alpha_k| >= |alpha_z|: side 0, (c, d) = F(|alpha_k / alpha_z|), scale = alpha_z;
 *   otherwise:              side 1, (c, d) = F(|alpha_z / alpha_k|), scale = alpha_k;
 * with c negated when alpha_z and alpha_k have opposite signs (a folded
 * normalisation with gamma < 0 has alpha_z < 0; for positive scales this is
 * the paper's rule, and scale = min(alpha_z, alpha_k)).
 * alpha_k has cout entries if alpha_k_per_channel, else one. INVALID for a
 * zero or non-finite scale, or a ratio outside aqd_approx_ratio's domain. */
aqd_status_t aqd_skip_params(int cout, const double *alpha_z, const double *alpha_k,
                             int alpha_k_per_channel, int32_t *c, int32_t *d, int32_t *side,
                             double *scale);

/* Requantisation to codes of step alpha_out (Eq. 2 applied to a sum of scale
 * `scale`): (mult, shift) = aqd_normalize_multiplier(scale / alpha_out), so
 * that RSM(u, mult, 31 + shift) is u * scale / alpha_out rounded to nearest
 * up to the dyadic error |mult / 2^(31+shift) - scale / alpha_out| <=
 * 2^-(32+shift). The split from aqd_fold_bn (which returns alpha_z, not a
 * multiplier) lets a skip add (aqd_skip_params) choose the sum's scale
 * between the fold and the requantisation. */
aqd_status_t aqd_requant_params(int cout, const double *scale, double alpha_out, int32_t *mult,
                                int32_t *shift);

#ifdef __cplusplus
}
#endif

#endif /* AQD_H */
