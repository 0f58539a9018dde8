// C-ABI host code: argument validation, handle creation (weight decoding and
// tiling, epilogue tables), kernel selection and launch, and the host-side
// parameter derivation helpers. Declarations and contracts: include/aqd.h.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "aqd.h"
#include "internal.h"

using namespace aqd;

namespace {

thread_local std::string g_err;

aqd_status_t fail(aqd_status_t st, const std::string &msg)
{
    g_err = msg;
    return st;
}

#define REQUIRE(cond, msg)                            \
    do {                                              \
        if (!(cond))                                  \
            return fail(AQD_ERR_INVALID, (msg));      \
    } while (0)

// code widths; 3-bit codes (Tables 2 and 4 of the paper) are stored one per
// 4-bit container, so that every kernel reads them as 4-bit codes
bool code_bits(int b) { return b == 2 || b == 3 || b == 4 || b == 8; }
int stored_bits(int b) { return b == 3 ? 4 : b; }

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

bool overlap(const void *a, size_t na, const void *b, size_t nb)
{
    uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return na && nb && a0 < b0 + nb && b0 < a0 + na;
}

// Positions of the 64 channels of one K step after the kernel's widening of
// packed codes (see qconv_mfma.hip): LDS byte p holds channel sigma(p);
// 8-bit codes are staged in channel order.
int widened_channel(int bits_in, int p)
{
    if (bits_in == 8)
        return p;
    if (bits_in == 4)
        return 8 * (p / 8) + 2 * (p % 4) + ((p / 4) % 2);
    return 16 * (p / 16) + 4 * (p % 4) + ((p / 4) % 4);  // bits_in == 2
}

// Channel (within a workgroup tile) of MFMA row rho: a wave slice has
// 4 * cpl_rows = 16 * MI rows; lane group g of accumulator tile i of slice w
// holds channel w * 16 * MI + cpl * g + 4i + e, where cpl = 4 * MI is the
// number of consecutive channels a lane owns per pixel.
int tile_row_channel(int rho, int cpl)
{
    const int slice = 4 * cpl;  // rows per wave slice
    int w = rho / slice, rr = rho % slice;
    int i = rr / 16, g = (rr % 16) / 4, e = rr % 4;
    return w * slice + cpl * g + 4 * i + e;
}

// FP4 path (qconv_fp4.hip): position kappa of a 256-channel stage in LDS
// holds channel fp4_channel(kappa). A copy lane spreads 32 packed 2-bit codes
// (channels 32c .. 32c+31) into 16-byte column c: word 0 = the even channels
// of the first 16, word 1 = their odd ones, words 2 and 3 the same for the
// second 16; nibble n of a word is its n-th channel.
int fp4_channel(int kappa)
{
    const int c = kappa / 32, wd = (kappa % 32) / 8, n = kappa % 8;
    return 32 * c + 16 * (wd >> 1) + 2 * n + (wd & 1);
}

// e2m1 nibble of a small integer (|v| <= 3: 0, 1, 2, 3 -> 0x0, 0x2, 0x4, 0x5;
// bit 3 = sign)
uint8_t e2m1_nibble(int v)
{
    static const uint8_t mag[4] = {0x0, 0x2, 0x4, 0x5};
    return (uint8_t)((v < 0 ? 0x8 : 0x0) | mag[v < 0 ? -v : v]);
}

int pick_tile(int cout, bool codes, int bits_in)
{
    if (bits_in == 4 && cout >= 256 && (!codes || cout % 32 == 0))
        return TILE_256x128;
    return cout > 64 ? TILE_128x256 : TILE_64x512;
}

// 256 zero bytes per device: the source of the kernel's copies for padding taps.
std::mutex g_zero_mu;
void *g_zero[64] = {};

const uint8_t *device_zero_page()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
        return nullptr;
    std::lock_guard<std::mutex> lock(g_zero_mu);
    if (!g_zero[dev]) {
        static const uint8_t zeros[256] = {};
        void *p = nullptr;
        if (hipMalloc(&p, sizeof zeros) != hipSuccess)
            return nullptr;
        if (hipMemcpy(p, zeros, sizeof zeros, hipMemcpyHostToDevice) != hipSuccess) {
            (void)hipFree(p);
            return nullptr;
        }
        g_zero[dev] = p;
    }
    return (const uint8_t *)g_zero[dev];
}

int weight_value(int field, int bits, int wenc)
{
    if (wenc == AQD_WENC_PAPER_ODD)
        return 2 * field - ((1 << bits) - 1);
    return field >= (1 << (bits - 1)) ? field - (1 << bits) : field;
}

}  // namespace

struct qconv_s {
    qconv_desc_t d;     // widths as stored (3-bit codes in 4-bit containers)
    int qmax;           // largest output code, 2^bits_out - 1 of the caller's bits_out
    bool mfma;
    int tile_cfg, blk_co, blk_px;
    int co_tiles, ksteps, cout_pad;
    void *w_dev;
    int32_t *epi_dev;  // [num_levels][EPI_FIELDS][cout_pad]
    int32_t *lut_dev;  // code skips: [num_levels][cout_pad][2^skip_bits] RSM(k, c, d), else null
    std::vector<int> fast;  // per level: every shift >= 2
    std::vector<int> side0; // per level: every skip side is 0
    const uint8_t *zero;    // the device's zero page
};

extern "C" {

const char *aqd_last_error(void) { return g_err.c_str(); }

static aqd_status_t validate_desc(const qconv_desc_t *d)
{
    REQUIRE(d->cin >= 1 && d->cout >= 1, "cin and cout must be >= 1");
    REQUIRE(d->cin <= 65536 && d->cout <= 65536, "cin and cout must be <= 65536");
    REQUIRE(d->kh >= 1 && d->kh <= 7 && d->kw >= 1 && d->kw <= 7, "kh and kw must be in 1..7");
    REQUIRE(d->stride >= 1 && d->stride <= 4, "stride must be in 1..4");
    REQUIRE(d->pad >= 0 && d->pad < d->kh && d->pad < d->kw, "pad must be in 0..k-1");
    REQUIRE(code_bits(d->bits_in), "bits_in must be 2, 3, 4 or 8");
    REQUIRE(code_bits(d->bits_w), "bits_w must be 2, 3, 4 or 8");
    REQUIRE(d->wenc == AQD_WENC_TWOS || d->wenc == AQD_WENC_PAPER_ODD, "unknown weight grid");
    REQUIRE(d->out_mode == AQD_OUT_CODES || d->out_mode == AQD_OUT_INT32, "unknown output mode");
    REQUIRE((d->cin * stored_bits(d->bits_in)) % 8 == 0, "cin * bits_in must be a multiple of 8");
    REQUIRE((d->cin * stored_bits(d->bits_w)) % 8 == 0, "cin * bits_w must be a multiple of 8");
    if (d->out_mode == AQD_OUT_CODES) {
        REQUIRE(code_bits(d->bits_out), "bits_out must be 2, 3, 4 or 8");
        REQUIRE((d->cout * stored_bits(d->bits_out)) % 8 == 0, "cout * bits_out must be a multiple of 8");
    }
    REQUIRE(d->skip_bits == 0 || code_bits(d->skip_bits) || d->skip_bits == 32,
            "skip_bits must be 0, 2, 3, 4, 8 or 32");
    if (d->skip_bits) {
        REQUIRE(d->out_mode == AQD_OUT_CODES, "a skip add needs code output");
        REQUIRE((d->cout * stored_bits(d->skip_bits)) % 8 == 0, "cout * skip_bits must be a multiple of 8");
    }
    REQUIRE(d->skip_up2 == 0 || (d->skip_up2 == 1 && d->skip_bits), "skip_up2 needs a skip");
    REQUIRE(d->num_levels >= 1 && d->num_levels <= 64, "num_levels must be in 1..64");
    const double steps[3] = {d->step_in, d->step_w, d->step_out};
    for (double st : steps)
        REQUIRE(std::isfinite(st) && st >= 0.0, "step sizes must be finite and >= 0 (0: not given)");
    return AQD_OK;
}

aqd_status_t qconv_create(const qconv_desc_t *desc, const uint8_t *w_packed,
                          const qconv_epilogue_t *levels, qconv_t *out)
{
    REQUIRE(desc && w_packed && levels && out, "null argument");
    *out = nullptr;
    aqd_status_t st = validate_desc(desc);
    if (st != AQD_OK)
        return st;
    const qconv_desc_t dc = *desc;  // the caller's widths
    const bool codes = dc.out_mode == AQD_OUT_CODES;
    qconv_desc_t d = dc;             // stored widths
    d.bits_in = stored_bits(dc.bits_in);
    d.bits_w = stored_bits(dc.bits_w);
    if (codes)
        d.bits_out = stored_bits(dc.bits_out);
    if (dc.skip_bits && dc.skip_bits != 32)
        d.skip_bits = stored_bits(dc.skip_bits);
    for (int l = 0; l < d.num_levels; ++l) {
        const qconv_epilogue_t &e = levels[l];
        REQUIRE(e.bias, "epilogue bias is null");
        if (codes) {
            REQUIRE(e.mult && e.shift, "epilogue mult/shift is null");
            for (int c = 0; c < d.cout; ++c)
                REQUIRE(e.shift[c] >= -31 && e.shift[c] <= 31, "shift outside [-31, 31]");
        }
        if (d.skip_bits) {
            REQUIRE(e.skip_c && e.skip_d && e.skip_side, "skip parameters are null");
            for (int c = 0; c < d.cout; ++c) {
                REQUIRE(e.skip_d[c] >= 0 && e.skip_d[c] <= 31, "skip_d outside [0, 31]");
                REQUIRE(e.skip_side[c] == 0 || e.skip_side[c] == 1, "skip_side must be 0 or 1");
            }
        }
    }
    // accumulator bound: K * max code * max |weight| < 2^31
    const long long K = (long long)d.kh * d.kw * d.cin;
    const long long wmax = dc.wenc == AQD_WENC_PAPER_ODD ? (1 << dc.bits_w) - 1 : (1 << (dc.bits_w - 1));
    if (K * ((1 << dc.bits_in) - 1) * wmax >= (1LL << 31))
        return fail(AQD_ERR_UNSUPPORTED, "accumulator could exceed int32 for this K and bitwidths");

    // decode weight fields
    const int wrow = d.cin * d.bits_w / 8;
    const int taps = d.kh * d.kw;
    std::vector<int16_t> wv((size_t)d.cout * taps * d.cin);
    for (int co = 0; co < d.cout; ++co)
        for (int t = 0; t < taps; ++t) {
            const uint8_t *row = w_packed + ((size_t)co * taps + t) * wrow;
            for (int ci = 0; ci < d.cin; ++ci) {
                int bit = ci * d.bits_w;
                int f = (row[bit >> 3] >> (bit & 7)) & ((1 << dc.bits_w) - 1);
                wv[((size_t)co * taps + t) * d.cin + ci] = (int16_t)weight_value(f, dc.bits_w, d.wenc);
            }
        }

    // MFMA kernel: 2/4-bit activations, weights that fit int8, 64-channel K
    // steps, output and skip codes of the input's width; the direct kernel
    // takes everything else
    const bool w_fits_i8 = dc.bits_w <= 4 || d.wenc == AQD_WENC_TWOS;
    // 8-bit codes with int32 outputs (the prediction convolutions of the
    // fully quantized networks): the int8 MFMA on codes re-centred by -128
    const bool b8 = dc.bits_in == 8 && !codes && d.skip_bits == 0 && d.cin % 128 == 0 && w_fits_i8 &&
                    d.cout % 4 == 0;
    // 4-bit codes in, 8-bit codes out (the last tower layer before 8-bit
    // prediction convolutions): the register-fed kernel's 8-bit epilogue
    const bool wv8 = d.bits_in == 4 && codes && dc.bits_out == 8 && d.skip_bits == 0 && d.cin % 256 == 0 &&
                     d.cout >= 256 && d.cout % 32 == 0 && w_fits_i8;
    // the ResNet stem (7x7, stride 2, pad 3) on a 3-channel 8-bit image
    const bool stem = dc.bits_in == 8 && d.cin == 3 && d.kh == 7 && d.kw == 7 && d.stride == 2 &&
                      d.pad == 3 && d.skip_bits == 0 && (!codes || dc.bits_out == 4) && d.cout % 64 == 0 &&
                      w_fits_i8;
    const bool mfma = b8 || wv8 || stem || ((d.bits_in == 2 || d.bits_in == 4) && d.cin % KC == 0 && w_fits_i8 &&
                             (codes ? (d.cout % 16 == 0 && d.bits_out == d.bits_in &&
                                       (d.skip_bits == 0 || d.skip_bits == d.bits_in || d.skip_bits == 32))
                                    : d.cout % 4 == 0));
    // 2-bit codes and weights in 256-channel chunks: the scaled FP4 MFMA, exact
    // while every partial sum stays below 2^24 (K * 3 * max|w| < 2^24)
    const char *no_fp4 = std::getenv("AQD_NO_FP4");
    const bool fp4 = mfma && !(no_fp4 && std::strcmp(no_fp4, "1") == 0) && dc.bits_in == 2 && dc.bits_w == 2 &&
                     d.cin % 256 == 0 && d.cout % 256 == 0 &&
                     (codes ? (dc.bits_out == 2 && (d.skip_bits == 0 || d.skip_bits == 2)) : d.skip_bits == 0) &&
                     K * 3 * wmax < (1LL << 24);
    qconv_s h{};
    h.d = d;
    h.qmax = codes ? (1 << dc.bits_out) - 1 : 0;
    h.mfma = mfma;
    int cpl = 0;
    h.tile_cfg = fp4 ? TILE_FP4 : b8 ? TILE_B8 : stem ? TILE_STEM : pick_tile(d.cout, codes, d.bits_in);
    mfma_tile_shape(h.tile_cfg, &h.blk_co, &h.blk_px, &cpl);
    const int BLK_CO = h.blk_co;
    h.co_tiles = mfma ? (d.cout + BLK_CO - 1) / BLK_CO : 1;
    h.cout_pad = mfma ? h.co_tiles * BLK_CO : d.cout;
    h.ksteps = stem ? 3 : mfma ? taps * (d.cin / KC) : 0;
    h.fast.assign(d.num_levels, 0);
    h.side0.assign(d.num_levels, 0);
    for (int l = 0; l < d.num_levels && d.skip_bits; ++l) {  // (stored widths from here on)
        int ok = 1;
        for (int c = 0; c < d.cout; ++c)
            ok &= levels[l].skip_side[c] == 0;
        h.side0[l] = ok;
    }
    for (int l = 0; l < d.num_levels && codes; ++l) {
        int ok = 1;
        for (int c = 0; c < d.cout; ++c)
            ok &= levels[l].shift[c] >= 2;
        h.fast[l] = ok;
    }

    std::vector<uint8_t> wbuf;
    if (stem) {
        // [co_tile][K step][row rho][64 B]: K byte k = window row k / 24, tap
        // (k % 24) / 3, channel k % 3 for k % 24 < 21, else zero; channel
        // tile_row_channel(rho) of the 64-channel tile
        wbuf.assign((size_t)h.co_tiles * 3 * 64 * KC, 0);
        for (int ct = 0; ct < h.co_tiles; ++ct)
            for (int rho = 0; rho < 64; ++rho) {
                const int co = ct * 64 + tile_row_channel(rho, cpl);
                for (int k = 0; k < 168; ++k) {
                    const int kh = k / 24, rem = k % 24;
                    if (rem >= 21)
                        continue;
                    const int kw = rem / 3, c = rem % 3;
                    wbuf[(((size_t)ct * 3 + k / KC) * 64 + rho) * KC + k % KC] =
                        (uint8_t)(int8_t)wv[((size_t)co * taps + kh * 7 + kw) * d.cin + c];
                }
            }
    } else if (fp4) {
        // tiles [co_tile][128-channel K step][row rho][64 bytes]: channel
        // tile_row_channel(rho) of the tile; nibble kappa (byte kappa / 2, low
        // nibble first) = e2m1 of the weight of input channel
        // fp4_channel(128 q + kappa) of the stage, q = K step % 2
        const int k4pt = d.cin / 128, ks4 = taps * k4pt;
        wbuf.assign((size_t)h.co_tiles * ks4 * 256 * 64, 0);
        for (int ct = 0; ct < h.co_tiles; ++ct)
            for (int ks = 0; ks < ks4; ++ks) {
                const int tap = ks / k4pt, c128 = ks % k4pt;
                const int stage0 = 256 * (c128 / 2), q = c128 % 2;
                for (int rho = 0; rho < 256; ++rho) {
                    const int co = ct * 256 + tile_row_channel(rho, cpl);
                    uint8_t *dst = wbuf.data() + (((size_t)ct * ks4 + ks) * 256 + rho) * 64;
                    const int16_t *src = wv.data() + ((size_t)co * taps + tap) * d.cin + stage0;
                    for (int kap = 0; kap < 128; ++kap)
                        dst[kap / 2] |= (uint8_t)(e2m1_nibble(src[fp4_channel(128 * q + kap)]) << (4 * (kap % 2)));
                }
            }
    } else if (mfma) {
        // tiles [co_tile][k step][row rho][byte p]: channel tile_row_channel(rho) of the tile,
        // input channel widened_channel(p) of the K step's 64-channel chunk
        const int kpt = d.cin / KC;
        wbuf.assign((size_t)h.co_tiles * h.ksteps * BLK_CO * KC, 0);
        for (int ct = 0; ct < h.co_tiles; ++ct)
            for (int ks = 0; ks < h.ksteps; ++ks) {
                const int tap = ks / kpt, cc = ks % kpt;
                for (int rho = 0; rho < BLK_CO; ++rho) {
                    const int co = ct * BLK_CO + tile_row_channel(rho, cpl);
                    if (co >= d.cout)
                        continue;
                    int8_t *dst = (int8_t *)wbuf.data() + (((size_t)ct * h.ksteps + ks) * BLK_CO + rho) * KC;
                    const int16_t *src = wv.data() + ((size_t)co * taps + tap) * d.cin + cc * KC;
                    for (int p = 0; p < KC; ++p)
                        dst[p] = (int8_t)src[widened_channel(d.bits_in, p)];
                }
            }
    } else {
        wbuf.resize(wv.size() * sizeof(int16_t));
        std::memcpy(wbuf.data(), wv.data(), wbuf.size());
    }
    // 8-bit codes on the MFMA enter as a - 128: the bias carries 128 * sum(w)
    // of the channel (every tap, padding included, enters as 0 - 128)
    std::vector<long long> recentre(d.cout, 0);
    if (b8 || stem)
        for (int co = 0; co < d.cout; ++co) {
            long long sw = 0;
            for (size_t k = 0; k < (size_t)taps * d.cin; ++k)
                sw += wv[(size_t)co * taps * d.cin + k];
            recentre[co] = 128 * sw;
        }
    std::vector<int32_t> epi((size_t)d.num_levels * EPI_FIELDS * h.cout_pad, 0);
    for (int l = 0; l < d.num_levels; ++l) {
        const qconv_epilogue_t &e = levels[l];
        int32_t *t = epi.data() + (size_t)l * EPI_FIELDS * h.cout_pad;
        for (int c = 0; c < d.cout; ++c) {
            const long long b = (long long)e.bias[c] + recentre[c];
            if (b < INT32_MIN || b > INT32_MAX)
                return fail(AQD_ERR_UNSUPPORTED, "bias + 128 * sum(w) exceeds int32 (8-bit codes)");
            t[EPI_BIAS * h.cout_pad + c] = (int32_t)b;
            if (codes) {
                const int sh = e.shift[c];
                t[EPI_MULT * h.cout_pad + c] = e.mult[c];
                t[EPI_SHIFT * h.cout_pad + c] = sh;
                t[EPI_SHR * h.cout_pad + c] = sh - 1;
                t[EPI_RND * h.cout_pad + c] = sh >= 2 ? (1 << (sh - 2)) : 0;
            }
            if (d.skip_bits) {
                t[EPI_SKIP_C * h.cout_pad + c] = e.skip_c[c];
                t[EPI_SKIP_D * h.cout_pad + c] = e.skip_d[c];
                t[EPI_SKIP_SIDE * h.cout_pad + c] = e.skip_side[c];
            }
        }
    }

    // code skips: per level and channel the skip operand's scaled value
    // RSM(k, c, d) for every code k (used when every side of the level is 0),
    // computed exactly and kept modulo 2^32 as the kernels' 32-bit sums are
    std::vector<int32_t> lut;
    const int nk = (d.skip_bits > 0 && d.skip_bits < 32) ? (1 << d.skip_bits) : 0;
    if (nk) {
        lut.assign((size_t)d.num_levels * h.cout_pad * nk, 0);
        for (int l = 0; l < d.num_levels; ++l)
            for (int c = 0; c < d.cout; ++c) {
                const long long cc = levels[l].skip_c[c];
                const int dd = levels[l].skip_d[c];
                for (int k = 0; k < nk; ++k) {
                    const long long p = (long long)k * cc;
                    const long long r = dd > 0 ? (p + (1LL << (dd - 1))) >> dd : p;
                    lut[((size_t)l * h.cout_pad + c) * nk + k] = (int32_t)(uint32_t)(uint64_t)r;
                }
            }
    }

    const char *inject = std::getenv("AQD_FAULT_INJECT");
    if (inject && std::strcmp(inject, "alloc") == 0)
        return fail(AQD_ERR_NOMEM, "device allocation failed (injected)");

    h.zero = device_zero_page();
    if (!h.zero)
        return fail(AQD_ERR_NOMEM, "could not allocate the device zero page");
    qconv_s *hp = new (std::nothrow) qconv_s(h);
    if (!hp)
        return fail(AQD_ERR_NOMEM, "host allocation failed");
    // MFMA weights: four K steps of 256-row tiles (64 KiB) of padding past the
    // end, which the register-fed kernel's look-ahead may read (never use)
    const size_t w_pad = mfma ? 4 * 256 * KC : 0;
    if (hipMalloc(&hp->w_dev, wbuf.size() + w_pad) != hipSuccess) {
        delete hp;
        return fail(AQD_ERR_NOMEM, "hipMalloc of the weights failed");
    }
    if (hipMalloc((void **)&hp->epi_dev, epi.size() * sizeof(int32_t)) != hipSuccess) {
        (void)hipFree(hp->w_dev);
        delete hp;
        return fail(AQD_ERR_NOMEM, "hipMalloc of the epilogue tables failed");
    }
    hp->lut_dev = nullptr;
    if (nk && hipMalloc((void **)&hp->lut_dev, lut.size() * sizeof(int32_t)) != hipSuccess) {
        (void)hipFree(hp->w_dev);
        (void)hipFree(hp->epi_dev);
        delete hp;
        return fail(AQD_ERR_NOMEM, "hipMalloc of the skip tables failed");
    }
    if (hipMemcpy(hp->w_dev, wbuf.data(), wbuf.size(), hipMemcpyHostToDevice) != hipSuccess ||
        hipMemcpy(hp->epi_dev, epi.data(), epi.size() * sizeof(int32_t), hipMemcpyHostToDevice) !=
            hipSuccess ||
        (nk && hipMemcpy(hp->lut_dev, lut.data(), lut.size() * sizeof(int32_t), hipMemcpyHostToDevice) !=
                   hipSuccess)) {
        (void)hipFree(hp->w_dev);
        (void)hipFree(hp->epi_dev);
        if (hp->lut_dev)
            (void)hipFree(hp->lut_dev);
        delete hp;
        return fail(AQD_ERR_DEVICE, "copy of the weights to the device failed");
    }
    *out = hp;
    return AQD_OK;
}

const char *qconv_path(qconv_t conv)
{
    if (!conv)
        return "invalid";
    if (!conv->mfma)
        return "direct";
    return conv->tile_cfg == TILE_FP4 ? "fp4-mfma" : "i8-mfma";  // TILE_B8 included
}

void qconv_destroy(qconv_t conv)
{
    if (!conv)
        return;
    (void)hipFree(conv->w_dev);
    (void)hipFree(conv->epi_dev);
    if (conv->lut_dev)
        (void)hipFree(conv->lut_dev);
    delete conv;
}

aqd_status_t qconv_out_shape(qconv_t conv, int h, int w, int *ho, int *wo)
{
    REQUIRE(conv && ho && wo, "null argument");
    REQUIRE(h >= 1 && w >= 1, "h and w must be >= 1");
    const qconv_desc_t &d = conv->d;
    REQUIRE(h + 2 * d.pad >= d.kh && w + 2 * d.pad >= d.kw, "input smaller than the filter");
    *ho = (h + 2 * d.pad - d.kh) / d.stride + 1;
    *wo = (w + 2 * d.pad - d.kw) / d.stride + 1;
    return AQD_OK;
}

aqd_status_t qconv_scales(qconv_t conv, double *alpha_conv, double *step_out)
{
    REQUIRE(conv, "null handle");
    REQUIRE(conv->d.step_in > 0.0 && conv->d.step_w > 0.0,
            "the handle was created without step_in / step_w");
    if (alpha_conv)
        *alpha_conv = conv->d.step_in * conv->d.step_w;
    if (step_out)
        *step_out = conv->d.step_out;
    return AQD_OK;
}

}  // extern "C"

namespace {

struct SegCheck {
    int ho, wo;
    size_t xbytes, sbytes, ybytes;
};

aqd_status_t check_seg(const qconv_seg_t &s, SegCheck *out)
{
    REQUIRE(s.conv, "null handle");
    const qconv_desc_t &d = s.conv->d;
    REQUIRE(s.level >= 0 && s.level < d.num_levels, "level out of range");
    REQUIRE(s.n >= 0, "n must be >= 0");
    int ho = 0, wo = 0;
    aqd_status_t st = qconv_out_shape(s.conv, s.h, s.w, &ho, &wo);
    if (st != AQD_OK)
        return st;
    REQUIRE((long long)s.n * ho * wo < (1LL << 31) && (long long)s.n * s.h * s.w < (1LL << 31),
            "too many pixels for one call");
    out->ho = ho;
    out->wo = wo;
    out->xbytes = (size_t)s.n * s.h * s.w * d.cin * d.bits_in / 8;
    out->ybytes = (size_t)s.n * ho * wo * d.cout * (d.out_mode == AQD_OUT_INT32 ? 32 : d.bits_out) / 8;
    out->sbytes = 0;
    if (s.n == 0)
        return AQD_OK;
    REQUIRE(s.x && s.y, "null tensor");
    REQUIRE(aligned16(s.x) && aligned16(s.y), "tensors must be 16-byte aligned");
    if (d.skip_bits) {
        REQUIRE(s.skip, "the handle has a skip but skip is null");
        REQUIRE(aligned16(s.skip), "skip must be 16-byte aligned");
        if (d.skip_up2)
            REQUIRE((ho - 1) / 2 < s.hs && (wo - 1) / 2 < s.ws && s.hs >= 1 && s.ws >= 1,
                    "upsampled skip too small for the output");
        else
            REQUIRE(s.hs == ho && s.ws == wo, "skip size must equal the output size");
        out->sbytes = (size_t)s.n * s.hs * s.ws * d.cout * d.skip_bits / 8;
    } else {
        REQUIRE(!s.skip, "skip given to a handle without a skip");
    }
    REQUIRE(!overlap(s.y, out->ybytes, s.x, out->xbytes), "output overlaps the input");
    REQUIRE(!overlap(s.y, out->ybytes, s.skip, out->sbytes), "output overlaps the skip");
    return AQD_OK;
}

bool same_config(const qconv_desc_t &a, const qconv_desc_t &b)
{
    return a.cin == b.cin && a.cout == b.cout && a.kh == b.kh && a.kw == b.kw &&
           a.stride == b.stride && a.pad == b.pad && a.bits_in == b.bits_in &&
           a.bits_w == b.bits_w && a.wenc == b.wenc && a.out_mode == b.out_mode &&
           (a.out_mode == AQD_OUT_INT32 || a.bits_out == b.bits_out) &&
           a.skip_bits == b.skip_bits && a.skip_up2 == b.skip_up2;
}

aqd_status_t launch_direct(const qconv_seg_t &s, const SegCheck &c, hipStream_t stream)
{
    const qconv_s &h = *s.conv;
    DirectArgs a{};
    a.x = (const uint8_t *)s.x;
    a.skip = s.skip;
    a.y = s.y;
    a.wt = (const int16_t *)h.w_dev;
    a.epi = h.epi_dev + (size_t)s.level * EPI_FIELDS * h.cout_pad;
    a.n = s.n;
    a.h = s.h;
    a.w = s.w;
    a.ho = c.ho;
    a.wo = c.wo;
    a.hs = s.hs;
    a.ws = s.ws;
    a.cin = h.d.cin;
    a.cout = h.d.cout;
    a.kh = h.d.kh;
    a.kw = h.d.kw;
    a.stride = h.d.stride;
    a.pad = h.d.pad;
    a.bits_in = h.d.bits_in;
    a.out_bits = h.d.out_mode == AQD_OUT_INT32 ? 32 : h.d.bits_out;
    a.qmax = h.qmax;
    a.skip_bits = h.d.skip_bits;
    a.up2 = h.d.skip_up2;
    if (launch_qconv_direct(a, stream) != hipSuccess)
        return fail(AQD_ERR_DEVICE, "direct conv launch failed");
    return AQD_OK;
}

}  // namespace

namespace {

// Checks a group and fills the MFMA launch description (everything but the
// split); *tiles receives the number of output tiles, *direct whether the
// group runs on the direct kernel.
aqd_status_t prepare_group(int count, const qconv_seg_t *segs, SegCheck *chk, MfmaArgs *out,
                           bool *direct)
{
    REQUIRE(segs && count >= 1 && count <= AQD_MAX_SEGS, "count must be in 1..AQD_MAX_SEGS");
    for (int i = 0; i < count; ++i) {
        aqd_status_t st = check_seg(segs[i], &chk[i]);
        if (st != AQD_OK)
            return st;
        REQUIRE(same_config(segs[0].conv->d, segs[i].conv->d) && segs[0].conv->qmax == segs[i].conv->qmax,
                "grouped handles must share shapes, bitwidths and modes");
    }
    for (int i = 0; i < count; ++i)
        for (int j = 0; j < count; ++j) {
            if (i == j || segs[j].n == 0 || segs[i].n == 0)
                continue;
            REQUIRE(!overlap(segs[i].y, chk[i].ybytes, segs[j].y, chk[j].ybytes) &&
                        !overlap(segs[i].y, chk[i].ybytes, segs[j].x, chk[j].xbytes) &&
                        !overlap(segs[i].y, chk[i].ybytes, segs[j].skip, chk[j].sbytes),
                    "a segment output overlaps another segment's tensors");
        }
    const qconv_s &h0 = *segs[0].conv;
    *direct = !h0.mfma;
    if (!h0.mfma)
        return AQD_OK;
    MfmaArgs &a = *out;
    a = MfmaArgs{};
    // launch tile for a handle laid out for 256-channel tiles: 1x1 convolutions
    // with cin <= 128 and code outputs on persistent 256 x 64 tiles (weights kept
    // in LDS, next tile's copies during the current epilogue); other short K
    // ranges with code outputs on 256 x 64 tiles three to a CU; launches with fewer
    // 256 x 128 tiles than CUs (but not tiny, and not so long in K that
    // splitting K is the better cure) on 256 x 64 tiles two to a CU (measured:
    // from ~260 tiles on, the larger tile is faster)
    int tile_cfg = h0.tile_cfg, blk_px = h0.blk_px;
    // the register-fed, FP4 and 8-bit kernels address each segment's input
    // with 32-bit buffer offsets
    bool x_small = true;
    for (int i = 0; i < count; ++i)
        x_small = x_small && chk[i].xbytes < (1ull << 31);
    REQUIRE(x_small || (tile_cfg != TILE_FP4 && tile_cfg != TILE_B8),
            "2-bit (FP4) and 8-bit MFMA layers take inputs of less than 2^31 bytes per segment");
    long long t_handle = 0;  // tiles at the handle's own tile shape
    for (int i = 0; i < count; ++i)
        t_handle += ((long long)segs[i].n * chk[i].ho * chk[i].wo + h0.blk_px - 1) / h0.blk_px * h0.co_tiles;
    if (h0.tile_cfg == TILE_256x128) {
        long long t128 = 0;
        for (int i = 0; i < count; ++i)
            t128 += ((long long)segs[i].n * chk[i].ho * chk[i].wo + 127) / 128 * h0.co_tiles;
        const bool short_codes = h0.ksteps <= 4 && h0.d.out_mode == AQD_OUT_CODES && h0.d.bits_in == 4 &&
                                 h0.d.bits_out == 4 && (h0.d.skip_bits == 0 || h0.d.skip_bits == 4);
        // 1x1 layers with 256 input channels and 4-bit code outputs (one
        // segment): weight-stationary persistent tiles
        const bool wvs = count == 1 && h0.d.out_mode == AQD_OUT_CODES && h0.d.bits_in == 4 &&
                         h0.d.bits_out == 4 && (h0.d.skip_bits == 0 || h0.d.skip_bits == 4) && h0.d.kh == 1 &&
                         h0.d.kw == 1 && h0.d.pad == 0 && h0.d.cin == 256 &&
                         h0.d.cout % 256 == 0 && h0.co_tiles <= 256 && x_small;
        if (h0.d.out_mode == AQD_OUT_CODES && h0.d.bits_out == 8) {
            // 8-bit code outputs: only the register-fed kernel writes them
            REQUIRE(x_small, "8-bit code outputs take inputs of less than 2^31 bytes per segment");
            tile_cfg = TILE_WV;
        } else if (wvs) {
            tile_cfg = TILE_WVS;
            blk_px = 64;
        } else if (short_codes && h0.ksteps <= 2 && h0.d.kh == 1 && h0.d.kw == 1 && h0.d.pad == 0 &&
                   h0.d.cout % 256 == 0) {
            tile_cfg = TILE_STREAM;
            blk_px = 64;
        } else if (short_codes && h0.d.kh == 1 && h0.d.kw == 1 && h0.d.pad == 0 && h0.d.cout % 256 == 0 &&
                   h0.co_tiles <= 128) {
            // 3-4 K steps: the weights of a 256-row tile do not fit twice in
            // LDS, its 128-row halves do (persistent 128 x 64 tiles; the
            // streaming launch takes at most 256 channel tiles)
            tile_cfg = TILE_STREAM_H128;
            blk_px = 64;
        } else if (short_codes) {
            tile_cfg = TILE_256x64S;
            blk_px = 64;
        } else if (t128 >= 64 && t128 < 200 && h0.ksteps <= 80 && h0.d.bits_in == 4 && h0.d.cin % 256 == 0 &&
                   h0.d.out_mode == AQD_OUT_CODES && (h0.d.skip_bits == 0 || h0.d.skip_bits == 4) && x_small) {
            // fewer 256 x 128 tiles than CUs, 256-channel input chunks, code
            // outputs: register-fed 256 x 64 tiles, one round at three per CU
            // (longer K ranges split K instead)
            tile_cfg = TILE_WV64;
            blk_px = 64;
        } else if (t128 >= 64 && t128 < 200 && h0.ksteps <= 80) {
            tile_cfg = TILE_256x64;
            blk_px = 64;
        } else if (h0.d.bits_in == 4 && h0.d.cin % 256 == 0 &&
                   (h0.d.out_mode == AQD_OUT_CODES ? (h0.d.skip_bits == 0 || h0.d.skip_bits == 4)
                                                   : h0.d.skip_bits == 0) &&
                   t128 >= 200 && x_small) {
            // 256-channel input chunks: weights read into registers (no LDS
            // traffic for them), activation codes staged in LDS four K steps
            // at a time
            tile_cfg = TILE_WV;
        }
    } else if ((h0.tile_cfg == TILE_128x256 || h0.tile_cfg == TILE_64x512) && h0.ksteps <= 4 &&
               h0.d.out_mode == AQD_OUT_CODES && h0.d.bits_in == 4 && h0.d.bits_out == 4 &&
               h0.d.skip_bits == 0 && h0.d.kh == 1 && h0.d.kw == 1 && h0.d.pad == 0 &&
               h0.d.cout % h0.blk_co == 0 && h0.co_tiles <= 256) {
        // 1x1 convolutions with cin <= 256 on 128- or 64-channel handles:
        // persistent streaming tiles (weights resident in LDS)
        tile_cfg = h0.tile_cfg == TILE_128x256 ? TILE_STREAM_C128 : TILE_STREAM_C64;
        blk_px = h0.tile_cfg == TILE_128x256 ? 64 : 128;
    } else if ((h0.tile_cfg == TILE_128x256 || h0.tile_cfg == TILE_64x512) && t_handle > 256 && h0.d.bits_in == 4 &&
               h0.d.skip_bits == 0 && (h0.d.out_mode == AQD_OUT_INT32 || h0.d.bits_out == 4)) {
        tile_cfg = h0.tile_cfg == TILE_128x256 ? TILE_128x128_O3 : TILE_64x256_O3;
        blk_px = h0.tile_cfg == TILE_128x256 ? 128 : 256;
    }
    if (tile_cfg == TILE_WV && h0.d.out_mode == AQD_OUT_CODES) {
        // a little above one round of 256 x 128 tiles at one workgroup per CU
        // (the CUs that get a second tile set the launch's time): 256 x 144
        // tiles, one round
        long long t128 = 0, t144 = 0;
        for (int i = 0; i < count; ++i) {
            const long long p = (long long)segs[i].n * chk[i].ho * chk[i].wo;
            t128 += (p + 127) / 128 * h0.co_tiles;
            t144 += (p + 143) / 144 * h0.co_tiles;
        }
        if (h0.ksteps <= 8) {
            // short K ranges: a tile's copies and epilogue outweigh its MFMAs;
            // 256 x 64 tiles, three workgroups per CU
            tile_cfg = TILE_WV64;
            blk_px = 64;
        } else if (t128 > 256 && t144 <= 256) {
            tile_cfg = TILE_WV144;
            blk_px = 144;
        }
    }
    // the half view splits each 256-channel tile in two
    const int co_tiles = tile_cfg == TILE_STREAM_H128 ? 2 * h0.co_tiles : h0.co_tiles;
    int tiles = 0;
    for (int i = 0; i < count; ++i) {
        const qconv_seg_t &s = segs[i];
        if (s.n == 0)
            continue;
        MfmaSeg &m = a.seg[a.nseg++];
        m.x = (const uint8_t *)s.x;
        m.skip = s.skip;
        m.y = s.y;
        m.wt = (const int8_t *)s.conv->w_dev;
        m.epi = s.conv->epi_dev + (size_t)s.level * EPI_FIELDS * s.conv->cout_pad;
        m.P = (long long)s.n * chk[i].ho * chk[i].wo;
        m.n = s.n;
        m.h = s.h;
        m.w = s.w;
        m.ho = chk[i].ho;
        m.wo = chk[i].wo;
        m.hs = s.hs;
        m.ws = s.ws;
        m.tile_begin = tiles;
        m.fast = s.conv->fast[s.level];
        m.side0 = s.conv->side0[s.level];
        m.lut = s.conv->lut_dev ? s.conv->lut_dev + (size_t)s.level * s.conv->cout_pad * (1 << h0.d.skip_bits)
                                : nullptr;
        const long long px_tiles = (m.P + blk_px - 1) / blk_px;
        REQUIRE(tiles + px_tiles * co_tiles < (1LL << 26), "too many tiles for one launch");
        tiles += (int)(px_tiles * co_tiles);
    }
    a.total_tiles = tiles;
    a.tiles_per_xcd = (tiles + 7) / 8;
    a.ksplit = 1;
    a.kchunk = h0.ksteps;
    a.part = 0;
    a.cin = h0.d.cin;
    a.cout = h0.d.cout;
    a.cout_pad = h0.cout_pad;
    a.kh = h0.d.kh;
    a.kw = h0.d.kw;
    a.stride = h0.d.stride;
    a.pad = h0.d.pad;
    a.co_tiles = co_tiles;
    a.ksteps = h0.ksteps;
    a.up2 = h0.d.skip_up2;
    a.tile_cfg = tile_cfg;
    a.bits_out = h0.d.out_mode == AQD_OUT_INT32 ? 32 : h0.d.bits_out;
    a.qmax = h0.qmax;
    a.skip_bits = h0.d.skip_bits;
    a.zero = h0.zero;
    return AQD_OK;
}

// Split of the K range: the number of parts minimising a simple model of the
// MI355X (256 CUs, two workgroups per CU), fitted to measured launches: a
// workgroup alone on its CU takes ~0.65 us per K step, two sharing a CU
// ~0.84 us (0.42 each), plus ~3 us of prologue and epilogue per pair of
// workgroups; the parts cost one write and one read of nparts x P x cout
// int32 (~5 TB/s) and the combining launch (~5 us). A split is taken only
// when the model gains 20%.
void plan_split(const MfmaArgs &a, int *nparts, int *kchunk)
{
    if (a.tile_cfg == TILE_256x64S || a.tile_cfg == TILE_256x64 || a.tile_cfg == TILE_STREAM ||
        a.tile_cfg == TILE_STREAM_C128 || a.tile_cfg == TILE_STREAM_C64 || a.tile_cfg == TILE_128x128_O3 ||
        a.tile_cfg == TILE_64x256_O3 || a.tile_cfg == TILE_STREAM_H128 || a.tile_cfg == TILE_WV || a.tile_cfg == TILE_WV144 || a.tile_cfg == TILE_WV64 || a.tile_cfg == TILE_WVS ||
        a.tile_cfg == TILE_STEM) {  // never split
        *nparts = 1;
        *kchunk = a.ksteps;
        return;
    }
    long long P = 0;
    for (int i = 0; i < a.nseg; ++i)
        P += a.seg[i].P;
    // the FP4 path: half the MFMA time per 64-channel step, parts of whole
    // 256-channel stages (4 steps)
    const bool fp4 = a.tile_cfg == TILE_FP4, b8 = a.tile_cfg == TILE_B8;
    const double step_scale = fp4 ? 0.5 : 1.0;
    const int align = fp4 ? 4 : b8 ? 2 : 1;
    auto cost = [&](int parts, int chunk) {
        const double units = (double)a.total_tiles * parts;
        const double per_cu = std::ceil(units / 256.0);
        double t = step_scale * chunk * (per_cu <= 1 ? 0.65 : 0.42 * per_cu) + 3.0 * std::ceil(per_cu / 2.0);
        if (parts > 1)
            t += (double)parts * P * a.cout * 8.0 / 5e6 + 5.0;
        return t;
    };
    *nparts = 1;
    *kchunk = a.ksteps;
    double best = cost(1, a.ksteps);
    static const int cand[] = {2, 3, 4, 6, 8, 12, 16};
    for (int c : cand) {
        const int chunk = ((a.ksteps + c - 1) / c + align - 1) / align * align;
        if (chunk < 2 || ((fp4 || b8) && chunk >= a.ksteps))
            break;
        const int parts = (a.ksteps + chunk - 1) / chunk;  // every part non-empty
        const double t = cost(parts, chunk);
        if (t < 0.8 * best) {
            best = t;
            *nparts = parts;
            *kchunk = chunk;
        }
    }
}

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

size_t split_bytes(const MfmaArgs &a, int nparts)
{
    size_t b = 0;
    for (int i = 0; i < a.nseg; ++i)
        b += align256((size_t)nparts * a.seg[i].P * a.cout * 4);
    return b;
}

}  // namespace

extern "C" {

aqd_status_t qconv_group_workspace(int count, const qconv_seg_t *segs, size_t *bytes)
{
    REQUIRE(bytes, "null bytes");
    *bytes = 0;
    SegCheck chk[AQD_MAX_SEGS];
    MfmaArgs a;
    bool direct = false;
    aqd_status_t st = prepare_group(count, segs, chk, &a, &direct);
    if (st != AQD_OK || direct || a.nseg == 0)
        return st;
    int nparts = 1, kchunk = 0;
    plan_split(a, &nparts, &kchunk);
    if (nparts > 1)
        *bytes = split_bytes(a, nparts);
    return AQD_OK;
}

}  // extern "C"

// Scratch of qconv_run_group_static: the split-K partial sums of callers that
// cannot allocate. Every GPU the library runs on holds its own copy until the
// process ends; host code reaches it only through the per-device address from
// hipGetSymbolAddress (the array's name is a host-side stand-in).
static __device__ __align__(256) uint8_t scratch[AQD_STATIC_SCRATCH_BYTES];

namespace {

std::mutex g_scratch_mu;
void *g_scratch[64] = {};

// Device address of the current device's scratch, looked up once per device
// (with that device current); nullptr if the lookup fails.
void *static_scratch()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
        return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
            (void)hipGetLastError();
            return nullptr;
        }
        g_scratch[dev] = p;
    }
    return g_scratch[dev];
}

// A group launch; the split-K partial sums go to `workspace` (the caller's,
// ws_bytes long, or null: no split), or with use_static to this device's
// scratch array (no allocation).
aqd_status_t run_group(int count, const qconv_seg_t *segs, void *workspace, size_t ws_bytes,
                       bool use_static, hipStream_t stream)
{
    SegCheck chk[AQD_MAX_SEGS];
    MfmaArgs a;
    bool direct = false;
    aqd_status_t st = prepare_group(count, segs, chk, &a, &direct);
    if (st != AQD_OK)
        return st;
    if (direct) {
        for (int i = 0; i < count; ++i)
            if (segs[i].n > 0) {
                st = launch_direct(segs[i], chk[i], stream);
                if (st != AQD_OK)
                    return st;
            }
        return AQD_OK;
    }
    if (a.nseg == 0)
        return AQD_OK;
    const qconv_s &h0 = *segs[0].conv;
    int nparts = 1, kchunk = a.ksteps;
    if (use_static) {
        plan_split(a, &nparts, &kchunk);
        if (nparts > 1) {
            const size_t need = split_bytes(a, nparts);
            if (need > AQD_STATIC_SCRATCH_BYTES)
                return fail(AQD_ERR_UNSUPPORTED,
                            "this group's split K reduction needs " + std::to_string(need) +
                                " bytes of scratch, more than the " +
                                std::to_string((size_t)AQD_STATIC_SCRATCH_BYTES) +
                                " of the static scratch; use qconv_run_group_ws with a workspace");
            workspace = static_scratch();
            if (!workspace)
                return fail(AQD_ERR_DEVICE, "the address of the static scratch could not be found");
        }
    } else if (workspace) {
        REQUIRE(((uintptr_t)workspace & 255) == 0, "workspace must be 256-byte aligned");
        plan_split(a, &nparts, &kchunk);
        if (nparts > 1 && ws_bytes < split_bytes(a, nparts))
            nparts = 1;
    }
    if (nparts == 1) {
        if (launch_qconv_mfma(h0.d.bits_in, a, stream) != hipSuccess)
            return fail(AQD_ERR_DEVICE, "MFMA conv launch failed");
        return AQD_OK;
    }
    // part sums of every segment into its workspace slice, then the combining epilogue
    SplitArgs e{};
    e.nseg = a.nseg;
    e.nparts = nparts;
    e.cout = a.cout;
    e.cout_pad = a.cout_pad;
    e.bits_out = a.bits_out;
    e.qmax = a.qmax;
    e.skip_bits = a.skip_bits;
    e.up2 = a.up2;
    const int cpt = a.bits_out == 32 ? 4 : 32 / a.bits_out;
    uint8_t *ws = (uint8_t *)workspace;
    long long items = 0;
    for (int i = 0; i < a.nseg; ++i) {
        MfmaSeg &m = a.seg[i];
        SplitSeg &q = e.seg[i];
        q.part = (const int32_t *)ws;
        q.skip = m.skip;
        q.y = m.y;
        q.epi = m.epi;
        q.P = m.P;
        q.ho = m.ho;
        q.wo = m.wo;
        q.hs = m.hs;
        q.ws = m.ws;
        q.item_begin = items;
        items += m.P * (a.cout / cpt);
        m.y = ws;
        m.skip = nullptr;
        ws += align256((size_t)nparts * m.P * a.cout * 4);
    }
    e.total_items = items;
    a.part = 1;
    a.ksplit = nparts;
    a.kchunk = kchunk;
    a.total_tiles *= nparts;
    a.tiles_per_xcd = (a.total_tiles + 7) / 8;
    a.bits_out = 32;
    a.skip_bits = 0;
    a.up2 = 0;
    if (launch_qconv_mfma(h0.d.bits_in, a, stream) != hipSuccess)
        return fail(AQD_ERR_DEVICE, "MFMA conv launch failed");
    if (launch_splitk_epilogue(e, stream) != hipSuccess)
        return fail(AQD_ERR_DEVICE, "split-K epilogue launch failed");
    return AQD_OK;
}

}  // namespace

extern "C" {

aqd_status_t qconv_run_group_ws(int count, const qconv_seg_t *segs, void *workspace, size_t ws_bytes,
                                aqd_stream_t stream)
{
    return run_group(count, segs, workspace, ws_bytes, false, (hipStream_t)stream);
}

aqd_status_t qconv_run_group_static(int count, const qconv_seg_t *segs, aqd_stream_t stream)
{
    return run_group(count, segs, nullptr, 0, true, (hipStream_t)stream);
}

aqd_status_t qconv_run_group(int count, const qconv_seg_t *segs, aqd_stream_t stream)
{
    return run_group(count, segs, nullptr, 0, false, (hipStream_t)stream);
}

aqd_status_t qconv_run_proj(qconv_t conv, qconv_t proj, int level, int n, int h, int w,
                            const void *x, int hp, int wp, const void *xp, void *y,
                            aqd_stream_t stream_)
{
    REQUIRE(conv && proj, "null handle");
    const qconv_desc_t &d = conv->d, &e = proj->d;
    REQUIRE(level >= 0 && level < d.num_levels && level < e.num_levels, "level out of range");
    REQUIRE(n >= 0, "n must be >= 0");
    int ho = 0, wo = 0, hpo = 0, wpo = 0;
    aqd_status_t st = qconv_out_shape(conv, h, w, &ho, &wo);
    if (st != AQD_OK)
        return st;
    st = qconv_out_shape(proj, hp, wp, &hpo, &wpo);
    if (st != AQD_OK)
        return st;
    REQUIRE(hpo == ho && wpo == wo, "the projection's output size differs from the convolution's");
    REQUIRE((long long)n * ho * wo < (1LL << 31) && (long long)n * h * w < (1LL << 31) &&
                (long long)n * hp * wp < (1LL << 31),
            "too many pixels for one call");
    if (!(conv->mfma && proj->mfma && d.out_mode == AQD_OUT_CODES && d.skip_bits == 32 && !d.skip_up2 &&
          e.out_mode == AQD_OUT_INT32 && e.skip_bits == 0 && e.kh == 1 && e.kw == 1 && e.pad == 0 &&
          d.bits_in == 4 && e.bits_in == 4 && d.bits_out == 4 && d.cout == e.cout &&
          conv->tile_cfg == TILE_256x128 && proj->tile_cfg == TILE_256x128))
        return fail(AQD_ERR_UNSUPPORTED, "this pair of handles has no fused launch; run them separately");
    if (n == 0)
        return AQD_OK;
    REQUIRE(x && xp && y, "null tensor");
    REQUIRE(aligned16(x) && aligned16(xp) && aligned16(y), "tensors must be 16-byte aligned");
    const size_t xbytes = (size_t)n * h * w * d.cin * d.bits_in / 8;
    const size_t pbytes = (size_t)n * hp * wp * e.cin * e.bits_in / 8;
    const size_t ybytes = (size_t)n * ho * wo * d.cout * d.bits_out / 8;
    REQUIRE(!overlap(y, ybytes, x, xbytes) && !overlap(y, ybytes, xp, pbytes),
            "output overlaps an input");
    MfmaArgs a{};
    a.nseg = 1;
    MfmaSeg &m = a.seg[0];
    m.x = (const uint8_t *)x;
    m.skip = nullptr;
    m.y = y;
    m.wt = (const int8_t *)conv->w_dev;
    m.epi = conv->epi_dev + (size_t)level * EPI_FIELDS * conv->cout_pad;
    m.P = (long long)n * ho * wo;
    m.n = n;
    m.h = h;
    m.w = w;
    m.ho = ho;
    m.wo = wo;
    m.hs = ho;
    m.ws = wo;
    m.tile_begin = 0;
    m.fast = conv->fast[level];
    m.side0 = 0;
    m.x2 = (const uint8_t *)xp;
    m.wt2 = (const int8_t *)proj->w_dev;
    m.epi2 = proj->epi_dev + (size_t)level * EPI_FIELDS * proj->cout_pad;
    m.h2 = hp;
    m.w2 = wp;
    const long long tiles = (m.P + PROJ_BLK_PX - 1) / PROJ_BLK_PX * conv->co_tiles;
    REQUIRE(tiles < (1LL << 26), "too many tiles for one launch");
    a.total_tiles = (int)tiles;
    a.tiles_per_xcd = (a.total_tiles + 7) / 8;
    a.ksplit = 1;
    a.kchunk = conv->ksteps;
    a.part = 0;
    a.cin = d.cin;
    a.cout = d.cout;
    a.cout_pad = conv->cout_pad;
    a.kh = d.kh;
    a.kw = d.kw;
    a.stride = d.stride;
    a.pad = d.pad;
    a.co_tiles = conv->co_tiles;
    a.ksteps = conv->ksteps;
    a.up2 = 0;
    a.tile_cfg = conv->tile_cfg;
    a.bits_out = d.bits_out;
    a.qmax = conv->qmax;
    a.skip_bits = 32;
    a.zero = conv->zero;
    a.cin2 = e.cin;
    a.stride2 = e.stride;
    a.ksteps2 = proj->ksteps;
    // one K step each (cin 64): persistent streaming tiles (same 256 x 64 tiles)
    const bool stream_tiles = conv->ksteps == 1 && proj->ksteps == 1 && d.kh == 1 && d.kw == 1 &&
                              d.pad == 0 && d.cout % 256 == 0;
    // both inputs in 256-channel chunks (the main one may have 128 channels:
    // one padded stage), 1x1 stride 1: register-fed 256 x 64 tiles (32-bit
    // buffer offsets: inputs below 2^31 bytes)
    const bool wv_tiles = (d.cin % 256 == 0 || d.cin == 128) && e.cin % 256 == 0 && d.kh == 1 && d.kw == 1 && d.stride == 1 &&
                          d.pad == 0 && xbytes < (1ull << 31) && pbytes < (1ull << 31);
    hipError_t err;
    if (stream_tiles) {
        a.tile_cfg = TILE_STREAM;
        err = launch_qconv_mfma(4, a, (hipStream_t)stream_);
    } else if (wv_tiles) {
        a.tile_cfg = TILE_WV64;
        err = launch_qconv_wv_proj(a, (hipStream_t)stream_);
    } else {
        err = launch_qconv_proj(a, (hipStream_t)stream_);
    }
    if (err != hipSuccess)
        return fail(AQD_ERR_DEVICE, "fused projection launch failed");
    return AQD_OK;
}

aqd_status_t qconv_run(qconv_t conv, int level, int n, int h, int w, const void *x, const void *skip,
                       int hs, int ws, void *y, aqd_stream_t stream)
{
    qconv_seg_t s{conv, level, n, h, w, x, skip, hs, ws, y};
    return qconv_run_group(1, &s, stream);
}

aqd_status_t qadd_run(const qadd_desc_t *desc, const void *a, const void *b, void *y,
                      const qadd_params_t *p, aqd_stream_t stream)
{
    REQUIRE(desc && p, "null argument");
    qadd_desc_t d = *desc;
    REQUIRE(d.n >= 0 && d.h >= 1 && d.w >= 1 && d.c >= 1, "bad tensor shape");
    REQUIRE(code_bits(d.bits_a) || d.bits_a == 32, "bits_a must be 2, 3, 4, 8 or 32");
    REQUIRE(code_bits(d.bits_b) || d.bits_b == 32, "bits_b must be 2, 3, 4, 8 or 32");
    REQUIRE(code_bits(d.bits_out), "bits_out must be 2, 3, 4 or 8");
    const int qmax = (1 << d.bits_out) - 1;
    d.bits_a = stored_bits(d.bits_a);  // widths as stored from here on
    d.bits_b = stored_bits(d.bits_b);
    d.bits_out = stored_bits(d.bits_out);
    REQUIRE((d.c * d.bits_a) % 8 == 0 && (d.c * d.bits_b) % 8 == 0 && (d.c * d.bits_out) % 8 == 0,
            "c * bits must be a multiple of 8");
    if (d.up2)
        REQUIRE(d.up2 == 1 && (d.h - 1) / 2 < d.hb && (d.w - 1) / 2 < d.wb && d.hb >= 1 && d.wb >= 1,
                "upsampled operand too small");
    else
        REQUIRE(d.hb == d.h && d.wb == d.w, "operand sizes differ");
    REQUIRE((long long)d.n * d.h * d.w < (1LL << 31), "too many pixels for one call");
    if (d.n == 0)
        return AQD_OK;
    REQUIRE(a && b && y, "null tensor");
    REQUIRE(aligned16(a) && aligned16(b) && aligned16(y), "tensors must be 16-byte aligned");
    REQUIRE(p->skip_c && p->skip_d && p->skip_side && p->mult && p->shift, "null parameter array");
    const size_t ab = (size_t)d.n * d.h * d.w * d.c * d.bits_a / 8;
    const size_t bb = (size_t)d.n * d.hb * d.wb * d.c * d.bits_b / 8;
    const size_t yb = (size_t)d.n * d.h * d.w * d.c * d.bits_out / 8;
    REQUIRE(!overlap(y, yb, a, ab) && !overlap(y, yb, b, bb), "output overlaps an input");
    QaddArgs q{};
    q.a = a;
    q.b = b;
    q.y = (uint8_t *)y;
    q.skip_c = p->skip_c;
    q.skip_d = p->skip_d;
    q.skip_side = p->skip_side;
    q.mult = p->mult;
    q.shift = p->shift;
    q.n = d.n;
    q.h = d.h;
    q.w = d.w;
    q.c = d.c;
    q.hb = d.hb;
    q.wb = d.wb;
    q.bits_a = d.bits_a;
    q.bits_b = d.bits_b;
    q.bits_out = d.bits_out;
    q.qmax = qmax;
    q.up2 = d.up2;
    if (launch_qadd(q, (hipStream_t)stream) != hipSuccess)
        return fail(AQD_ERR_DEVICE, "qadd launch failed");
    return AQD_OK;
}

aqd_status_t aqd_channel_sums(const int32_t *v, int64_t rows, int c, int64_t *sums,
                              aqd_stream_t stream)
{
    REQUIRE(rows >= 0 && c >= 1, "bad shape");
    if (rows == 0)
        return AQD_OK;
    REQUIRE(v && sums, "null pointer");
    if (launch_channel_sums(v, rows, c, (long long *)sums, (hipStream_t)stream) != hipSuccess)
        return fail(AQD_ERR_DEVICE, "channel sums launch failed");
    return AQD_OK;
}

aqd_status_t aqd_mfma_probe(int workgroups, int iters, int32_t *out, aqd_stream_t stream)
{
    REQUIRE(workgroups >= 1 && workgroups <= (1 << 20) && iters >= 1, "workgroups in 1..2^20, iters >= 1");
    REQUIRE(out, "null pointer");
    if (launch_mfma_probe(workgroups, iters, out, (hipStream_t)stream) != hipSuccess)
        return fail(AQD_ERR_DEVICE, "probe launch failed");
    return AQD_OK;
}

aqd_status_t aqd_maxpool_run(const aqd_maxpool_desc_t *desc, const void *x, void *y,
                             aqd_stream_t stream)
{
    REQUIRE(desc, "null argument");
    aqd_maxpool_desc_t d = *desc;
    REQUIRE(d.n >= 0 && d.h >= 1 && d.w >= 1 && d.c >= 1, "bad tensor shape");
    REQUIRE(code_bits(d.bits), "bits must be 2, 3, 4 or 8");
    d.bits = stored_bits(d.bits);
    REQUIRE((d.c * d.bits) % 8 == 0, "c * bits must be a multiple of 8");
    REQUIRE(d.k >= 1 && d.k <= 7 && d.stride >= 1 && d.stride <= 4 && d.pad >= 0 && d.pad < d.k,
            "k must be in 1..7, stride in 1..4, pad in 0..k-1");
    const int ho = (d.h + 2 * d.pad - d.k) / d.stride + 1;
    const int wo = (d.w + 2 * d.pad - d.k) / d.stride + 1;
    REQUIRE(d.h + 2 * d.pad >= d.k && d.w + 2 * d.pad >= d.k && ho >= 1 && wo >= 1,
            "input smaller than the window");
    REQUIRE((long long)d.n * d.h * d.w < (1LL << 31), "too many pixels for one call");
    if (d.n == 0)
        return AQD_OK;
    REQUIRE(x && y, "null tensor");
    const size_t xb = (size_t)d.n * d.h * d.w * d.c * d.bits / 8;
    const size_t yb = (size_t)d.n * ho * wo * d.c * d.bits / 8;
    REQUIRE(!overlap(y, yb, x, xb), "output overlaps the input");
    PoolArgs a{};
    a.x = (const uint8_t *)x;
    a.y = (uint8_t *)y;
    a.n = d.n;
    a.h = d.h;
    a.w = d.w;
    a.c = d.c;
    a.bits = d.bits;
    a.k = d.k;
    a.stride = d.stride;
    a.pad = d.pad;
    a.ho = ho;
    a.wo = wo;
    if (launch_maxpool(a, (hipStream_t)stream) != hipSuccess)
        return fail(AQD_ERR_DEVICE, "max-pooling launch failed");
    return AQD_OK;
}

// ------------------------------------------------------------------ graph capture
aqd_status_t aqd_graph_begin(aqd_stream_t stream)
{
    REQUIRE(stream, "capture needs a stream other than the null stream");
    hipStreamCaptureStatus st = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing((hipStream_t)stream, &st) != hipSuccess)
        return fail(AQD_ERR_DEVICE, "stream query failed");
    REQUIRE(st == hipStreamCaptureStatusNone, "the stream is already capturing");
    if (hipStreamBeginCapture((hipStream_t)stream, hipStreamCaptureModeThreadLocal) != hipSuccess)
        return fail(AQD_ERR_DEVICE, "stream capture could not start");
    return AQD_OK;
}

aqd_status_t aqd_graph_end(aqd_stream_t stream, void **graph_exec)
{
    REQUIRE(stream && graph_exec, "null stream or output pointer");
    *graph_exec = nullptr;
    hipGraph_t g = nullptr;
    if (hipStreamEndCapture((hipStream_t)stream, &g) != hipSuccess || !g) {
        (void)hipGetLastError();
        return fail(AQD_ERR_DEVICE, "stream capture failed (an operation was not capturable)");
    }
    hipGraphExec_t e = nullptr;
    const hipError_t r = hipGraphInstantiate(&e, g, nullptr, nullptr, 0);
    (void)hipGraphDestroy(g);
    if (r != hipSuccess || !e)
        return fail(AQD_ERR_DEVICE, "graph instantiation failed");
    *graph_exec = (void *)e;
    return AQD_OK;
}

aqd_status_t aqd_graph_launch(void *graph_exec, aqd_stream_t stream)
{
    REQUIRE(graph_exec, "null graph");
    if (hipGraphLaunch((hipGraphExec_t)graph_exec, (hipStream_t)stream) != hipSuccess)
        return fail(AQD_ERR_DEVICE, "graph launch failed");
    return AQD_OK;
}

void aqd_graph_destroy(void *graph_exec)
{
    if (graph_exec)
        (void)hipGraphExecDestroy((hipGraphExec_t)graph_exec);
}

// ------------------------------------------------------------------ host helpers
aqd_status_t aqd_pack_codes(const uint8_t *codes, int64_t rows, int c, int bits, uint8_t *out)
{
    REQUIRE(codes && out && rows >= 0 && c >= 1 && code_bits(bits) && (c * stored_bits(bits)) % 8 == 0,
            "bad arguments");
    const int sb = stored_bits(bits);
    const int rb = c * sb / 8;
    const int mask = (1 << bits) - 1;
    for (int64_t r = 0; r < rows; ++r) {
        uint8_t *o = out + r * rb;
        std::memset(o, 0, rb);
        for (int ch = 0; ch < c; ++ch) {
            const int v = codes[r * c + ch];
            REQUIRE(v <= mask, "code out of range for the bitwidth");
            const int bit = ch * sb;
            o[bit >> 3] |= (uint8_t)(v << (bit & 7));
        }
    }
    return AQD_OK;
}

aqd_status_t aqd_unpack_codes(const uint8_t *packed, int64_t rows, int c, int bits, uint8_t *out)
{
    REQUIRE(packed && out && rows >= 0 && c >= 1 && code_bits(bits) && (c * stored_bits(bits)) % 8 == 0,
            "bad arguments");
    const int sb = stored_bits(bits);
    const int rb = c * sb / 8;
    for (int64_t r = 0; r < rows; ++r)
        for (int ch = 0; ch < c; ++ch) {
            const int bit = ch * sb;
            out[r * c + ch] = (packed[r * rb + (bit >> 3)] >> (bit & 7)) & ((1 << bits) - 1);
        }
    return AQD_OK;
}

aqd_status_t aqd_approx_ratio(double r, int32_t *c_out, int32_t *d_out)
{
    REQUIRE(c_out && d_out, "null argument");
    REQUIRE(std::isfinite(r) && r >= 1.0 && r < 1073741824.0, "ratio must be in [1, 2^30)");
    bool have = false;
    double best_err = 0.0;
    int32_t bc = 0, bd = 0;
    for (int d = 1; d <= 31; ++d) {
        const double x = std::ldexp(r, d);
        if (x + 0.5 >= 2147483648.0)
            break;
        const double c = std::floor(x + 0.5);
        const double err = std::fabs(r - std::ldexp(c, -d));
        if (!have || err < best_err) {
            have = true;
            best_err = err;
            bc = (int32_t)c;
            bd = d;
        }
    }
    *c_out = bc;
    *d_out = bd;
    return AQD_OK;
}

aqd_status_t aqd_normalize_multiplier(double r, int32_t *mult, int32_t *shift)
{
    REQUIRE(mult && shift, "null argument");
    REQUIRE(std::isfinite(r) && r != 0.0, "scale must be finite and non-zero");
    const double a = std::fabs(r);
    int e = 0;
    (void)std::frexp(a, &e);  // a = m * 2^e, m in [0.5, 1)
    int d = 31 - e;           // a * 2^d in [2^30, 2^31)
    double c = std::floor(std::ldexp(a, d) + 0.5);
    if (c == 2147483648.0) {
        c = 1073741824.0;
        d -= 1;
    }
    const int sh = d - 31;
    REQUIRE(sh >= -31 && sh <= 31, "scale out of range for the dyadic form");
    *mult = r < 0 ? -(int32_t)c : (int32_t)c;
    *shift = sh;
    return AQD_OK;
}

aqd_status_t aqd_bn_stats_from_sums(int cout, const int64_t *s1, const int64_t *s2, int64_t count,
                                    double alpha_conv, double *mean, double *var)
{
    REQUIRE(cout >= 1 && s1 && s2 && mean && var && count >= 1, "bad arguments");
    for (int i = 0; i < cout; ++i) {
        const double m = (double)s1[i] / (double)count;
        const double va = (double)s2[i] / (double)count - m * m;
        mean[i] = alpha_conv * m;
        var[i] = (alpha_conv * alpha_conv) * va;
    }
    return AQD_OK;
}

aqd_status_t aqd_fold_bn(int cout, const double *gamma, const double *beta, const double *mean,
                         const double *var, double eps, double alpha_conv, int32_t *bias,
                         double *alpha_z)
{
    REQUIRE(cout >= 1 && gamma && beta && mean && var && bias && alpha_z, "bad arguments");
    REQUIRE(std::isfinite(alpha_conv) && alpha_conv > 0.0, "alpha_conv must be positive");
    for (int i = 0; i < cout; ++i) {
        REQUIRE(gamma[i] != 0.0 && var[i] + eps > 0.0, "gamma must be non-zero and var + eps > 0");
        const double sd = std::sqrt(var[i] + eps);
        const double s = (beta[i] * sd / gamma[i] - mean[i]) / alpha_conv;
        const double rb = std::floor(s + 0.5);
        REQUIRE(rb > -2147483648.0 && rb < 2147483648.0, "folded bias outside int32");
        bias[i] = (int32_t)rb;
        alpha_z[i] = alpha_conv * gamma[i] / sd;
    }
    return AQD_OK;
}

aqd_status_t aqd_skip_params(int cout, const double *alpha_z, const double *alpha_k,
                             int alpha_k_per_channel, int32_t *c, int32_t *d, int32_t *side,
                             double *scale)
{
    REQUIRE(cout >= 1 && alpha_z && alpha_k && c && d && side && scale, "bad arguments");
    for (int i = 0; i < cout; ++i) {
        const double az = alpha_z[i];
        const double ak = alpha_k_per_channel ? alpha_k[i] : alpha_k[0];
        REQUIRE(std::isfinite(az) && std::isfinite(ak) && az != 0.0 && ak != 0.0,
                "scales must be finite and non-zero");
        // opposite signs (a normalisation with gamma < 0): the numerator is negated
        const bool neg = (az < 0.0) != (ak < 0.0);
        aqd_status_t st;
        if (std::fabs(ak) >= std::fabs(az)) {
            st = aqd_approx_ratio(std::fabs(ak / az), &c[i], &d[i]);
            side[i] = 0;
            scale[i] = az;
        } else {
            st = aqd_approx_ratio(std::fabs(az / ak), &c[i], &d[i]);
            side[i] = 1;
            scale[i] = ak;
        }
        if (st != AQD_OK)
            return st;
        if (neg)
            c[i] = -c[i];
    }
    return AQD_OK;
}

aqd_status_t aqd_requant_params(int cout, const double *scale, double alpha_out, int32_t *mult,
                                int32_t *shift)
{
    REQUIRE(cout >= 1 && scale && mult && shift, "bad arguments");
    REQUIRE(std::isfinite(alpha_out) && alpha_out > 0.0, "alpha_out must be positive");
    for (int i = 0; i < cout; ++i) {
        aqd_status_t st = aqd_normalize_multiplier(scale[i] / alpha_out, &mult[i], &shift[i]);
        if (st != AQD_OK)
            return st;
    }
    return AQD_OK;
}

}  // extern "C"
