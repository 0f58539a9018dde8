// The 7x7 stride-2 input convolution (ResNet-50 stem) of the paper's fully
// quantized networks (Sec. 4: input and output layers at 8 bits): 8-bit codes
// of a 3-channel image, 8-bit two's-complement weights, on the int8 MFMA
// (v_mfma_i32_16x16x64_i8). GEMM view of Eq. 4 (Sec. 3.2.1): rows = output
// channels, columns = output pixels, K = the 7 x 7 x 3 window.
//
// With three input channels a K step cannot be a tap's channels, so the K
// axis is the whole window, laid out as 7 window rows of 24 bytes (7 taps x
// 3 channels and 3 bytes whose weights are zero) and padded to 192 = 3 K
// steps. A workgroup gathers the windows of its 128 output pixels into LDS
// (two threads per pixel, window rows 0-3 and 4-6: per window row 7 aligned
// dwords of the image row, shifted into place), re-centred as a - 128 like
// the other 8-bit path (the bias folded at create carries 128 * sum(w)); the
// weights of its 64 output channels stay in registers. Taps outside the image
// are code 0 (-128 after re-centring, as the correction assumes). Small
// workgroups (32 KiB of LDS, four to a CU) overlap one's gather with
// another's MFMAs and stores.
//
// Tile 64 channels x 128 pixels, 4 waves, wave w owning pixels 32w .. 32w+31
// (2 column tiles) and all 64 channels (4 accumulator tiles); lane group g
// holds channels 16g .. 16g+15 of a pixel (rows permuted at create), so the
// epilogue packs them into one 8-byte store of 4-bit codes or four 16-byte
// stores of int32.

#include "epilogue.h"
#include "internal.h"
#include "mfma_common.h"

namespace aqd {
namespace {

constexpr int ST_BCO = 64;      // channels per workgroup tile
constexpr int ST_BPX = 128;     // pixels per workgroup tile
constexpr int ST_ROW = 256;     // LDS bytes per pixel (192 used), 16-byte columns XOR-swizzled
constexpr int ST_KW = 24;       // K bytes per window row
constexpr int ST_K = 192;       // K bytes per window (7 x 24, padded to 3 K steps)

// OUTK: 0 = 4-bit codes, 1 = int32 (v = acc + bias); FAST: every shift >= 2
template <int OUTK, int FAST>
__global__ void __launch_bounds__(256, 4) qconv_stem_kernel(MfmaArgs A)
{
    constexpr int MI = 4, NJ = 2, QMAX = 15;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[ST_BPX * ST_ROW];

    const int bid = blockIdx.x;
    const int tile = (bid & 7) * A.tiles_per_xcd + (bid >> 3);
    if (tile >= A.total_tiles)
        return;
    int s = 0;
#pragma unroll
    for (int i = 1; i < AQD_MAX_SEGS; ++i)
        if (i < A.nseg && tile >= A.seg[i].tile_begin)
            s = i;
    const MfmaSeg &S = A.seg[s];
    const int t_in_seg = tile - S.tile_begin;
    const int co_tile = t_in_seg % A.co_tiles;
    const int px_tile = t_in_seg / A.co_tiles;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane & 15, g = lane >> 4;

    // ---- weights of the tile's 64 channels: accumulator tile i, K step q
    // (row r, 16-byte column g), from [co_tile][K step][64 rows][64 B]
    v4i fa[3][MI];
#pragma unroll
    for (int q = 0; q < 3; ++q)
#pragma unroll
        for (int i = 0; i < MI; ++i)
            fa[q][i] = *(const v4i *)(S.wt + (((long long)co_tile * 3 + q) * ST_BCO + 16 * i + r) * KC + 16 * g);

    // ---- gather: threads 2t and 2t + 1 build window rows 0-3 and 4-6 of
    // pixel px_tile * 128 + t (byte offsets in 32 bits: the image has fewer
    // than 2^31 bytes, checked on the host)
    {
        const int pl = tid >> 1, half = tid & 1;
        const int total = S.n * S.h * S.w * 3;      // image bytes (>= 147)
        const unsigned p = (unsigned)(px_tile * ST_BPX + pl);
        const bool ok = p < (unsigned)S.P;
        const unsigned hw = (unsigned)(S.ho * S.wo);
        const unsigned pn = ok ? p / hw : 0u;
        const unsigned prem = ok ? p - pn * hw : 0u;
        const int oh = (int)(prem / (unsigned)S.wo), ow = (int)(prem - (prem / (unsigned)S.wo) * S.wo);
        const int ih0 = oh * 2 - 3, iw0 = ow * 2 - 3;
        // valid bytes of a window row: taps kw in [kw0, kw1), bytes [3 kw0, 3 kw1);
        // bytes 21-23 meet zero weights, so an interior window needs no mask
        const int kw0 = max(0, -iw0), kw1 = min(7, S.w - iw0);
        uint32_t cmask[6] = {~0u, ~0u, ~0u, ~0u, ~0u, ~0u};
        if (!ok || kw0 > 0 || kw1 < 7) {
#pragma unroll
            for (int d = 0; d < 6; ++d) {
                const int lo = min(max(3 * kw0 - 4 * d, 0), 4), hi = min(max(3 * kw1 - 4 * d, 0), 4);
                const uint32_t below_hi = hi >= 4 ? ~0u : (1u << (8 * hi)) - 1u;
                const uint32_t from_lo = lo >= 4 ? 0u : ~0u << (8 * lo);
                cmask[d] = ok ? (below_hi & from_lo) : 0u;
            }
        }
        uint8_t *row = lds + pl * ST_ROW;
        auto put = [&](int d, uint32_t v) {  // dword d of the window (K bytes 4d .. 4d+3)
            *(uint32_t *)(row + 16 * ((d >> 2) ^ (pl & 7)) + 4 * (d & 3)) = v ^ 0x80808080u;
        };
        const int img0 = (int)pn * S.h;
#pragma unroll
        for (int kr = 0; kr < 4; ++kr) {
            const int kh = 4 * half + kr;
            if (kh >= 7)
                break;
            const int ih = ih0 + kh;
            const bool rin = ok && (unsigned)ih < (unsigned)S.h;
            // bytes [b, b + 24) of the image hold the window row (21 bytes used)
            const int b = ((img0 + ih) * S.w + iw0) * 3;
            const int a0 = b & ~3;
            const int sh = b - a0;
            uint32_t w[7] = {0, 0, 0, 0, 0, 0, 0};
            if (!rin) {
                // a window row above or below the image: padding
            } else if (a0 >= 0 && a0 + 28 <= total) {
                // the whole row segment lies inside the image (every window
                // row but those touching the image's first or last bytes):
                // seven loads, issued back to back
#pragma unroll
                for (int d = 0; d < 7; ++d)
                    w[d] = *(const uint32_t *)(S.x + a0 + 4 * d);
            } else {
                // near either end of the image: the bytes inside, one by one
#pragma unroll
                for (int d = 0; d < 7; ++d) {
                    uint32_t v = 0;
                    for (int bb = 0; bb < 4; ++bb) {
                        const int at = a0 + 4 * d + bb;
                        if (at >= 0 && at < total)
                            v |= (uint32_t)S.x[at] << (8 * bb);
                    }
                    w[d] = v;
                }
            }
#pragma unroll
            for (int d = 0; d < 6; ++d) {
                const uint32_t v = (uint32_t)(((uint64_t)w[d + 1] << 32 | w[d]) >> (8 * sh));
                put(6 * kh + d, v & cmask[d]);
            }
        }
        if (half)
#pragma unroll
            for (int d = 42; d < ST_K / 4; ++d)
                put(d, 0);  // K positions 168 .. 191: zero weights
    }
    __syncthreads();

    // ---- MFMAs: 3 K steps x 2 column tiles x 4 accumulator tiles
    v4i acc[MI][NJ];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
            acc[i][j] = v4i{0, 0, 0, 0};
#pragma unroll
    for (int q = 0; q < 3; ++q)
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int p = 32 * wave + 16 * j + r;
            const v4i b = *(const v4i *)(lds + p * ST_ROW + 16 * ((4 * q + g) ^ (p & 7)));
#pragma unroll
            for (int i = 0; i < MI; ++i)
                acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[q][i], b, acc[i][j], 0, 0, 0);
        }

    // ---- epilogue: lane group g holds channels 16g + 4i + e of pixel 16j + r
    // of its wave's 32 pixels; per channel group i its table entries are read
    // once for both pixels
    const int co_glob = co_tile * ST_BCO + 16 * g;
    const int32_t *epi = S.epi;
    const int cp = A.cout_pad;
    long long px[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j)
        px[j] = (long long)px_tile * ST_BPX + 32 * wave + 16 * j + r;
    if constexpr (OUTK == 1) {
#pragma unroll
        for (int i = 0; i < MI; ++i) {
            const v4i bias = *(const v4i *)(epi + EPI_BIAS * cp + co_glob + 4 * i);
#pragma unroll
            for (int j = 0; j < NJ; ++j)
                if (px[j] < S.P)
                    *(v4i *)((int32_t *)S.y + px[j] * A.cout + co_glob + 4 * i) = acc[i][j] + bias;
        }
    } else {
        uint32_t out[NJ][2] = {};
#pragma unroll
        for (int i = 0; i < MI; ++i) {
            const int c = co_glob + 4 * i;
            const v4i bias = *(const v4i *)(epi + EPI_BIAS * cp + c);
            const v4i mult = *(const v4i *)(epi + EPI_MULT * cp + c);
            const v4i shf = *(const v4i *)(epi + (FAST ? EPI_SHR : EPI_SHIFT) * cp + c);
            const v4i rnd = *(const v4i *)(epi + EPI_RND * cp + c);
#pragma unroll
            for (int j = 0; j < NJ; ++j)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int v = acc[i][j][e] + bias[e];
                    int y;
                    if constexpr (FAST) {
                        y = requant32(v, mult[e], (long long)rnd[e] << 32, shf[e]);
                        y = y < 0 ? 0 : (y > QMAX ? QMAX : y);
                    } else {
                        y = (int)requant_clamp(v, mult[e], shf[e], QMAX);
                        asm volatile("" : "+v"(y));  // one 64-bit product alive at a time
                    }
                    const int bit = 4 * (4 * i + e);
                    out[j][bit >> 5] |= (uint32_t)y << (bit & 31);
                }
        }
#pragma unroll
        for (int j = 0; j < NJ; ++j)
            if (px[j] < S.P)
                *(uint2 *)((uint8_t *)S.y + px[j] * (A.cout / 2) + co_glob / 2) = make_uint2(out[j][0], out[j][1]);
    }
}

}  // namespace

hipError_t launch_qconv_stem(const MfmaArgs &a, hipStream_t stream)
{
    for (int i = 0; i < a.nseg; ++i)
        if ((long long)a.seg[i].n * a.seg[i].h * a.seg[i].w * 3 >= (1LL << 31))
            return hipErrorInvalidValue;   // byte offsets of the image in 32 bits
    if (a.cin != 3 || a.kh != 7 || a.kw != 7 || a.stride != 2 || a.pad != 3 || a.skip_bits != 0 ||
        (a.bits_out != 4 && a.bits_out != 32) || a.cout % ST_BCO != 0 || a.co_tiles * ST_BCO != a.cout ||
        a.ksplit != 1 || a.part != 0)
        return hipErrorInvalidValue;
    dim3 grid(8 * a.tiles_per_xcd), block(256);
    bool fast = true;
    for (int i = 0; i < a.nseg; ++i)
        fast = fast && a.seg[i].fast;
    if (a.bits_out == 32)
        hipLaunchKernelGGL((qconv_stem_kernel<1, 1>), grid, block, 0, stream, a);
    else if (fast)
        hipLaunchKernelGGL((qconv_stem_kernel<0, 1>), grid, block, 0, stream, a);
    else
        hipLaunchKernelGGL((qconv_stem_kernel<0, 0>), grid, block, 0, stream, a);
    return hipGetLastError();
}

}  // namespace aqd
