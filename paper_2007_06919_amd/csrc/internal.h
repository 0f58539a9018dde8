// Internal interface between the C-ABI host code and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "aqd.h"

namespace aqd {

// ---- implicit-GEMM MFMA kernel (qconv_mfma.hip) ----------------------------
// One K step is KC input channels of one filter tap. Workgroup tile shapes
// (output channels x output pixels), chosen per handle from cout:
enum { TILE_256x128 = 0, TILE_128x256 = 1, TILE_64x512 = 2,
       // launch-time choices for handles laid out for 256x128 (same weight layout):
       TILE_256x64S = 3,   // short K, code outputs: three workgroups per CU
       TILE_256x64 = 4,    // launches with too few 256x128 tiles to fill the GPU
       TILE_STREAM = 5,    // 1x1, cin <= 128, code outputs: persistent 256 x 64 tiles
       // 1x1, cin <= 256, code outputs, no skip, for handles laid out for 128-
       // and 64-channel tiles: persistent 128 x 64 and 64 x 128 tiles
       TILE_STREAM_C128 = 6, TILE_STREAM_C64 = 7,
       // half-width pixel tiles, three workgroups per CU, on 128/64-channel handles
       TILE_128x128_O3 = 8, TILE_64x256_O3 = 9,
       // 1x1, 3-4 K steps, code outputs, no skip or a code skip, on handles laid
       // out for 256-channel tiles: persistent 128 x 64 tiles reading each
       // 256-row weight tile as two halves
       TILE_STREAM_H128 = 10,
       // cin a multiple of 256, code outputs: 256 x 128 tiles with the weights
       // read into registers (qconv_wv.hip), same weight layout as 256x128
       TILE_WV = 11,
       // 2-bit codes and 2-bit weights, cin and cout multiples of 256: 256 x 128
       // tiles on the scaled FP4 MFMA (qconv_b16.hip), weights stored as e2m1
       // nibbles at create (64 bytes per row and 128-channel K step)
       TILE_FP4 = 12,
       // 8-bit codes, cin a multiple of 128, int32 outputs: 256 x 128 tiles on
       // the int8 MFMA (qconv_b16.hip), weights in channel order at create
       TILE_B8 = 13,
       // the 7x7 stride-2 stem on a 3-channel 8-bit image: 64 x 128 tiles, K =
       // the whole window (qconv_stem.hip)
       TILE_STEM = 14,
       // TILE_WV's kernel on 256 x 144 tiles, one workgroup per CU: code
       // outputs of launches a little above one round of 256 x 128 tiles
       TILE_WV144 = 15,
       // TILE_WV's kernel on 256 x 64 tiles, three workgroups per CU: code
       // outputs with at most 8 K steps
       TILE_WV64 = 16,
       // 1x1, cin 256, 4-bit code outputs, cout a multiple of 256, one
       // segment: weight-stationary persistent 256 x 64 tiles (qconv_wvs.hip)
       TILE_WVS = 17 };
constexpr int KC = 64;

// tile shape of a configuration, and the channels one lane holds per pixel
void mfma_tile_shape(int tile_cfg, int *blk_co, int *blk_px, int *chan_per_lane);

// Epilogue table of one level: EPI_FIELDS arrays of cout_pad int32.
enum {
    EPI_BIAS = 0, EPI_MULT = 1, EPI_SHIFT = 2,            // v = acc + bias; requant M / 2^(31+shift)
    EPI_SKIP_C = 3, EPI_SKIP_D = 4, EPI_SKIP_SIDE = 5,    // Eq. 7-8 alignment
    EPI_SHR = 6, EPI_RND = 7,                             // shift - 1 and 2^(shift-2) (shift >= 2)
    EPI_FIELDS = 8
};

struct MfmaSeg {
    const uint8_t *x;    // [n][h][w][cin] codes
    const void *skip;    // [n][hs][ws][cout] or null
    void *y;             // [n][ho][wo][cout]
    const int8_t *wt;    // weight tiles [co_tiles][ksteps][blk_co][KC]
    const int32_t *epi;  // epilogue table [EPI_FIELDS][cout_pad] of this segment's level
    long long P;         // n * ho * wo
    int n, h, w, ho, wo, hs, ws;
    int tile_begin;      // first workgroup tile of this segment
    int fast;            // every shift of the level >= 2: 32-bit requantisation
    int side0;           // every skip side of the level is 0 (code skips use a table)
    const int32_t *lut;  // code skips: [cout_pad][2^bits] RSM(k, c, d) of the level
    // projection shortcut (fused launch only): 1x1 conv of x2 whose int32 output is the skip
    const uint8_t *x2;   // [n][h2][w2][cin2] codes
    const int8_t *wt2;   // its weight tiles (same tile layout)
    const int32_t *epi2; // its epilogue table (bias)
    int h2, w2;
};

struct MfmaArgs {
    MfmaSeg seg[AQD_MAX_SEGS];
    int nseg;
    int total_tiles;     // work units: output tiles x ksplit
    int tiles_per_xcd;   // grid = 8 * tiles_per_xcd workgroups
    int ksplit;          // parts of the K range per output tile (1: no split)
    int kchunk;          // K steps per part (the last part may have fewer)
    int part;            // 1: write int32 partial sums (part 0 with the bias) to y + part * P * cout
    int tile_cfg;
    int cin, cout, cout_pad;
    int kh, kw, stride, pad;
    int co_tiles, ksteps;
    int bits_out;        // 2, 4, 8 or 32 (int32 output), as stored
    int qmax;            // largest output code (7 for 3-bit codes in 4-bit containers)
    int skip_bits;       // 0, 2, 4, 8 or 32
    int up2;
    const uint8_t *zero; // >= 16 zero bytes in device memory (source of padding taps)
    int cin2, stride2, ksteps2;  // projection shortcut (fused launch only)
};

// bits_in in {2, 4}, or 8 with TILE_B8
hipError_t launch_qconv_mfma(int bits_in, const MfmaArgs &a, hipStream_t stream);
// fused projection shortcut (4-bit, 256 x 64 tiles): tile counts use blk_px = 64
constexpr int PROJ_BLK_PX = 64;
hipError_t launch_qconv_proj(const MfmaArgs &a, hipStream_t stream);
// the matrix-core rate probe (mfma_probe.hip): workgroups x 4 waves x iters
// x 16 MFMAs of 16x16x64 int8; out: workgroups x 256 ints
hipError_t launch_mfma_probe(int workgroups, int iters, int *out, hipStream_t stream);
// TILE_WVS launches (qconv_wvs.hip)
hipError_t launch_qconv_wvs(const MfmaArgs &a, hipStream_t stream);
// TILE_WV launches (qconv_wv.hip)
hipError_t launch_qconv_wv(const MfmaArgs &a, hipStream_t stream);
// fused projection shortcut, both 1x1 with cin and cin2 multiples of 256, on
// TILE_WV64's 256 x 64 tiles (qconv_wv.hip)
hipError_t launch_qconv_wv_proj(const MfmaArgs &a, hipStream_t stream);
// TILE_FP4 (code_bits 2) and TILE_B8 (code_bits 8) launches (qconv_b16.hip);
// a.ksteps and a.kchunk in 64-channel steps, multiples of a stage (4 and 2)
hipError_t launch_qconv_b16(int code_bits, const MfmaArgs &a, hipStream_t stream);
// TILE_STEM launches (qconv_stem.hip); weights [co_tile][3][64 rows][64 B]
hipError_t launch_qconv_stem(const MfmaArgs &a, hipStream_t stream);

// ---- split-K combine + epilogue (qconv_splitk.hip) ---------------------------
struct SplitSeg {
    const int32_t *part;  // [nparts][P][cout] int32 partial sums
    const void *skip;     // as MfmaSeg
    void *y;
    const int32_t *epi;   // [EPI_FIELDS][cout_pad]
    long long P;
    int ho, wo, hs, ws;
    long long item_begin; // first work item (pixel x channel group) of this segment
};
struct SplitArgs {
    SplitSeg seg[AQD_MAX_SEGS];
    int nseg;
    long long total_items;
    int nparts, cout, cout_pad;
    int bits_out, skip_bits, up2;  // bits_out 32: int32 output
    int qmax;                      // largest output code
};
hipError_t launch_splitk_epilogue(const SplitArgs &a, hipStream_t stream);

// ---- direct kernel (qconv_direct.hip): any shape the ABI allows -------------
struct DirectArgs {
    const uint8_t *x;
    const void *skip;
    void *y;
    const int16_t *wt;   // [cout][kh][kw][cin] decoded values
    const int32_t *epi;  // [6][cout]
    int n, h, w, ho, wo, hs, ws;
    int cin, cout, kh, kw, stride, pad;
    int bits_in, out_bits, skip_bits, up2;
    int qmax;  // largest output code
};
hipError_t launch_qconv_direct(const DirectArgs &a, hipStream_t stream);

// ---- standalone add (qadd.hip) ----------------------------------------------
struct QaddArgs {
    const void *a, *b;
    uint8_t *y;
    const int32_t *skip_c, *skip_d, *skip_side, *mult, *shift;
    int n, h, w, c, hb, wb;
    int bits_a, bits_b, bits_out, up2;
    int qmax;  // largest output code
};
hipError_t launch_qadd(const QaddArgs &a, hipStream_t stream);

// ---- max-pooling (qpool.hip) --------------------------------------------------
struct PoolArgs {
    const uint8_t *x;
    uint8_t *y;
    int n, h, w, c, bits, k, stride, pad, ho, wo;
};
hipError_t launch_maxpool(const PoolArgs &a, hipStream_t stream);

// ---- per-channel sums (qadd.hip) ----------------------------------------------
hipError_t launch_channel_sums(const int32_t *v, long long rows, int c, long long *sums,
                               hipStream_t stream);

}  // namespace aqd
