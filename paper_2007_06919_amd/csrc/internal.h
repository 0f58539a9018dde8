// Internal interface between the C-ABI host code and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "aqd.h"

namespace aqd {

// ---- implicit-GEMM MFMA kernel (qconv_mfma.hip) ----------------------------
// Output tile of one workgroup: BLK_CO output channels x BLK_PX output pixels;
// one K step is KC input channels of one filter tap.
constexpr int BLK_CO = 128;
constexpr int BLK_PX = 256;
constexpr int KC = 64;

struct MfmaSeg {
    const uint8_t *x;    // [n][h][w][cin] codes
    const void *skip;    // [n][hs][ws][cout] or null
    void *y;             // [n][ho][wo][cout]
    const int8_t *wt;    // weight tiles [co_tiles][ksteps][BLK_CO][KC]
    const int32_t *epi;  // epilogue table [6][cout_pad] of this segment's level
    long long P;         // n * ho * wo
    int n, h, w, ho, wo, hs, ws;
    int tile_begin;      // first workgroup tile of this segment
};

struct MfmaArgs {
    MfmaSeg seg[AQD_MAX_SEGS];
    int nseg;
    int total_tiles;
    int tiles_per_xcd;   // grid = 8 * tiles_per_xcd workgroups
    int cin, cout, cout_pad;
    int kh, kw, stride, pad;
    int co_tiles, ksteps;
    int up2;
};

// bits_in in {2, 4}; out_bits in {2, 4, 8} or 32 (int32 output); skip_bits in {0, 2, 4, 8, 32}
hipError_t launch_qconv_mfma(int bits_in, int out_bits, int skip_bits, const MfmaArgs &a,
                             hipStream_t stream);

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
};
hipError_t launch_qconv_direct(const DirectArgs &a, hipStream_t stream);

// ---- standalone add (qadd.hip) ----------------------------------------------
struct QaddArgs {
    const void *a, *b;
    uint8_t *y;
    const int32_t *skip_c, *skip_d, *skip_side, *mult, *shift;
    int n, h, w, c, hb, wb;
    int bits_a, bits_b, bits_out, up2;
};
hipError_t launch_qadd(const QaddArgs &a, hipStream_t stream);

// ---- per-channel sums (qadd.hip) ----------------------------------------------
hipError_t launch_channel_sums(const int32_t *v, long long rows, int c, long long *sums,
                               hipStream_t stream);

}  // namespace aqd
