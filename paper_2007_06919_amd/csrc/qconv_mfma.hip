// Implicit-GEMM integer convolution on the gfx950 int8 MFMA
// (v_mfma_i32_16x16x64_i8), with the integer epilogue fused.
//
// GEMM view of a convolution (Sec. 3.2.1, Eq. 4): rows = output channels
// (weights, operand A), columns = output pixels n*ho*wo (operand B, gathered
// from the NHWC input per filter tap), K = taps x input channels.
//
// Workgroup: 256 threads = 4 waves in a 2 x 2 arrangement; tile 128 channels
// x 256 pixels; each wave owns 64 channels x 128 pixels = 4 x 8 MFMA tiles of
// 16 x 16 (128 int32 accumulators per lane). One K step = 64 input channels
// of one tap, double-buffered in LDS.
//
// Operand staging:
//  * activations: each thread loads one pixel's 64 packed b-bit codes
//    (32 B at 4 bit, 16 B at 2 bit) with 16-byte loads, widens them to int8
//    with mask/shift word operations and writes one 64-byte LDS row. The
//    widening leaves the codes in a fixed permutation sigma of the 64
//    channels; the weights were stored in the same permutation at create,
//    so every MFMA dot product is unchanged.
//  * weights: int8 tiles prepared at create ([co_tile][k step][128][64]);
//    each thread copies 32 B into LDS.
//  LDS rows are 80 B apart (64 B + 16 B pad), which spreads the 16-byte
//  reads of 16 consecutive rows over distinct banks.
//
// Epilogue: the weight rows of each 64-channel wave slice were permuted at
// create so that lane group g (lanes 16g..16g+15) of a 16 x 16 accumulator
// tile i holds channels 16g + 4i + e (e = 0..3): each lane ends with 16
// consecutive channels of one pixel per column tile and packs their b-bit
// codes into one 4/8/16-byte store without cross-lane traffic.
//
// Workgroup order: consecutive workgroup ids are dispatched round-robin over
// the 8 XCDs; ids are remapped so that each XCD receives a contiguous range
// of tiles (neighbouring pixel tiles of all channel tiles), which keeps the
// gathered input rows and the weights in that XCD's L2.

#include "epilogue.h"
#include "internal.h"

namespace aqd {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int NT = 256;
constexpr int LDS_ROW = 80;
constexpr int A_STAGE = BLK_CO * LDS_ROW;            // 10 KiB
constexpr int B_STAGE = BLK_PX * LDS_ROW;            // 20 KiB
constexpr int PRM_OFF = 2 * (A_STAGE + B_STAGE);     // parameter table after both stages
constexpr int LDS_BYTES = PRM_OFF + 6 * BLK_CO * 4;  // 64512 B

template <int BI, int BO, int SK>
__global__ void __launch_bounds__(NT, 2) qconv_mfma_kernel(MfmaArgs A)
{
    __shared__ __attribute__((aligned(16))) uint8_t lds[LDS_BYTES];

    const int bid = blockIdx.x;
    const int logical = (bid & 7) * A.tiles_per_xcd + (bid >> 3);
    if (logical >= A.total_tiles)
        return;

    // segment of this tile (uniform over the workgroup)
    int s = 0;
#pragma unroll
    for (int i = 1; i < AQD_MAX_SEGS; ++i)
        if (i < A.nseg && logical >= A.seg[i].tile_begin)
            s = i;
    const MfmaSeg &S = A.seg[s];
    const int t_in_seg = logical - S.tile_begin;
    const int co_tile = t_in_seg % A.co_tiles;
    const int px_tile = t_in_seg / A.co_tiles;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wc = wave >> 1;  // channel half of the tile
    const int wp = wave & 1;   // pixel half of the tile

    constexpr int CHUNK = KC * BI / 8;  // packed bytes of one K step per pixel
    const int row_bytes = A.cin * BI / 8;
    const int kpt = A.cin / KC;         // K steps per tap
    const int KS = A.ksteps;

    // pixel gathered by this thread
    const long long p = (long long)px_tile * BLK_PX + tid;
    const bool pvalid = p < S.P;
    const int hw = S.ho * S.wo;
    const int pn = pvalid ? (int)(p / hw) : 0;
    const int prem = pvalid ? (int)(p - (long long)pn * hw) : 0;
    const int poh = prem / S.wo;
    const int pow_ = prem - poh * S.wo;
    const int ih0 = poh * A.stride - A.pad;
    const int iw0 = pow_ * A.stride - A.pad;
    const uint8_t *xn = S.x + (long long)pn * S.h * S.w * row_bytes;

    const int8_t *wtile = S.wt + (long long)co_tile * KS * (BLK_CO * KC);

    // epilogue parameters of this channel tile -> LDS
    {
        int32_t *prm = (int32_t *)(lds + PRM_OFF);
        constexpr int NP = (BO == 32) ? 1 : (SK ? 6 : 3);
        for (int i = tid; i < NP * BLK_CO; i += NT) {
            int which = i / BLK_CO, c = i - which * BLK_CO;
            prm[which * BLK_CO + c] = S.epi[which * A.cout_pad + co_tile * BLK_CO + c];
        }
    }

    uint4 breg[CHUNK / 16];
    uint4 areg[2];

    auto load_b = [&](int ks) {
        int tap = ks / kpt;
        int cc = ks - tap * kpt;
        int r = tap / A.kw;
        int q = tap - r * A.kw;
        int ih = ih0 + r, iw = iw0 + q;
        bool ok = pvalid && (unsigned)ih < (unsigned)S.h && (unsigned)iw < (unsigned)S.w;
        if (ok) {
            const uint4 *src = (const uint4 *)(xn + ((long long)ih * S.w + iw) * row_bytes + cc * CHUNK);
#pragma unroll
            for (int u = 0; u < CHUNK / 16; ++u)
                breg[u] = src[u];
        } else {
#pragma unroll
            for (int u = 0; u < CHUNK / 16; ++u)
                breg[u] = make_uint4(0, 0, 0, 0);
        }
    };
    auto store_b = [&](int stage) {
        uint8_t *dst = lds + 2 * A_STAGE + stage * B_STAGE + tid * LDS_ROW;
        uint32_t in[CHUNK / 4];
#pragma unroll
        for (int u = 0; u < CHUNK / 16; ++u) {
            in[4 * u + 0] = breg[u].x;
            in[4 * u + 1] = breg[u].y;
            in[4 * u + 2] = breg[u].z;
            in[4 * u + 3] = breg[u].w;
        }
        uint32_t o[16];
        if constexpr (BI == 4) {
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                o[2 * i] = in[i] & 0x0F0F0F0Fu;
                o[2 * i + 1] = (in[i] >> 4) & 0x0F0F0F0Fu;
            }
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    o[4 * i + j] = (in[i] >> (2 * j)) & 0x03030303u;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
            *(uint4 *)(dst + 16 * u) = make_uint4(o[4 * u], o[4 * u + 1], o[4 * u + 2], o[4 * u + 3]);
    };
    auto load_a = [&](int ks) {
        const uint4 *src = (const uint4 *)(wtile + (long long)ks * (BLK_CO * KC)) + tid * 2;
        areg[0] = src[0];
        areg[1] = src[1];
    };
    auto store_a = [&](int stage) {
        uint8_t *dst = lds + stage * A_STAGE + (tid >> 1) * LDS_ROW + (tid & 1) * 32;
        *(uint4 *)dst = areg[0];
        *(uint4 *)(dst + 16) = areg[1];
    };

    v4i acc[4][8];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j)
            acc[i][j] = v4i{0, 0, 0, 0};

    load_a(0);
    load_b(0);
    store_a(0);
    store_b(0);
    __syncthreads();

    const int a_off = (wc * 64 + (lane & 15)) * LDS_ROW + (lane >> 4) * 16;
    const int b_off = 2 * A_STAGE + (wp * 128 + (lane & 15)) * LDS_ROW + (lane >> 4) * 16;

    for (int ks = 0; ks < KS; ++ks) {
        const int cur = ks & 1;
        const bool more = ks + 1 < KS;
        if (more) {
            load_a(ks + 1);
            load_b(ks + 1);
        }
        const uint8_t *ab = lds + cur * A_STAGE + a_off;
        const uint8_t *bb = lds + cur * B_STAGE + b_off;
        v4i af[4], bf[8];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            af[i] = *(const v4i *)(ab + i * 16 * LDS_ROW);
#pragma unroll
        for (int j = 0; j < 8; ++j)
            bf[j] = *(const v4i *)(bb + j * 16 * LDS_ROW);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 8; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[i], bf[j], acc[i][j], 0, 0, 0);
        if (more) {
            store_a(cur ^ 1);
            store_b(cur ^ 1);
        }
        __syncthreads();
    }

    // ---------------------------------------------------------------- epilogue
    const int g = lane >> 4;
    const int co_loc = wc * 64 + 16 * g;           // first of this lane's 16 channels
    const int co_glob = co_tile * BLK_CO + co_loc;
    const int32_t *prm = (const int32_t *)(lds + PRM_OFF);
    constexpr int QMAX = (BO == 32) ? 0 : (1 << BO) - 1;

    if (BO != 32 && co_glob >= A.cout)
        return;

#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const long long px = (long long)px_tile * BLK_PX + wp * 128 + j * 16 + (lane & 15);
        if (px >= S.P)
            continue;
        // skip row of this pixel
        long long spix = px;
        if (SK && A.up2) {
            int n_ = (int)(px / hw);
            int rem = (int)(px - (long long)n_ * hw);
            int oh = rem / S.wo, ow = rem - oh * S.wo;
            spix = ((long long)n_ * S.hs + (oh >> 1)) * S.ws + (ow >> 1);
        }
        uint32_t skw[4] = {0, 0, 0, 0};  // packed skip codes of the 16 channels
        if constexpr (SK == 2) {
            skw[0] = *(const uint32_t *)((const uint8_t *)S.skip + spix * (A.cout / 4) + co_glob / 4);
        } else if constexpr (SK == 4) {
            uint2 t = *(const uint2 *)((const uint8_t *)S.skip + spix * (A.cout / 2) + co_glob / 2);
            skw[0] = t.x;
            skw[1] = t.y;
        } else if constexpr (SK == 8) {
            uint4 t = *(const uint4 *)((const uint8_t *)S.skip + spix * A.cout + co_glob);
            skw[0] = t.x;
            skw[1] = t.y;
            skw[2] = t.z;
            skw[3] = t.w;
        }
        uint32_t outw[(BO == 32) ? 1 : BO / 2];
#pragma unroll
        for (int u = 0; u < ((BO == 32) ? 1 : BO / 2); ++u)
            outw[u] = 0;

#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int cl = co_loc + 4 * i;
            const int4 bias4 = *(const int4 *)(prm + cl);
            const int bias[4] = {bias4.x, bias4.y, bias4.z, bias4.w};
            if constexpr (BO == 32) {
                if (co_glob + 4 * i < A.cout) {
                    int4 o;
                    o.x = acc[i][j][0] + bias[0];
                    o.y = acc[i][j][1] + bias[1];
                    o.z = acc[i][j][2] + bias[2];
                    o.w = acc[i][j][3] + bias[3];
                    *(int4 *)((int32_t *)S.y + px * A.cout + co_glob + 4 * i) = o;
                }
            } else {
                const int4 m4 = *(const int4 *)(prm + BLK_CO + cl);
                const int4 s4 = *(const int4 *)(prm + 2 * BLK_CO + cl);
                const int mult[4] = {m4.x, m4.y, m4.z, m4.w};
                const int shf[4] = {s4.x, s4.y, s4.z, s4.w};
                int kv[4] = {0, 0, 0, 0}, sc[4] = {0, 0, 0, 0}, sd[4] = {0, 0, 0, 0}, sside[4] = {0, 0, 0, 0};
                if constexpr (SK != 0) {
                    const int4 c4 = *(const int4 *)(prm + 3 * BLK_CO + cl);
                    const int4 d4 = *(const int4 *)(prm + 4 * BLK_CO + cl);
                    const int4 e4 = *(const int4 *)(prm + 5 * BLK_CO + cl);
                    sc[0] = c4.x; sc[1] = c4.y; sc[2] = c4.z; sc[3] = c4.w;
                    sd[0] = d4.x; sd[1] = d4.y; sd[2] = d4.z; sd[3] = d4.w;
                    sside[0] = e4.x; sside[1] = e4.y; sside[2] = e4.z; sside[3] = e4.w;
                    if constexpr (SK == 32) {
                        const int4 k4 = *(const int4 *)((const int32_t *)S.skip + spix * A.cout + co_glob + 4 * i);
                        kv[0] = k4.x; kv[1] = k4.y; kv[2] = k4.z; kv[3] = k4.w;
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int bit = (4 * i + e) * SK;
                            kv[e] = (skw[bit >> 5] >> (bit & 31)) & ((1 << SK) - 1);
                        }
                    }
                }
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int v = acc[i][j][e] + bias[e];
                    long long u = v;
                    if constexpr (SK != 0)
                        u = align_add(v, kv[e], sc[e], sd[e], sside[e]);
                    const uint32_t code = requant_clamp(u, mult[e], shf[e], QMAX);
                    const int bit = (4 * i + e) * BO;
                    outw[bit >> 5] |= code << (bit & 31);
                }
            }
        }
        if constexpr (BO == 2) {
            *(uint32_t *)((uint8_t *)S.y + px * (A.cout / 4) + co_glob / 4) = outw[0];
        } else if constexpr (BO == 4) {
            *(uint2 *)((uint8_t *)S.y + px * (A.cout / 2) + co_glob / 2) = make_uint2(outw[0], outw[1]);
        } else if constexpr (BO == 8) {
            *(uint4 *)((uint8_t *)S.y + px * A.cout + co_glob) = make_uint4(outw[0], outw[1], outw[2], outw[3]);
        }
    }
}

template <int BI, int BO, int SK>
hipError_t launch_t(const MfmaArgs &a, hipStream_t stream)
{
    dim3 grid(8 * a.tiles_per_xcd), block(NT);
    hipLaunchKernelGGL((qconv_mfma_kernel<BI, BO, SK>), grid, block, 0, stream, a);
    return hipGetLastError();
}

template <int BI, int BO>
hipError_t launch_skip(int skip_bits, const MfmaArgs &a, hipStream_t stream)
{
    switch (skip_bits) {
    case 0: return launch_t<BI, BO, 0>(a, stream);
    case 2: return launch_t<BI, BO, 2>(a, stream);
    case 4: return launch_t<BI, BO, 4>(a, stream);
    case 8: return launch_t<BI, BO, 8>(a, stream);
    case 32: return launch_t<BI, BO, 32>(a, stream);
    }
    return hipErrorInvalidValue;
}

template <int BI>
hipError_t launch_out(int out_bits, int skip_bits, const MfmaArgs &a, hipStream_t stream)
{
    switch (out_bits) {
    case 2: return launch_skip<BI, 2>(skip_bits, a, stream);
    case 4: return launch_skip<BI, 4>(skip_bits, a, stream);
    case 8: return launch_skip<BI, 8>(skip_bits, a, stream);
    case 32: return skip_bits ? hipErrorInvalidValue : launch_t<BI, 32, 0>(a, stream);
    }
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_qconv_mfma(int bits_in, int out_bits, int skip_bits, const MfmaArgs &a,
                             hipStream_t stream)
{
    if (bits_in == 4)
        return launch_out<4>(out_bits, skip_bits, a, stream);
    if (bits_in == 2)
        return launch_out<2>(out_bits, skip_bits, a, stream);
    return hipErrorInvalidValue;
}

}  // namespace aqd
