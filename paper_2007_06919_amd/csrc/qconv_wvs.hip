// Weight-stationary, persistent form of the register-fed int8-MFMA
// convolution (Eq. 4 as an implicit GEMM, Sec. 3.2.1) for 1x1 layers with 256
// input channels: 4-bit codes in and out, 4 K steps, cout a multiple of 256,
// no skip or a 4-bit code skip (Eq. 7-8, optionally 2x-upsampled): ResNet-50's
// res4 conv3. These layers move more bytes than they multiply: a workgroup
// that did one tile would spend its time on its copies, its prologue and its
// epilogue.
//
// Each workgroup keeps one 256-channel tile of weights in registers for the
// whole launch (wave w: rows 64w .. 64w+63, 16 VGPRs per K step, 64 in all)
// and walks over 64-pixel tiles with a stride, two workgroups per CU. With
// 512 input channels (twice the weight registers) only one workgroup fits a
// CU, which measured slower than the register-fed kernel's 256 x 64 tiles
// (FPN P3 lateral 43 -> 61 us); the template keeps the stage count general. The activation codes of all
// its tiles form one continuous stream of stages (a stage = one tile's 256
// channels, 128 B per pixel) through a ring of four LDS stages: stage G + 2
// is copied during stage G whichever tile it belongs to, so the copies of a
// tile's first stages run during the previous tile's last stage and
// epilogue. The epilogue tables (and the side-0 skip table) are loaded into
// LDS once; a tile's skip codes are loaded into registers when its first
// stage starts and used in its epilogue; its output codes leave through an
// LDS staging area as whole 16-byte chunks of contiguous pixel rows.
//
// Copies, fragment reads, the widening of the 4-bit codes and the MFMA
// schedule are those of the register-fed kernel (qconv_wv.hip): buffer loads
// (zeros past the input's end), 8-byte columns XOR-swizzled by pixel, one
// barrier per stage, the next column's widening between the current column's
// MFMAs.

#include "epilogue.h"
#include "internal.h"
#include "mfma_common.h"

namespace aqd {
namespace {

constexpr int WS_BCO = 256;                       // channels per workgroup tile
constexpr int WS_BPX = 64;                        // pixels per tile
constexpr int WS_ROW = 128;                       // bytes of one stage per pixel
constexpr int WS_STAGE = WS_BPX * WS_ROW;         // 8 KiB
constexpr int WS_RING = 4 * WS_STAGE;             // 32 KiB
constexpr int WS_TAB = WS_RING;                   // [EPI_FIELDS][256] int32, then [256][16] (side-0 skip table)
constexpr int WS_OUT = WS_TAB + (EPI_FIELDS + 16) * WS_BCO * 4;  // output staging: 64 pixels x 128 B
constexpr int WS_LDS = WS_OUT + WS_BPX * 128;     // 64 KiB

// NST: stages per tile (cin / 256; launched with 1); SKK: 0 = no skip, 1 =
// 4-bit code skip; FAST: every shift >= 2 (32-bit requantisation)
template <int NST, int SKK, int FAST>
__global__ void __launch_bounds__(256, 2) qconv_wvs_kernel(MfmaArgs A)
{
    constexpr int BI = 4, MI = 4, NJ = 4, KS = 4 * NST, QMAX = 15, RA = 2;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[WS_LDS];

    const MfmaSeg &S = A.seg[0];
    const int co_tile = blockIdx.x % A.co_tiles;
    const int nstream = gridDim.x / A.co_tiles;
    const int qtiles = A.total_tiles / A.co_tiles;
    int q = blockIdx.x / A.co_tiles;              // this workgroup's current pixel tile
    if (q >= qtiles)
        return;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane & 15, g = lane >> 4;
    const int row_bytes = A.cin * BI / 8;
    const int hw = S.ho * S.wo;

    // ---- weights: all K steps of this wave's 64 rows, once (the layout of
    // the 256 x 128 tiles: step k, accumulator tile i at k * 16 KiB + i * 1 KiB)
    const buf_rsrc wr = make_rsrc(S.wt + (long long)co_tile * KS * WS_BCO * KC, KS * WS_BCO * KC);
    const int w_lane = (64 * wave + r) * KC + 16 * g;
    v4i fa[KS][MI];
#pragma unroll
    for (int k = 0; k < KS; ++k)
#pragma unroll
        for (int i = 0; i < MI; ++i)
            fa[k][i] = load_b128(wr, w_lane + i * 1024, k * (WS_BCO * KC));

    // ---- tables, once: [EPI_FIELDS][256] and the side-0 skip table [256][16]
    int32_t *prm = (int32_t *)(lds + WS_TAB);
    int32_t *lut = prm + EPI_FIELDS * WS_BCO;
    const bool use_lut = SKK == 1 && S.side0;
#pragma unroll
    for (int t = 0; t < EPI_FIELDS; ++t)
        prm[tid + 256 * t] = S.epi[t * A.cout_pad + co_tile * WS_BCO + tid];
    if (use_lut) {
#pragma unroll
        for (int t = 0; t < 16; ++t)
            lut[tid + 256 * t] = S.lut[co_tile * WS_BCO * 16 + tid + 256 * t];
    }

    // ---- the copy stream: stage cs of pixel tile cq; piece m of a stage =
    // pixels 32m .. 32m+31 of the tile, lane tid copying 16-byte chunk
    // tid % 8 of pixel 32m + tid / 8 (an offset past the input's end for
    // pixels past the last tile)
    const int c16 = tid & 7, wp = tid >> 3;
    const buf_rsrc xr = make_rsrc(S.x, S.n * S.h * S.w * row_bytes);
    int cq = q, cs = 0;
    int cbase[2];
    auto copy_tile = [&]() {
#pragma unroll
        for (int m = 0; m < 2; ++m) {
            const long long p = (long long)cq * WS_BPX + 32 * m + wp;
            int off = (int)0x80000000;
            if (cq < qtiles && p < S.P) {  // 1x1, no padding: the input pixel is inside
                int in_px = (int)p;
                if (A.stride != 1) {
                    const int n_ = (int)p / hw;
                    const int rem = (int)p - n_ * hw;
                    const int oh = rem / S.wo, ow = rem - oh * S.wo;
                    in_px = (n_ * S.h + oh * A.stride) * S.w + ow * A.stride;
                }
                off = in_px * row_bytes + 16 * c16;
            }
            cbase[m] = off;
        }
    };
    copy_tile();
    auto load_piece = [&](int m) -> v4i {
        return load_b128(xr, cbase[m] < 0 ? (int)0x80000000 : cbase[m] + WS_ROW * cs, 0);
    };
    auto advance_copy = [&]() {
        if (++cs == NST) {
            cs = 0;
            cq += nstream;
            copy_tile();
        }
    };
    // LDS: eight-byte column c of pixel p at 128 p + 8 (c ^ (p & 15))
    const uint32_t wo0 = WS_ROW * wp + 8 * ((2 * c16) ^ (wp & 15));
    const uint32_t wo1 = WS_ROW * wp + 8 * ((2 * c16 + 1) ^ (wp & 15));
    auto write_piece = [&](int buf, int m, const v4i v) {
        uint8_t *base = lds + buf * WS_STAGE + m * (32 * WS_ROW);
        *(uint2 *)(base + wo0) = make_uint2((uint32_t)v.x, (uint32_t)v.y);
        *(uint2 *)(base + wo1) = make_uint2((uint32_t)v.z, (uint32_t)v.w);
    };
    // fragment of K step qq of a stage: pixel 16j + r, eight-byte column 4qq + g
    auto ro = [&](int qq) -> uint32_t { return WS_ROW * r + 8 * ((4 * qq + g) ^ r); };
    auto widen = [](const uint2 w) -> v4i {
        return v4i{(int)(w.x & 0x0F0F0F0Fu), (int)((w.x >> 4) & 0x0F0F0F0Fu),
                   (int)(w.y & 0x0F0F0F0Fu), (int)((w.y >> 4) & 0x0F0F0F0Fu)};
    };

    // ---- prologue: stream stages 0 and 1 in LDS
#pragma unroll
    for (int m = 0; m < 2; ++m)
        write_piece(0, m, load_piece(m));
    advance_copy();
#pragma unroll
    for (int m = 0; m < 2; ++m)
        write_piece(1, m, load_piece(m));
    advance_copy();  // copy stream: stage 2
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    uint2 fb[NJ];
#pragma unroll
    for (int j = 0; j < RA; ++j)
        fb[j] = *(const uint2 *)(lds + 2048 * j + ro(0));
    v4i bw = widen(fb[0]);
    v4i rb[2];

    // lane group g of wave w holds channels 128 (w >> 1) + 32 g + 16 (w & 1) + 4 i + e
    const int co_loc = 128 * (wave >> 1) + 32 * g + 16 * (wave & 1);
    const int co_glob = co_tile * WS_BCO + co_loc;
    const int32_t *lut_l = lut + (co_loc << BI);
    int G = 0;  // stream stage being multiplied (buffer G % 4)

    // one stage: the MFMAs of its 4 K steps (weights of step 4s + qq), the
    // copy of stream stage G + 2 (pieces loaded at the start of steps 0 and 1,
    // written at the end of steps 1 and 2), a barrier in the last step before
    // the first fragment read of stage G + 1 (which makes it visible; the
    // barrier of stage G - 1 ordered every read of stage G - 2 before the
    // writes into its buffer)
    v4i acc[MI][NJ];
    auto stage = [&](auto sc) {
        constexpr int s = decltype(sc)::value;
        const int buf = G & 3;
        static_for<4>([&](auto qc) {
            constexpr int qq = decltype(qc)::value;
            if constexpr (qq < 2)
                rb[qq] = load_piece(qq);
            __builtin_amdgcn_sched_barrier(0);
            const uint32_t r_this = ro(qq) + buf * WS_STAGE;
            const uint32_t r_next = qq < 3 ? ro(qq + 1) + buf * WS_STAGE : ro(0) + ((buf + 1) & 3) * WS_STAGE;
            static_for<NJ>([&](auto jc) {
                constexpr int j = decltype(jc)::value;
                if constexpr (qq == 3 && j == NJ - RA)
                    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
                const v4i bn = widen(fb[(j + 1) % NJ]);
#pragma unroll
                for (int i = 0; i < MI; ++i)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[4 * s + qq][i], bw, acc[i][j], 0, 0, 0);
                if constexpr (j + RA < NJ)
                    fb[j + RA] = *(const uint2 *)(lds + 2048 * (j + RA) + r_this);
                else
                    fb[j + RA - NJ] = *(const uint2 *)(lds + 2048 * (j + RA - NJ) + r_next);
                bw = bn;
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
                __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);  // VALU
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_barrier(0);
            });
            if constexpr (qq == 1 || qq == 2)
                write_piece((buf + 2) & 3, qq - 1, rb[qq - 1]);
            if constexpr (qq == 3)
                advance_copy();
        });
        ++G;
    };

    for (;;) {
        const long long px0 = (long long)q * WS_BPX + r;
        bool okj[NJ];
#pragma unroll
        for (int j = 0; j < NJ; ++j)
            okj[j] = px0 + 16 * j < S.P;
        // this tile's skip codes (16 channels of 8 pixels per lane), used in
        // the epilogue
        uint32_t skw[NJ][2];
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            skw[j][0] = skw[j][1] = 0;
            if constexpr (SKK == 1) {
                if (okj[j]) {
                    const long long px = px0 + 16 * j;
                    long long spix = px;
                    if (A.up2) {
                        const int n_ = (int)(px / hw);
                        const int rem = (int)(px - (long long)n_ * hw);
                        const int oh = rem / S.wo, ow = rem - oh * S.wo;
                        spix = ((long long)n_ * S.hs + (oh >> 1)) * S.ws + (ow >> 1);
                    }
                    const uint2 t = *(const uint2 *)((const uint8_t *)S.skip + spix * (A.cout * BI / 8) +
                                                     co_glob * BI / 8);
                    skw[j][0] = t.x;
                    skw[j][1] = t.y;
                }
            }
        }
        // accumulators start at the bias (Eq. 6)
#pragma unroll
        for (int i = 0; i < MI; ++i) {
            const v4i b = *(const v4i *)(prm + EPI_BIAS * WS_BCO + co_loc + 4 * i);
#pragma unroll
            for (int j = 0; j < NJ; ++j)
                acc[i][j] = b;
        }
        static_for<NST>([&](auto sc) { stage(sc); });

        // ---- epilogue (Eq. 6-8, Eq. 2 on integers): requantised 4-bit codes,
        // 16 consecutive channels of 4 pixels per lane
        uint32_t outw[NJ][2];
#pragma unroll
        for (int j = 0; j < NJ; ++j)
            outw[j][0] = outw[j][1] = 0;
        auto group = [&](auto lut_c, auto ic) {
            constexpr bool LUT = decltype(lut_c)::value;
            constexpr int i = decltype(ic)::value;
            const int cl = co_loc + 4 * i;
            const int4 m4 = *(const int4 *)(prm + EPI_MULT * WS_BCO + cl);
            const int4 s4 = *(const int4 *)(prm + (FAST ? EPI_SHR : EPI_SHIFT) * WS_BCO + cl);
            const int mult[4] = {m4.x, m4.y, m4.z, m4.w};
            const int shf[4] = {s4.x, s4.y, s4.z, s4.w};
            long long rnd[4] = {0, 0, 0, 0};  // 2^(shift-2) in the high word
            if constexpr (FAST) {
                const int4 r4 = *(const int4 *)(prm + EPI_RND * WS_BCO + cl);
                rnd[0] = (long long)r4.x << 32; rnd[1] = (long long)r4.y << 32;
                rnd[2] = (long long)r4.z << 32; rnd[3] = (long long)r4.w << 32;
            }
            int sc[4] = {0, 0, 0, 0}, sd[4] = {0, 0, 0, 0}, sside[4] = {0, 0, 0, 0};
            long long srnd[4] = {0, 0, 0, 0};  // rounding terms of the alignment
            if constexpr (SKK != 0 && !LUT) {
                const int4 c4 = *(const int4 *)(prm + EPI_SKIP_C * WS_BCO + cl);
                const int4 d4 = *(const int4 *)(prm + EPI_SKIP_D * WS_BCO + cl);
                const int4 e4 = *(const int4 *)(prm + EPI_SKIP_SIDE * WS_BCO + cl);
                sc[0] = c4.x; sc[1] = c4.y; sc[2] = c4.z; sc[3] = c4.w;
                sd[0] = d4.x; sd[1] = d4.y; sd[2] = d4.z; sd[3] = d4.w;
                srnd[0] = rsm_rnd(d4.x); srnd[1] = rsm_rnd(d4.y); srnd[2] = rsm_rnd(d4.z); srnd[3] = rsm_rnd(d4.w);
                sside[0] = e4.x; sside[1] = e4.y; sside[2] = e4.z; sside[3] = e4.w;
            }
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int v = acc[i][j][e];  // acc + bias
                    const int bit = (4 * i + e) * BI;
                    int kv = 0;
                    if constexpr (SKK == 1)
                        kv = (int)__builtin_amdgcn_ubfe(skw[j][bit >> 5], bit & 31, BI);
                    int y;
                    if constexpr (FAST) {
                        int u = v;
                        // u fits in int32, so sums modulo 2^32 are exact
                        if constexpr (LUT) {
                            u = (int)((unsigned)v + (unsigned)lut_l[((4 * i + e) << BI) + kv]);
                        } else if constexpr (SKK != 0) {
                            const int scaled = rsm32r(sside[e] ? v : kv, sc[e], srnd[e], sd[e]);
                            u = (int)((unsigned)scaled + (unsigned)(sside[e] ? kv : v));
                        }
                        y = requant32(u, mult[e], rnd[e], shf[e]);
                        y = y < 0 ? 0 : (y > QMAX ? QMAX : y);
                    } else {
                        long long u = v;
                        if constexpr (LUT)
                            u = (int)((unsigned)v + (unsigned)lut_l[((4 * i + e) << BI) + kv]);
                        else if constexpr (SKK != 0)
                            u = align_add(v, kv, sc[e], sd[e], sside[e]);
                        y = (int)requant_clamp(u, mult[e], shf[e], QMAX);
                        asm volatile("" : "+v"(y));  // one 64-bit product alive at a time
                    }
                    outw[j][bit >> 5] |= (uint32_t)y << (bit & 31);
                }
            }
        };
        if (use_lut)
            static_for<MI>([&](auto ic) { group(std::true_type{}, ic); });
        else
            static_for<MI>([&](auto ic) { group(std::false_type{}, ic); });
        if (A.qmax == 7) {  // 3-bit codes (the epilogue clamped to 15)
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                outw[j][0] = sat7_nibbles(outw[j][0]);
                outw[j][1] = sat7_nibbles(outw[j][1]);
            }
        }
        // the tile's codes through the staging area (every wave's copy-out
        // of the last tile came before the barriers of this tile's stages):
        // pixel row p of 128 B, 16-byte chunk c at position c ^ (p & 7)
        const int c0 = co_loc / 2;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int p = 16 * j + r;
            *(uint2 *)(lds + WS_OUT + p * 128 + 16 * ((c0 >> 4) ^ (p & 7)) + (c0 & 8)) =
                make_uint2(outw[j][0], outw[j][1]);
        }
        __syncthreads();
        const long long rowg = (long long)A.cout * BI / 8;
#pragma unroll
        for (int it = 0; it < WS_BPX * 8 / 256; ++it) {
            const int idx = it * 256 + tid;
            const int p = idx >> 3, c = idx & 7;
            const long long px = (long long)q * WS_BPX + p;
            if (px < S.P)
                *(uint4 *)((uint8_t *)S.y + px * rowg + co_tile * 128 + 16 * c) =
                    *(const uint4 *)(lds + WS_OUT + p * 128 + 16 * (c ^ (p & 7)));
        }
        q += nstream;
        if (q >= qtiles)
            break;
    }
}

template <int NST>
void launch_wvs_modes(const MfmaArgs &a, bool fast, dim3 grid, hipStream_t stream)
{
    const dim3 block(256);
    if (a.skip_bits == 0) {
        if (fast)
            hipLaunchKernelGGL((qconv_wvs_kernel<NST, 0, 1>), grid, block, 0, stream, a);
        else
            hipLaunchKernelGGL((qconv_wvs_kernel<NST, 0, 0>), grid, block, 0, stream, a);
    } else {
        if (fast)
            hipLaunchKernelGGL((qconv_wvs_kernel<NST, 1, 1>), grid, block, 0, stream, a);
        else
            hipLaunchKernelGGL((qconv_wvs_kernel<NST, 1, 0>), grid, block, 0, stream, a);
    }
}

}  // namespace

hipError_t launch_qconv_wvs(const MfmaArgs &a, hipStream_t stream)
{
    if (a.nseg != 1 || a.bits_out != 4 || (a.skip_bits != 0 && a.skip_bits != 4) || a.kh != 1 || a.kw != 1 ||
        a.pad != 0 || a.cin != 256 || a.ksteps != a.cin / KC || a.cout % WS_BCO != 0 ||
        a.co_tiles * WS_BCO != a.cout || a.co_tiles < 1 || a.co_tiles > 256 || a.ksplit != 1 || a.part != 0)
        return hipErrorInvalidValue;
    // 32-bit buffer offsets: the input below 2^31 bytes
    if ((long long)a.seg[0].n * a.seg[0].h * a.seg[0].w * (a.cin / 2) >= (1LL << 31))
        return hipErrorInvalidValue;
    const int qtiles = a.total_tiles / a.co_tiles;
    if (qtiles <= 0)
        return hipSuccess;
    // two workgroups per CU, every channel tile on its own workgroups
    const int nstream = qtiles < 512 / a.co_tiles ? qtiles : 512 / a.co_tiles;
    const dim3 grid((nstream < 1 ? 1 : nstream) * a.co_tiles);
    launch_wvs_modes<1>(a, a.seg[0].fast, grid, stream);
    return hipGetLastError();
}

}  // namespace aqd
