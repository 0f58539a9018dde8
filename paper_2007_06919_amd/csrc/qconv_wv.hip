// Implicit-GEMM integer convolution on the gfx950 int8 MFMA
// (v_mfma_i32_16x16x64_i8) for layers with 256-channel input chunks (cin a
// multiple of 256) and 4-bit activation codes, with code outputs (the
// detection heads' 3x3 256 -> 256 towers, the FPN's 3x3 outputs, ResNet-50's
// res4/res5 3x3 and 1x1 layers with cin >= 512) or int32 outputs (the class
// predictor). The GEMM view is that of Eq. 4
// (Sec. 3.2.1): rows = output channels (weights), columns = output pixels,
// K = taps x input channels, one K step = 64 input channels of one tap.
//
// Workgroup tile 256 channels x 128 pixels, 4 waves; wave w owns channel rows
// 64w .. 64w+63 (4 accumulator tiles of 16) for all 128 pixels (8 column
// tiles of 16), so no two waves share a weight row:
//  * weights (int8, decoded and tiled at create exactly as for the 256 x 128
//    kernel) go from global memory (L2) straight into registers, two K steps
//    ahead of their MFMAs, one 16-byte buffer load per column tile during the
//    first four column tiles of a step: no LDS traffic for the larger operand;
//  * activation codes (4-bit, packed as stored) go through LDS in stages of
//    four K steps (one tap's 256 channels, 128 B per pixel: whole cache
//    lines), a ring of four stages; each lane copies 16 B per K step through
//    registers: loaded at the start of a step, written at the end of the
//    next. Buffer loads return zeros past the end of the input, so padding
//    taps cost no branch and no mask. In LDS a pixel row's eight-byte columns
//    are XOR-swizzled with the pixel index, so that the fragment reads (8 B
//    per lane, 16 pixels per lane group) and the copies' writes are free of
//    bank conflicts;
//  * one barrier per stage (four K steps);
//  * each column tile is one scheduling region: its 4 MFMAs with the widening
//    of the next column's fragment (mask/shift of the packed codes to int8, in
//    the byte order the weights were stored in at create) between them, so
//    that the VALU work issues while the matrix core runs;
//  * the channel tile's epilogue table is fetched before the last stage.
//
// Epilogue (Sec. 3.2.2-3.2.3, Eq. 6-8, and Eq. 2 on integers): the
// accumulators start at the folded bias; a lane holds 16 consecutive channels
// of 8 pixels and packs their requantised codes. The LDS ring holds the
// channel tile's epilogue table and the side-0 skip table after the last K
// step, then the tile's packed codes, which leave as 16-byte chunks of
// contiguous pixel rows (a partial channel tile stores from registers).

#include "epilogue.h"
#include "internal.h"
#include "mfma_common.h"

namespace aqd {
namespace {

constexpr int WV_BCO = 256;              // channels per workgroup tile
constexpr int WV_ROW = 128;              // bytes of one stage per pixel (256 codes of 4 bits)
constexpr int WV_NBUF = 4;

// OUTK: 0 = 4-bit codes, 1 = int32 v = acc + bias (then SKK = 0), 2 = 8-bit
// codes (the last tower layer of the fully quantized heads; then SKK = 0);
// SKK: 0 = no skip, 1 = code skip (4-bit), 2 = a residual block's projection
// shortcut fused in (1x1 convolutions both, 256 x 64 tiles, 4-bit codes out:
// two accumulator sets, two workgroups per CU); FAST: every shift >= 2 (32-bit
// requantisation); NJ: column tiles of 16 pixels, 8 (256 x 128 tiles, two
// workgroups per CU), 9 (256 x 144 tiles, one per CU: launches a little
// above one round of the smaller tile fit in one round) or 4 (256 x 64
// tiles, three per CU: short K ranges, where a tile's copies and epilogue
// outweigh its MFMAs); 9 and 4 for code outputs only
template <int OUTK, int SKK, int FAST, int NJ>
__global__ void __launch_bounds__(256, NJ == 8 ? 2 : NJ == 4 ? (SKK == 2 ? 2 : 3) : 1) qconv_wv_kernel(MfmaArgs A)
{
    static_assert(OUTK == 0 || SKK == 0, "int32 and 8-bit outputs have no skip");
    static_assert(SKK != 2 || NJ == 4, "the fused projection runs on 256 x 64 tiles");
    static_assert(NJ == 8 || ((NJ == 9 || NJ == 4) && OUTK != 1), "256 x 144 and 256 x 64 tiles: code outputs");
    constexpr int BI = 4, MI = 4;
    constexpr int WV_BPX = 16 * NJ;                // pixels per workgroup tile
    constexpr int NPC = (WV_BPX + 31) / 32;        // copy pieces of 32 pixels per stage (2, 4 or 5)
    constexpr int WV_STAGE = 32 * NPC * WV_ROW;    // 8, 16 or 20 KiB (rows past the tile unused)
    constexpr int WV_LDS = WV_NBUF * WV_STAGE;
    constexpr int BO = OUTK == 2 ? 8 : 4;          // output code width
    constexpr int QMAX = (1 << BO) - 1, OW = BO / 2;  // words of a lane's 16 channels
    __shared__ __attribute__((aligned(1024))) uint8_t lds[WV_LDS];

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

    const int KS = A.ksteps;
    // stages (KS is a multiple of 4; under SKK 2 the main 1x1 convolution may
    // have 128 input channels: one stage whose K steps 2-3 read the next
    // pixel's codes against weights past the buffer's end, zeros)
    const int NST = (KS + 3) / 4;
    const int hw = S.ho * S.wo;
    // the fused projection shortcut (SKK 2): its 1x1 convolution of x2 (cin2
    // channels, stride2, no padding) runs first, over K steps 0 .. KS2 - 1,
    // into a second accumulator set; the main 1x1 convolution follows
    const int KS2 = SKK == 2 ? A.ksteps2 : 0;
    const int NST2 = KS2 / 4;
    const int NSTT = NST2 + NST;                 // stages of both

    // ---- activation copies: piece m of a stage = pixels 32m .. 32m+31 of the
    // tile, lane tid copying 16-byte chunk tid % 8 of pixel 32m + tid / 8.
    // Buffer loads: a tap in the padding, a pixel past the end and a stage
    // past the last read at an offset past the buffer's size and get zeros
    // (code 0), with no branch and no mask on the data.
    const int c16 = tid & 7;
    // per piece: the byte offset of its pixel's window origin (negative at the
    // top and left borders) and which window rows (bit t) and columns (bit
    // 16 + t) lie inside the image (none for pixels past the end); the input
    // holds n * h * w * row_bytes < 2^31 bytes (checked on the host)
    int xbase[NPC];
    uint32_t xvalid[NPC];
    // geometry of the input being copied (the projection's x2 first under SKK 2)
    int row_bytes = 0, spt = 0, c_w = 0;
    buf_rsrc xr;
    auto set_copy = [&](const bool proj) {
        const uint8_t *src = proj ? S.x2 : S.x;
        const int ch = proj ? A.cin2 : A.cin, ih = proj ? S.h2 : S.h, iw = proj ? S.w2 : S.w;
        const int st = proj ? A.stride2 : A.stride, pd = proj ? 0 : A.pad;
        const int kh = proj ? 1 : A.kh, kw = proj ? 1 : A.kw;
        row_bytes = ch * BI / 8;
        spt = (ch + 255) / 256;                  // stages per tap
        c_w = iw;
#pragma unroll
        for (int m = 0; m < NPC; ++m) {
            const unsigned pl = (unsigned)(32 * m + (tid >> 3));    // pixel within the tile
            const unsigned p = (unsigned)(px_tile * WV_BPX) + pl;
            const bool ok = p < (unsigned)S.P && pl < (unsigned)WV_BPX;
            const unsigned pn = ok ? p / (unsigned)hw : 0u;
            const unsigned prem = ok ? p - pn * (unsigned)hw : 0u;
            const int oh = (int)(prem / (unsigned)S.wo), ow = (int)prem - oh * S.wo;
            const int ih0 = oh * st - pd, iw0 = ow * st - pd;
            uint32_t v = 0;
            for (int t = 0; t < kh; ++t)
                v |= ((unsigned)(ih0 + t) < (unsigned)ih ? 1u : 0u) << t;
            for (int t = 0; t < kw; ++t)
                v |= ((unsigned)(iw0 + t) < (unsigned)iw ? 1u : 0u) << (16 + t);
            xvalid[m] = ok ? v : 0u;
            xbase[m] = (((int)pn * ih + ih0) * iw + iw0) * row_bytes + 16 * c16;
        }
        xr = make_rsrc(src, S.n * ih * iw * row_bytes);
    };
    set_copy(SKK == 2);
    // LDS byte offsets: eight-byte column c of pixel p at 128 p + 8 (c ^ (p & 15))
    const int wp = tid >> 3;                      // pixel within a piece (p & 15 == wp & 15)
    const uint32_t wo0 = WV_ROW * wp + 8 * ((2 * c16) ^ (wp & 15));
    const uint32_t wo1 = WV_ROW * wp + 8 * ((2 * c16 + 1) ^ (wp & 15));
    // fragment of K step q: pixel 16j + r, eight-byte column 4q + g
    auto ro = [&](int q) -> uint32_t { return WV_ROW * r + 8 * ((4 * q + g) ^ r); };

    // copy state of the stage being loaded (uniform): tap (tr, tq), 128-byte
    // chunk th; its byte offset from a window origin and the window bits it needs
    int tr = 0, tq = 0, th = 0;
    bool c_proj = SKK == 2;                       // the projection's stages are being copied
    int x_off = 0;
    uint32_t x_need = 0x10001u;
    auto advance = [&]() {
        if (++th == spt) {
            th = 0;
            if (++tq == (c_proj ? 1 : A.kw)) {
                tq = 0;
                ++tr;
            }
        }
        if constexpr (SKK == 2) {
            if (c_proj && tr == 1) {             // past the projection's one tap: the main input
                c_proj = false;
                tr = 0;
                set_copy(false);
            }
        }
        x_off = (tr * c_w + tq) * row_bytes + WV_ROW * th;
        x_need = (1u << tr) | (1u << (16 + tq));
    };
    auto load_piece = [&](int m) -> v4i {
        const int off = (xvalid[m] & x_need) == x_need ? xbase[m] + x_off : (int)0x80000000;
        return load_b128(xr, off, 0);
    };
    auto write_piece = [&](int buf, int m, const v4i v) {
        uint8_t *base = lds + buf * WV_STAGE + m * (32 * WV_ROW);
        *(uint2 *)(base + wo0) = make_uint2((uint32_t)v.x, (uint32_t)v.y);
        *(uint2 *)(base + wo1) = make_uint2((uint32_t)v.z, (uint32_t)v.w);
    };

    // ---- weights: this wave's rows of K step k, accumulator tile i at
    // k * 16 KiB + i * 1 KiB from the channel tile's first step (lane: row r,
    // 16-byte column g; in global memory the columns are in order, only LDS
    // copies swizzle them); the look-ahead past the last step reads past the
    // buffer's size and gets zeros, which no MFMA uses
    const buf_rsrc wr = make_rsrc(S.wt + (long long)co_tile * KS * WV_BCO * KC, KS * WV_BCO * KC);
    const int w_lane = (64 * wave + r) * KC + 16 * g;
    // under SKK 2, K steps 0 .. KS2 - 1 are the projection's (same tile layout)
    buf_rsrc wr2 = wr;
    if constexpr (SKK == 2)
        wr2 = make_rsrc(S.wt2 + (long long)co_tile * KS2 * WV_BCO * KC, KS2 * WV_BCO * KC);
    auto load_w = [&](int k, int i) -> v4i {
        if constexpr (SKK == 2) {
            if (k < KS2)
                return load_b128(wr2, w_lane + i * 1024, k * (WV_BCO * KC));
            return load_b128(wr, w_lane + i * 1024, (k - KS2) * (WV_BCO * KC));
        }
        return load_b128(wr, w_lane + i * 1024, k * (WV_BCO * KC));
    };

    // ---- accumulators start at the bias (Eq. 6): lane group g of wave w holds
    // channels 128 (w >> 1) + 32 g + 16 (w & 1) + 4 i + e of the tile
    const int co_loc = 128 * (wave >> 1) + 32 * g + 16 * (wave & 1);
    const int co_glob = co_tile * WV_BCO + co_loc;
    v4i acc[MI][NJ];
    v4i acc2[SKK == 2 ? MI : 1][SKK == 2 ? NJ : 1];  // the projection's, from its own bias
#pragma unroll
    for (int i = 0; i < MI; ++i) {
        const v4i b = *(const v4i *)(S.epi + EPI_BIAS * A.cout_pad + co_glob + 4 * i);
#pragma unroll
        for (int j = 0; j < NJ; ++j)
            acc[i][j] = b;
        if constexpr (SKK == 2) {
            const v4i b2 = *(const v4i *)(S.epi2 + EPI_BIAS * A.cout_pad + co_glob + 4 * i);
#pragma unroll
            for (int j = 0; j < NJ; ++j)
                acc2[i][j] = b2;
        }
    }

    // ---- prologue: stage 0 and pieces 0-2 of stage 1 in LDS (pieces 3 and 4
    // are written at the end of the first K step, as every stage's last ones
    // are), weights of steps 0-1 in registers
    v4i rb[NPC];
#pragma unroll
    for (int m = 0; m < NPC; ++m)
        write_piece(0, m, load_piece(m));
    advance();
#pragma unroll
    for (int m = 0; m < (NPC < 3 ? NPC : 3); ++m)
        write_piece(1, m, load_piece(m));
#pragma unroll
    for (int m = 3; m < NPC; ++m)
        rb[m] = load_piece(m);
#pragma unroll
    for (int m = 0; m < (NPC < 3 ? NPC : 3); ++m)
        rb[m] = rb[NPC - 1];
    advance();  // copy state: stage 2
    v4i fa[4][MI];
#pragma unroll
    for (int i = 0; i < MI; ++i) {
        fa[0][i] = load_w(0, i);
        fa[1][i] = load_w(1, i);
    }
    uint2 fb[NJ];   // packed fragment j of the current step, or of the next one once read ahead

    auto widen = [](const uint2 w) -> v4i {
        return v4i{(int)(w.x & 0x0F0F0F0Fu), (int)((w.x >> 4) & 0x0F0F0F0Fu),
                   (int)(w.y & 0x0F0F0F0Fu), (int)((w.y >> 4) & 0x0F0F0F0Fu)};
    };
    constexpr int RA = NJ == 4 ? 2 : 3;  // fragments are read RA column tiles ahead of their MFMAs
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
#pragma unroll
    for (int j = 0; j < RA; ++j)
        fb[j] = *(const uint2 *)(lds + 2048 * j + ro(0));
    v4i bw = widen(fb[0]);  // the widened fragment of the next column tile's MFMAs

    // ---- main loop, one stage (four K steps) per call: stage g lives in
    // buffer g % 4; during stage g the pieces of stage g + 2 are loaded (piece
    // q at the start of K step q, piece 4 too in the last step) and written at
    // the end of the next K step (the last step's at the end of the first
    // step of stage g + 1), into the buffer of stage g - 2. The weights of step k + 2 are loaded during the first
    // four column tiles of step k. Fragment (k, j) is read RA column tiles
    // ahead (during step k, or k - 1) and widened during the MFMAs of column
    // tile j - 1. A barrier in the last step, before the first read of the
    // next stage, makes that stage visible; the barrier of stage g - 1 orders
    // every wave's reads of stage g - 2 before the writes of stage g + 2 into
    // its buffer. Loads and writes for stages past the last go to buffers
    // nobody reads again.
    // Each column tile is one scheduling region, in the order: MFMA, weight
    // load, fragment read, then the widening of the next fragment (two
    // instructions) between each of the other three MFMAs; the VALU work
    // then issues while the matrix core runs.
    auto stage = [&](const int gs, auto main_c) {
        constexpr bool MAIN = decltype(main_c)::value;  // false: the projection's accumulators
        const int buf = gs & 3;
        static_for<4>([&](auto qc) {
            constexpr int q = decltype(qc)::value;
            const int k = 4 * gs + q;
            if constexpr (q < NPC)
                rb[q] = load_piece(q);  // pieces of stage gs + 2
            if constexpr (q == 3 && NPC == 5)
                rb[4] = load_piece(4);
            __builtin_amdgcn_sched_barrier(0);
            const uint32_t r_this = ro(q) + buf * WV_STAGE;
            const uint32_t r_next = q < 3 ? ro(q + 1) + buf * WV_STAGE : ro(0) + ((buf + 1) & 3) * WV_STAGE;
            static_for<NJ>([&](auto jc) {
                constexpr int j = decltype(jc)::value;
                if constexpr (q == 3 && j == NJ - RA)
                    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
                if constexpr (j < MI)
                    fa[(q + 2) & 3][j] = load_w(k + 2, j);  // set (q + 2) % 4 was step k - 2's
                const v4i bn = widen(fb[(j + 1) % NJ]);
#pragma unroll
                for (int i = 0; i < MI; ++i) {
                    if constexpr (MAIN)
                        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[q][i], bw, acc[i][j], 0, 0, 0);
                    else
                        acc2[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[q][i], bw, acc2[i][j], 0, 0, 0);
                }
                if constexpr (j + RA < NJ)
                    fb[j + RA] = *(const uint2 *)(lds + 2048 * (j + RA) + r_this);
                else
                    fb[j + RA - NJ] = *(const uint2 *)(lds + 2048 * (j + RA - NJ) + r_next);
                bw = bn;
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
                __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM read
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
                __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);  // VALU
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_barrier(0);
            });
            // the pieces loaded one step earlier (at q = 0: the last ones of
            // stage gs + 1)
            if constexpr (q >= 1) {
                if constexpr (q - 1 < NPC)
                    write_piece((buf + 2) & 3, q - 1, rb[q - 1]);
            } else {
#pragma unroll
                for (int m = 3; m < NPC; ++m)
                    write_piece((buf + 1) & 3, m, rb[m]);
            }
            if constexpr (q == 3)
                advance();
        });
    };
    int gs0 = 0;
    if constexpr (SKK == 2)
        for (; gs0 < NST2; ++gs0)
            stage(gs0, std::false_type{});
    for (int gs = gs0; gs < NSTT - 1; ++gs)
        stage(gs, std::true_type{});
    // the channel tile's epilogue table does not depend on the accumulators:
    // its loads are issued before the last stage, whose MFMAs hide their
    // latency (after it on 256 x 64 tiles, within their register budget)
    constexpr int PRM_PER = EPI_FIELDS * WV_BCO / 256;
    int prm_r[PRM_PER];
    auto load_prm = [&]() {
#pragma unroll
        for (int t = 0; t < PRM_PER; ++t) {
            const int i = tid + 256 * t;
            const int which = i / WV_BCO, c = i - which * WV_BCO;
            prm_r[t] = S.epi[which * A.cout_pad + co_tile * WV_BCO + c];
        }
    };
    if constexpr (OUTK != 1 && NJ != 4)
        load_prm();
    stage(NSTT - 1, std::true_type{});
    if constexpr (OUTK != 1 && NJ == 4)
        load_prm();

    if constexpr (OUTK == 1) {
        // int32 outputs v = acc + bias (the bias is in the accumulators), in
        // two passes of 64 pixels (column tiles 4p .. 4p+3): each lane's 16
        // channels x 4 pixels go to LDS as rows of 256 int32 (1 KiB per pixel;
        // 16-byte chunk c of pixel p at position c ^ (p & 7), so that neither
        // the writes nor the reads conflict), then every thread stores 16-byte
        // chunks of whole rows: 1 KiB of contiguous output per wave and
        // instruction
        const int valid_chunks = (A.cout - co_tile * WV_BCO < WV_BCO ? A.cout - co_tile * WV_BCO : WV_BCO) / 4;
        static_for<2>([&](auto pc) {
            constexpr int pass = decltype(pc)::value;
            __syncthreads();  // the ring, or the last pass's rows, are no longer read
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const int p = 16 * jj + r;
#pragma unroll
                for (int i = 0; i < MI; ++i) {
                    const int c = co_loc / 4 + i;
                    *(v4i *)(lds + p * 1024 + 16 * (c ^ (p & 7))) = acc[i][4 * pass + jj];
                }
            }
            __syncthreads();
#pragma unroll
            for (int it = 0; it < 16; ++it) {
                const int idx = it * 256 + tid;
                const int p = idx >> 6, c = idx & 63;
                const long long px = (long long)px_tile * WV_BPX + 64 * pass + p;
                if (px < S.P && c < valid_chunks)
                    *(v4i *)((int32_t *)S.y + px * A.cout + co_tile * WV_BCO + 4 * c) =
                        *(const v4i *)(lds + p * 1024 + 16 * (c ^ (p & 7)));
            }
        });
        return;
    }

    // ---------------------------------------------------------------- epilogue
    const long long px0 = (long long)px_tile * WV_BPX + r;
    const bool co_ok = co_glob < A.cout;          // a lane's 16 channels are all valid or all padding
    bool okj[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j)
        okj[j] = co_ok && px0 + 16 * j < S.P;
    // skip codes: issued before the tables go to LDS, so that the two overlap
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
                const uint2 t = *(const uint2 *)((const uint8_t *)S.skip + spix * (A.cout * BI / 8) + co_glob * BI / 8);
                skw[j][0] = t.x;
                skw[j][1] = t.y;
            }
        }
    }
    int32_t *prm = (int32_t *)lds;                 // [EPI_FIELDS][256]
    int32_t *lut = prm + EPI_FIELDS * WV_BCO;      // [256][16]: RSM(k, c, d) of the side-0 skip codes
    const bool use_lut = SKK == 1 && S.side0;
    constexpr int LUT_PER = SKK == 1 ? WV_BCO * (QMAX + 1) / 256 : 1;
    int lut_r[LUT_PER];
    if (use_lut) {
#pragma unroll
        for (int t = 0; t < LUT_PER; ++t)
            lut_r[t] = S.lut[co_tile * WV_BCO * (QMAX + 1) + tid + 256 * t];
    }
    __syncthreads();  // every wave is done with the ring
#pragma unroll
    for (int t = 0; t < PRM_PER; ++t)
        prm[tid + 256 * t] = prm_r[t];
    if (use_lut) {
#pragma unroll
        for (int t = 0; t < LUT_PER; ++t)
            lut[tid + 256 * t] = lut_r[t];
    }
    __syncthreads();
    static_assert((EPI_FIELDS + 16) * WV_BCO * 4 <= WV_LDS, "tables fit in the ring");

    const int32_t *lut_l = lut + (co_loc << BI);  // this lane's 16 channels
    uint32_t outw[NJ][OW];
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int o = 0; o < OW; ++o)
            outw[j][o] = 0;
    // per channel group i: the requantisation parameters, read once for all
    // columns
    auto group = [&](auto lut_c, auto ic, int j0, int j1) {
        constexpr bool LUT = decltype(lut_c)::value;
        constexpr int i = decltype(ic)::value;
        const int cl = co_loc + 4 * i;
        const int4 m4 = *(const int4 *)(prm + EPI_MULT * WV_BCO + cl);
        const int4 s4 = *(const int4 *)(prm + (FAST ? EPI_SHR : EPI_SHIFT) * WV_BCO + cl);
        const int mult[4] = {m4.x, m4.y, m4.z, m4.w};
        const int shf[4] = {s4.x, s4.y, s4.z, s4.w};
        long long rnd[4] = {0, 0, 0, 0};  // 2^(shift-2) in the high word
        if constexpr (FAST) {
            const int4 r4 = *(const int4 *)(prm + EPI_RND * WV_BCO + cl);
            rnd[0] = (long long)r4.x << 32; rnd[1] = (long long)r4.y << 32;
            rnd[2] = (long long)r4.z << 32; rnd[3] = (long long)r4.w << 32;
        }
        int sc[4] = {0, 0, 0, 0}, sd[4] = {0, 0, 0, 0}, sside[4] = {0, 0, 0, 0};
        long long srnd[4] = {0, 0, 0, 0};  // rounding terms of the alignment
        if constexpr (SKK != 0 && !LUT) {
            const int4 c4 = *(const int4 *)(prm + EPI_SKIP_C * WV_BCO + cl);
            const int4 d4 = *(const int4 *)(prm + EPI_SKIP_D * WV_BCO + cl);
            const int4 e4 = *(const int4 *)(prm + EPI_SKIP_SIDE * WV_BCO + cl);
            sc[0] = c4.x; sc[1] = c4.y; sc[2] = c4.z; sc[3] = c4.w;
            sd[0] = d4.x; sd[1] = d4.y; sd[2] = d4.z; sd[3] = d4.w;
            srnd[0] = rsm_rnd(d4.x); srnd[1] = rsm_rnd(d4.y); srnd[2] = rsm_rnd(d4.z); srnd[3] = rsm_rnd(d4.w);
            sside[0] = e4.x; sside[1] = e4.y; sside[2] = e4.z; sside[3] = e4.w;
        }
#pragma unroll
        for (int j = j0; j < j1; ++j) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int v = acc[i][j][e];  // acc + bias
                const int bit = (4 * i + e) * BO, kbit = (4 * i + e) * BI;
                int kv = 0;
                if constexpr (SKK == 1)
                    kv = (int)__builtin_amdgcn_ubfe(skw[j][kbit >> 5], kbit & 31, BI);
                else if constexpr (SKK == 2)
                    kv = acc2[i][j][e];  // the projection's int32 output (Eq. 7-8: the skip)
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
    auto body = [&](auto lut_c) { static_for<MI>([&](auto ic) { group(lut_c, ic, 0, NJ); }); };
    if (use_lut)
        body(std::true_type{});
    else
        body(std::false_type{});
    if (OUTK == 0 && A.qmax == 7) {  // 3-bit codes (the epilogue clamped to 15)
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            outw[j][0] = sat7_nibbles(outw[j][0]);
            outw[j][1] = sat7_nibbles(outw[j][1]);
        }
    }
    // the packed words are complete here: the compiler would otherwise sink
    // their last steps into the conditional stores and keep every 64-bit
    // product alive until then
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int o = 0; o < OW; ++o)
            asm volatile("" : "+v"(outw[j][o]));
    // a whole channel tile's codes go through LDS (free again once every wave
    // has read its tables) and out as 16-byte chunks of contiguous pixel rows
    constexpr int ROWB = WV_BCO * BO / 8;         // bytes of a pixel's 256 channels
    constexpr int CPR = ROWB / 16;                // 16-byte chunks per row (8 or 16)
    if (A.cout - co_tile * WV_BCO >= WV_BCO) {
        __syncthreads();
        const int c0 = co_loc * BO / 8;           // this lane's byte offset in a row
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int p = 16 * j + r;
            uint8_t *d = lds + p * ROWB + 16 * ((c0 >> 4) ^ (p & (CPR - 1))) + (c0 & 8);
            if constexpr (BO == 8)
                *(uint4 *)d = make_uint4(outw[j][0], outw[j][1], outw[j][2], outw[j][3]);
            else
                *(uint2 *)d = make_uint2(outw[j][0], outw[j][1]);
        }
        __syncthreads();
        const long long rowg = (long long)A.cout * BO / 8;
#pragma unroll
        for (int it = 0; it < (WV_BPX * CPR + 255) / 256; ++it) {
            const int idx = it * 256 + tid;
            const int p = idx / CPR, c = idx % CPR;
            const long long px = (long long)px_tile * WV_BPX + p;
            if (px < S.P && p < WV_BPX)
                *(uint4 *)((uint8_t *)S.y + px * rowg + co_tile * ROWB + 16 * c) =
                    *(const uint4 *)(lds + p * ROWB + 16 * (c ^ (p & (CPR - 1))));
        }
        return;
    }
#pragma unroll
    for (int j = 0; j < NJ; ++j)
        if (okj[j]) {
            uint8_t *dst = (uint8_t *)S.y + (px0 + 16 * j) * (A.cout * BO / 8) + co_glob * BO / 8;
            if constexpr (BO == 8)
                *(uint4 *)dst = make_uint4(outw[j][0], outw[j][1], outw[j][2], outw[j][3]);
            else
                *(uint2 *)dst = make_uint2(outw[j][0], outw[j][1]);
        }
}

template <int NJ>
void launch_wv_modes(const MfmaArgs &a, bool fast, dim3 grid, hipStream_t stream)
{
    const dim3 block(256);
    if constexpr (NJ == 8) {
        if (a.bits_out == 32) {
            hipLaunchKernelGGL((qconv_wv_kernel<1, 0, 1, NJ>), grid, block, 0, stream, a);
            return;
        }
    }
    if (a.bits_out == 8) {
        if (fast)
            hipLaunchKernelGGL((qconv_wv_kernel<2, 0, 1, NJ>), grid, block, 0, stream, a);
        else
            hipLaunchKernelGGL((qconv_wv_kernel<2, 0, 0, NJ>), grid, block, 0, stream, a);
    } else if (a.skip_bits == 0) {
        if (fast)
            hipLaunchKernelGGL((qconv_wv_kernel<0, 0, 1, NJ>), grid, block, 0, stream, a);
        else
            hipLaunchKernelGGL((qconv_wv_kernel<0, 0, 0, NJ>), grid, block, 0, stream, a);
    } else {
        if (fast)
            hipLaunchKernelGGL((qconv_wv_kernel<0, 1, 1, NJ>), grid, block, 0, stream, a);
        else
            hipLaunchKernelGGL((qconv_wv_kernel<0, 1, 0, NJ>), grid, block, 0, stream, a);
    }
}

}  // namespace

// fused projection shortcut on the register-fed 256 x 64 tiles: main and
// projection 1x1 with cin and cin2 multiples of 256, 4-bit codes out
hipError_t launch_qconv_wv_proj(const MfmaArgs &a, hipStream_t stream)
{
    if (a.bits_out != 4 || a.skip_bits != 32 || (a.cin % 256 != 0 && a.cin != 128) || a.cin2 % 256 != 0 ||
        (a.ksteps % 4 != 0 && a.cin != 128) ||
        a.ksteps2 % 4 != 0 || a.ksteps != a.cin / KC || a.ksteps2 != a.cin2 / KC || a.kh != 1 || a.kw != 1 ||
        a.pad != 0 || a.ksplit != 1 || a.part != 0 || a.nseg != 1 || a.up2)
        return hipErrorInvalidValue;
    const MfmaSeg &m = a.seg[0];
    if ((long long)m.n * m.h * m.w * (a.cin / 2) >= (1LL << 31) ||
        (long long)m.n * m.h2 * m.w2 * (a.cin2 / 2) >= (1LL << 31) ||
        (long long)a.co_tiles * a.ksteps2 * WV_BCO * KC >= (1LL << 31) ||
        (long long)a.co_tiles * a.ksteps * WV_BCO * KC >= (1LL << 31))
        return hipErrorInvalidValue;
    const dim3 grid(8 * a.tiles_per_xcd), block(256);
    if (m.fast)
        hipLaunchKernelGGL((qconv_wv_kernel<0, 2, 1, 4>), grid, block, 0, stream, a);
    else
        hipLaunchKernelGGL((qconv_wv_kernel<0, 2, 0, 4>), grid, block, 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_qconv_wv(const MfmaArgs &a, hipStream_t stream)
{
    const bool wide = a.tile_cfg == TILE_WV144, narrow = a.tile_cfg == TILE_WV64;
    if ((a.bits_out != 4 && a.bits_out != 8 && a.bits_out != 32) || ((wide || narrow) && a.bits_out == 32) ||
        (a.skip_bits != 0 && (a.skip_bits != 4 || a.bits_out != 4)) || a.cin % 256 != 0 ||
        a.ksteps % 4 != 0 || a.ksplit != 1 || a.part != 0 || a.kh > 16 || a.kw > 16)
        return hipErrorInvalidValue;
    // 32-bit buffer offsets and sizes: inputs and weights below 2^31 bytes
    for (int i = 0; i < a.nseg; ++i)
        if ((long long)a.seg[i].n * a.seg[i].h * a.seg[i].w * (a.cin / 2) >= (1LL << 31) ||
            (long long)a.co_tiles * a.ksteps * WV_BCO * KC >= (1LL << 31))
            return hipErrorInvalidValue;
    const dim3 grid(8 * a.tiles_per_xcd);
    bool fast = true;
    for (int i = 0; i < a.nseg; ++i)
        fast = fast && a.seg[i].fast;
    if (wide)
        launch_wv_modes<9>(a, fast, grid, stream);
    else if (narrow)
        launch_wv_modes<4>(a, fast, grid, stream);
    else
        launch_wv_modes<8>(a, fast, grid, stream);
    return hipGetLastError();
}

}  // namespace aqd
