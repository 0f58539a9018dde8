// Implicit-GEMM integer convolution on the gfx950 int8 MFMA
// (v_mfma_i32_16x16x64_i8), with the integer epilogue fused.
//
// GEMM view of a convolution (Sec. 3.2.1, Eq. 4): rows = output channels
// (weights, operand A), columns = output pixels n*ho*wo (operand B, gathered
// from the NHWC input per filter tap), K = taps x input channels; one K step
// is 64 input channels of one tap.
//
// Workgroup: 4 waves in a WC x WP grid; a wave owns MI x NJ accumulator tiles
// of 16 x 16, i.e. 16*MI channels x 16*NJ pixels; the workgroup tile is
// WC*16*MI x WP*16*NJ. Two workgroups share a CU.
//
// Operand path: every K step is copied from global memory straight into LDS
// (global_load_lds_dwordx4, no VGPR staging) into a ring of NSTAGE stages; a
// stage is refilled as soon as every wave has read it, so copies run NSTAGE
// steps ahead of the MFMAs:
//  * weights: int8, decoded and tiled at create ([co_tile][k step][rows][64]),
//    64-byte rows whose 16-byte columns are XOR-swizzled;
//  * activations: the packed b-bit codes as stored in HBM (32 B per pixel and
//    K step at 4 bit, 16 B at 2 bit), 4-bit rows with swizzled 16-byte halves;
//    padding taps copy zeros from a zero page.
// Each wave reads its fragments for step k+1 from LDS into a second register
// set while the MFMAs of step k run, and widens the packed codes to int8 with
// mask/shift word operations. The widening leaves a fixed permutation of the
// 16 channels of a fragment; the weights were stored at create in the same
// permutation, so every dot product is unchanged.
//
// Epilogue: weight rows were permuted at create so that lane group g (lanes
// 16g..16g+15) of accumulator tile i holds channels 4*MI*g + 4i + e
// (e = 0..3): each lane owns 4*MI consecutive channels of one pixel per
// column tile and packs their codes into one store without cross-lane
// traffic. Output codes and skip codes have the input's bitwidth. The
// requantisation uses 32-bit operations when every shift is >= 2: with
// d = 31 + shift, floor((u*M + 2^(d-1)) / 2^d) = (mulhi(u, M) + 2^(d-33)) >>
// (d-32) exactly (u*M = hi*2^32 + lo with 0 <= lo < 2^32 cannot carry into
// the quotient); other levels take the 64-bit path. int32 outputs and int32
// skips pass through LDS so that global accesses cover whole channel runs.
//
// Variants: a part of a split K range writes raw int32 partial sums (summed
// and finished by the split-K epilogue kernel); the fused projection
// shortcut (DUAL) runs a second 1x1 convolution into a second accumulator set
// before the main one and aligns the two in the epilogue.
//
// Workgroup order: consecutive workgroup ids are dispatched round-robin over
// the 8 XCDs; ids are remapped so that each XCD receives a contiguous range
// of tiles (neighbouring pixel tiles of all channel tiles), which keeps the
// gathered input rows and the weights in that XCD's L2.

#include <type_traits>
#include <utility>

#include "epilogue.h"
#include "internal.h"
#include "mfma_common.h"

namespace aqd {
namespace {

// OCC: workgroups per CU the tile is built for (0: two, or one when a wave
// holds 256 accumulators or the workgroup has 8 waves)
template <int BI, int MI, int NJ, int WC, int WP, int OCC = 0>
struct Cfg {
    static constexpr int WPC = WP;                // waves along pixels
    static constexpr int NW = WC * WP;            // waves per workgroup
    static constexpr int NTH = 64 * NW;           // threads per workgroup
    static constexpr int TM = 16 * MI;            // channels per wave
    static constexpr int TN = 16 * NJ;            // pixels per wave
    static constexpr int BCO = WC * TM;           // channels per workgroup
    static constexpr int BPX = WP * TN;           // pixels per workgroup
    static constexpr int PB = KC * BI / 8;        // packed bytes per pixel and K step (32 / 16)
    static constexpr int A_STAGE = BCO * KC;      // int8 weight rows of 64 B
    static constexpr int B_STAGE = BPX * PB;      // packed code rows of PB bytes
    static constexpr int STAGE = A_STAGE + B_STAGE;
    // one workgroup per CU when a wave holds 256 accumulators (they live in the
    // AGPRs: 512 registers per lane at one wave per SIMD), else two
    static constexpr int WG_PER_CU = OCC ? OCC : ((MI * NJ >= 64 || NW == 8) ? 1 : 2);
    static constexpr int WAVES_PER_SIMD = NW / 4 * WG_PER_CU;  // occupancy the register budget targets
    // ring depth: the workgroup's share of the CU's 160 KiB of LDS; the
    // epilogue table reuses the ring after the last K step
    static constexpr int LDS_BUDGET = 163840 / WG_PER_CU / 1024 * 1024;
    static constexpr int NSTAGE = LDS_BUDGET / STAGE < 6 ? LDS_BUDGET / STAGE : 6;
    static constexpr int A_PER = A_STAGE / 1024 / NW;      // 1 KiB copies per wave and K step
    // activation copies: 1 KiB each, or one copy per wave with only BLANES
    // lanes active when the stage is smaller than 1 KiB per wave
    static constexpr int BCH = B_STAGE / NW < 1024 ? B_STAGE / NW : 1024;
    static constexpr int BLANES = BCH / 16;
    static constexpr int B_PER = B_STAGE / BCH / NW;
    static constexpr int NOPS = A_PER + B_PER;             // copy instructions per lane and K step
    static constexpr int BPC = BCH / PB;                   // pixels per copy
    static constexpr int LPP = PB / 16;                    // lanes per pixel row (2 / 1)
    static constexpr int CPL = 4 * MI;                     // channels per lane and pixel (epilogue)
    static constexpr int OW = CPL * BI / 32;               // packed output dwords per lane and pixel
    static_assert(A_STAGE % (1024 * NW) == 0 && B_STAGE % (BCH * NW) == 0 && BCH % PB == 0,
                  "a stage splits into copies, the same number per wave");
    static_assert(NSTAGE >= 2, "ring of at least two stages");
    static_assert(NSTAGE * STAGE >= EPI_FIELDS * BCO * 4, "epilogue table fits in the ring");
};

// OUTK: 0 = codes of width BI, 1 = int32.
// SKK: 0 = none, 1 = codes of width BI, 2 = int32.
// FAST: every segment's shifts are >= 2 (32-bit requantisation).
// DUAL: the int32 skip is a second convolution computed in the same
//   workgroup (a residual block's projection shortcut, 1x1 with stride
//   A.stride2 on the block input x2): its K steps run first into a second
//   accumulator set, then the main convolution's; the epilogue aligns
//   v = acc + bias with v2 = acc2 + bias2 (Eq. 7-8) from registers.
template <int BI, int MI, int NJ, int WC, int WP, int OUTK, int SKK, int FAST, int DUAL = 0, int OCC = 0>
__global__ void __launch_bounds__(64 * WC * WP, (Cfg<BI, MI, NJ, WC, WP, OCC>::WAVES_PER_SIMD)) qconv_mfma_kernel(MfmaArgs A)
{
    static_assert(!DUAL || (OUTK == 0 && SKK == 2), "the projection is an int32 skip of a codes output");
    using C = Cfg<BI, MI, NJ, WC, WP, OCC>;
    constexpr int NT = C::NTH;
    __shared__ __attribute__((aligned(1024))) uint8_t lds_stages[C::NSTAGE * C::STAGE];

    const int bid = blockIdx.x;
    const int logical = (bid & 7) * A.tiles_per_xcd + (bid >> 3);
    if (logical >= A.total_tiles)
        return;
    // work unit -> output tile and part of its K range (the parts of a tile are
    // consecutive units, hence on one XCD)
    const int tile = logical / A.ksplit;
    const int kpart = logical - tile * A.ksplit;

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
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: SGPR arithmetic
    const int wc = wave / C::WPC;
    const int wp = wave % C::WPC;

    const int row_bytes = A.cin * BI / 8;
    const int kpt = A.cin / KC;
    const int kb = kpart * A.kchunk;                   // first K step of this part
    const int KSM = A.ksteps - kb < A.kchunk ? A.ksteps - kb : A.kchunk;  // >= 1 (host)
    const int KS1 = DUAL ? A.ksteps2 : 0;              // projection steps (first)
    const int KS = KS1 + KSM;
    const int hw = S.ho * S.wo;

    // Copies: chunk q of a stage (1 KiB) belongs to wave q % NW; which source
    // bytes a lane fetches implements the LDS swizzle.
    //  weights: chunk q = rows 16q .. 16q+15; lane L -> row 16q + L/4, LDS
    //           column L%4 holding logical column (L%4) ^ swz_a(row)
    //  codes:   chunk q = pixels BPC*q ..; lane L -> pixel BPC*q + L/LPP, LDS
    //           16-byte part L%LPP holding logical part (L%LPP) ^ swz_b4(pixel)
    int a_src[C::A_PER];
#pragma unroll
    for (int t = 0; t < C::A_PER; ++t) {
        const int row = 16 * (C::NW * t + wave) + (lane >> 2);
        a_src[t] = row * KC + 16 * ((lane & 3) ^ swz_a(row));
    }
    int ih0[C::B_PER], iw0[C::B_PER];
    const uint8_t *xb[C::B_PER];
    const uint8_t *xb2[DUAL ? C::B_PER : 1];
    bool pv[C::B_PER];
#pragma unroll
    for (int t = 0; t < C::B_PER; ++t) {
        const int ploc = C::BPC * (C::NW * t + wave) + lane / C::LPP;
        const int part = lane % C::LPP;
        const long long p = (long long)px_tile * C::BPX + ploc;
        pv[t] = p < S.P && lane < C::BLANES;
        const int pn = pv[t] ? (int)(p / hw) : 0;
        const int prem = pv[t] ? (int)(p - (long long)pn * hw) : 0;
        const int oh = prem / S.wo, ow = prem - oh * S.wo;
        const int sw = 16 * (BI == 4 ? (part ^ swz_b4(ploc)) : part);
        ih0[t] = oh * A.stride - A.pad;
        iw0[t] = ow * A.stride - A.pad;
        xb[t] = S.x + (long long)pn * S.h * S.w * row_bytes + sw;
        if constexpr (DUAL)  // 1x1 projection, no padding: always inside its input
            xb2[t] = pv[t] ? S.x2 + (((long long)pn * S.h2 + oh * A.stride2) * S.w2 + ow * A.stride2) *
                                        (A.cin2 * BI / 8) + sw
                           : nullptr;
    }

    // Copy state: steps are issued in order, so the per-pixel source of the
    // current tap is computed once per tap (bsrc; null for padding taps).
    const int8_t *a_next = S.wt + ((long long)co_tile * A.ksteps + kb) * C::A_STAGE;
    const int8_t *a2_next = DUAL ? S.wt2 + (long long)co_tile * KS1 * C::A_STAGE : nullptr;
    int issued = 0;  // steps issued (the first KS1 are the projection's)
    const uint32_t lds_base = lds_addr(lds_stages);
    int tap_next = kb / kpt, cc_next = kb - (kb / kpt) * kpt, st_next = 0;
    const uint8_t *bsrc[C::B_PER];
    // per-pixel sources of tap tap_next (null: the tap falls in the padding)
    auto tap_sources = [&]() {
        const int r = tap_next / A.kw;
        const int q = tap_next - r * A.kw;
#pragma unroll
        for (int t = 0; t < C::B_PER; ++t) {
            const int ih = ih0[t] + r, iw = iw0[t] + q;
            const bool ok = pv[t] && (unsigned)ih < (unsigned)S.h && (unsigned)iw < (unsigned)S.w;
            bsrc[t] = ok ? xb[t] + ((long long)ih * S.w + iw) * row_bytes : nullptr;
        }
    };
    // a part of a split K range may start inside a tap: its sources are set here
    tap_sources();
    // A step's copies are issued in three parts: issue_begin (the tap's
    // sources, at a tap change), issue_copy<d> for d = 0 .. NOPS-1
    // (activation copies first), issue_end (advance to the next step).
    uint32_t st_cur = 0;
    auto issue_begin = [&]() {
        if (!(DUAL && issued < KS1) && cc_next == 0)
            tap_sources();
        st_cur = lds_base + st_next * C::STAGE;
    };
    auto issue_copy = [&](auto d_c) {
        constexpr int d = decltype(d_c)::value;
        const bool proj = DUAL && issued < KS1;
        if constexpr (d < C::B_PER) {
            const uint8_t *src = proj ? (xb2[DUAL ? d : 0] ? xb2[DUAL ? d : 0] + issued * C::PB : A.zero)
                                      : (bsrc[d] ? bsrc[d] + cc_next * C::PB : A.zero);
            if (C::BLANES == 64 || lane < C::BLANES)
                dma16(src, st_cur + C::A_STAGE + (C::NW * d + wave) * C::BCH);
        } else {
            dma16((proj ? a2_next : a_next) + a_src[d - C::B_PER], st_cur + (C::NW * (d - C::B_PER) + wave) * 1024);
        }
    };
    auto issue_end = [&]() {
        if (++st_next == C::NSTAGE)
            st_next = 0;
        if (DUAL && issued < KS1) {
            a2_next += C::A_STAGE;
        } else {
            a_next += C::A_STAGE;
            if (++cc_next == kpt) {
                cc_next = 0;
                ++tap_next;
            }
        }
        if constexpr (DUAL)
            ++issued;
    };
    auto issue = [&]() {
        issue_begin();
        static_for<C::NOPS>([&](auto d_c) { issue_copy(d_c); });
        issue_end();
    };
    // wait until at most `steps` K steps of copies are outstanding
    auto wait_steps = [&](int steps) {
        switch (steps) {
        case 0: wait_vmcnt<0>(); break;
        case 1: wait_vmcnt<C::NOPS>(); break;
        case 2: wait_vmcnt<2 * C::NOPS>(); break;
        case 3: wait_vmcnt<3 * C::NOPS>(); break;
        default: wait_vmcnt<4 * C::NOPS>(); break;
        }
    };

    // accumulators start at the bias (Eq. 6: v = acc + bias, one add per output
    // saved): lane group g of tile i holds channels CPL*g + 4i + e of the wave's
    // rows; a part of a split K range other than the first starts at zero
    v4i acc[MI][NJ];
    v4i acc2[DUAL ? MI : 1][DUAL ? NJ : 1];  // projection accumulators (DUAL)
    {
        const int ch0 = co_tile * C::BCO + wc * C::TM + C::CPL * (lane >> 4);
        const bool with_bias = !(A.part && kpart > 0);
#pragma unroll
        for (int i = 0; i < MI; ++i) {
            v4i b = v4i{0, 0, 0, 0};
            if (with_bias)
                b = *(const v4i *)(S.epi + EPI_BIAS * A.cout_pad + ch0 + 4 * i);
            v4i b2 = v4i{0, 0, 0, 0};
            if constexpr (DUAL)
                b2 = *(const v4i *)(S.epi2 + EPI_BIAS * A.cout_pad + ch0 + 4 * i);
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                acc[i][j] = b;
                if constexpr (DUAL)
                    acc2[i][j] = b2;
            }
        }
    }

    // fragment addresses inside a stage (swizzled as written above)
    const int a_off = (wc * C::TM + (lane & 15)) * KC + 16 * ((lane >> 4) ^ swz_a(lane & 15));
    int b_off;
    if constexpr (BI == 4)
        b_off = C::A_STAGE + (wp * C::TN + (lane & 15)) * C::PB + 8 * ((lane >> 4) ^ (swz_b4(lane & 15) << 1));
    else
        b_off = C::A_STAGE + (wp * C::TN + (lane & 15)) * C::PB + 4 * (lane >> 4);

    using BW = typename std::conditional<BI == 4, uint2, uint32_t>::type;
    v4i fa[2][MI];
    BW fb[2][NJ];
    auto read_a = [&](int stage, v4i *dst, int i) {
        dst[i] = *(const v4i *)(lds_stages + stage * C::STAGE + a_off + i * 16 * KC);
    };
    auto read_b = [&](int stage, BW *dst, int j) {
        dst[j] = *(const BW *)(lds_stages + stage * C::STAGE + b_off + j * 16 * C::PB);
    };
    auto widen = [&](const BW w) -> v4i {
        if constexpr (BI == 4)
            return v4i{(int)(w.x & 0x0F0F0F0Fu), (int)((w.x >> 4) & 0x0F0F0F0Fu),
                       (int)(w.y & 0x0F0F0F0Fu), (int)((w.y >> 4) & 0x0F0F0F0Fu)};
        else
            return v4i{(int)(w & 0x03030303u), (int)((w >> 2) & 0x03030303u),
                       (int)((w >> 4) & 0x03030303u), (int)((w >> 6) & 0x03030303u)};
    };

    // prologue: copies for steps 0 .. NSTAGE-1 (every stage), fragments of step 0
    const int pre = KS < C::NSTAGE ? KS : C::NSTAGE;
    for (int k = 0; k < pre; ++k)
        issue();

    // this channel tile's epilogue table does not depend on the accumulators:
    // it is fetched now, so that its latency hides behind the K loop, and goes
    // to LDS after the last step
    constexpr int PRM_PER = EPI_FIELDS * C::BCO / NT;
    static_assert(EPI_FIELDS * C::BCO % NT == 0, "epilogue table splits evenly over the threads");
    int prm_r[PRM_PER];
#pragma unroll
    for (int t = 0; t < PRM_PER; ++t) {
        const int i = tid + t * NT;
        const int which = i / C::BCO, c = i - which * C::BCO;
        prm_r[t] = S.epi[which * A.cout_pad + co_tile * C::BCO + c];
    }

    constexpr int CPL = C::CPL;
    const int g = lane >> 4;
    const int co_loc = wc * C::TM + CPL * g;      // first of this lane's CPL channels (in the tile)
    const int co_glob = co_tile * C::BCO + co_loc;
    const long long px0 = (long long)px_tile * C::BPX + wp * C::TN + (lane & 15);
    const bool co_ok = co_glob < A.cout;          // CPL channels are all valid or all padding
    bool okj[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j)
        okj[j] = co_ok && px0 + j * 16 < S.P;

    wait_steps(pre - 1);
    __syncthreads();
#pragma unroll
    for (int j = 0; j < NJ; ++j)
        read_b(0, fb[0], j);
#pragma unroll
    for (int i = 0; i < MI; ++i)
        read_a(0, fa[0], i);

    // step ks: MFMAs on register set ks & 1 while the fragments of step ks + 1
    // are read into the other set (after the last step these reads fetch
    // unused data). The stage of step ks was read into registers during step
    // ks - 1; once every wave has those reads back (lgkmcnt(0) + barrier) it is
    // refilled with step ks + NSTAGE, so copies run NSTAGE steps ahead.
    int st_read = 1 % C::NSTAGE;  // stage of step ks + 1
    // steps [kbeg, kend) into the accumulator set ac; register set P = ks & 1
    auto steps = [&](auto &ac, int kbeg, int kend) {
        auto one = [&](auto pc, int ks) {
            constexpr int P = decltype(pc)::value;
            if (ks + 1 < KS) {
                // step ks + 1 landed: copies up to step min(ks + NSTAGE - 1, KS - 1) were issued
                const int last = ks + C::NSTAGE - 1 < KS - 1 ? ks + C::NSTAGE - 1 : KS - 1;
                wait_steps(last - (ks + 1));
                // this wave's fragment reads of stage ks are back
                asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
                // stage ks + 1 visible to every wave, and no wave reads stage ks any more
                asm volatile("s_barrier" ::: "memory");
                if (ks + C::NSTAGE < KS)
                    issue();
            }
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                const v4i bj = widen(fb[P][j]);
#pragma unroll
                for (int i = 0; i < MI; ++i)
                    ac[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[P][i], bj, ac[i][j], 0, 0, 0);
                read_b(st_read, fb[P ^ 1], j);
                if (j < MI)
                    read_a(st_read, fa[P ^ 1], j);
            }
#pragma unroll
            for (int i = NJ; i < MI; ++i)
                read_a(st_read, fa[P ^ 1], i);
            // schedule: per column tile, its widening, then its MI MFMAs with
            // the next step's fragment reads spread between them, so that the
            // LDS latency hides under the matrix cores
            static_for<NJ>([&](auto jc) {
                constexpr int j = decltype(jc)::value;
                constexpr int RD = MI + NJ;                       // fragment reads per step
                constexpr int lo = RD * j / NJ, hi = RD * (j + 1) / NJ;
                __builtin_amdgcn_sched_group_barrier(0x002, BI == 4 ? 6 : 7, 0);  // VALU
                static_for<MI>([&](auto ic) {
                    constexpr int i = decltype(ic)::value;
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);            // MFMA
                    if constexpr (i < hi - lo)
                        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);        // DS read
                });
            });
            if (++st_read == C::NSTAGE)
                st_read = 0;
        };
        using P0 = std::integral_constant<int, 0>;
        using P1 = std::integral_constant<int, 1>;
        int ks = kbeg;
        if ((ks & 1) && ks < kend)
            one(P1{}, ks++);
        for (; ks < kend; ks += 2) {
            one(P0{}, ks);
            if (ks + 1 < kend)
                one(P1{}, ks + 1);
        }
    };
    if constexpr (DUAL)
        steps(acc2, 0, KS1);
    steps(acc, KS1, KS);

    // ---------------------------------------------------------------- epilogue
    // The ring is idle after the last step; it now holds this channel tile's
    // epilogue table, the side-0 skip table and the int32 output staging.
    constexpr int QMAX = (1 << BI) - 1;
    int32_t *prm = (int32_t *)lds_stages;
    int32_t *lut = prm + EPI_FIELDS * C::BCO;            // [BCO][2^BI]: RSM(k, c, d)
    const int32_t *lut_l = lut + (co_loc << BI);         // this lane's channels
    const bool use_lut = SKK == 1 && S.side0;            // uniform over the workgroup
    // skip codes: issued before the table goes to LDS, so that the two overlap
    uint32_t skw[NJ][C::OW];
    static_for<NJ>([&](auto jc) {
        constexpr int j = decltype(jc)::value;
#pragma unroll
        for (int u = 0; u < C::OW; ++u)
            skw[j][u] = 0;
        if constexpr (OUTK == 0 && SKK == 1) {
            if (okj[j]) {
                const long long px = px0 + j * 16;
                long long spix = px;
                if (A.up2) {
                    const int n_ = (int)(px / hw);
                    const int rem = (int)(px - (long long)n_ * hw);
                    const int oh = rem / S.wo, ow = rem - oh * S.wo;
                    spix = ((long long)n_ * S.hs + (oh >> 1)) * S.ws + (ow >> 1);
                }
                load_words<C::OW>((const uint8_t *)S.skip + spix * (A.cout * BI / 8) + co_glob * BI / 8, skw[j]);
            }
        }
    });
    // every skip operand is a b-bit code scaled by c / 2^d (side 0): the
    // channel tile's table of RSM(k, c, d) (built at create) goes to LDS too
    constexpr int LUT_PER = SKK == 1 ? (C::BCO * (QMAX + 1) + NT - 1) / NT : 1;
    int lut_r[LUT_PER];
    if (use_lut) {
#pragma unroll
        for (int t = 0; t < LUT_PER; ++t) {
            const int i = tid + t * NT;
            lut_r[t] = i < C::BCO * (QMAX + 1) ? S.lut[co_tile * C::BCO * (QMAX + 1) + i] : 0;
        }
    }
    __syncthreads();  // every wave is done with the ring
#pragma unroll
    for (int t = 0; t < PRM_PER; ++t)
        prm[tid + t * NT] = prm_r[t];
    if (use_lut) {
#pragma unroll
        for (int t = 0; t < LUT_PER; ++t)
            if (tid + t * NT < C::BCO * (QMAX + 1))
                lut[tid + t * NT] = lut_r[t];
    }
    __syncthreads();

    // int32 tiles (outputs, int32 skips) move between HBM and registers through
    // a per-wave LDS staging area, JP column tiles (16 JP pixel rows) at a time,
    // so that global accesses cover whole contiguous channel runs of a pixel row
    constexpr int ROWB = C::TM * 4 + 16;          // staged row: TM channels + pad (bank spread)
    // column tiles per pass: two when the staging fits in the ring, else one
    constexpr int JP = EPI_FIELDS * C::BCO * 4 + C::NW * 32 * ROWB <= C::NSTAGE * C::STAGE ? 2 : 1;
    constexpr int LPR = C::TM / 4;                // lanes per staged row (16 B each)
    constexpr int RPI = 64 / LPR;                 // rows per instruction
    static_assert((OUTK == 0 && (SKK != 2 || DUAL)) ||
                      EPI_FIELDS * C::BCO * 4 + C::NW * 16 * JP * ROWB <= C::NSTAGE * C::STAGE,
                  "int32 staging fits in the ring");
    static_assert((EPI_FIELDS + 1) * C::BCO * 4 <= C::NSTAGE * C::STAGE, "epilogue tables fit in the ring");
    static_assert(SKK != 1 || (EPI_FIELDS + (QMAX + 1)) * C::BCO * 4 <= C::NSTAGE * C::STAGE,
                  "the skip table fits in the ring");
    uint8_t *stg = lds_stages + EPI_FIELDS * C::BCO * 4 + wave * (16 * JP * ROWB);

    if constexpr (OUTK == 1) {
        static_for<NJ / JP>([&](auto pc) {
            constexpr int pass = decltype(pc)::value;
            static_for<JP>([&](auto jc) {
                constexpr int jj = decltype(jc)::value;
                constexpr int j = pass * JP + jj;
#pragma unroll
                for (int i = 0; i < MI; ++i) {
                    int4 o;  // v = acc + bias (the bias is in the accumulators)
                    o.x = acc[i][j][0];
                    o.y = acc[i][j][1];
                    o.z = acc[i][j][2];
                    o.w = acc[i][j][3];
                    *(int4 *)(stg + (jj * 16 + (lane & 15)) * ROWB + (CPL * g + 4 * i) * 4) = o;
                }
            });
            __syncthreads();
#pragma unroll
            for (int r = 0; r < 16 * JP; r += RPI) {
                const int row = r + lane / LPR;
                const int cw = (lane % LPR) * 4;                       // channel within the wave
                const long long px = (long long)px_tile * C::BPX + wp * C::TN + pass * JP * 16 + row;
                const int ch = co_tile * C::BCO + wc * C::TM + cw;
                const int4 v = *(const int4 *)(stg + row * ROWB + cw * 4);
                if (px < S.P && ch < A.cout)
                    *(int4 *)((int32_t *)S.y + (kpart * S.P + px) * A.cout + ch) = v;
            }
            __syncthreads();  // staging is rewritten by the next pass
        });
        return;
    }

    // packed output codes per pixel column
    uint32_t outw[NJ][C::OW];
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int u = 0; u < C::OW; ++u)
            outw[j][u] = 0;

    // columns [J0, J0 + JN): channel group outer (parameters read once), column inner
    auto body = [&](auto lut_c, auto j0_c, auto jn_c) {
        constexpr bool LUT = decltype(lut_c)::value;
        constexpr int J0 = decltype(j0_c)::value, JN = decltype(jn_c)::value;
        static_for<MI>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            const int cl = co_loc + 4 * i;
            const int4 m4 = *(const int4 *)(prm + EPI_MULT * C::BCO + cl);
            const int4 s4 = *(const int4 *)(prm + (FAST ? EPI_SHR : EPI_SHIFT) * C::BCO + cl);
            const int mult[4] = {m4.x, m4.y, m4.z, m4.w};
            const int shf[4] = {s4.x, s4.y, s4.z, s4.w};
            long long rnd[4] = {0, 0, 0, 0};  // 2^(shift-2) in the high word
            if constexpr (FAST) {
                const int4 r4 = *(const int4 *)(prm + EPI_RND * C::BCO + cl);
                rnd[0] = (long long)r4.x << 32; rnd[1] = (long long)r4.y << 32;
                rnd[2] = (long long)r4.z << 32; rnd[3] = (long long)r4.w << 32;
            }
            int sc[4] = {0, 0, 0, 0}, sd[4] = {0, 0, 0, 0}, sside[4] = {0, 0, 0, 0};
            long long srnd[4] = {0, 0, 0, 0};  // rounding terms of the alignment
            if constexpr (SKK != 0 && !LUT) {
                const int4 c4 = *(const int4 *)(prm + EPI_SKIP_C * C::BCO + cl);
                const int4 d4 = *(const int4 *)(prm + EPI_SKIP_D * C::BCO + cl);
                const int4 e4 = *(const int4 *)(prm + EPI_SKIP_SIDE * C::BCO + cl);
                sc[0] = c4.x; sc[1] = c4.y; sc[2] = c4.z; sc[3] = c4.w;
                sd[0] = d4.x; sd[1] = d4.y; sd[2] = d4.z; sd[3] = d4.w;
                srnd[0] = rsm_rnd(d4.x); srnd[1] = rsm_rnd(d4.y); srnd[2] = rsm_rnd(d4.z); srnd[3] = rsm_rnd(d4.w);
                sside[0] = e4.x; sside[1] = e4.y; sside[2] = e4.z; sside[3] = e4.w;
            }
            static_for<JN>([&](auto jc) {
                constexpr int j = J0 + decltype(jc)::value;
                if (!okj[j])
                    return;
                int kv[4] = {0, 0, 0, 0};
                if constexpr (DUAL) {
                    // v2 = acc2 (its bias included), the projection's int32 output
                    kv[0] = acc2[i][j][0];
                    kv[1] = acc2[i][j][1];
                    kv[2] = acc2[i][j][2];
                    kv[3] = acc2[i][j][3];
                } else if constexpr (SKK == 2) {
                    const int4 k4 = *(const int4 *)(stg + ((j - J0) * 16 + (lane & 15)) * ROWB + (CPL * g + 4 * i) * 4);
                    kv[0] = k4.x; kv[1] = k4.y; kv[2] = k4.z; kv[3] = k4.w;
                } else if constexpr (SKK == 1) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int bit = (4 * i + e) * BI;
                        kv[e] = (int)__builtin_amdgcn_ubfe(skw[j][bit >> 5], bit & 31, BI);
                    }
                }
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int v = acc[i][j][e];  // acc + bias
                    int y;
                    if constexpr (FAST) {
                        int u = v;
                        // u fits in int32, so the sum modulo 2^32 is exact
                        if constexpr (LUT) {
                            u = (int)((unsigned)v + (unsigned)lut_l[((4 * i + e) << BI) + kv[e]]);
                        } else if constexpr (SKK != 0) {
                            const int scaled = rsm32r(sside[e] ? v : kv[e], sc[e], srnd[e], sd[e]);
                            u = (int)((unsigned)scaled + (unsigned)(sside[e] ? kv[e] : v));
                        }
                        y = requant32(u, mult[e], rnd[e], shf[e]);
                        y = y < 0 ? 0 : (y > QMAX ? QMAX : y);
                    } else {
                        long long u = v;
                        if constexpr (LUT)
                            u = (int)((unsigned)v + (unsigned)lut_l[((4 * i + e) << BI) + kv[e]]);
                        else if constexpr (SKK != 0)
                            u = align_add(v, kv[e], sc[e], sd[e], sside[e]);
                        y = (int)requant_clamp(u, mult[e], shf[e], QMAX);
                        asm volatile("" : "+v"(y));  // one 64-bit product alive at a time
                    }
                    const int bit = (4 * i + e) * BI;
                    outw[j][bit >> 5] |= (uint32_t)y << (bit & 31);
                }
            });
        });
    };
    using I0 = std::integral_constant<int, 0>;
    using INJ = std::integral_constant<int, NJ>;
    if constexpr (DUAL) {
        body(std::false_type{}, I0{}, INJ{});
    } else if constexpr (SKK == 2) {
        // int32 skip: JP column tiles per pass, staged with row-contiguous loads
        static_for<NJ / JP>([&](auto pc) {
            constexpr int pass = decltype(pc)::value;
#pragma unroll
            for (int r = 0; r < 16 * JP; r += RPI) {
                const int row = r + lane / LPR;
                const int cw = (lane % LPR) * 4;
                const long long px = (long long)px_tile * C::BPX + wp * C::TN + pass * JP * 16 + row;
                const int ch = co_tile * C::BCO + wc * C::TM + cw;
                int4 v = make_int4(0, 0, 0, 0);
                if (px < S.P && ch < A.cout) {
                    long long spix = px;
                    if (A.up2) {
                        const int n_ = (int)(px / hw);
                        const int rem = (int)(px - (long long)n_ * hw);
                        const int oh = rem / S.wo, ow = rem - oh * S.wo;
                        spix = ((long long)n_ * S.hs + (oh >> 1)) * S.ws + (ow >> 1);
                    }
                    v = *(const int4 *)((const int32_t *)S.skip + spix * A.cout + ch);
                }
                *(int4 *)(stg + row * ROWB + cw * 4) = v;
            }
            __syncthreads();
            body(std::false_type{}, std::integral_constant<int, pass * JP>{},
                 std::integral_constant<int, JP>{});
            __syncthreads();  // staging is rewritten by the next pass
        });
    } else if constexpr (SKK == 1) {
        if (use_lut)
            body(std::true_type{}, I0{}, INJ{});
        else
            body(std::false_type{}, I0{}, INJ{});
    } else {
        body(std::false_type{}, I0{}, INJ{});
    }

    if (BI == 4 && A.qmax == 7) {  // 3-bit codes (the epilogue clamped to 15)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
            for (int u = 0; u < C::OW; ++u)
                outw[j][u] = sat7_nibbles(outw[j][u]);
    }
    static_for<NJ>([&](auto jc) {
        constexpr int j = decltype(jc)::value;
        if (okj[j])
            store_words<C::OW>((uint8_t *)S.y + (px0 + j * 16) * (A.cout * BI / 8) + co_glob * BI / 8, outw[j]);
    });
}

// ------------------------------------------------------------------ streaming
// 1x1 convolutions with at most ST_KMAX K steps (cin <= 128), 4-bit code
// outputs and no skip or a code skip: per 256 x 64 tile the matrix cores have
// little to do, and a workgroup that does one tile spends its time waiting for
// its copies and in the epilogue. This persistent variant runs two
// workgroups per CU; each keeps its channel tile's weights (every K step) in
// LDS and walks over pixel tiles, copying the activation codes and skip codes
// of its next tile into the other half of a double buffer while the current
// tile's MFMAs and epilogue run. Everything a tile's epilogue reads (table,
// skip table, skip codes) is in LDS, so that the only waits for global memory
// are the explicit ones at the top of each tile.
// SKK: 0 = no skip, 1 = code skip, 2 = a residual block's projection shortcut
// fused in (1x1 of x2 with one K step, int32, aligned with v as in Eq. 7-8;
// the main convolution then has one K step too): its weights and codes use
// the second K-step slots of the weight and code buffers.
// Shapes (4 waves, two workgroups per CU, 32 pixels per wave): MI = 8, WC = 2:
// 256 channels x 64 pixels, up to 2 K steps (handles laid out for 256-channel
// tiles); MI = 4, WC = 2: 128 x 64, up to 4 K steps; MI = 4, WC = 1: 64 x 128,
// up to 4 K steps (the latter two without skip).
// HV = 1 (MI = 4, WC = 2): a handle laid out for 256-channel tiles read as two
// 128-channel tiles (weights of a 256-row tile: rows 128h .. 128h+127 of
// each K step), up to 4 K steps, with or without a code skip: a lane of
// lane group g in wave wc holds channels 32g + 16wc .. 32g + 16wc + 15.
template <int SKK, int FAST, int MI = 8, int WC = 2, int HV = 0>
__global__ void __launch_bounds__(256, 2) qconv_stream_kernel(MfmaArgs A)
{
    constexpr int BI = 4, NJ = 2, WPC = 4 / WC, NT = 256;
    constexpr int TM = 16 * MI, TN = 32, BCO = WC * TM, BPX = TN * WPC, PB = KC * BI / 8;
    constexpr int ST_KMAX = BCO == 256 ? 2 : 4;
    constexpr int PPW = BPX / 4;                   // pixels each wave copies (16 or 32)
    static_assert(!HV || (MI == 4 && WC == 2), "the half view reads 128-row halves of 256-row tiles");
    static_assert(SKK == 0 || BCO == 256 || (HV && SKK == 1), "skips on 256-channel tiles or the half view");
    constexpr int CPL = 4 * MI, OW = CPL * BI / 32, QMAX = (1 << BI) - 1;
    constexpr int A_STEP = BCO * KC;               // int8 weight rows of one K step (16 KiB)
    constexpr int B_STEP = BPX * PB;               // packed codes of one K step (2 KiB)
    constexpr int SK_TILE = BPX * BCO * BI / 8;    // skip codes of one tile (8 KiB; 4 KiB for the half view)
    constexpr int OFF_B = ST_KMAX * A_STEP;
    constexpr int OFF_S = OFF_B + 2 * ST_KMAX * B_STEP;
    constexpr int OFF_P = OFF_S + (SKK == 1 ? 2 * SK_TILE : 0);
    constexpr int OFF_L = OFF_P + EPI_FIELDS * BCO * 4;   // skip table (SKK 1) or the shortcut's bias (SKK 2)
    constexpr int LDS_BYTES = OFF_L + (SKK == 1 ? BCO * (QMAX + 1) * 4 : SKK == 2 ? BCO * 4 : 0);
    static_assert(LDS_BYTES <= 81920, "two workgroups per CU");
    __shared__ __attribute__((aligned(1024))) uint8_t lds[LDS_BYTES];
    int32_t *prm = (int32_t *)(lds + OFF_P);
    int32_t *lut = (int32_t *)(lds + OFF_L);       // [BCO][2^BI]: RSM(k, c, d)
    int32_t *bias2 = (int32_t *)(lds + OFF_L);     // [BCO]: the shortcut's bias

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wc = wave / WPC, wp = wave % WPC;
    const int g = lane >> 4;
    // workgroup -> channel tile (fixed) and a stride-nstream walk over the
    // pixel tiles of every segment
    const int co_tile = blockIdx.x % A.co_tiles;
    const int nstream = gridDim.x / A.co_tiles;
    const int qtiles = A.total_tiles / A.co_tiles;
    const int K = A.ksteps;
    const uint32_t lbase = lds_addr(lds);

    auto seg_of = [&](int q) {
        int s = 0;
#pragma unroll
        for (int i = 1; i < AQD_MAX_SEGS; ++i)
            if (i < A.nseg && q * A.co_tiles >= A.seg[i].tile_begin)
                s = i;
        return s;
    };

    // copies of pixel tile q into buffer b: K steps of codes (wave w: pixels
    // 16w .. 16w+15, 32 lanes, swizzled halves as in the main kernel) and the
    // tile's skip codes (128 B per pixel, 16-byte chunk c of pixel p at
    // position c ^ (p & 7))
    auto issue_tile = [&](int q, int b) {
        const MfmaSeg &S = A.seg[seg_of(q)];
        const int pq = q - S.tile_begin / A.co_tiles;
        const int hw = S.ho * S.wo;
        {
            const int ploc = PPW * wave + (lane >> 1);
            const long long p = (long long)pq * BPX + ploc;
            const uint8_t *src = nullptr;
            if (p < S.P) {  // P < 2^31 (host): 32-bit index arithmetic
                if (A.stride == 1) {  // 1x1, no padding: input pixel p
                    src = S.x + p * (A.cin * BI / 8) + 16 * ((lane & 1) ^ swz_b4(ploc));
                } else {
                    const int n_ = (int)p / hw;
                    const int rem = (int)p - n_ * hw;
                    const int oh = rem / S.wo, ow = rem - oh * S.wo;
                    src = S.x + (((long long)n_ * S.h + oh * A.stride) * S.w + ow * A.stride) * (A.cin * BI / 8) +
                          16 * ((lane & 1) ^ swz_b4(ploc));
                }
            }
            for (int k = 0; k < K; ++k)
                if (PPW == 32 || lane < 2 * PPW)
                    dma16(src ? src + k * PB : A.zero,
                          lbase + OFF_B + (b * ST_KMAX + k) * B_STEP + wave * (PPW * PB));
            if constexpr (SKK == 2) {
                // the shortcut's input pixel (1x1, stride A.stride2, always inside x2)
                const uint8_t *src2 = A.zero;
                if (p < S.P) {
                    if (A.stride2 == 1) {  // x2 has the output's size: pixel p
                        src2 = S.x2 + p * (A.cin2 * BI / 8) + 16 * ((lane & 1) ^ swz_b4(ploc));
                    } else {
                        const int n_ = (int)p / hw;
                        const int rem = (int)p - n_ * hw;
                        const int oh = rem / S.wo, ow = rem - oh * S.wo;
                        src2 = S.x2 + (((long long)n_ * S.h2 + oh * A.stride2) * S.w2 + ow * A.stride2) *
                                          (A.cin2 * BI / 8) + 16 * ((lane & 1) ^ swz_b4(ploc));
                    }
                }
                if (lane < 32)
                    dma16(src2, lbase + OFF_B + (b * ST_KMAX + 1) * B_STEP + wave * 512);
            }
        }
        if constexpr (SKK == 1 && HV) {
            // 64 B per pixel: 4 lanes per pixel, 16 pixels per wave, 16-byte
            // chunk c of pixel p at position c ^ (p & 3)
            const int ploc = wave * 16 + (lane >> 2);
            const long long p = (long long)pq * BPX + ploc;
            const uint8_t *src = A.zero;
            if (p < S.P) {
                long long spix = p;
                if (A.up2) {
                    const int n_ = (int)p / hw;
                    const int rem = (int)p - n_ * hw;
                    const int oh = rem / S.wo, ow = rem - oh * S.wo;
                    spix = ((long long)n_ * S.hs + (oh >> 1)) * S.ws + (ow >> 1);
                }
                src = (const uint8_t *)S.skip + spix * (A.cout * BI / 8) + co_tile * (BCO * BI / 8) +
                      16 * ((lane & 3) ^ (ploc & 3));
            }
            dma16(src, lbase + OFF_S + b * SK_TILE + wave * 1024);
        } else if constexpr (SKK == 1) {
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                const int ploc = (2 * wave + c) * 8 + (lane >> 3);
                const long long p = (long long)pq * BPX + ploc;
                const uint8_t *src = A.zero;
                if (p < S.P) {
                    long long spix = p;
                    if (A.up2) {
                        const int n_ = (int)p / hw;
                        const int rem = (int)p - n_ * hw;
                        const int oh = rem / S.wo, ow = rem - oh * S.wo;
                        spix = ((long long)n_ * S.hs + (oh >> 1)) * S.ws + (ow >> 1);
                    }
                    src = (const uint8_t *)S.skip + spix * (A.cout * BI / 8) + co_tile * (BCO * BI / 8) +
                          16 * ((lane & 7) ^ (ploc & 7));
                }
                dma16(src, lbase + OFF_S + b * SK_TILE + (2 * wave + c) * 1024);
            }
        }
    };

    // fragment addresses (the main kernel's swizzles)
    const int a_off = (wc * TM + (lane & 15)) * KC + 16 * ((lane >> 4) ^ swz_a(lane & 15));
    const int b_off = OFF_B + (wp * TN + (lane & 15)) * PB + 8 * ((lane >> 4) ^ (swz_b4(lane & 15) << 1));
    // first of this lane's CPL channels (in the tile)
    const int co_loc = HV ? 32 * g + 16 * wc : wc * TM + CPL * g;
    const int co_glob = co_tile * BCO + co_loc;

    int q = blockIdx.x / A.co_tiles;
    int cur = -1, buf = 0;
    if (q < qtiles)
        issue_tile(q, 0);
    for (; q < qtiles; q += nstream, buf ^= 1) {
        const int s = seg_of(q);
        const MfmaSeg &S = A.seg[s];
        wait_vmcnt<0>();   // this tile's copies (and the last tile's stores) are done
        __syncthreads();   // ... for every wave, and every wave is done with the last tile
        if (s != cur) {
            // the segment's weights (every K step) and tables
            for (int k = 0; k < K; ++k)
#pragma unroll
                for (int t = 0; t < BCO / 64; ++t) {
                    const int row = 16 * (4 * t + wave) + (lane >> 2);
                    // the half view: half (co_tile & 1) of a 256-row tile (the row
                    // swizzle depends on the row modulo 8 only)
                    const long long step = HV ? ((long long)(co_tile >> 1) * A.ksteps + k) * 2 + (co_tile & 1)
                                              : (long long)co_tile * A.ksteps + k;
                    dma16(S.wt + step * A_STEP + row * KC + 16 * ((lane & 3) ^ swz_a(row)),
                          lbase + k * A_STEP + (4 * t + wave) * 1024);
                }
#pragma unroll
            for (int t = 0; t < EPI_FIELDS * BCO / NT; ++t) {
                const int i = tid + t * NT;
                const int which = i / BCO, c = i - which * BCO;
                prm[i] = S.epi[which * A.cout_pad + co_tile * BCO + c];
            }
            if (SKK == 1 && S.side0) {
#pragma unroll
                for (int t = 0; t < BCO * (QMAX + 1) / NT; ++t)
                    lut[tid + t * NT] = S.lut[co_tile * BCO * (QMAX + 1) + tid + t * NT];
            }
            if constexpr (SKK == 2) {
                // the shortcut's weights in the second K-step slot, its bias
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const int row = 16 * (4 * t + wave) + (lane >> 2);
                    dma16(S.wt2 + (long long)co_tile * A.ksteps2 * A_STEP + row * KC + 16 * ((lane & 3) ^ swz_a(row)),
                          lbase + A_STEP + (4 * t + wave) * 1024);
                }
                bias2[tid] = S.epi2[EPI_BIAS * A.cout_pad + co_tile * BCO + tid];
            }
            wait_vmcnt<0>();
            __syncthreads();
            cur = s;
        }
        if (q + nstream < qtiles)
            issue_tile(q + nstream, buf ^ 1);

        // the shortcut first: v2 = acc2 + bias2
        v4i acc2[SKK == 2 ? MI : 1][SKK == 2 ? NJ : 1];
        if constexpr (SKK == 2) {
#pragma unroll
            for (int i = 0; i < MI; ++i) {
                const v4i b = *(const v4i *)(bias2 + co_loc + 4 * i);
#pragma unroll
                for (int j = 0; j < NJ; ++j)
                    acc2[i][j] = b;
            }
            v4i fa[MI];
            uint2 fb[NJ];
#pragma unroll
            for (int j = 0; j < NJ; ++j)
                fb[j] = *(const uint2 *)(lds + b_off + (buf * ST_KMAX + 1) * B_STEP + j * 16 * PB);
#pragma unroll
            for (int i = 0; i < MI; ++i)
                fa[i] = *(const v4i *)(lds + A_STEP + a_off + i * 16 * KC);
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                const uint2 w = fb[j];
                const v4i bj = v4i{(int)(w.x & 0x0F0F0F0Fu), (int)((w.x >> 4) & 0x0F0F0F0Fu),
                                   (int)(w.y & 0x0F0F0F0Fu), (int)((w.y >> 4) & 0x0F0F0F0Fu)};
#pragma unroll
                for (int i = 0; i < MI; ++i)
                    acc2[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[i], bj, acc2[i][j], 0, 0, 0);
            }
        }

        // MFMAs: accumulators start at the bias (v = acc + bias)
        v4i acc[MI][NJ];
#pragma unroll
        for (int i = 0; i < MI; ++i) {
            const v4i b = *(const v4i *)(prm + EPI_BIAS * BCO + co_loc + 4 * i);
#pragma unroll
            for (int j = 0; j < NJ; ++j)
                acc[i][j] = b;
        }
#pragma unroll
        for (int k = 0; k < (SKK == 2 ? 1 : ST_KMAX); ++k) {
            if (k < K) {
                v4i fa[MI];
                uint2 fb[NJ];
#pragma unroll
                for (int j = 0; j < NJ; ++j)
                    fb[j] = *(const uint2 *)(lds + b_off + (buf * ST_KMAX + k) * B_STEP + j * 16 * PB);
#pragma unroll
                for (int i = 0; i < MI; ++i)
                    fa[i] = *(const v4i *)(lds + k * A_STEP + a_off + i * 16 * KC);
#pragma unroll
                for (int j = 0; j < NJ; ++j) {
                    const uint2 w = fb[j];
                    const v4i bj = v4i{(int)(w.x & 0x0F0F0F0Fu), (int)((w.x >> 4) & 0x0F0F0F0Fu),
                                       (int)(w.y & 0x0F0F0F0Fu), (int)((w.y >> 4) & 0x0F0F0F0Fu)};
#pragma unroll
                    for (int i = 0; i < MI; ++i)
                        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[i], bj, acc[i][j], 0, 0, 0);
                }
            }
        }

        // epilogue
        const int pq = q - S.tile_begin / A.co_tiles;
        const long long px0 = (long long)pq * BPX + wp * TN + (lane & 15);
        const bool co_ok = co_glob < A.cout;
        const bool use_lut = SKK == 1 && S.side0;
        const int32_t *lut_l = lut + (co_loc << BI);  // this lane's channels
        const uint32_t lut_base = (uint32_t)(OFF_L + (co_loc << (BI + 2)));
        uint32_t outw[NJ][OW];
        uint32_t skw[NJ][OW];
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
#pragma unroll
            for (int u = 0; u < OW; ++u)
                outw[j][u] = skw[j][u] = 0;
            if constexpr (SKK == 1 && HV) {
                // this lane's 16 channels: logical chunk g, half wc
                const int ploc = wp * TN + j * 16 + (lane & 15);
                const uint2 t = *(const uint2 *)(lds + OFF_S + buf * SK_TILE + ploc * (BCO * BI / 8) +
                                                 16 * (g ^ (ploc & 3)) + 8 * wc);
                skw[j][0] = t.x;
                skw[j][1] = t.y;
            } else if constexpr (SKK == 1) {
                const int ploc = wp * TN + j * 16 + (lane & 15);
                const uint4 t = *(const uint4 *)(lds + OFF_S + buf * SK_TILE + ploc * (BCO * BI / 8) +
                                                 16 * ((wc * 4 + g) ^ (ploc & 7)));
                skw[j][0] = t.x;
                skw[j][1] = t.y;
                skw[j][2] = t.z;
                skw[j][3] = t.w;
            }
        }
        auto body = [&](auto lut_c) {
            constexpr bool LUT = decltype(lut_c)::value;
            // table byte offsets 4k of the skip codes, one per byte: even
            // nibbles of each word in kev, odd ones in kod
            uint32_t kev[NJ][OW], kod[NJ][OW];
#pragma unroll
            for (int j = 0; j < NJ; ++j)
#pragma unroll
                for (int u = 0; u < OW; ++u) {
                    kev[j][u] = (skw[j][u] << 2) & 0x3C3C3C3Cu;
                    kod[j][u] = (skw[j][u] >> 2) & 0x3C3C3C3Cu;
                }
            static_for<MI>([&](auto ic) {
                constexpr int i = decltype(ic)::value;
                const int cl = co_loc + 4 * i;
                const int4 m4 = *(const int4 *)(prm + EPI_MULT * BCO + cl);
                const int4 s4 = *(const int4 *)(prm + (FAST ? EPI_SHR : EPI_SHIFT) * BCO + cl);
                const int mult[4] = {m4.x, m4.y, m4.z, m4.w};
                const int shf[4] = {s4.x, s4.y, s4.z, s4.w};
                long long rnd[4] = {0, 0, 0, 0};
                if constexpr (FAST) {
                    const int4 r4 = *(const int4 *)(prm + EPI_RND * BCO + cl);
                    rnd[0] = (long long)r4.x << 32; rnd[1] = (long long)r4.y << 32;
                    rnd[2] = (long long)r4.z << 32; rnd[3] = (long long)r4.w << 32;
                }
                int sc[4] = {0, 0, 0, 0}, sd[4] = {0, 0, 0, 0}, sside[4] = {0, 0, 0, 0};
                long long srnd[4] = {0, 0, 0, 0};  // rounding terms of the alignment
                if constexpr (SKK != 0 && !LUT) {
                    const int4 c4 = *(const int4 *)(prm + EPI_SKIP_C * BCO + cl);
                    const int4 d4 = *(const int4 *)(prm + EPI_SKIP_D * BCO + cl);
                    const int4 e4 = *(const int4 *)(prm + EPI_SKIP_SIDE * BCO + cl);
                    sc[0] = c4.x; sc[1] = c4.y; sc[2] = c4.z; sc[3] = c4.w;
                    sd[0] = d4.x; sd[1] = d4.y; sd[2] = d4.z; sd[3] = d4.w;
                    srnd[0] = rsm_rnd(d4.x); srnd[1] = rsm_rnd(d4.y); srnd[2] = rsm_rnd(d4.z); srnd[3] = rsm_rnd(d4.w);
                    sside[0] = e4.x; sside[1] = e4.y; sside[2] = e4.z; sside[3] = e4.w;
                }
                static_for<NJ>([&](auto jc) {
                    constexpr int j = decltype(jc)::value;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int v = acc[i][j][e];  // acc + bias
                        const int bit = (4 * i + e) * BI;
                        int kv = 0;
                        if constexpr (SKK == 1 && !LUT)
                            kv = (int)__builtin_amdgcn_ubfe(skw[j][bit >> 5], bit & 31, BI);
                        else if constexpr (SKK == 2)
                            kv = acc2[i][j][e];  // v2 = acc2 + bias2
                        // the table entry of this channel and code (LUT)
                        auto lut_at = [&]() {
                            const int n = (4 * i + e) & 7;  // nibble in its word (a constant once unrolled)
                            const uint32_t w = (n & 1) ? kod[j][bit >> 5] : kev[j][bit >> 5];
                            const uint32_t a = add_byte(lut_base, w, n >> 1);
                            return *(const int32_t *)((const uint8_t *)lds + a + ((4 * i + e) << (BI + 2)));
                        };
                        int y;
                        if constexpr (FAST) {
                            int u = v;
                            // u fits in int32, so the sum modulo 2^32 is exact
                            if constexpr (LUT) {
                                u = (int)((unsigned)v + (unsigned)lut_at());
                            } else if constexpr (SKK != 0) {
                                const int scaled = rsm32r(sside[e] ? v : kv, sc[e], srnd[e], sd[e]);
                                u = (int)((unsigned)scaled + (unsigned)(sside[e] ? kv : v));
                            }
                            y = requant32(u, mult[e], rnd[e], shf[e]);
                            y = y < 0 ? 0 : (y > QMAX ? QMAX : y);
                        } else {
                            long long u = v;
                            if constexpr (LUT)
                                u = (int)((unsigned)v + (unsigned)lut_at());
                            else if constexpr (SKK != 0)
                                u = align_add(v, kv, sc[e], sd[e], sside[e]);
                            y = (int)requant_clamp(u, mult[e], shf[e], QMAX);
                            asm volatile("" : "+v"(y));  // one 64-bit product alive at a time
                        }
                        outw[j][bit >> 5] |= (uint32_t)y << (bit & 31);
                    }
                });
            });
        };
        if (use_lut)
            body(std::true_type{});
        else
            body(std::false_type{});
        if (A.qmax == 7) {  // 3-bit codes (the epilogue clamped to 15)
#pragma unroll
            for (int j = 0; j < NJ; ++j)
#pragma unroll
                for (int u = 0; u < OW; ++u)
                    outw[j][u] = sat7_nibbles(outw[j][u]);
        }
#pragma unroll
        for (int j = 0; j < NJ; ++j)
            if (co_ok && px0 + j * 16 < S.P)
                store_words<OW>((uint8_t *)S.y + (px0 + j * 16) * (A.cout * BI / 8) + co_glob * BI / 8, outw[j]);
    }
}

template <int BI, int MI, int NJ, int WC, int WP, int OUTK, int SKK, int OCC = 0>
hipError_t launch_t(const MfmaArgs &a, hipStream_t stream)
{
    dim3 grid(8 * a.tiles_per_xcd), block(64 * WC * WP);
    bool fast = true;
    for (int i = 0; i < a.nseg; ++i)
        fast = fast && a.seg[i].fast;
    if (OUTK == 1 || fast)
        hipLaunchKernelGGL((qconv_mfma_kernel<BI, MI, NJ, WC, WP, OUTK, SKK, 1, 0, OCC>), grid, block, 0, stream, a);
    else
        hipLaunchKernelGGL((qconv_mfma_kernel<BI, MI, NJ, WC, WP, OUTK, SKK, 0, 0, OCC>), grid, block, 0, stream, a);
    return hipGetLastError();
}

// half-width pixel tiles, three workgroups per CU, for handles laid out for
// 128- and 64-channel tiles (same weight layout): outputs without skip
template <int MI, int NJ, int WC, int WP>
hipError_t launch_occ3(const MfmaArgs &a, hipStream_t stream)
{
    if (a.skip_bits != 0)
        return hipErrorInvalidValue;
    if (a.bits_out == 32)
        return launch_t<4, MI, NJ, WC, WP, 1, 0, 3>(a, stream);
    if (a.bits_out != 4)
        return hipErrorInvalidValue;
    return launch_t<4, MI, NJ, WC, WP, 0, 0, 3>(a, stream);
}

template <int BI, int MI, int NJ, int WC, int WP>
hipError_t launch_modes(const MfmaArgs &a, hipStream_t stream)
{
    if (a.bits_out == 32)
        return a.skip_bits ? hipErrorInvalidValue : launch_t<BI, MI, NJ, WC, WP, 1, 0>(a, stream);
    if (a.bits_out != BI)
        return hipErrorInvalidValue;
    if (a.skip_bits == 0)
        return launch_t<BI, MI, NJ, WC, WP, 0, 0>(a, stream);
    if (a.skip_bits == 32)
        return launch_t<BI, MI, NJ, WC, WP, 0, 2>(a, stream);
    if (a.skip_bits == BI)
        return launch_t<BI, MI, NJ, WC, WP, 0, 1>(a, stream);
    return hipErrorInvalidValue;
}

}  // namespace

void mfma_tile_shape(int tile_cfg, int *blk_co, int *blk_px, int *chan_per_lane)
{
    switch (tile_cfg) {
    case TILE_256x128: *blk_co = 256; *blk_px = 128; *chan_per_lane = 32; return;
    case TILE_WV: *blk_co = 256; *blk_px = 128; *chan_per_lane = 16; return;
    case TILE_WV144: *blk_co = 256; *blk_px = 144; *chan_per_lane = 16; return;
    case TILE_WV64:
    case TILE_WVS: *blk_co = 256; *blk_px = 64; *chan_per_lane = 16; return;
    case TILE_FP4:
    case TILE_B8: *blk_co = 256; *blk_px = 128; *chan_per_lane = 32; return;
    case TILE_STEM: *blk_co = 64; *blk_px = 128; *chan_per_lane = 16; return;
    case TILE_256x64S:
    case TILE_256x64:
    case TILE_STREAM: *blk_co = 256; *blk_px = 64; *chan_per_lane = 32; return;
    case TILE_STREAM_C128: *blk_co = 128; *blk_px = 64; *chan_per_lane = 16; return;
    case TILE_STREAM_H128: *blk_co = 128; *blk_px = 64; *chan_per_lane = 32; return;
    case TILE_STREAM_C64: *blk_co = 64; *blk_px = 128; *chan_per_lane = 16; return;
    case TILE_128x128_O3: *blk_co = 128; *blk_px = 128; *chan_per_lane = 16; return;
    case TILE_64x256_O3: *blk_co = 64; *blk_px = 256; *chan_per_lane = 16; return;
    case TILE_128x256: *blk_co = 128; *blk_px = 256; *chan_per_lane = 16; return;
    default: *blk_co = 64; *blk_px = 512; *chan_per_lane = 16; return;
    }
}

// 256 x 64 tiles, three workgroups per CU: short K ranges (up to 4 steps)
// with code outputs, where the epilogue, not the matrix cores, sets the pace
hipError_t launch_qconv_short(const MfmaArgs &a, hipStream_t stream)
{
    constexpr int BI = 4, MI = 8, NJ = 2, WC = 2, WP = 2, OCC = 3;
    if (a.bits_out != BI || (a.skip_bits != 0 && a.skip_bits != BI))
        return hipErrorInvalidValue;
    dim3 grid(8 * a.tiles_per_xcd), block(64 * WC * WP);
    bool fast = true;
    for (int i = 0; i < a.nseg; ++i)
        fast = fast && a.seg[i].fast;
    if (a.skip_bits == 0) {
        if (fast)
            hipLaunchKernelGGL((qconv_mfma_kernel<BI, MI, NJ, WC, WP, 0, 0, 1, 0, OCC>), grid, block, 0, stream, a);
        else
            hipLaunchKernelGGL((qconv_mfma_kernel<BI, MI, NJ, WC, WP, 0, 0, 0, 0, OCC>), grid, block, 0, stream, a);
    } else {
        if (fast)
            hipLaunchKernelGGL((qconv_mfma_kernel<BI, MI, NJ, WC, WP, 0, 1, 1, 0, OCC>), grid, block, 0, stream, a);
        else
            hipLaunchKernelGGL((qconv_mfma_kernel<BI, MI, NJ, WC, WP, 0, 1, 0, 0, OCC>), grid, block, 0, stream, a);
    }
    return hipGetLastError();
}

// streaming 256 x 64 tiles: two persistent workgroups per CU (a multiple of
// the channel tiles, each workgroup on one channel tile)
hipError_t launch_qconv_stream(const MfmaArgs &a, hipStream_t stream)
{
    // skip_bits 32: the fused projection shortcut, one K step each
    const bool dual = a.skip_bits == 32;
    const bool hv = a.tile_cfg == TILE_STREAM_H128;
    const int bco = a.tile_cfg == TILE_STREAM ? 256 : (a.tile_cfg == TILE_STREAM_C128 || hv) ? 128 : 64;
    const int kmax = bco == 256 ? 2 : 4;
    if (a.ksteps > kmax || a.bits_out != 4 || (a.skip_bits != 0 && a.skip_bits != 4 && !dual) ||
        (bco != 256 && a.skip_bits != 0 && !(hv && a.skip_bits == 4)) ||
        (dual && (a.ksteps != 1 || a.ksteps2 != 1 || a.cin2 != KC || a.up2)) || a.kh != 1 || a.kw != 1 ||
        a.pad != 0 || a.cout % bco != 0 || a.co_tiles < 1 || a.co_tiles > 256)
        return hipErrorInvalidValue;
    const int qtiles = a.total_tiles / a.co_tiles;
    if (qtiles <= 0)
        return hipSuccess;
    // workgroups per CU: two on 256-channel tiles and the half view (LDS), three on the others
    const int slots = (bco == 256 || hv) ? 512 : 768;
    const int nstream = qtiles < slots / a.co_tiles ? qtiles : slots / a.co_tiles;
    dim3 grid(nstream * a.co_tiles), block(256);
    bool fast = true;
    for (int i = 0; i < a.nseg; ++i)
        fast = fast && a.seg[i].fast;
    if (hv) {
        if (a.skip_bits == 0) {
            if (fast)
                hipLaunchKernelGGL((qconv_stream_kernel<0, 1, 4, 2, 1>), grid, block, 0, stream, a);
            else
                hipLaunchKernelGGL((qconv_stream_kernel<0, 0, 4, 2, 1>), grid, block, 0, stream, a);
        } else {
            if (fast)
                hipLaunchKernelGGL((qconv_stream_kernel<1, 1, 4, 2, 1>), grid, block, 0, stream, a);
            else
                hipLaunchKernelGGL((qconv_stream_kernel<1, 0, 4, 2, 1>), grid, block, 0, stream, a);
        }
    } else if (bco != 256) {
        if (bco == 128) {
            if (fast)
                hipLaunchKernelGGL((qconv_stream_kernel<0, 1, 4, 2>), grid, block, 0, stream, a);
            else
                hipLaunchKernelGGL((qconv_stream_kernel<0, 0, 4, 2>), grid, block, 0, stream, a);
        } else {
            if (fast)
                hipLaunchKernelGGL((qconv_stream_kernel<0, 1, 4, 1>), grid, block, 0, stream, a);
            else
                hipLaunchKernelGGL((qconv_stream_kernel<0, 0, 4, 1>), grid, block, 0, stream, a);
        }
    } else if (dual) {
        if (fast)
            hipLaunchKernelGGL((qconv_stream_kernel<2, 1>), grid, block, 0, stream, a);
        else
            hipLaunchKernelGGL((qconv_stream_kernel<2, 0>), grid, block, 0, stream, a);
    } else if (a.skip_bits == 0) {
        if (fast)
            hipLaunchKernelGGL((qconv_stream_kernel<0, 1>), grid, block, 0, stream, a);
        else
            hipLaunchKernelGGL((qconv_stream_kernel<0, 0>), grid, block, 0, stream, a);
    } else {
        if (fast)
            hipLaunchKernelGGL((qconv_stream_kernel<1, 1>), grid, block, 0, stream, a);
        else
            hipLaunchKernelGGL((qconv_stream_kernel<1, 0>), grid, block, 0, stream, a);
    }
    return hipGetLastError();
}

hipError_t launch_qconv_proj(const MfmaArgs &a, hipStream_t stream)
{
    // 256 x 64 tiles (two accumulator sets per wave), the 256-channel weight layout
    constexpr int BI = 4, MI = 8, NJ = 2, WC = 2, WP = 2;
    if (a.bits_out != BI || a.skip_bits != 32)
        return hipErrorInvalidValue;
    dim3 grid(8 * a.tiles_per_xcd), block(64 * WC * WP);
    bool fast = true;
    for (int i = 0; i < a.nseg; ++i)
        fast = fast && a.seg[i].fast;
    if (fast)
        hipLaunchKernelGGL((qconv_mfma_kernel<BI, MI, NJ, WC, WP, 0, 2, 1, 1>), grid, block, 0, stream, a);
    else
        hipLaunchKernelGGL((qconv_mfma_kernel<BI, MI, NJ, WC, WP, 0, 2, 0, 1>), grid, block, 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_qconv_mfma(int bits_in, const MfmaArgs &a, hipStream_t stream)
{
    if (bits_in == 4) {
        switch (a.tile_cfg) {
        case TILE_256x128: return launch_modes<4, 8, 4, 2, 2>(a, stream);
        case TILE_WV:
        case TILE_WV144:
        case TILE_WV64: return launch_qconv_wv(a, stream);
        case TILE_WVS: return launch_qconv_wvs(a, stream);
        case TILE_256x64S: return launch_qconv_short(a, stream);
        case TILE_256x64: return launch_modes<4, 8, 2, 2, 2>(a, stream);
        case TILE_STREAM:
        case TILE_STREAM_H128:
        case TILE_STREAM_C128:
        case TILE_STREAM_C64: return launch_qconv_stream(a, stream);
        case TILE_128x128_O3: return launch_occ3<4, 4, 2, 2>(a, stream);
        case TILE_64x256_O3: return launch_occ3<4, 4, 1, 4>(a, stream);
        case TILE_128x256: return launch_modes<4, 4, 8, 2, 2>(a, stream);
        case TILE_64x512: return launch_modes<4, 4, 8, 1, 4>(a, stream);
        }
    } else if ((bits_in == 2 && a.tile_cfg == TILE_FP4) || (bits_in == 8 && a.tile_cfg == TILE_B8)) {
        return launch_qconv_b16(bits_in, a, stream);
    } else if (bits_in == 8 && a.tile_cfg == TILE_STEM) {
        return launch_qconv_stem(a, stream);
    } else if (bits_in == 2) {
        switch (a.tile_cfg) {
        case TILE_128x256: return launch_modes<2, 4, 8, 2, 2>(a, stream);
        case TILE_64x512: return launch_modes<2, 4, 8, 1, 4>(a, stream);
        }
    }
    return hipErrorInvalidValue;
}

}  // namespace aqd
