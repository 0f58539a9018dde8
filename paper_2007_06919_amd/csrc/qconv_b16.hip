// Implicit-GEMM integer convolution whose MFMA operand row of a K step is
// 16 bytes of staged codes, used as they are (no widening in the main loop):
//  * 2-bit codes with 2-bit weights on the gfx950 scaled FP4 MFMA
//    (v_mfma_scale_f32_16x16x128_f8f6f4, e2m1 operands, K step = 128 input
//    channels), for layers with cin and cout multiples of 256: the ResNet-50
//    res4/res5 layers, the FPN and the heads of the paper's 2-bit detectors;
//  * 8-bit codes (the input and output layers of the paper's fully quantized
//    networks, Sec. 4) on the int8 MFMA (v_mfma_i32_16x16x64_i8, K step = 64
//    input channels), for cin a multiple of 128, int32 outputs (the
//    prediction convolutions).
// GEMM view of Eq. 4 (Sec. 3.2.1): rows = output channels, columns = output
// pixels, K = taps x input channels.
//
// Exactness, FP4. Every operand is a small integer that e2m1 holds exactly: a
// 2-bit weight value (odd grid -3, -1, 1, 3 or two's complement -2 .. 1) is
// stored as its e2m1 nibble with block scale 1, an activation code k in
// {0, 1, 2, 3} as the nibble k itself, which e2m1 reads as k / 2, with block
// scale 2. Each product is then an integer, the MFMA sums them in fp32, and
// every partial sum is bounded by K * 3 * 3 < 2^24 (checked at create), so
// the fp32 accumulator holds the exact integer sum; its conversion to int32
// is exact too.
// Exactness, int8. An 8-bit code a in [0, 255] does not fit int8; the staging
// copy stores a - 128 (the byte a XOR 0x80, read as signed), padding taps
// included (code 0 -> -128), and the bias folded at create carries
// 128 * sum(w) of the channel, so v = acc + bias is the exact sum of Eq. 6.
// The epilogue is the integer one of Eq. 6-8 and Eq. 2.
//
// Workgroup tile 256 channels x 128 pixels, 4 waves; wave w owns channel rows
// 64w .. 64w+63 (4 accumulator tiles of 16) for all 128 pixels (8 column
// tiles), as in the register-fed int8 kernel:
//  * weights (tiled at create, 64 bytes per row and K step: 128 e2m1 nibbles
//    or 64 int8) go from global memory straight into registers, three K steps
//    ahead of their MFMAs;
//  * activation codes go through LDS in stages of 128 bytes per pixel (one
//    tap's 256 2-bit or 128 8-bit channels; two K steps). A copy lane takes 8
//    bytes of packed 2-bit codes and spreads them into 16 bytes of nibbles
//    with two masks and a shift (even channels of a word in one word of
//    nibbles, odd ones in the next; the weights were stored in that channel
//    order at create), or 16 bytes of 8-bit codes and flips their top bits.
//    A pixel's 128 bytes are 16-byte columns XOR-swizzled with the pixel
//    index, so that the copies' writes and the fragment reads (16 bytes per
//    lane) are free of bank conflicts. A stage is loaded one stage ahead of
//    its use and written during the stage before it (two-buffer ring, one
//    barrier per stage).
//  * A part of a split K range (whole stages) writes int32 partial sums, the
//    first part with the bias, for the split-K combining epilogue.

#include "epilogue.h"
#include "internal.h"
#include "mfma_common.h"

namespace aqd {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));

constexpr int F4_BCO = 256;                   // channels per workgroup tile
constexpr int F4_BPX = 128;                   // pixels per workgroup tile
constexpr int F4_ROW = 128;                   // LDS bytes of one stage per pixel (256 nibbles)
constexpr int F4_STAGE = F4_BPX * F4_ROW;     // 16 KiB
constexpr int F4_TAB = 2 * F4_STAGE;          // epilogue tables after the ring of two stages
constexpr int F4_LDS = 4 * F4_STAGE;          // int32 staging uses all 64 KiB
constexpr int F4_KROW = 64;                   // weight bytes per row and K step
constexpr int F4_SCALE_W = 127;               // E8M0 block scales: 2^0 for the weights,
constexpr int F4_SCALE_X = 128;               // 2^1 for the codes (nibble k reads as k / 2)

// c += a * b on the scaled FP4 MFMA (formats 4 = e2m1 for both operands, block
// scales sa, sb as E8M0 exponents), accumulating in place. Inline assembly
// because the compiler's form of this instruction never writes its
// accumulator in place, and 128 accumulator registers rotating through fresh
// ones do not fit. The compiler therefore does not see an MFMA here: the
// wait states it would insert around one are the caller's (a VALU write of an
// operand needs 2 before the MFMA reads it, a read of the result 18 after),
// and a hazard scan of the built code is part of the tests.
__device__ __forceinline__ void mfma_fp4(const v4i a, const v4i b, v4f &c, int sa, int sb)
{
    asm volatile("v_mfma_scale_f32_16x16x128_f8f6f4 %0, %1, %2, %0, %3, %4 op_sel_hi:[0,0,0] cbsz:4 blgp:4"
                 : "+v"(c) : "v"(a), "v"(b), "v"(sa), "v"(sb));
}

// Wait states around the inline MFMAs, and a fence the compiler cannot move
// the accumulators' other uses across: every accumulator is an operand
template <int MI, int NJ>
__device__ __forceinline__ void mfma_fence(v4f (&acc)[MI][NJ])
{
    static_assert(MI * NJ == 32, "two groups of 16 operands");
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7"
                 : "+v"(acc[0][0]), "+v"(acc[0][1]), "+v"(acc[0][2]), "+v"(acc[0][3]),
                   "+v"(acc[0][4]), "+v"(acc[0][5]), "+v"(acc[0][6]), "+v"(acc[0][7]),
                   "+v"(acc[1][0]), "+v"(acc[1][1]), "+v"(acc[1][2]), "+v"(acc[1][3]),
                   "+v"(acc[1][4]), "+v"(acc[1][5]), "+v"(acc[1][6]), "+v"(acc[1][7]));
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7"
                 : "+v"(acc[2][0]), "+v"(acc[2][1]), "+v"(acc[2][2]), "+v"(acc[2][3]),
                   "+v"(acc[2][4]), "+v"(acc[2][5]), "+v"(acc[2][6]), "+v"(acc[2][7]),
                   "+v"(acc[3][0]), "+v"(acc[3][1]), "+v"(acc[3][2]), "+v"(acc[3][3]),
                   "+v"(acc[3][4]), "+v"(acc[3][5]), "+v"(acc[3][6]), "+v"(acc[3][7]));
}

// CB: input code width, 2 (FP4 MFMA) or 8 (int8 MFMA); OUTK: 0 = 2-bit codes
// (CB 2 only), 1 = int32 (v = acc + bias, or a split part's sums); SKK: 0 = no
// skip, 1 = 2-bit code skip; FAST: every shift >= 2 (32-bit requantisation)
template <int CB, int OUTK, int SKK, int FAST>
__global__ void __launch_bounds__(256, 2) qconv_b16_kernel(MfmaArgs A)
{
    static_assert(CB == 2 || CB == 8, "2-bit or 8-bit input codes");
    static_assert(OUTK == 0 || SKK == 0, "int32 outputs have no skip");
    static_assert(CB == 2 || OUTK == 1, "8-bit inputs: int32 outputs");
    constexpr bool FP4 = CB == 2;
    constexpr int MI = 4, NJ = 8, QMAX = 3, BO = 2;
    constexpr int SPS = FP4 ? 4 : 2;            // 64-channel steps per stage
    constexpr int SCH = FP4 ? 256 : 128;        // input channels per stage
    using acc_t = typename std::conditional<FP4, v4f, v4i>::type;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[F4_LDS];

    const int bid = blockIdx.x;
    const int logical = (bid & 7) * A.tiles_per_xcd + (bid >> 3);
    if (logical >= A.total_tiles)
        return;
    // work unit -> output tile and part of its K range (consecutive units)
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
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane & 15, g = lane >> 4;

    // K range of this part in stages (one tap's SCH channels; A.ksteps and
    // A.kchunk count 64-channel steps, multiples of SPS on this path); the
    // kernel's K steps are two per stage
    const int row_bytes = A.cin * CB / 8;
    const int spt = A.cin / SCH;                           // stages per tap
    const int st0 = kpart * (A.kchunk / SPS);
    const int NST = min(A.kchunk, A.ksteps - kpart * A.kchunk) / SPS;  // >= 1 (host)
    const int KSK = 2 * (A.ksteps / SPS);                  // kernel K steps of the whole range
    const int hw = S.ho * S.wo;

    // ---- activation copies: piece m of a stage = pixels 32m .. 32m+31, lane
    // tid copying stage bytes 8c .. 8c+7 (2-bit: channels 32c .. 32c+31) or
    // 16c .. 16c+15 (8-bit: channels 16c .. 16c+15) of pixel 32m + tid / 8,
    // c = tid % 8
    const int c8 = tid & 7;
    // per piece: the byte offset of its pixel's window origin (negative at the
    // top and left borders) and which window rows (bit t) and columns (bit
    // 16 + t) lie inside the image (none for pixels past the end); the input
    // holds n * h * w * row_bytes < 2^31 bytes (checked on the host)
    int xbase[4];
    uint32_t xvalid[4];
#pragma unroll
    for (int m = 0; m < 4; ++m) {
        const unsigned p = (unsigned)(px_tile * F4_BPX + 32 * m + (tid >> 3));
        const bool ok = p < (unsigned)S.P;
        const unsigned pn = ok ? p / (unsigned)hw : 0u;
        const unsigned prem = ok ? p - pn * (unsigned)hw : 0u;
        const int oh = (int)(prem / (unsigned)S.wo), ow = (int)prem - oh * S.wo;
        const int ih0 = oh * A.stride - A.pad, iw0 = ow * A.stride - A.pad;
        uint32_t v = 0;
        for (int t = 0; t < A.kh; ++t)
            v |= ((unsigned)(ih0 + t) < (unsigned)S.h ? 1u : 0u) << t;
        for (int t = 0; t < A.kw; ++t)
            v |= ((unsigned)(iw0 + t) < (unsigned)S.w ? 1u : 0u) << (16 + t);
        xvalid[m] = ok ? v : 0u;
        xbase[m] = (((int)pn * S.h + ih0) * S.w + iw0) * row_bytes + (FP4 ? 8 : 16) * c8;
    }
    const buf_rsrc xr = make_rsrc(S.x, S.n * S.h * S.w * row_bytes);
    // LDS: 16-byte column c of pixel p at 128 p + 16 (c ^ (p & 7))
    const int wp = tid >> 3;
    const uint32_t wofs = F4_ROW * wp + 16 * (c8 ^ (wp & 7));
    // fragment of K step q of a stage: pixel 16j + r, column 4q + g
    auto ro = [&](int q) -> uint32_t { return F4_ROW * r + 16 * ((4 * q + g) ^ (r & 7)); };

    // copy state of the stage being loaded (uniform): tap (tr, tq), SCH-channel
    // chunk th; its byte offset from a window origin and the window bits it needs
    int th = st0 % spt, tr, tq;
    {
        const int tap = st0 / spt;
        tr = tap / A.kw;
        tq = tap - tr * A.kw;
    }
    int x_off = 0;
    uint32_t x_need = 0;
    auto set_copy = [&]() {
        x_off = (tr * S.w + tq) * row_bytes + (SCH * CB / 8) * th;
        x_need = (1u << tr) | (1u << (16 + tq));
    };
    set_copy();
    auto advance = [&]() {
        if (++th == spt) {
            th = 0;
            if (++tq == A.kw) {
                tq = 0;
                ++tr;
            }
        }
        set_copy();
    };
    // buffer loads: taps in the padding, pixels past the end and stages past
    // the last read past the end of the input and get zeros (code 0)
    using piece_t = typename std::conditional<FP4, uint2, uint4>::type;
    auto load_piece = [&](int m) -> piece_t {
        const int off = (xvalid[m] & x_need) == x_need ? xbase[m] + x_off : (int)0x80000000;
        if constexpr (FP4) {
            return load_b64(xr, off, 0);
        } else {
            const v4i v = load_b128(xr, off, 0);
            return make_uint4((uint32_t)v.x, (uint32_t)v.y, (uint32_t)v.z, (uint32_t)v.w);
        }
    };
    // 2-bit: 32 packed codes -> 32 nibbles, word 2h holding the even channels
    // of packed word h, word 2h + 1 the odd ones; 8-bit: code a -> a - 128
    auto write_piece = [&](int buf, int m, const piece_t v) {
        uint4 n;
        if constexpr (FP4)
            n = make_uint4(v.x & 0x33333333u, (v.x >> 2) & 0x33333333u,
                           v.y & 0x33333333u, (v.y >> 2) & 0x33333333u);
        else
            n = make_uint4(v.x ^ 0x80808080u, v.y ^ 0x80808080u, v.z ^ 0x80808080u, v.w ^ 0x80808080u);
        *(uint4 *)(lds + buf * F4_STAGE + m * (32 * F4_ROW) + wofs) = n;
    };

    // ---- weights: this wave's rows of K step k, accumulator tile i at
    // k * 16 KiB + i * 1 KiB from the channel tile's first step (lane: row r,
    // 16-byte column g); the look-ahead reads up to three steps past the
    // part's last (inside the tile range, or past the buffer's size: zeros),
    // never used
    const buf_rsrc wr = make_rsrc(S.wt + (long long)co_tile * KSK * F4_BCO * F4_KROW, KSK * F4_BCO * F4_KROW);
    const int w_lane = (64 * wave + r) * F4_KROW + 16 * g;
    const int k0 = 2 * st0;
    auto load_a = [&](int k, v4i *dst) {
#pragma unroll
        for (int i = 0; i < MI; ++i)
            dst[i] = load_b128(wr, w_lane + i * 1024, (k0 + k) * (F4_BCO * F4_KROW));
    };

    // lane group g of wave w holds channels 128 (w >> 1) + 32 g + 16 (w & 1) + 4 i + e
    const int co_loc = 128 * (wave >> 1) + 32 * g + 16 * (wave & 1);
    const int co_glob = co_tile * F4_BCO + co_loc;
    acc_t acc[MI][NJ];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
            acc[i][j] = acc_t{0, 0, 0, 0};
    if constexpr (FP4)
        mfma_fence(acc);  // the zeros are written before the first MFMA reads them
    // block scales in registers the compiler cannot rematerialise next to an MFMA
    int scale_w = F4_SCALE_W, scale_x = F4_SCALE_X;
    asm volatile("" : "+v"(scale_w), "+v"(scale_x));

    // ---- the channel tile's epilogue table (and the side-0 skip table) go to
    // LDS past the ring before the prologue: nothing holds them in registers
    // through the main loop
    int32_t *prm = (int32_t *)(lds + F4_TAB);      // [EPI_FIELDS][256]
    int32_t *lut = prm + EPI_FIELDS * F4_BCO;      // [256][4]: RSM(k, c, d) of the side-0 skip codes
    const bool use_lut = SKK == 1 && S.side0;
    if constexpr (OUTK == 0) {
#pragma unroll
        for (int u = 0; u < EPI_FIELDS; ++u)
            prm[tid + 256 * u] = S.epi[u * A.cout_pad + co_tile * F4_BCO + tid];
        if (use_lut) {
#pragma unroll
            for (int u = 0; u < QMAX + 1; ++u)
                lut[tid + 256 * u] = S.lut[co_tile * F4_BCO * (QMAX + 1) + tid + 256 * u];
        }
    }
    static_assert(F4_TAB + (EPI_FIELDS + QMAX + 1) * F4_BCO * 4 <= F4_LDS, "tables fit past the ring");

    // ---- prologue: stage 0 in LDS, stage 1 in registers, weights of steps 0-2
    piece_t rb[4];
#pragma unroll
    for (int m = 0; m < 4; ++m)
        write_piece(0, m, load_piece(m));
    advance();
#pragma unroll
    for (int m = 0; m < 4; ++m)
        rb[m] = load_piece(m);
    advance();  // copy state: stage 2
    v4i fa[4][MI];
    load_a(0, fa[0]);
    load_a(1, fa[1]);
    load_a(2, fa[2]);
    v4i fb[NJ];
    int kstep = 0;         // K step of this part being multiplied
    constexpr int RA = FP4 ? 3 : 2;  // fragments are read RA column tiles ahead of their MFMAs
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
#pragma unroll
    for (int j = 0; j < RA; ++j)
        fb[j] = *(const v4i *)(lds + 2048 * j + ro(0));

    // ---- main loop, one stage (two K steps) per call: stage t lives in buffer
    // t % 2 (the parity P, a compile-time constant, so that the weight sets
    // (K step % 4) are registers). During stage t the pieces of stage t + 1
    // (loaded during stage t - 1) are written into buffer (t + 1) % 2, two per
    // K step, each right before the load of the same piece of stage t + 2
    // reuses its registers. The barrier in the last K step, before the first
    // read of stage t + 1, makes that stage visible; every read of stage t - 1
    // (the buffer's previous contents) came before the barrier of stage t - 1.
    auto stage = [&](auto pc) {
        constexpr int P = decltype(pc)::value;
        static_for<2>([&](auto qc) {
            constexpr int q = decltype(qc)::value;
            constexpr int kq = 2 * P + q;  // K step % 4
            write_piece(P ^ 1, 2 * q, rb[2 * q]);
            write_piece(P ^ 1, 2 * q + 1, rb[2 * q + 1]);
            rb[2 * q] = load_piece(2 * q);
            rb[2 * q + 1] = load_piece(2 * q + 1);
            load_a(kstep + 3, fa[(kq + 3) & 3]);
            const uint32_t r_this = ro(q) + P * F4_STAGE;
            const uint32_t r_next = q == 0 ? ro(1) + P * F4_STAGE : ro(0) + (P ^ 1) * F4_STAGE;
            static_for<NJ>([&](auto jc) {
                constexpr int j = decltype(jc)::value;
                if constexpr (q == 1 && j == NJ - RA)
                    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
#pragma unroll
                for (int i = 0; i < MI; ++i) {
                    if constexpr (FP4)
                        mfma_fp4(fa[kq][i], fb[j], acc[i][j], scale_w, scale_x);
                    else
                        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[kq][i], fb[j], acc[i][j], 0, 0, 0);
                }
                if constexpr (j + RA < NJ)
                    fb[j + RA] = *(const v4i *)(lds + 2048 * (j + RA) + r_this);
                else
                    fb[j + RA - NJ] = *(const v4i *)(lds + 2048 * (j + RA - NJ) + r_next);
            });
            ++kstep;
            if constexpr (q == 1)
                advance();
        });
    };
    // pairs of stages (even, odd parity); the odd stage of the last pair may
    // be past the end
    for (int t = 0; t < NST; t += 2) {
        stage(std::integral_constant<int, 0>{});
        if (t + 1 < NST)
            stage(std::integral_constant<int, 1>{});
    }

    if constexpr (FP4)
        mfma_fence(acc);  // the last MFMAs have written the accumulators
    // exact integer sums (see the header), converted where they are used;
    // the bias of Eq. 6 joins there
    if constexpr (OUTK == 1) {
        // int32 outputs (or part sums at y + kpart * P * cout), in two passes
        // of 64 pixels through LDS rows of 256 int32 (16-byte chunk c of pixel
        // p at c ^ (p & 7)); every thread then stores 16-byte chunks of whole rows
        int32_t *ybase = (int32_t *)S.y + (long long)kpart * S.P * A.cout;
        // the tile's valid 16-byte chunks (a partial last channel tile)
        const int valid_chunks = min(A.cout - co_tile * F4_BCO, F4_BCO) / 4;
        const bool with_bias = !(A.part && kpart > 0);
        v4i bias[MI];
#pragma unroll
        for (int i = 0; i < MI; ++i)
            bias[i] = with_bias ? *(const v4i *)(S.epi + EPI_BIAS * A.cout_pad + co_glob + 4 * i)
                                : v4i{0, 0, 0, 0};
        static_for<2>([&](auto pc) {
            constexpr int pass = decltype(pc)::value;
            __syncthreads();  // the ring, or the last pass's rows, are no longer read
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const int p = 16 * jj + r;
#pragma unroll
                for (int i = 0; i < MI; ++i) {
                    const int c = co_loc / 4 + i;
                    const acc_t a = acc[i][4 * pass + jj];
                    *(v4i *)(lds + p * 1024 + 16 * (c ^ (p & 7))) =
                        v4i{(int)a.x, (int)a.y, (int)a.z, (int)a.w} + bias[i];
                }
            }
            __syncthreads();
#pragma unroll
            for (int it = 0; it < 16; ++it) {
                const int idx = it * 256 + tid;
                const int p = idx >> 6, c = idx & 63;
                const long long px = (long long)px_tile * F4_BPX + 64 * pass + p;
                if (px < S.P && c < valid_chunks)
                    *(v4i *)(ybase + px * A.cout + co_tile * F4_BCO + 4 * c) =
                        *(const v4i *)(lds + p * 1024 + 16 * (c ^ (p & 7)));
            }
        });
        return;
    }

    // ---------------------------------------------------------------- epilogue
    const long long px0 = (long long)px_tile * F4_BPX + r;
    bool okj[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j)
        okj[j] = px0 + 16 * j < S.P;
    // a lane's 16 channels of a pixel: one word of 2-bit codes
    uint32_t skw[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        skw[j] = 0;
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
                skw[j] = *(const uint32_t *)((const uint8_t *)S.skip + spix * (A.cout / 4) + co_glob / 4);
            }
        }
    }
    const int32_t *lut_l = lut + co_loc * (QMAX + 1);  // this lane's 16 channels
    uint32_t outw[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j)
        outw[j] = 0;
    auto group = [&](auto lut_c, auto ic) {
        constexpr bool LUT = decltype(lut_c)::value;
        constexpr int i = decltype(ic)::value;
        const int cl = co_loc + 4 * i;
        const int4 m4 = *(const int4 *)(prm + EPI_MULT * F4_BCO + cl);
        const int4 s4 = *(const int4 *)(prm + (FAST ? EPI_SHR : EPI_SHIFT) * F4_BCO + cl);
        const int4 b4 = *(const int4 *)(prm + EPI_BIAS * F4_BCO + cl);
        const int mult[4] = {m4.x, m4.y, m4.z, m4.w};
        const int shf[4] = {s4.x, s4.y, s4.z, s4.w};
        const int bias[4] = {b4.x, b4.y, b4.z, b4.w};
        long long rnd[4] = {0, 0, 0, 0};
        if constexpr (FAST) {
            const int4 r4 = *(const int4 *)(prm + EPI_RND * F4_BCO + cl);
            rnd[0] = (long long)r4.x << 32; rnd[1] = (long long)r4.y << 32;
            rnd[2] = (long long)r4.z << 32; rnd[3] = (long long)r4.w << 32;
        }
        int sc[4] = {0, 0, 0, 0}, sd[4] = {0, 0, 0, 0}, sside[4] = {0, 0, 0, 0};
        long long srnd[4] = {0, 0, 0, 0};  // rounding terms of the alignment
        if constexpr (SKK != 0 && !LUT) {
            const int4 c4 = *(const int4 *)(prm + EPI_SKIP_C * F4_BCO + cl);
            const int4 d4 = *(const int4 *)(prm + EPI_SKIP_D * F4_BCO + cl);
            const int4 e4 = *(const int4 *)(prm + EPI_SKIP_SIDE * F4_BCO + cl);
            sc[0] = c4.x; sc[1] = c4.y; sc[2] = c4.z; sc[3] = c4.w;
            sd[0] = d4.x; sd[1] = d4.y; sd[2] = d4.z; sd[3] = d4.w;
            srnd[0] = rsm_rnd(d4.x); srnd[1] = rsm_rnd(d4.y); srnd[2] = rsm_rnd(d4.z); srnd[3] = rsm_rnd(d4.w);
            sside[0] = e4.x; sside[1] = e4.y; sside[2] = e4.z; sside[3] = e4.w;
        }
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int v = (int)acc[i][j][e] + bias[e];
                const int bit = (4 * i + e) * BO;
                int kv = 0;
                if constexpr (SKK == 1)
                    kv = (int)__builtin_amdgcn_ubfe(skw[j], bit, BO);
                int y;
                if constexpr (FAST) {
                    int u = v;
                    if constexpr (LUT) {
                        u = (int)((unsigned)v + (unsigned)lut_l[(4 * i + e) * (QMAX + 1) + kv]);
                    } else if constexpr (SKK != 0) {
                        const int scaled = rsm32r(sside[e] ? v : kv, sc[e], srnd[e], sd[e]);
                        u = (int)((unsigned)scaled + (unsigned)(sside[e] ? kv : v));
                    }
                    y = requant32(u, mult[e], rnd[e], shf[e]);
                    y = y < 0 ? 0 : (y > QMAX ? QMAX : y);
                } else {
                    long long u = v;
                    if constexpr (LUT)
                        u = (int)((unsigned)v + (unsigned)lut_l[(4 * i + e) * (QMAX + 1) + kv]);
                    else if constexpr (SKK != 0)
                        u = align_add(v, kv, sc[e], sd[e], sside[e]);
                    y = (int)requant_clamp(u, mult[e], shf[e], QMAX);
                    asm volatile("" : "+v"(y));  // one 64-bit product alive at a time
                }
                outw[j] |= (uint32_t)y << bit;
            }
        }
    };
    auto body = [&](auto lut_c) { static_for<MI>([&](auto ic) { group(lut_c, ic); }); };
    if (use_lut)
        body(std::true_type{});
    else
        body(std::false_type{});
    // the packed words are complete here: the compiler would otherwise sink
    // their last steps into the conditional stores and keep every 64-bit
    // product alive until then
#pragma unroll
    for (int j = 0; j < NJ; ++j)
        asm volatile("" : "+v"(outw[j]));
#pragma unroll
    for (int j = 0; j < NJ; ++j)
        if (okj[j])
            *(uint32_t *)((uint8_t *)S.y + (px0 + 16 * j) * (A.cout / 4) + co_glob / 4) = outw[j];
}

}  // namespace

hipError_t launch_qconv_b16(int code_bits, const MfmaArgs &a, hipStream_t stream)
{
    dim3 grid(8 * a.tiles_per_xcd), block(256);
    if ((a.part == 0 && a.ksplit != 1) || a.kh > 16 || a.kw > 16)
        return hipErrorInvalidValue;
    // 32-bit buffer offsets and sizes: inputs and weights below 2^31 bytes
    for (int i = 0; i < a.nseg; ++i)
        if ((long long)a.seg[i].n * a.seg[i].h * a.seg[i].w * a.cin * code_bits / 8 >= (1LL << 31) ||
            (long long)a.co_tiles * (2 * (a.ksteps / (code_bits == 2 ? 4 : 2))) * F4_BCO * F4_KROW >= (1LL << 31))
            return hipErrorInvalidValue;
    if (code_bits == 8) {
        // int32 outputs (or split parts); a partial last channel tile
        if (a.bits_out != 32 || a.skip_bits != 0 || a.cin % 128 != 0 || a.co_tiles * F4_BCO < a.cout ||
            a.cout % 4 != 0 || a.ksteps % 2 != 0 || a.kchunk % 2 != 0 || a.kchunk < 2)
            return hipErrorInvalidValue;
        hipLaunchKernelGGL((qconv_b16_kernel<8, 1, 0, 1>), grid, block, 0, stream, a);
        return hipGetLastError();
    }
    if (code_bits != 2 || (a.bits_out != 2 && a.bits_out != 32) ||
        (a.skip_bits != 0 && (a.skip_bits != 2 || a.bits_out == 32)) || a.cin % 256 != 0 ||
        a.cout % 256 != 0 || a.co_tiles * F4_BCO != a.cout || a.ksteps % 4 != 0 || a.kchunk % 4 != 0 ||
        a.kchunk < 4 || (a.part && a.bits_out != 32))
        return hipErrorInvalidValue;
    bool fast = true;
    for (int i = 0; i < a.nseg; ++i)
        fast = fast && a.seg[i].fast;
    if (a.bits_out == 32)
        hipLaunchKernelGGL((qconv_b16_kernel<2, 1, 0, 1>), grid, block, 0, stream, a);
    else if (a.skip_bits == 0) {
        if (fast)
            hipLaunchKernelGGL((qconv_b16_kernel<2, 0, 0, 1>), grid, block, 0, stream, a);
        else
            hipLaunchKernelGGL((qconv_b16_kernel<2, 0, 0, 0>), grid, block, 0, stream, a);
    } else {
        if (fast)
            hipLaunchKernelGGL((qconv_b16_kernel<2, 0, 1, 1>), grid, block, 0, stream, a);
        else
            hipLaunchKernelGGL((qconv_b16_kernel<2, 0, 1, 0>), grid, block, 0, stream, a);
    }
    return hipGetLastError();
}

}  // namespace aqd
