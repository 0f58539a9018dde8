// Second half of a split-K convolution: the int32 partial sums of the parts
// of the K range (Sec. 3.2.1, Eq. 4: acc is an integer sum over taps and input
// channels, so adding the parts gives acc exactly; the first part started at
// the bias, so the sum is v = acc + bias, Eq. 6) are added, and the rest of
// the integer epilogue runs on the result: the optional skip alignment
// (Eq. 7-8), requantisation and clamp.
//
// One work item = one output pixel x CPT consecutive channels: one packed
// 32-bit word of b-bit codes (CPT = 32 / b) or four int32 outputs. The
// partial sums are read as 16-byte vectors (rows of cout int32 per pixel);
// the launches that are split are small, so the epilogue uses the general
// 64-bit arithmetic for every shift.

#include "epilogue.h"
#include "internal.h"

namespace aqd {
namespace {

template <int BO, int SB>
__global__ void __launch_bounds__(256) splitk_epilogue_kernel(SplitArgs A)
{
    const long long item = (long long)blockIdx.x * 256 + threadIdx.x;
    if (item >= A.total_items)
        return;
    int s = 0;
#pragma unroll
    for (int i = 1; i < AQD_MAX_SEGS; ++i)
        if (i < A.nseg && item >= A.seg[i].item_begin)
            s = i;
    const SplitSeg &S = A.seg[s];

    constexpr int CPT = BO == 32 ? 4 : 32 / BO;
    const int groups = A.cout / CPT;
    const long long it = item - S.item_begin;
    const long long px = it / groups;
    const int c0 = (int)(it - px * groups) * CPT;

    int acc[CPT];
#pragma unroll
    for (int q = 0; q < CPT; q += 4) {
        int4 t = *(const int4 *)(S.part + px * A.cout + c0 + q);
        for (int p = 1; p < A.nparts; ++p) {
            const int4 u = *(const int4 *)(S.part + ((long long)p * S.P + px) * A.cout + c0 + q);
            t.x += u.x;
            t.y += u.y;
            t.z += u.z;
            t.w += u.w;
        }
        acc[q] = t.x;
        acc[q + 1] = t.y;
        acc[q + 2] = t.z;
        acc[q + 3] = t.w;
    }
    if constexpr (BO == 32) {
        *(int4 *)((int32_t *)S.y + px * A.cout + c0) = make_int4(acc[0], acc[1], acc[2], acc[3]);
    } else {
        long long spix = px;
        if (SB != 0 && A.up2) {
            const int hw = S.ho * S.wo;
            const int n_ = (int)(px / hw);
            const int rem = (int)(px - (long long)n_ * hw);
            const int oh = rem / S.wo, ow = rem - oh * S.wo;
            spix = ((long long)n_ * S.hs + (oh >> 1)) * S.ws + (ow >> 1);
        }
        uint32_t word = 0;
#pragma unroll
        for (int e = 0; e < CPT; ++e) {
            const int c = c0 + e;
            const int v = acc[e];
            long long u = v;
            if constexpr (SB == 32) {
                const int k = ((const int32_t *)S.skip)[spix * A.cout + c];
                u = align_add(v, k, S.epi[EPI_SKIP_C * A.cout_pad + c], S.epi[EPI_SKIP_D * A.cout_pad + c],
                              S.epi[EPI_SKIP_SIDE * A.cout_pad + c]);
            } else if constexpr (SB != 0) {
                const int k = load_code((const uint8_t *)S.skip + spix * (A.cout * SB / 8), c, SB);
                u = align_add(v, k, S.epi[EPI_SKIP_C * A.cout_pad + c], S.epi[EPI_SKIP_D * A.cout_pad + c],
                              S.epi[EPI_SKIP_SIDE * A.cout_pad + c]);
            }
            const uint32_t y = requant_clamp(u, S.epi[EPI_MULT * A.cout_pad + c], S.epi[EPI_SHIFT * A.cout_pad + c], A.qmax);
            word |= y << (e * BO);
        }
        *(uint32_t *)((uint8_t *)S.y + px * (A.cout * BO / 8) + c0 * BO / 8) = word;
    }
}

template <int BO, int SB>
hipError_t launch_t(const SplitArgs &a, hipStream_t stream)
{
    const long long blocks = (a.total_items + 255) / 256;
    hipLaunchKernelGGL((splitk_epilogue_kernel<BO, SB>), dim3((unsigned)blocks), dim3(256), 0, stream, a);
    return hipGetLastError();
}

template <int BO>
hipError_t launch_skip(const SplitArgs &a, hipStream_t stream)
{
    switch (a.skip_bits) {
    case 0: return launch_t<BO, 0>(a, stream);
    case 2: return launch_t<BO, 2>(a, stream);
    case 4: return launch_t<BO, 4>(a, stream);
    case 8: return launch_t<BO, 8>(a, stream);
    case 32: return launch_t<BO, 32>(a, stream);
    }
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_splitk_epilogue(const SplitArgs &a, hipStream_t stream)
{
    if (a.total_items <= 0)
        return hipSuccess;
    switch (a.bits_out) {
    case 2: return launch_skip<2>(a, stream);
    case 4: return launch_skip<4>(a, stream);
    case 8: return launch_skip<8>(a, stream);
    case 32: return a.skip_bits ? hipErrorInvalidValue : launch_t<32, 0>(a, stream);
    }
    return hipErrorInvalidValue;
}

}  // namespace aqd
