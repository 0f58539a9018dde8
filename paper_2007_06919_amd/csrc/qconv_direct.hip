// Direct integer convolution for shapes the MFMA kernel does not take
// (8-bit activation codes, input channels not a multiple of 64, output
// channels not a multiple of 16, 8-bit odd-grid weights).
//
// One thread computes the channels of one output pixel that share an output
// byte (8 / b_out channels for codes, one channel for int32 output): the
// accumulation of Eq. 4 over the taps inside the image, then the shared
// integer epilogue. Weights are decoded values, int16 [cout][kh][kw][cin].

#include "epilogue.h"
#include "internal.h"

namespace aqd {
namespace {

__global__ void __launch_bounds__(256) qconv_direct_kernel(DirectArgs A)
{
    const int per = A.out_bits == 32 ? 1 : 8 / A.out_bits;  // channels per thread
    const int groups = (A.cout + per - 1) / per;
    const long long P = (long long)A.n * A.ho * A.wo;
    const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= P * groups)
        return;
    const long long px = idx / groups;
    const int grp = (int)(idx - px * groups);
    const int hw = A.ho * A.wo;
    const int n = (int)(px / hw);
    const int rem = (int)(px - (long long)n * hw);
    const int oh = rem / A.wo, ow = rem - oh * A.wo;
    const int row_bytes = A.cin * A.bits_in / 8;
    const int32_t *bias = A.epi, *mult = A.epi + A.cout, *shift = A.epi + 2 * A.cout;
    const int32_t *sc = A.epi + 3 * A.cout, *sd = A.epi + 4 * A.cout, *sside = A.epi + 5 * A.cout;
    const int qmax = A.out_bits == 32 ? 0 : A.qmax;

    uint32_t packed = 0;
    for (int e = 0; e < per; ++e) {
        const int co = grp * per + e;
        if (co >= A.cout)
            break;
        int acc = 0;
        for (int r = 0; r < A.kh; ++r) {
            const int ih = oh * A.stride - A.pad + r;
            if ((unsigned)ih >= (unsigned)A.h)
                continue;
            for (int q = 0; q < A.kw; ++q) {
                const int iw = ow * A.stride - A.pad + q;
                if ((unsigned)iw >= (unsigned)A.w)
                    continue;
                const uint8_t *xr = A.x + (((long long)n * A.h + ih) * A.w + iw) * row_bytes;
                const int16_t *wr = A.wt + (((long long)co * A.kh + r) * A.kw + q) * A.cin;
                for (int ci = 0; ci < A.cin; ++ci)
                    acc += load_code(xr, ci, A.bits_in) * (int)wr[ci];
            }
        }
        const int v = acc + bias[co];
        if (A.out_bits == 32) {
            ((int32_t *)A.y)[px * A.cout + co] = v;
            continue;
        }
        long long u = v;
        if (A.skip_bits) {
            long long spix = px;
            if (A.up2)
                spix = ((long long)n * A.hs + (oh >> 1)) * A.ws + (ow >> 1);
            int k;
            if (A.skip_bits == 32)
                k = ((const int32_t *)A.skip)[spix * A.cout + co];
            else
                k = load_code((const uint8_t *)A.skip + spix * (A.cout * A.skip_bits / 8), co,
                              A.skip_bits);
            u = align_add(v, k, sc[co], sd[co], sside[co]);
        }
        packed |= requant_clamp(u, mult[co], shift[co], qmax) << (e * A.out_bits);
    }
    if (A.out_bits != 32)
        ((uint8_t *)A.y)[px * (A.cout * A.out_bits / 8) + grp] = (uint8_t)packed;
}

}  // namespace

hipError_t launch_qconv_direct(const DirectArgs &a, hipStream_t stream)
{
    const int per = a.out_bits == 32 ? 1 : 8 / a.out_bits;
    const long long total = (long long)a.n * a.ho * a.wo * ((a.cout + per - 1) / per);
    if (total == 0)
        return hipSuccess;
    const long long blocks = (total + 255) / 256;
    if (blocks > 0x7fffffffLL)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(qconv_direct_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace aqd
