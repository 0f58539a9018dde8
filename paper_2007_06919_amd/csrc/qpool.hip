// Max-pooling of b-bit code tensors (Sec. 3.2.4: pooling leaves the scale
// factor of its input unchanged, so the codes are pooled as they are, with no
// arithmetic beyond comparisons). Window positions outside the input are
// skipped (codes are >= 0, so this equals pooling over a zero-padded input
// whenever the window holds at least one input position, which the host
// checks).

#include "internal.h"

namespace aqd {
namespace {

// One thread per output byte: 8 / b channels of one output pixel.
__global__ void __launch_bounds__(256) maxpool_kernel(PoolArgs A)
{
    const int per = 8 / A.bits;
    const int groups = A.c / per;
    const long long P = (long long)A.n * A.ho * A.wo;
    const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= P * groups)
        return;
    const long long px = idx / groups;
    const int grp = (int)(idx - px * groups);
    const int hw = A.ho * A.wo;
    const int n = (int)(px / hw);
    const int rem = (int)(px - (long long)n * hw);
    const int i = rem / A.wo, j = rem - i * A.wo;
    const int row_bytes = A.c * A.bits / 8;
    const int mask = (1 << A.bits) - 1;
    int best[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int dy = 0; dy < A.k; ++dy) {
        const int ih = i * A.stride - A.pad + dy;
        if ((unsigned)ih >= (unsigned)A.h)
            continue;
        for (int dx = 0; dx < A.k; ++dx) {
            const int iw = j * A.stride - A.pad + dx;
            if ((unsigned)iw >= (unsigned)A.w)
                continue;
            const int v = A.x[(((long long)n * A.h + ih) * A.w + iw) * row_bytes + grp];
            for (int e = 0; e < per; ++e) {
                const int code = (v >> (e * A.bits)) & mask;
                best[e] = code > best[e] ? code : best[e];
            }
        }
    }
    uint32_t packed = 0;
    for (int e = 0; e < per; ++e)
        packed |= (uint32_t)best[e] << (e * A.bits);
    A.y[px * row_bytes + grp] = (uint8_t)packed;
}

}  // namespace

hipError_t launch_maxpool(const PoolArgs &a, hipStream_t stream)
{
    const long long items = (long long)a.n * a.ho * a.wo * (a.c * a.bits / 8);
    if (items <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(maxpool_kernel, dim3((unsigned)((items + 255) / 256)), dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace aqd
