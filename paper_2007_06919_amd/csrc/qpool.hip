// Max-pooling of b-bit code tensors (Sec. 3.2.4: pooling leaves the scale
// factor of its input unchanged, so the codes are pooled as they are, with no
// arithmetic beyond comparisons). Window positions outside the input are
// skipped (codes are >= 0, so this equals pooling over a zero-padded input
// whenever the window holds at least one input position, which the host
// checks).

#include "internal.h"

namespace aqd {
namespace {

// One thread per output byte: 8 / b channels of one output pixel (rows whose
// byte count is not a multiple of 16).
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

// Lane-wise max of packed b-bit codes in a word: the codes are spread into
// lanes twice as wide as the largest code needs (even and odd codes in turn),
// so a lane's top bit is free for the borrow of a - b: set when a >= b.
template <int B>
__device__ __forceinline__ uint32_t packed_max(uint32_t a, uint32_t b)
{
    constexpr int LANE = B == 8 ? 16 : 8;                      // lane width of a phase
    constexpr uint32_t TOP = LANE == 16 ? 0x80008000u : 0x80808080u;
    constexpr uint32_t M = B == 8 ? 0x00FF00FFu : B == 4 ? 0x0F0F0F0Fu : 0x03030303u;
    uint32_t out = 0;
#pragma unroll
    for (int sh = 0; sh < LANE; sh += B) {
        const uint32_t x = (a >> sh) & M, y = (b >> sh) & M;
        const uint32_t ge = ((x | TOP) - y) & TOP;              // top bit of lanes with x >= y
        const uint32_t sel = (ge >> (LANE - 1)) * ((1u << LANE) - 1);   // all ones in those lanes
        out |= ((x & sel) | (y & ~sel)) << sh;
    }
    return out;
}

// 16 bytes of one output pixel per thread (rows of a multiple of 16 bytes):
// per window position one 16-byte load, packed lane-wise maxima.
template <int B>
__global__ void __launch_bounds__(256) maxpool16_kernel(PoolArgs A)
{
    const int chunks = A.c * B / 128;
    const long long P = (long long)A.n * A.ho * A.wo;
    const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= P * chunks)
        return;
    const long long px = idx / chunks;
    const int ch = (int)(idx - px * chunks);
    const int hw = A.ho * A.wo;
    const int n = (int)(px / hw);
    const int rem = (int)(px - (long long)n * hw);
    const int i = rem / A.wo, j = rem - i * A.wo;
    const int row_bytes = A.c * B / 8;
    uint4 best = make_uint4(0, 0, 0, 0);   // codes are >= 0, and the window holds an input position
    for (int dy = 0; dy < A.k; ++dy) {
        const int ih = i * A.stride - A.pad + dy;
        if ((unsigned)ih >= (unsigned)A.h)
            continue;
        for (int dx = 0; dx < A.k; ++dx) {
            const int iw = j * A.stride - A.pad + dx;
            if ((unsigned)iw >= (unsigned)A.w)
                continue;
            const uint4 v = *(const uint4 *)(A.x + (((long long)n * A.h + ih) * A.w + iw) * row_bytes + 16 * ch);
            best = make_uint4(packed_max<B>(best.x, v.x), packed_max<B>(best.y, v.y),
                              packed_max<B>(best.z, v.z), packed_max<B>(best.w, v.w));
        }
    }
    *(uint4 *)(A.y + px * row_bytes + 16 * ch) = best;
}

}  // namespace

hipError_t launch_maxpool(const PoolArgs &a, hipStream_t stream)
{
    const int row_bytes = a.c * a.bits / 8;
    if (row_bytes % 16 == 0 && ((uintptr_t)a.x & 15) == 0 && ((uintptr_t)a.y & 15) == 0) {
        const long long items = (long long)a.n * a.ho * a.wo * (row_bytes / 16);
        if (items <= 0)
            return hipSuccess;
        const dim3 grid((unsigned)((items + 255) / 256)), block(256);
        if (a.bits == 2)
            hipLaunchKernelGGL(maxpool16_kernel<2>, grid, block, 0, stream, a);
        else if (a.bits == 4)
            hipLaunchKernelGGL(maxpool16_kernel<4>, grid, block, 0, stream, a);
        else
            hipLaunchKernelGGL(maxpool16_kernel<8>, grid, block, 0, stream, a);
        return hipGetLastError();
    }
    const long long items = (long long)a.n * a.ho * a.wo * (a.c * a.bits / 8);
    if (items <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(maxpool_kernel, dim3((unsigned)((items + 255) / 256)), dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace aqd
