// Standalone integer skip connection (Sec. 3.2.3, Eq. 7) with nearest 2x
// upsample of the coarser operand (Sec. 3.2.4), and exact per-channel sums of
// an int32 tensor (the statistics a BN layer keeps, Sec. 3.2.2).

#include "epilogue.h"
#include "internal.h"

namespace aqd {
namespace {

__device__ __forceinline__ int load_value(const void *base, long long pix, int c, int ch, int bits)
{
    if (bits == 32)
        return ((const int32_t *)base)[pix * c + ch];
    return load_code((const uint8_t *)base + pix * (c * bits / 8), ch, bits);
}

// One thread per output byte: 8 / b_out channels of one pixel.
__global__ void __launch_bounds__(256) qadd_kernel(QaddArgs A)
{
    const int per = 8 / A.bits_out;
    const int groups = A.c / per;
    const long long P = (long long)A.n * A.h * A.w;
    const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= P * groups)
        return;
    const long long px = idx / groups;
    const int grp = (int)(idx - px * groups);
    long long bpix = px;
    if (A.up2) {
        const int hw = A.h * A.w;
        const int n = (int)(px / hw);
        const int rem = (int)(px - (long long)n * hw);
        const int y = rem / A.w, x = rem - y * A.w;
        bpix = ((long long)n * A.hb + (y >> 1)) * A.wb + (x >> 1);
    }
    const int qmax = A.qmax;
    uint32_t packed = 0;
    for (int e = 0; e < per; ++e) {
        const int ch = grp * per + e;
        const int a = load_value(A.a, px, A.c, ch, A.bits_a);
        const int b = load_value(A.b, bpix, A.c, ch, A.bits_b);
        const long long u = align_add(a, b, A.skip_c[ch], A.skip_d[ch], A.skip_side[ch]);
        packed |= requant_clamp(u, A.mult[ch], A.shift[ch], qmax) << (e * A.bits_out);
    }
    A.y[px * (A.c * A.bits_out / 8) + grp] = (uint8_t)packed;
}

// Workgroup: 256 consecutive channels x a strip of rows; int64 partial sums
// per thread, one atomic add per channel and workgroup (integer addition is
// associative, so the result is exact and order independent).
__global__ void __launch_bounds__(256) channel_sums_kernel(const int32_t *v, long long rows, int c,
                                                          long long rows_per_block, long long *sums)
{
    const int ch = blockIdx.x * 256 + threadIdx.x;
    if (ch >= c)
        return;
    const long long r0 = (long long)blockIdx.y * rows_per_block;
    long long r1 = r0 + rows_per_block;
    if (r1 > rows)
        r1 = rows;
    long long s1 = 0, s2 = 0;
    for (long long r = r0; r < r1; ++r) {
        const long long x = v[r * c + ch];
        s1 += x;
        s2 += x * x;
    }
    atomicAdd((unsigned long long *)&sums[ch], (unsigned long long)s1);
    atomicAdd((unsigned long long *)&sums[c + ch], (unsigned long long)s2);
}

}  // namespace

hipError_t launch_qadd(const QaddArgs &a, hipStream_t stream)
{
    const long long total = (long long)a.n * a.h * a.w * (a.c / (8 / a.bits_out));
    if (total == 0)
        return hipSuccess;
    const long long blocks = (total + 255) / 256;
    if (blocks > 0x7fffffffLL)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(qadd_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_channel_sums(const int32_t *v, long long rows, int c, long long *sums,
                               hipStream_t stream)
{
    if (rows == 0)
        return hipSuccess;
    // at most 4096 row strips (grid.y limit is 65535)
    long long rows_per_block = (rows + 4095) / 4096;
    if (rows_per_block < 256)
        rows_per_block = 256;
    const long long ystrips = (rows + rows_per_block - 1) / rows_per_block;
    dim3 grid((c + 255) / 256, (unsigned)ystrips);
    hipLaunchKernelGGL(channel_sums_kernel, grid, dim3(256), 0, stream, v, rows, c, rows_per_block,
                       sums);
    return hipGetLastError();
}

}  // namespace aqd
