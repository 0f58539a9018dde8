// Sustained int8 matrix-core rate of the GPU this library runs on: a kernel
// of v_mfma_i32_16x16x64_i8 instructions alone (no memory traffic in the
// loop), on register operands of the magnitudes the convolutions multiply
// (4-bit weights in -15..15 and codes in 0..15, drawn per lane), so that the
// rate is the one the matrix cores sustain under that load. It is the
// measured ceiling next to the 5.0 POPS dense int8 figure.

#include "internal.h"
#include "mfma_common.h"

namespace aqd {
namespace {

constexpr int PROBE_ACC = 16;  // independent accumulators per wave

__global__ void __launch_bounds__(256, 2) mfma_probe_kernel(int iters, int *out)
{
    // per-lane operands from a 32-bit linear congruential sequence
    unsigned s = 2654435761u * (blockIdx.x * 256 + threadIdx.x + 1);
    auto next = [&]() { s = s * 1664525u + 1013904223u; return s; };
    v4i a[4], b[4];
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            unsigned wa = 0, wb = 0;
#pragma unroll
            for (int byte = 0; byte < 4; ++byte) {
                wa |= (unsigned)(uint8_t)(int8_t)((int)(next() >> 27) - 15) << (8 * byte);  // -15..16
                wb |= ((next() >> 28) & 15u) << (8 * byte);                                   // 0..15
            }
            a[t][e] = (int)wa;
            b[t][e] = (int)wb;
        }
    v4i acc[PROBE_ACC];
#pragma unroll
    for (int i = 0; i < PROBE_ACC; ++i)
        acc[i] = v4i{0, 0, 0, 0};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int i = 0; i < PROBE_ACC; ++i)
            acc[i] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[i & 3], b[(i >> 2) & 3], acc[i], 0, 0, 0);
    }
    int x = 0;
#pragma unroll
    for (int i = 0; i < PROBE_ACC; ++i)
        x ^= acc[i][0] ^ acc[i][1] ^ acc[i][2] ^ acc[i][3];
    out[blockIdx.x * 256 + threadIdx.x] = x;
}

}  // namespace

hipError_t launch_mfma_probe(int workgroups, int iters, int *out, hipStream_t stream)
{
    hipLaunchKernelGGL(mfma_probe_kernel, dim3(workgroups), dim3(256), 0, stream, iters, out);
    return hipGetLastError();
}

}  // namespace aqd
