// Integer epilogue of one output element, shared by every kernel.
//
//   v  = acc + bias                                   (Sec. 3.2.2, Eq. 6)
//   u  = v + RSM(k, c, d)      side 0                 (Sec. 3.2.3, Eq. 7-8)
//      = RSM(v, c, d) + k      side 1
//   y  = clamp(RSM(u, M, 31 + sh), 0, qmax)           (Eq. 2 on integers)
//
// RSM(a, c, d) = floor((a*c + 2^(d-1)) / 2^d), and a*c for d = 0. With
// |a| < 2^31 and |c| < 2^31 the product stays below 2^62 and the rounding
// constant below 2^61, so the 64-bit sum cannot overflow; an arithmetic
// right shift of a signed 64-bit value is the floor division.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace aqd {

__device__ __forceinline__ long long rsm(long long a, long long c, int d)
{
    long long p = a * c;
    return d > 0 ? ((p + (1LL << (d - 1))) >> d) : p;
}

__device__ __forceinline__ long long align_add(int v, int k, int c, int d, int side)
{
    return side == 0 ? (long long)v + rsm(k, c, d) : rsm(v, c, d) + (long long)k;
}

__device__ __forceinline__ uint32_t requant_clamp(long long u, int mult, int shift, int qmax)
{
    long long y = rsm(u, mult, 31 + shift);
    y = y < 0 ? 0 : y;
    y = y > qmax ? qmax : y;
    return (uint32_t)y;
}

// Code of channel c of a packed row (bits in {2, 4, 8}).
__device__ __forceinline__ int load_code(const uint8_t *row, int c, int bits)
{
    int bit = c * bits;
    return (row[bit >> 3] >> (bit & 7)) & ((1 << bits) - 1);
}

}  // namespace aqd
