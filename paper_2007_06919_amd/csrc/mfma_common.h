// Device helpers shared by the MFMA convolution kernels: compile-time loops,
// the 32-bit forms of the integer epilogue's rounding steps, LDS swizzles and
// addressing, the LDS-DMA copy, raw buffer loads, and packed-word loads and
// stores.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

namespace aqd {
namespace {

// f(integral_constant<int, 0>) ... f(integral_constant<int, N-1>): compile-time
// indices, so register arrays indexed by them stay in registers.
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F &&f, std::integer_sequence<int, I...>)
{
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F &&f)
{
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

typedef int v4i __attribute__((ext_vector_type(4)));

// Raw buffer loads (buffer_load_dwordx4 / _dwordx2 ... offen): 16 or 8 bytes
// at byte offset voff + soff of the resource's base. The hardware checks the offset against
// the resource's size and returns zeros for an access at or past it (no
// memory is touched), which the kernels use for padding taps and look-ahead
// past the last K step. Word 3 of the descriptor: 32-bit data format, as a
// raw (untyped) buffer on gfx9-family GPUs needs.
typedef __amdgpu_buffer_rsrc_t buf_rsrc;
__device__ __forceinline__ buf_rsrc make_rsrc(const void *p, int bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, bytes, 0x00020000);
}
__device__ __forceinline__ v4i load_b128(buf_rsrc r, int voff, int soff)
{
    return (v4i)__builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
}
__device__ __forceinline__ uint2 load_b64(buf_rsrc r, int voff, int soff)
{
    typedef unsigned v2u __attribute__((ext_vector_type(2)));
    const v2u v = __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0);
    return make_uint2(v.x, v.y);
}


// round(a * c / 2^d), ties up, d in [0, 31], result modulo 2^32: one 64-bit
// multiply-add (exact: |a*c| < 2^62) and a funnel shift. The rounding term
// 2^(d-1) (0 for d = 0) is (2^d) / 2 in 32 bits (below 2^31: a zero high
// word), the addend of the multiply-add.
__device__ __forceinline__ long long rsm_rnd(int d) { return (long long)((1u << d) >> 1); }
// with the rounding term computed once per channel (rnd = rsm_rnd(d))
__device__ __forceinline__ int rsm32r(int a, int c, long long rnd, int d)
{
    long long t;
    asm("v_mad_i64_i32 %0, vcc, %1, %2, %3" : "=v"(t) : "v"(a), "v"(c), "v"(rnd) : "vcc");
    return (int)__builtin_amdgcn_alignbit((unsigned)((unsigned long long)t >> 32), (unsigned)t, (unsigned)d);
}
__device__ __forceinline__ int rsm32(int a, int c, int d) { return rsm32r(a, c, rsm_rnd(d), d); }

// Requantisation of u with shift >= 2, before the clamp: with d = 31 + shift,
// floor((u*M + 2^(d-1)) / 2^d) = (high word of u*M + 2^(d-33) * 2^32) >> (d - 32),
// the high word taken exactly from one 64-bit multiply-add (rnd = 2^(shift-2),
// shr = shift - 1).
// (written as one v_mad_i64_i32: left to itself the compiler splits it into a
// high multiply and an add)
__device__ __forceinline__ int requant32(int u, int m, long long rnd_hi, int shr)
{
    long long t;
    asm("v_mad_i64_i32 %0, vcc, %1, %2, %3" : "=v"(t) : "v"(u), "v"(m), "v"(rnd_hi) : "vcc");
    return (int)(t >> 32) >> shr;
}


// XOR swizzle of the 16-byte columns of weight row r (64-byte rows): the
// 16-byte reads of 16 consecutive rows at one logical column hit distinct
// banks whether 8 or 16 lanes are served per cycle.
__device__ __forceinline__ int swz_a(int r) { return ((r >> 1) ^ (r >> 2)) & 3; }
// XOR swizzle of the 16-byte halves of a 32-byte packed 4-bit code row.
__device__ __forceinline__ int swz_b4(int p) { return (p >> 3) & 1; }

// 16 bytes per lane from global memory straight into LDS at byte address
// la + 16 * lane (la wave-uniform, kept in SGPRs, in M0). Issued as inline
// assembly so that the compiler does not track it: every wait for these
// copies is an explicit wait_vmcnt (the counter retires in issue order, so the
// compiler's own waits for later loads stay correct, only stricter).
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(const void *g, uint32_t la)
{
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
                 ::"s"(__builtin_amdgcn_readfirstlane(la)), "v"(g) : "memory", "m0");
}
#pragma clang diagnostic pop

// LDS byte address of a shared-memory pointer
__device__ __forceinline__ uint32_t lds_addr(const void *p)
{
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint8_t *)p;
}

// a + byte b of w (b a constant once unrolled), one SDWA add: kept out of the
// compiler's reach, which otherwise rebuilds the byte as a shift and a mask
__device__ __forceinline__ uint32_t add_byte(uint32_t a, uint32_t w, int b)
{
    uint32_t r;
    switch (b) {
    case 0: asm("v_add_u32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_0"
                : "=v"(r) : "v"(a), "v"(w)); break;
    case 1: asm("v_add_u32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_1"
                : "=v"(r) : "v"(a), "v"(w)); break;
    case 2: asm("v_add_u32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_2"
                : "=v"(r) : "v"(a), "v"(w)); break;
    default: asm("v_add_u32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_3"
                 : "=v"(r) : "v"(a), "v"(w)); break;
    }
    return r;
}

// 3-bit outputs in 4-bit containers: min(code, 7) in each nibble of a word
// of 4-bit codes already clamped to [0, 15] (a nibble >= 8 has bit 3 set)
__device__ __forceinline__ uint32_t sat7_nibbles(uint32_t w)
{
    const uint32_t m = (w >> 3) & 0x11111111u;
    return (w & ~((m << 4) - m)) | ((m << 3) - m);  // m * 15, m * 7 without carries
}

template <int N>
__device__ __forceinline__ void wait_vmcnt()
{
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

template <int W>
__device__ __forceinline__ void load_words(const uint8_t *p, uint32_t *w)
{
    if constexpr (W == 1) {
        w[0] = *(const uint32_t *)p;
    } else if constexpr (W == 2) {
        const uint2 t = *(const uint2 *)p;
        w[0] = t.x;
        w[1] = t.y;
    } else {
#pragma unroll
        for (int u = 0; u < W; u += 4) {
            const uint4 t = *(const uint4 *)(p + 4 * u);
            w[u] = t.x;
            w[u + 1] = t.y;
            w[u + 2] = t.z;
            w[u + 3] = t.w;
        }
    }
}

template <int W>
__device__ __forceinline__ void store_words(uint8_t *p, const uint32_t *w)
{
    if constexpr (W == 1) {
        *(uint32_t *)p = w[0];
    } else if constexpr (W == 2) {
        *(uint2 *)p = make_uint2(w[0], w[1]);
    } else {
#pragma unroll
        for (int u = 0; u < W; u += 4)
            *(uint4 *)(p + 4 * u) = make_uint4(w[u], w[u + 1], w[u + 2], w[u + 3]);
    }
}

}  // namespace
}  // namespace aqd
