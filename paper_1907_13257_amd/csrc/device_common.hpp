// device_common.hpp -- storage types, conversions, gate non-linearities and
// matrix-core (MFMA) wrappers shared by the gfx950 kernels of liblstm355.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lstm355 {

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// Storage types: bf16 values travel as their 16-bit patterns.
typedef uint16_t bf16_t;

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16_t v) { return __uint_as_float(((unsigned)v) << 16); }

// fp32 -> bf16, round to nearest even; NaN stays a NaN.  gfx950 converts in
// one instruction (v_cvt_pk_bf16_f32, rounding per the default RNE mode).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }

// fp16 (binary16) storage of the forward's input projection (the gate
// pre-activations x W^T + b): three more mantissa bits than bf16.  The
// conversion rounds to nearest even and saturates at +-65504, where every
// gate function is flat to fp32 precision; NaN stays a NaN.
typedef _Float16 f16_t;
__device__ __forceinline__ float to_f32(f16_t v) { return (float)v; }
__device__ __forceinline__ f16_t f32_to_f16_sat(float f)
{
    return (f16_t)(f == f ? __builtin_fminf(__builtin_fmaxf(f, -65504.0f), 65504.0f) : f);
}

template <typename TI> __device__ __forceinline__ TI from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) { return f32_to_bf16(v); }
template <> __device__ __forceinline__ f16_t from_f32<f16_t>(float v) { return f32_to_f16_sat(v); }

// Gate non-linearities in fp32.  sigma(u) = 1/(1+e^-u); tanh(u) = 2 sigma(2u) - 1.
// The reciprocal is the hardware's (v_rcp_f32, within 1 ulp) rather than an
// IEEE division sequence.  Both saturate correctly: e^-u overflows to +inf
// for very negative u, and rcp(+inf) = 0.
__device__ __forceinline__ float sigmoid_f(float u) { return __builtin_amdgcn_rcpf(1.0f + __expf(-u)); }
__device__ __forceinline__ float tanh_f(float u) { return 2.0f * __builtin_amdgcn_rcpf(1.0f + __expf(-2.0f * u)) - 1.0f; }

// ---------------------------------------------------------------------------
// MFMA wrappers.  A "fragment" is the 16 bytes one lane contributes per
// operand: 8 bf16 or 4 fp32 values consecutive along k.
//
// 16x16 output block (C[16][16], 4 fp32 per lane: row 4*(lane/16)+v, col lane%16).
//   Operand row (A: output row, B: output col) = lane % 16, and lane group
//   q = lane / 16 (0..3) supplies k = q*E .. q*E+E-1 of a 4E-wide k chunk
//   (E = elements per fragment).  bf16: one v_mfma_f32_16x16x32_bf16 covers
//   the 32-wide chunk.  fp32: four v_mfma_f32_16x16x4f32, element e of every
//   lane group in the e-th instruction.  The sum over k does not depend on
//   which lane holds which k, so A and B only have to agree, which they do
//   by construction.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void mfma16(f32x4 &acc, u32x4 a, u32x4 b, bf16_t)
{
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                  acc, 0, 0, 0);
}
__device__ __forceinline__ void mfma16(f32x4 &acc, u32x4 a, u32x4 b, float)
{
    f32x4 fa = __builtin_bit_cast(f32x4, a), fb = __builtin_bit_cast(f32x4, b);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[0], fb[0], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[1], fb[1], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[2], fb[2], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[3], fb[3], acc, 0, 0, 0);
}

// 32x32 output block (16 fp32 per lane: row 8*(v/4) + 4*(lane/32) + v%4,
// col lane%32).  Operand row = lane % 32; lane group q = lane / 32 (0..1)
// supplies k = q*E .. q*E+E-1 of a 2E-wide chunk.
__device__ __forceinline__ void mfma32(f32x16 &acc, u32x4 a, u32x4 b, bf16_t)
{
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                  acc, 0, 0, 0);
}
__device__ __forceinline__ void mfma32(f32x16 &acc, u32x4 a, u32x4 b, float)
{
    f32x4 fa = __builtin_bit_cast(f32x4, a), fb = __builtin_bit_cast(f32x4, b);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[0], fb[0], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[1], fb[1], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[2], fb[2], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[3], fb[3], acc, 0, 0, 0);
}

__device__ __forceinline__ u32x4 ldg16(const void *p) { return *reinterpret_cast<const u32x4 *>(p); }
__device__ __forceinline__ u32x4 zero16() { return u32x4{0u, 0u, 0u, 0u}; }

// ---------------------------------------------------------------------------
// Direct global -> LDS loads.  A buffer descriptor covers [base, base+bytes);
// loads past its end return zero.  buffer_load_dwordx4 ... lds writes lane
// l's 16 bytes to LDS byte M0 + 16*l, so one wave fills 1 KiB per
// instruction.  It is issued as inline asm so that the compiler does not
// wait for it before unrelated LDS accesses; callers order it themselves
// with s_waitcnt vmcnt and barriers.
// ---------------------------------------------------------------------------
__device__ __forceinline__ u32x4 buffer_desc(const void *base, long bytes)
{
    const unsigned nrec = bytes > 0x7fffffffL ? 0x7fffffffu : (unsigned)bytes;
    const uintptr_t b = reinterpret_cast<uintptr_t>(base);
    return u32x4{(unsigned)b, (unsigned)(b >> 32) & 0xffffu, nrec, 0x00020000u};
}

__device__ __forceinline__ unsigned lds_addr(const void *p) { return (unsigned)(uintptr_t)p; }

// M0 is a register the compiler reserves; naming it as clobbered draws a
// warning but still orders the compiler's own M0 loads around the asm (the
// generated code differs without it), so it stays and the warning is off here.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(u32x4 rsrc, unsigned lds_byte, unsigned voff)
{
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                 :
                 : "s"(lds_byte), "v"(voff), "s"(rsrc)
                 : "memory", "m0");
}

// The same at device (agent) scope: the load misses the CU's L1 and reads the
// L2, so it observes stores other CUs of the same XCD made after an earlier
// read of the same line.
__device__ __forceinline__ void dma16_sc1(u32x4 rsrc, unsigned lds_byte, unsigned voff)
{
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen sc1 lds"
                 :
                 : "s"(lds_byte), "v"(voff), "s"(rsrc)
                 : "memory", "m0");
}
#pragma clang diagnostic pop

// s_waitcnt vmcnt(N) with expcnt and lgkmcnt not waited on (gfx9 encoding:
// vmcnt bits [3:0] and [15:14], expcnt [6:4], lgkmcnt [11:8]).
template <int N>
__device__ __forceinline__ void waitcnt_vm()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 0xf) | (0x7 << 4) | (0xf << 8) | ((N >> 4) << 14));
}

}  // namespace lstm355
