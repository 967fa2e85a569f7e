// Shared device helpers of the gfx950 kernels (MFMA wrappers, vector types,
// LDS swizzles, 8x8 half transposes).  Internal to liblt; not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lt {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half4 __attribute__((ext_vector_type(4)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// D[32x32] += A[32x16] * B[16x32], fp16 in, fp32 accumulate.
// Operand lane layout: lane l supplies row/column (l % 32) and 8 consecutive
// reduction indices selected by (l / 32); A and B use the same reduction
// index mapping, so any consistent permutation of the reduction axis is
// allowed.  Result: lane l holds column (l % 32), rows
// 8*(r/4) + 4*(l/32) + (r%4) for r = 0..15.
__device__ __forceinline__ f32x16 mfma32(half8 a, half8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// D[16x16] += A[16x32] * B[32x16], fp16 in, fp32 accumulate.
// Operand lane layout: lane l supplies row/column (l % 16) and 8 consecutive
// reduction indices 8*(l/16) + 0..7 (any consistent permutation of the
// reduction axis is allowed).  Result: lane l holds column (l % 16), rows
// 4*(l/16) + r for r = 0..3.  At equal FLOPs it draws less power than the
// 32x32x16 form, which sustains a higher clock under full load.
__device__ __forceinline__ f32x4 mfma16(half8 a, half8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// Registers loaded from global memory before a loop are marked as used at
// this point: the compiler then waits for their loads here, once, instead of
// before their first use inside the loop.  That in-loop wait would be a
// vmcnt(0) executed every iteration, and vmcnt also counts the direct-to-LDS
// prefetches issued inside the loop (opaque to the compiler), so each
// iteration would wait for its own prefetch.  Call it after an explicit
// vmcnt(0), where it costs nothing.
template <class T>
__device__ __forceinline__ void loaded_here(const T& v) {
  asm volatile("" ::"v"(v));
}

__device__ __forceinline__ half8 as_half8(u32x4 v) {
  return __builtin_bit_cast(half8, v);
}
__device__ __forceinline__ u32x4 as_u32x4(half8 v) {
  return __builtin_bit_cast(u32x4, v);
}

// 16-byte global load / store helpers.
__device__ __forceinline__ u32x4 ld16(const void* p) {
  return *reinterpret_cast<const u32x4*>(p);
}
__device__ __forceinline__ void st16(void* p, u32x4 v) {
  *reinterpret_cast<u32x4*>(p) = v;
}

// Transpose an 8x8 block of halves held as 8 rows of 16 bytes:
// in[r] holds elements (r, 0..7); out[c] receives elements (0..7, c).
__device__ __forceinline__ void transpose8x8(const u32x4 in[8], u32x4 out[8]) {
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const int w = c >> 1;
    const bool hi = c & 1;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t a = in[2 * q][w];
      const uint32_t b = in[2 * q + 1][w];
      out[c][q] = hi ? ((a >> 16) | (b & 0xffff0000u)) : ((a & 0xffffu) | (b << 16));
    }
  }
}

// Pack 8 fp32 values into 8 fp16 (round to nearest even).
__device__ __forceinline__ half8 pack8(float a0, float a1, float a2, float a3,
                                       float a4, float a5, float a6, float a7) {
  half8 h;
  h[0] = (_Float16)a0; h[1] = (_Float16)a1; h[2] = (_Float16)a2; h[3] = (_Float16)a3;
  h[4] = (_Float16)a4; h[5] = (_Float16)a5; h[6] = (_Float16)a6; h[7] = (_Float16)a7;
  return h;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// ---- buffer resources, direct global->LDS loads, LDS transpose reads ----
typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef short v4s __attribute__((ext_vector_type(4)));
#define LT_LDS __attribute__((address_space(3)))

// Raw buffer over `bytes` bytes at p: loads at offsets >= bytes return 0.
__device__ __forceinline__ rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
// Offset that is always out of range: the load returns zeros.
constexpr uint32_t kOOB = 0x80000000u;

// Direct load of 16 bytes per lane into LDS: lane l's bytes land at
// lds + 16*l (one contiguous KiB per wave).  lds must be wave-uniform.
__device__ __forceinline__ void lds_dma16(rsrc_t r, void* lds, uint32_t voff, uint32_t soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (LT_LDS void*)lds, 16, (int)voff, (int)soff, 0, 0);
}

// Same load, issued as an opaque instruction pair (M0 = LDS address, then the
// buffer load).  The compiler does not see the LDS write, so it adds no
// conservative vmcnt wait before later LDS reads of *other* buffers; the
// caller orders the data with an explicit s_waitcnt vmcnt + barrier.  Raw
// buffer descriptor: 48-bit base, stride 0, num_records bytes.
__device__ __forceinline__ void lds_dma16_opaque(const void* base, uint32_t nrec, void* lds,
                                                 uint32_t voff) {
  const uint64_t b = (uint64_t)base;
  u32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane((uint32_t)b);
  r[1] = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32) & 0xffffu);
  r[2] = __builtin_amdgcn_readfirstlane(nrec);
  r[3] = 0x00020000u;
  const uint32_t m0v = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(m0v), "v"(voff), "s"(r)
               : "memory");
}

// 4 bytes per lane (lane l's dword lands at lds + 4*l); otherwise as above.
__device__ __forceinline__ void lds_dma4_opaque(const void* base, uint32_t nrec, void* lds,
                                                uint32_t voff) {
  const uint64_t b = (uint64_t)base;
  u32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane((uint32_t)b);
  r[1] = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32) & 0xffffu);
  r[2] = __builtin_amdgcn_readfirstlane(nrec);
  r[3] = 0x00020000u;
  const uint32_t m0v = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dword %1, %2, 0 offen lds"
               :
               : "s"(m0v), "v"(voff), "s"(r)
               : "memory");
}

// ds_read_b64_tr_b16: within each 16-lane group, lane l receives element
// (l % 4) of the 8-byte chunks read by lanes (l/4) + 4q, q = 0..3.
__device__ __forceinline__ v4s lds_read_tr16(const void* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((LT_LDS v4s*)(p));
}

__device__ __forceinline__ u32x4 pack_v4s_pair(v4s a, v4s b) {
  u32x4 w;
  w[0] = (uint32_t)(uint16_t)a[0] | ((uint32_t)(uint16_t)a[1] << 16);
  w[1] = (uint32_t)(uint16_t)a[2] | ((uint32_t)(uint16_t)a[3] << 16);
  w[2] = (uint32_t)(uint16_t)b[0] | ((uint32_t)(uint16_t)b[1] << 16);
  w[3] = (uint32_t)(uint16_t)b[2] | ((uint32_t)(uint16_t)b[3] << 16);
  return w;
}

}  // namespace lt
