// Device helpers shared by the gfx950 kernels: vector types, 16-byte memory moves, bf16
// packing and the matrix-core wrappers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pkv {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;

constexpr int kBlockSize = 16;  // tokens per KV block (the only supported block size)
constexpr float kLn2 = 0.69314718055994530942f;
constexpr float kLog2e = 1.44269504088896340736f;

__device__ __forceinline__ u32x4 ld16(const void* p) {
  return *reinterpret_cast<const u32x4*>(p);
}
__device__ __forceinline__ void st16(void* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }
// 16-byte store with the non-temporal hint (streaming data the launch does not read again)
__device__ __forceinline__ void st16_nt(void* p, u32x4 v) {
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
}
__device__ __forceinline__ u32x2 ld8(const void* p) {
  return *reinterpret_cast<const u32x2*>(p);
}
__device__ __forceinline__ void st8(void* p, u32x2 v) { *reinterpret_cast<u32x2*>(p) = v; }

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Two floats -> two bf16 (round to nearest even) packed low/high in one 32-bit word.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
  bf16x2 v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// 16x16x32 bf16 matrix-core product, fp32 accumulate: D = A(16x32) B(32x16) + C.
// Lane l holds A[l%16][8(l/16) .. 8(l/16)+7], B[8(l/16) .. +7][l%16], and D[4(l/16)+r][l%16].
__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// 32x32x16 bf16 matrix-core product, fp32 accumulate: D = A(32x16) B(16x32) + C.
// Lane l holds A[l%32][8(l/32) .. +7], B[8(l/32) .. +7][l%32], and D[8(i/4)+4(l/32)+i%4][l%32]
// in register i (0..15).
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Fourth word of a raw buffer resource on gfx9-family parts: 32-bit data format, no
// swizzle, no index stride -- a plain byte-addressed buffer.
constexpr int kBufferFlags = 0x00020000;

// Direct global -> LDS load of 16 bytes per lane through a buffer resource whose base is
// `base` and which holds `bytes` bytes (the hardware bounds-checks `voffset`): lane i's
// 16 bytes land at lds + 16 i. The buffer form, unlike the global form, leaves the
// compiler's LDS-read wait counting exact. The builtins exist for the device target only,
// so the body is compiled in the device pass.
__device__ __forceinline__ void lds_load16(const void* base, int bytes, int voffset, void* lds) {
#if __HIP_DEVICE_COMPILE__
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, kBufferFlags);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (__attribute__((address_space(3))) void*)lds,
                                           16, voffset, 0, 0, 0);
#endif
}

// 16- and 8-byte loads through a buffer resource: wave-uniform `base` (kept in scalar
// registers) plus a 32-bit per-lane byte offset, so a load needs one address register
// instead of two. Offsets at or past `bytes` read zero.
__device__ __forceinline__ u32x4 buf_ld16(const void* base, int bytes, int voffset) {
#if __HIP_DEVICE_COMPILE__
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, kBufferFlags);
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, voffset, 0, 0));
#else
  return u32x4{0u, 0u, 0u, 0u};
#endif
}
__device__ __forceinline__ u32x2 buf_ld8(const void* base, int bytes, int voffset) {
#if __HIP_DEVICE_COMPILE__
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, kBufferFlags);
  return __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(rsrc, voffset, 0, 0));
#else
  return u32x2{0u, 0u};
#endif
}

}  // namespace pkv
