// common.h -- device-side building blocks for the gfx950 (CDNA4) kernels:
// vector types, buffer-resource loads/stores with hardware bounds checking,
// bf16 packing and the two bf16 MFMA shapes used.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dash {

typedef __bf16 bf16x8 __attribute__((__vector_size__(16)));
typedef float f32x16 __attribute__((__vector_size__(64)));
typedef float f32x4 __attribute__((__vector_size__(16)));
typedef unsigned u32x4 __attribute__((__vector_size__(16)));
typedef unsigned u32x2 __attribute__((__vector_size__(8)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Buffer resource over `bytes` bytes at p: loads past the end return 0 and
// stores past the end are dropped, which masks ragged row tails for free.
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

// cache-policy immediates for the buffer builtins (gfx950): bit 4 = SC1, i.e.
// coherent at agent (device) scope across XCDs; 0 = default policy.
constexpr int kCoherent = 16;

__device__ inline u32x4 ld16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}
__device__ inline u32x4 ld16_coherent(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kCoherent);
}
__device__ inline void st16(__amdgpu_buffer_rsrc_t r, uint32_t off, u32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, 0);
}
__device__ inline void st16_coherent(__amdgpu_buffer_rsrc_t r, uint32_t off, u32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, kCoherent);
}
__device__ inline void st8(__amdgpu_buffer_rsrc_t r, uint32_t off, u32x2 v) {
  __builtin_amdgcn_raw_buffer_store_b64(v, r, off, 0, 0);
}
__device__ inline unsigned short ld2(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0);
}
__device__ inline void st2(__amdgpu_buffer_rsrc_t r, uint32_t off, unsigned short v) {
  __builtin_amdgcn_raw_buffer_store_b16(v, r, off, 0, 0);
}
__device__ inline float ld4f(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
__device__ inline void st4f(__amdgpu_buffer_rsrc_t r, uint32_t off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), r, off, 0, 0);
}

// P = 2^x clamped to [0, 1]; the clamp is the exp instruction's own output
// modifier, so it costs nothing.  For a real key x = S*log2(e) - L*log2(e) <= 0
// up to rounding (a score never exceeds its row's logsumexp), so the clamp
// only removes rounding excess.  A padded key of a ragged last KV tile has
// S = 0 (its K row reads as zero): 2^(-L*log2(e)) would overflow to inf for a
// row whose logsumexp is below about -88, and inf * 0 would put NaN into dQ;
// clamped it is 1, and every product it enters has a zero K or V factor.
__device__ inline float exp2_unit(float x) {
  return __builtin_amdgcn_fmed3f(__builtin_amdgcn_exp2f(x), 0.f, 1.f);
}

// fp32 -> bf16 with round-to-nearest-even (hardware v_cvt_pk_bf16_f32)
__device__ inline unsigned pack_bf16(float lo, float hi) {
  typedef __bf16 bf16x2 __attribute__((__vector_size__(4)));
  bf16x2 r = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(unsigned, r);
}
__device__ inline unsigned short to_bf16(float x) {
  return __builtin_bit_cast(unsigned short, (__bf16)x);
}
__device__ inline float bf16_to_f32(unsigned short h) {
  return __builtin_bit_cast(float, (unsigned)h << 16);
}

// two 16-bit lanes of a and b at the same position: e even -> low halves
__device__ inline unsigned pick16(unsigned a, unsigned b, int odd) {
  return odd ? __builtin_amdgcn_perm(b, a, 0x07060302u) : __builtin_amdgcn_perm(b, a, 0x05040100u);
}

__device__ inline f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ inline bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }
__device__ inline bf16x8 as_bf16x8(u32x2 lo, u32x2 hi) {
  u32x4 v = {lo[0], lo[1], hi[0], hi[1]};
  return __builtin_bit_cast(bf16x8, v);
}

// 8 consecutive accumulator values -> one bf16x8 MFMA operand
__device__ inline bf16x8 pack8(const f32x16& a, int base) {
  u32x4 v = {pack_bf16(a[base + 0], a[base + 1]), pack_bf16(a[base + 2], a[base + 3]),
             pack_bf16(a[base + 4], a[base + 5]), pack_bf16(a[base + 6], a[base + 7])};
  return __builtin_bit_cast(bf16x8, v);
}

// LDS chunk swizzle for the [row][64] transposed tiles: 8-byte chunk c of row
// `row` lives at chunk c ^ f(row); writes along rows 8 apart and reads along
// 32 consecutive rows both spread over all banks.
__device__ inline int tswz(int row) { return ((row >> 3) ^ ((row & 7) << 1)) & 15; }

}  // namespace dash
