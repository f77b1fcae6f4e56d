// bwd_common.h -- device pieces shared by the backward main kernels: the
// ordering wait, transposed LDS reads, direct global->LDS loads and the
// packed per-chain step table.
#pragma once
#include "common.h"
#include "kernels.h"

namespace dash {

// ---------------------------------------------------------------- ordering
// Spin until *ctr >= want (relaxed, device-coherent loads).  Wave-uniform.
// A block's counter advances by one per wave of each contributor, so rank r
// holds the turn once it reads at least (waves per workgroup) * r.  The test
// is "at least", not "equal": the other waves of the same workgroup share the
// rank and bump the counter as soon as their own slices are stored, so a wave
// that polls late sees up to waves - 1 more; it cannot see (waves) * (r + 1),
// which needs its own bump.
// Returns false after `limit` polls; the caller then skips its update.
__device__ inline bool wait_turn(const int* ctr, int want, int limit) {
  for (int n = 0;; ++n) {
    const int v = __builtin_amdgcn_readfirstlane(__hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
    if (v >= want) break;
    if (n >= limit) return false;
    __builtin_amdgcn_s_sleep(2);
  }
  __atomic_signal_fence(__ATOMIC_SEQ_CST);  // keep the data loads after the wait
  return true;
}

// 4 bf16 of one column from 4 consecutive rows (gfx950 transpose read): within
// each group of 16 lanes, lane L addresses row L/4, columns 4*(L%4)..+3 of a
// 4 x 16 tile and receives column L of it.
__device__ inline u32x2 tr_read(const __bf16* p) {
  typedef short s16x4 __attribute__((__vector_size__(8)));
  s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(p));
  return __builtin_bit_cast(u32x2, v);
}

// Direct global -> LDS load of 16 (or 4) bytes per lane: lane i of the wave
// writes bytes [16i, 16i+16) after the wave-uniform LDS base `dst`.
typedef __attribute__((address_space(3))) void* lds_ptr;
__device__ inline void lds_load16(__amdgpu_buffer_rsrc_t r, void* dst, uint32_t off) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr)dst, 16, off, 0, 0, 0);
}
__device__ inline void lds_load16_coherent(__amdgpu_buffer_rsrc_t r, void* dst, uint32_t off) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr)dst, 16, off, 0, 0, kCoherent);
}
__device__ inline void lds_load4(__amdgpu_buffer_rsrc_t r, void* dst, uint32_t off) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr)dst, 4, off, 0, 0, 0);
}

// One step of a chain, packed for the LDS step table: 64-row block pb (12
// bits), KV tile j (9), rank in the block's summation order (10), last (1).
// kNoStep marks a step whose block or KV tile lies past N.
constexpr unsigned kNoStep = 0xffffffffu;
__device__ inline unsigned pack_step(int pb, int j, int rank, bool last) {
  return (unsigned)pb | ((unsigned)j << 12) | ((unsigned)rank << 21) | ((unsigned)last << 31);
}

}  // namespace dash
