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

// Ordering-wait statistics (instrumented kernels only).  Each wave counts
// its late wave-steps (the turn was not visible at the early look) and the
// real-time clock ticks their waits took in its own registers, and publishes
// them, with its lifetime, by three atomic adds of lane 0 when it exits: an
// atomic on the shared counters at every late step would serialize the waves
// on those addresses and distort the waits being measured.
struct WaitStats {
  unsigned long long begin = 0, late = 0, ticks = 0;
};
__device__ inline unsigned long long clock_now() { return (unsigned long long)__builtin_amdgcn_s_memrealtime(); }
__device__ inline void stats_wave_begin(WaitStats& w) { w.begin = clock_now(); }
__device__ inline void stats_wait(WaitStats& w, unsigned long long t0) {
  w.late += 1;
  w.ticks += clock_now() - t0;
}
__device__ inline void stats_wave_end(const WaitStats& w, unsigned long long* st, int lane) {
  if (lane == 0) {
    atomicAdd(&st[0], w.late);
    atomicAdd(&st[1], w.ticks);
    atomicAdd(&st[2], clock_now() - w.begin);
  }
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

// The same direct loads issued from inline assembly, so the compiler's
// wait-count pass does not see them.  The builtins above make it guard every
// later LDS read that it cannot prove disjoint from the target (it cannot for
// a double buffer with a run-time index, nor through the transposed-read
// pointer casts) with a full vmcnt(0), which drains the next block's prefetch
// and the accumulator fetch in the middle of a step.  With these, the caller
// owns the ordering: before reading the landed bytes it waits with
// s_waitcnt vmcnt (vm_wait, vm_wait_le), and a workgroup barrier follows when
// other waves read them.  `lds` is the wave-uniform LDS byte address of the
// copy (lane i writes bytes [lds + 16i, lds + 16i + 16)); m0 is saved and
// restored around it.
__device__ inline uint32_t lds_base(const void* p) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)p);
}
__device__ inline void dma16(__amdgpu_buffer_rsrc_t r, uint32_t lds, uint32_t off) {
  uint32_t save;
  asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\tbuffer_load_dwordx4 %2, %3, 0 offen lds\n\ts_mov_b32 m0, %0"
               : "=&s"(save) : "s"(lds), "v"(off), "s"(r) : "memory");
}
// ... device-coherent (SC1), with a wave-uniform byte offset added in the
// scalar offset field, so a run of copies at fixed strides shares one
// per-lane offset register
__device__ inline void dma16_coherent(__amdgpu_buffer_rsrc_t r, uint32_t lds, uint32_t off, uint32_t soff) {
  uint32_t save;
  asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\tbuffer_load_dwordx4 %2, %3, %4 offen sc1 lds\n\ts_mov_b32 m0, %0"
               : "=&s"(save) : "s"(lds), "v"(off), "s"(r), "s"(soff) : "memory");
}
// Runs of copies sharing one m0.  The instruction offset field moves both
// the global address and the LDS target, so four 1 KB copies at +0, +1 KB,
// +2 KB and +3 KB of both take one m0 value (x4 forms).  A Q chunk and the
// dO chunk at the same offset go to two LDS targets (pair form).
#define DASH_DMA16X4(name, bits)                                                                  \
  __device__ inline void name(__amdgpu_buffer_rsrc_t r, uint32_t lds, uint32_t off, uint32_t soff) { \
    uint32_t save;                                                                                \
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\t"                                     \
                 "buffer_load_dwordx4 %2, %3, %4 offen " bits " lds\n\t"                          \
                 "buffer_load_dwordx4 %2, %3, %4 offen offset:1024 " bits " lds\n\t"              \
                 "buffer_load_dwordx4 %2, %3, %4 offen offset:2048 " bits " lds\n\t"              \
                 "buffer_load_dwordx4 %2, %3, %4 offen offset:3072 " bits " lds\n\t"              \
                 "s_mov_b32 m0, %0"                                                               \
                 : "=&s"(save) : "s"(lds), "v"(off), "s"(r), "s"(soff) : "memory");               \
  }
DASH_DMA16X4(dma16x4_coherent, "sc1")
#undef DASH_DMA16X4
__device__ inline void dma16_pair(__amdgpu_buffer_rsrc_t r0, __amdgpu_buffer_rsrc_t r1, uint32_t lds0, uint32_t lds1,
                                  uint32_t off, uint32_t soff) {
  uint32_t save;
  asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\tbuffer_load_dwordx4 %3, %4, %6 offen lds\n\t"
               "s_mov_b32 m0, %2\n\tbuffer_load_dwordx4 %3, %5, %6 offen lds\n\ts_mov_b32 m0, %0"
               : "=&s"(save) : "s"(lds0), "s"(lds1), "v"(off), "s"(r0), "s"(r1), "s"(soff) : "memory");
}
__device__ inline void dma4(__amdgpu_buffer_rsrc_t r, uint32_t lds, uint32_t off) {
  uint32_t save;
  asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\tbuffer_load_dword %2, %3, 0 offen lds\n\ts_mov_b32 m0, %0"
               : "=&s"(save) : "s"(lds), "v"(off), "s"(r) : "memory");
}
__device__ inline void dma4_coherent(__amdgpu_buffer_rsrc_t r, uint32_t lds, uint32_t off) {  // SC1: device-coherent
  uint32_t save;
  asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\tbuffer_load_dword %2, %3, 0 offen sc1 lds\n\ts_mov_b32 m0, %0"
               : "=&s"(save) : "s"(lds), "v"(off), "s"(r) : "memory");
}
// The XCD (accelerator complex die, with its own L2) this wave runs on.
__device__ inline int xcc_id() {
  unsigned x;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(x));
  return (int)(x & 15);
}

// The lane index, read afresh where it is called.  Per-lane offsets derived
// from it are rebuilt in a step instead of being hoisted out of the loop and
// spilled: a spill reload waits for every vector memory operation in flight,
// including the copies, stores and atomics the wave has just issued.
__device__ inline int fresh_lane() {
  unsigned lane;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(lane));
  return (int)lane;
}

// Wait until at most N of this wave's vector memory operations are in flight.
// A real s_waitcnt (the compiler's wait-count pass sees it and drops waits of
// its own that it makes redundant), then a compiler memory fence so that no
// LDS read of landed bytes moves above it.  Encoding (gfx9 family): vmcnt in
// bits 3:0 and 15:14, expcnt 6:4 and lgkmcnt 11:8 left at their maxima.
template <int N>
__device__ inline void vm_wait() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
  asm volatile("" ::: "memory");
}
// Wait until at most n (wave-uniform, any value) are in flight: n is rounded
// down to a supported count, which only waits longer.  Vector memory
// operations of a wave complete in issue order, so this guarantees that
// everything issued before the last n of them has completed.
__device__ inline void vm_wait_le(int n) {
  // three levels: the common counts of the callers are 16-17 (a step's
  // prefetch and accumulator copies or stores); the rare others wait longer
  if (n >= 16) vm_wait<16>();
  else if (n >= 8) vm_wait<8>();
  else vm_wait<0>();
}

// Launch a main-kernel instantiation on the persistent grid.  Shift and
// Symmetric Shift chains wait on each other in a cycle, so every workgroup of
// their grid must be resident at once: they launch cooperatively, and a grid
// the device cannot keep resident fails at launch (instead of spinning into
// the wait watchdog).  The others wait only on earlier tickets.
template <typename Kernel>
hipError_t launch_main_grid(Kernel kernel, const BwdArgs& a, int grid, int threads, hipStream_t stream) {
  if (a.G.sched == S_SHIFT || a.G.sched == S_SYMSHIFT) {
    BwdArgs copy = a;  // the arguments are copied at launch
    void* args[] = {&copy};
    return hipLaunchCooperativeKernel((const void*)kernel, dim3(grid), dim3(threads), args, 0, stream);
  }
  hipLaunchKernelGGL(kernel, dim3(grid), dim3(threads), 0, stream, a);
  return hipGetLastError();
}

// One step of a chain, packed for the LDS step table: 64-row block pb (12
// bits), KV tile j (9), rank in the block's summation order (10), last (1).
// kNoStep marks a step whose block or KV tile lies past N.
constexpr unsigned kNoStep = 0xffffffffu;
__device__ inline unsigned pack_step(int pb, int j, int rank, bool last) {
  return (unsigned)pb | ((unsigned)j << 12) | ((unsigned)rank << 21) | ((unsigned)last << 31);
}

}  // namespace dash
