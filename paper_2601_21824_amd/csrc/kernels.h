// kernels.h -- interface between the C ABI layer and the HIP kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "schedule.h"

namespace dash {

constexpr int kCtrStride = 32;        // ints per ordering counter (one 128-byte line each)
constexpr int kPoison = -0x40000000;  // counter start value below every rank's turn
constexpr int kCtrlTicket = 0;        // ctrl[] slot: next work item
constexpr int kCtrlError = 16;        // ctrl[] slot: set to 1 when a wait timed out
constexpr int kCtrlXcdTicket = 32;    // ctrl[] slots 32 + x: next work item of XCD x (XCD-local placement)
constexpr int kMaxXcd = 16;           // XCD queues the ctrl block holds
constexpr size_t kCtrlBytes = 256;    // ctrl block at the start of the workspace
constexpr int kMaxChainSteps = 1040;  // 64-row blocks one workgroup chain may visit

struct FwdArgs {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  float* lse;
  int bh, n, causal;
  float scale;
};

// what the main backward kernel does with a KV tile's dQ partial
constexpr int kModeAtomic = 0;    // fp32 atomic adds into dQacc (non-deterministic comparison)
constexpr int kModeOrdered = 1;   // the ordered reduction (every DASH schedule)
constexpr int kModePartials = 2;  // store it in its own buffer; bwd_sum_partials adds them in KV order
constexpr int kModeNoDq = 3;      // no dQ at all: dK, dV only (SPLIT's first pass)
constexpr int kModeOrderedXcd = 4;  // the ordered reduction with every chain of a head on one XCD

struct BwdArgs {
  const void* q;
  const void* k;
  const void* v;
  const void* o;
  const void* dO;
  const float* lse;
  void* dq;
  void* dk;
  void* dv;
  float* dqacc;   // fp32 accumulator (PARTIALS: one per KV tile)
  float* dvec;    // [bh][N] D = rowsum(dO o O)
  float* lse2;    // [bh][N] L * log2(e)
  int* counters;  // [bh][nblk] ordering counters, kCtrStride ints apart
  int* ctrl;      // ticket / error flag
  unsigned* steps;  // [chains][step_cap]: per chain its length, then its packed steps (bwd_pre writes them)
  int step_cap;
  int* order;       // [items][2]: work ticket -> (head, chain) (bwd_pre writes it); XCD-local
                   // placement: XCD x's tickets at [x * xcd_cap, x * xcd_cap + its items)
  int nxcd;         // XCD-local placement: number of XCDs (head bh runs on XCD bh % nxcd); 0: one queue
  int xcd_cap;      // work items per XCD segment of `order`
  int32_t* witness;
  float* partials;
  float* dq_accum;
  int bh, n, nblk, tc;  // tc = real KV tiles per head (ceil(N/bc))
  float scale;
  int spin_limit;
  int poison;
  Geom G;
  hipEvent_t ev_begin, ev_end;  // optional, recorded around bwd_main
  int* status;      // optional caller-owned device int: bwd_pre writes 0, a wait timeout 1
  unsigned long long* wait_stats;  // optional ordering-wait statistics (see dash_bwd_options_t)
};

hipError_t launch_attn_fwd(const FwdArgs& a, int d, hipStream_t stream);
hipError_t launch_bwd(const BwdArgs& a, int d, int grid_main, hipStream_t stream);
hipError_t launch_dq(const BwdArgs& a, int d, hipStream_t stream);  // SPLIT's dQ pass (attn_dq.hip)
int bwd_main_occupancy(int d);
// head dim 64: 128-row KV tiles (attn_bwd_d64.hip) and 256-row tiles (attn_bwd64w.hip)
hipError_t launch_main64(const BwdArgs& a, int grid_main, hipStream_t stream);
int main64_occupancy();
hipError_t launch_main64w(const BwdArgs& a, int grid_main, hipStream_t stream);
int bwd_main64w_occupancy();
// head dim 256 (attn_bwd256.hip)
hipError_t launch_main256(const BwdArgs& a, int grid_main, hipStream_t stream);
int bwd_main256_occupancy();
// measured MFMA throughput (mfma_peak.hip): grid workgroups of 4 waves
void launch_mfma_peak(int grid, int iters, float* sink, hipStream_t stream);
double mfma_peak_flops_per_launch(int grid, int iters);

}  // namespace dash
