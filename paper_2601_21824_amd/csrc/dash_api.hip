// dash_api.hip -- the C ABI declared in include/dash.h: argument checking,
// schedule resolution, workspace layout, kernel launches and error reporting.
// Host code only; the kernels live in attn_fwd.hip and attn_bwd.hip.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <tuple>

#include "dag_model.h"
#include "dash.h"
#include "kernels.h"
#include "model_calibration.h"
#include "schedule.h"

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(DASH_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct Layout {
  size_t ctrl, dqacc, dvec, lse2, counters, steps, order, total;
  int step_cap;
};

// ctrl first so that dash_bwd_check can find it without the problem size.
// The layout depends on the schedule only through PARTIALS, which keeps one
// accumulator-sized buffer per KV tile: the step and ticket tables are sized
// for the longest chains and the most chains of any schedule and mask, so a
// workspace sized for one schedule serves every other one (and both masks).
Layout layout(int B, int H, int N, int d, int sched) {
  Layout L;
  const size_t bh = (size_t)B * H;
  const size_t nblk = ((size_t)N + dash::kBlockRows - 1) / dash::kBlockRows;
  const int bc_f = dash::kv_tile_rows(d, 0, N, (long)bh), bc_c = dash::kv_tile_rows(d, 1, N, (long)bh);
  const size_t bc = (size_t)(bc_f < bc_c ? bc_f : bc_c);  // PARTIALS: the more tiles of either mask
  const size_t copies = sched == DASH_SCHED_PARTIALS ? ((size_t)N + bc - 1) / bc : 1;
  size_t off = 0;
  L.ctrl = off;
  off += dash::kCtrlBytes;
  L.dqacc = off;
  off += align256(copies * bh * nblk * dash::kBlockRows * d * sizeof(float));  // >= N rows per head
  L.dvec = off;
  off += align256(bh * N * sizeof(float));
  L.lse2 = off;
  off += align256(bh * N * sizeof(float));
  L.counters = off;
  off += align256(bh * nblk * dash::kCtrStride * sizeof(int));
  // per-chain step tables: at most T_c + 1 chains (Symmetric Shift pads T_c
  // to even), each its length and at most (T_r + 1) * nsub steps (full mask:
  // 64-row Q tiles; causal: Symmetric Shift's padded T_r + 1 tasks); then the
  // ticket order
  const dash::Geom G = dash::make_geom(dash::S_SHIFT, 0, N, d, (long)bh);
  const dash::Geom Gc = dash::make_geom(dash::S_SYMSHIFT, 1, N, d, (long)bh);
  const int cap_f = (G.t_r + 1) * G.nsub, cap_c = (Gc.t_r + 1) * Gc.nsub;
  L.step_cap = 1 + (cap_f > cap_c ? cap_f : cap_c);
  const size_t chains = (size_t)(G.t_c > Gc.t_c ? G.t_c : Gc.t_c) + 1;
  L.steps = off;
  off += align256(chains * L.step_cap * sizeof(unsigned));
  L.order = off;
  off += align256((bh + dash::kMaxXcd) * chains * 2 * sizeof(int));  // XCD segments round up per XCD
  L.total = off;
  return L;
}

struct DeviceInfo {
  int device = -1;
  int cus = 0;
  int occ64 = 0, occ128 = 0, occ256 = 0;
  bool probed = false;  // nxcd is known (the probe allocates, so it runs only when XCD placement is asked for)
  int nxcd = 0;  // XCDs, when workgroup i runs on XCD i % nxcd (0: not usable for XCD-local placement)
};

// A call with no rows still reports "no timeout": one lane stores 0 into the
// workspace's error flag and / or the caller's status word (a kernel, not a
// memset, so that the call stays capturable into a HIP graph).
__global__ void clear_flags_kernel(int* flag, int* status) {
  if (threadIdx.x == 0) {
    if (flag) *flag = 0;
    if (status) *status = 0;
  }
}

int clear_flags(int* flag, int* status, void* stream);

// Each workgroup records the XCD it runs on.
__global__ void xcc_probe_kernel(int* out) {
  unsigned x;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(x));
  if (threadIdx.x == 0) out[blockIdx.x] = (int)(x & 15);
}

// Number of XCDs if the dispatcher deals workgroups out to them round-robin
// (what the XCD-local placement relies on to give every XCD its share of a
// persistent grid whose size is a multiple of the XCD count), else 0.  The
// deal may start at any XCD: it continues from the previous dispatch.
int probe_xcds() {
  constexpr int kWg = 64;
  int* d = nullptr;
  if (hipMalloc(&d, kWg * sizeof(int)) != hipSuccess) return 0;
  int h[kWg];
  hipLaunchKernelGGL(xcc_probe_kernel, dim3(kWg), dim3(64), 0, nullptr, d);
  const bool ok = hipGetLastError() == hipSuccess && hipMemcpy(h, d, sizeof(h), hipMemcpyDeviceToHost) == hipSuccess;
  (void)hipFree(d);
  if (!ok) return 0;
  int n = 0;
  for (int i = 0; i < kWg; ++i) n = h[i] + 1 > n ? h[i] + 1 : n;
  if (n < 1 || n > dash::kMaxXcd) return 0;
  for (int i = 0; i < kWg; ++i)
    if (h[i] != (h[0] + i) % n) return 0;
  return n;
}

std::mutex g_mu;
DeviceInfo g_dev[64];

// bytes of dash_attn_bwd_noalloc's fixed workspace on each device
constexpr size_t kScratchBytes = (size_t)256 << 20;

}  // namespace

// dash_attn_bwd_noalloc's workspace: each device holds its own copy from
// module load until the process ends.
static __device__ __align__(256) unsigned char dash_scratch[kScratchBytes];

namespace {

// The current device's properties (queried once per device).  With xcd, also
// whether XCD-local placement is usable: that probe runs a kernel on a small
// buffer it allocates, so only calls that ask for XCD placement run it.
int device_info(DeviceInfo* out, bool xcd = false) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(DASH_ERR_NO_DEVICE, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= 64) return fail(DASH_ERR_NO_DEVICE, "device index out of range");
  std::lock_guard<std::mutex> lk(g_mu);
  DeviceInfo& di = g_dev[dev];
  if (di.device < 0) {
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDeviceProperties");
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
      return fail(DASH_ERR_NO_DEVICE, std::string("libdash is built for gfx950, device is ") + prop.gcnArchName);
    di.cus = prop.multiProcessorCount;
    di.occ64 = dash::bwd_main_occupancy(64);
    di.occ128 = dash::bwd_main_occupancy(128);
    di.occ256 = dash::bwd_main_occupancy(256);
    if (di.occ64 <= 0 || di.occ128 <= 0 || di.occ256 <= 0) return fail(DASH_ERR_HIP, "occupancy query failed");
    di.device = dev;
  }
  if (xcd && !di.probed) {
    di.nxcd = probe_xcds();
    di.probed = true;
  }
  *out = di;
  return DASH_OK;
}

int check_shape(int B, int H, int N, int d) {
  if (B < 0 || H < 0 || N < 0) return fail(DASH_ERR_INVALID_ARG, "B, H and N must be >= 0");
  if (d != 64 && d != 128 && d != 256) return fail(DASH_ERR_INVALID_ARG, "head dim d must be 64, 128 or 256");
  if ((double)N * d * 4 >= 2147483648.0) return fail(DASH_ERR_INVALID_ARG, "N*d too large (per-head fp32 > 2 GiB)");
  if ((double)B * H >= 2147483647.0 / 1024) return fail(DASH_ERR_INVALID_ARG, "B*H too large");
  // the interface's documented row limit (row counts stay far inside int range)
  if ((double)B * H * N >= 1073741824.0) return fail(DASH_ERR_INVALID_ARG, "B*H*N too large (at most 2^30 - 1 rows)");
  return DASH_OK;
}

int resolve(int schedule, int d, int causal) {
  switch (schedule) {
    case DASH_SCHED_AUTO:
      return causal ? DASH_SCHED_DESCENDING : DASH_SCHED_SHIFT;
    case DASH_SCHED_SHIFT:
      return causal ? DASH_SCHED_SYMSHIFT : DASH_SCHED_SHIFT;
    default:
      return schedule;
  }
}

int check_schedule(int schedule, int causal) {
  if (schedule < DASH_SCHED_ATOMIC || schedule > DASH_SCHED_SPLIT)
    return fail(DASH_ERR_INVALID_ARG, "unknown schedule");
  if (schedule == DASH_SCHED_SYMSHIFT && !causal)
    return fail(DASH_ERR_UNSUPPORTED, "symmetric shift is the causal-mask schedule; use SHIFT for a full mask");
  return DASH_OK;
}

// everything about a backward call that can be checked without the device
int check_bwd(const void* q, const void* k, const void* v, const void* o, const void* dO, const float* lse,
              const void* dq, const void* dk, const void* dv, int B, int H, int N, int d, int causal,
              int schedule, float scale) {
  int rc = check_shape(B, H, N, d);
  if (rc) return rc;
  if ((rc = check_schedule(schedule, causal))) return rc;
  if ((schedule == DASH_SCHED_PARTIALS || schedule == DASH_SCHED_SPLIT) && d > 128)
    return fail(DASH_ERR_UNSUPPORTED, "the partials and split comparison variants are built for d = 64 and 128");
  if ((size_t)B * H * N == 0) return DASH_OK;
  if (!q || !k || !v || !o || !dO || !lse || !dq || !dk || !dv)
    return fail(DASH_ERR_INVALID_ARG, "null tensor pointer");
  if (!(scale > 0.f) || !std::isfinite(scale)) return fail(DASH_ERR_INVALID_ARG, "scale must be finite and > 0");
  return DASH_OK;
}

int occupancy(const DeviceInfo& di, int d) { return d == 64 ? di.occ64 : d == 128 ? di.occ128 : di.occ256; }

// XCD-local placement (every chain of a head on one XCD, see place_on_xcds)
// serves the ordered schedules when the chains that must run at once fit the
// workgroups one XCD keeps resident.  AUTO takes it when every XCD gets at
// least one head (otherwise one queue spreads a few heads over all XCDs), a
// Shift head has at most 8 groups, and
// a caller's workgroup cap leaves every XCD those chains -- except that a cap
// never changes the summation order: where the placement decides Shift's
// groups, a cap too small for XCD placement is rejected instead.
int choose_placement(const DeviceInfo& di, int sched, int causal, int N, int d, long heads, int want, bool* xcd) {
  *xcd = false;
  if (want != DASH_PLACEMENT_XCD) return DASH_OK;
  // Automatic placement is global: with the accumulator read and written
  // device-coherently under both placements, XCD-local placement measured
  // within 2% of global at d = 64 and 128 under both masks (either way), and
  // it caps a Shift group at the chains one XCD keeps resident.
  const bool ordered = sched == DASH_SCHED_NAIVE || sched == DASH_SCHED_DESCENDING || sched == DASH_SCHED_SHIFT ||
                       sched == DASH_SCHED_SYMSHIFT;
  dash::Geom Gx = dash::make_geom(sched, causal, N, d, heads);
  dash::place_on_xcds(Gx);
  const long per_xcd = di.nxcd > 0 ? (long)occupancy(di, d) * di.cus / di.nxcd : 0;
  const long together = sched == DASH_SCHED_SHIFT ? Gx.grp : sched == DASH_SCHED_SYMSHIFT ? Gx.chains : 1;
  if (!(di.nxcd > 0 && ordered && together <= per_xcd))
    return fail(DASH_ERR_UNSUPPORTED, "XCD-local placement needs an ordered schedule and the co-running chains "
                                      "within one XCD's resident workgroups");
  *xcd = true;
  return DASH_OK;
}

// DASH_TICKETS_AUTO's ticket order.  Chain-major while a head has fewer
// chains than resident workgroups: head-major would put all of a head's
// chains on the GPU at once, and with naive / Descending every one of them
// waits out the whole pipeline fill of the head (chain j's first turn comes j
// steps late); chain-major keeps few chains per head in flight and starts the
// longest first.  The variants without ordering waits only gain the
// longest-first balance, so they go chain-major under a causal mask only.
// Once one head's chains fill the GPU, head-major keeps the resident
// workgroups on one head's Q / dO and wins.  (Measured over d = 64 / 128 /
// 256 and both masks.)  Under XCD-local placement an XCD's queue holds several
// heads whose chains outnumber its resident workgroups: chain-major keeps the
// naive pipeline fill short there as well, and for Descending except with a
// causal mask at d = 128, where its chains all start at the last Q tile and
// head-major measured better.  Shift and Symmetric Shift are head-major.
bool auto_chain_major(int sched, int causal, int d, long chains, long resident, bool xcd) {
  if (sched == DASH_SCHED_SHIFT || sched == DASH_SCHED_SYMSHIFT) return false;
  const bool waits = sched == DASH_SCHED_NAIVE || sched == DASH_SCHED_DESCENDING;
  if (xcd) return sched == DASH_SCHED_NAIVE || (sched == DASH_SCHED_DESCENDING && (!causal || d < 128));
  return chains < resident && (waits || causal);
}

// ---- the DAG model (Section 3.1) and DASH_SCHED_AUTO

// Measured time of one block step of `sched` at (d, mask) for `heads` heads of
// length N, interpolated log-linearly between the calibrated shapes (first in
// the number of heads at the two calibrated lengths around N, then in N) and
// held constant beyond them; < 0 when nothing was calibrated at (d, mask).
double step_us_at(int d, int causal, int sched, int n, long heads) {
  double h0 = -1, u0 = 0, h1 = -1, u1 = 0;  // nearest calibrated head counts below / above
  for (const dash::StepCost& e : dash::kStepCosts) {
    if (e.d != d || e.causal != causal || e.sched != sched || e.n != n) continue;
    if (e.heads <= heads && (h0 < 0 || e.heads > h0)) h0 = e.heads, u0 = e.us;
    if (e.heads >= heads && (h1 < 0 || e.heads < h1)) h1 = e.heads, u1 = e.us;
  }
  if (h0 < 0) return u1;
  if (h1 < 0 || h1 == h0) return u0;
  const double f = std::log2((double)heads / h0) / std::log2(h1 / h0);
  return u0 + f * (u1 - u0);
}

double step_us(int d, int causal, int sched, int N, long heads) {
  double n0 = -1, n1 = -1;  // nearest calibrated lengths at or below / at or above N
  for (const dash::StepCost& e : dash::kStepCosts) {
    if (e.d != d || e.causal != causal || e.sched != sched || e.n <= 0) continue;
    if (e.n <= N && (n0 < 0 || e.n > n0)) n0 = e.n;
    if (e.n >= N && (n1 < 0 || e.n < n1)) n1 = e.n;
  }
  if (n0 < 0 && n1 < 0) return -1.0;
  if (n0 < 0) return step_us_at(d, causal, sched, (int)n1, heads);
  if (n1 < 0 || n1 == n0) return step_us_at(d, causal, sched, (int)n0, heads);
  const double u0 = step_us_at(d, causal, sched, (int)n0, heads), u1 = step_us_at(d, causal, sched, (int)n1, heads);
  const double f = std::log2((double)N / n0) / std::log2(n1 / n0);
  return u0 + f * (u1 - u0);
}

// Makespan of B*H heads on `workers` workgroups with compute c and reduction
// r per block step.  With `head_cap` > 0 and more than 2 * head_cap heads,
// head_cap and 2 * head_cap heads are simulated and the makespan is
// extrapolated linearly in the number of heads: once the workgroups are
// full, every further head adds the same time, while the pipeline fill and
// the last partial round are paid once (scaling one simulation by
// B*H / head_cap would charge those once per head_cap heads).  Where the
// fill shrinks as heads are added (chain-major tickets spread it over more
// heads), the line can fall below what the steps alone need: the result is
// kept at or above that bound, every workgroup busy from start to end (and
// no less than the longest chain).  Returns < 0 if the model deadlocks.
double model_makespan(int sched, int B, int H, int N, int d, int causal, long workers, int tickets, double c,
                      double r, long head_cap) {
  dash::Geom G = dash::make_geom(sched, causal, N, d, (long)B * H);
  G.chain_major = tickets != DASH_TICKETS_AUTO ? tickets == DASH_TICKETS_CHAIN_MAJOR
                                               : auto_chain_major(sched, causal, d, G.chains, workers, false);
  const dash::HeadDag hd = dash::build_head_dag(G, N);
  const long heads = (long)B * H;
  if (head_cap <= 0 || heads <= 2 * head_cap) return dash::simulate_dag(G, hd, (int)heads, (int)workers, c, r);
  const double m1 = dash::simulate_dag(G, hd, (int)head_cap, (int)workers, c, r);
  const double m2 = dash::simulate_dag(G, hd, (int)(2 * head_cap), (int)workers, c, r);
  if (m1 < 0 || m2 < 0) return -1.0;
  const double line = m2 + (m2 - m1) * (double)(heads - 2 * head_cap) / (double)head_cap;
  int longest = 0;
  for (int w = 0; w < G.chains; ++w) longest = std::max(longest, hd.off[w + 1] - hd.off[w]);
  const double bound = std::max((double)hd.off[G.chains] * (double)heads * (c + r) / (double)workers,
                                (double)longest * (c + r));
  return std::max(line, bound);
}

// Head cap of DASH_SCHED_AUTO's simulations: enough heads to fill the
// workgroups three times (and twice that for the extrapolation).
long model_head_cap(long chains, long resident) {
  const long cap = (3 * resident + chains - 1) / chains;
  return cap > 0 ? cap : 1;
}

// DASH_SCHED_AUTO: the deterministic schedule with the shortest makespan the
// calibrated model predicts for this shape (ties: the mask's default, Shift /
// Descending).  Candidates the device cannot run (a Shift group or a head's
// Symmetric Shift chains beyond the resident workgroups) are left out.  A
// shape is simulated once per process while the cache holds it (up to
// kAutoCacheShapes shapes; then it starts over, which only costs the
// simulations again: the pick is a pure function of the shape and the
// device); a call with many heads is simulated at enough heads to fill the
// workgroups three and six times and extrapolated (model_makespan).
constexpr size_t kAutoCacheShapes = 4096;
std::mutex g_auto_mu;
std::map<std::tuple<int, int, int, int, int, long>, std::pair<int, double>> g_auto;

int auto_pick(int B, int H, int N, int d, int causal, long resident, int* sched, double* ms) {
  const auto key = std::make_tuple(B, H, N, d, causal, resident);
  {
    std::lock_guard<std::mutex> lk(g_auto_mu);
    auto it = g_auto.find(key);
    if (it != g_auto.end()) {
      *sched = it->second.first;
      if (ms) *ms = it->second.second;
      return DASH_OK;
    }
  }
  const int cand[3] = {causal ? DASH_SCHED_DESCENDING : DASH_SCHED_SHIFT, DASH_SCHED_NAIVE,
                       causal ? DASH_SCHED_SYMSHIFT : DASH_SCHED_DESCENDING};
  int best = cand[0];
  double best_us = -1.0;
  if ((long)B * H * N > 0 && resident > 0) {
    for (int s : cand) {
      const dash::Geom G = dash::make_geom(s, causal, N, d, (long)B * H);
      const long together = s == DASH_SCHED_SHIFT ? G.grp : s == DASH_SCHED_SYMSHIFT ? G.chains : 1;
      if (together > resident) continue;
      const double us = step_us(d, causal, s, N, (long)B * H);
      if (us <= 0) continue;
      const long cap = model_head_cap(G.chains, resident);
      const double m = model_makespan(s, B, H, N, d, causal, resident, DASH_TICKETS_AUTO,
                                      dash::kModelComputeShare * us, (1.0 - dash::kModelComputeShare) * us,
                                      cap);
      if (m < 0) continue;
      if (best_us < 0 || m < best_us * (1.0 - 1e-9)) best = s, best_us = m;
    }
  }
  const double best_ms = best_us < 0 ? -1.0 : best_us * 1e-3;
  std::lock_guard<std::mutex> lk(g_auto_mu);
  if (g_auto.size() >= kAutoCacheShapes) g_auto.clear();
  g_auto[key] = {best, best_ms};
  *sched = best;
  if (ms) *ms = best_ms;
  return DASH_OK;
}

// The workspace of the non-_ex backward, one per device (grown on demand,
// freed by dash_release_workspace): a call uses the current device's.
struct CachedWorkspace {
  void* p = nullptr;
  size_t bytes = 0;
};
CachedWorkspace g_ws[64];
std::mutex g_ws_mu;

}  // namespace

extern "C" {

const char* dash_last_error(void) { return g_err.c_str(); }

int dash_resolve_schedule(int schedule, int d, int causal) { return resolve(schedule, d, causal); }

size_t dash_bwd_workspace_size(int B, int H, int N, int d, int schedule) {
  if (check_shape(B, H, N, d) != DASH_OK) return 0;
  if (schedule < DASH_SCHED_ATOMIC || schedule > DASH_SCHED_SPLIT) return 0;
  return layout(B, H, N, d, resolve(schedule, d, 0)).total;
}

int dash_attn_fwd_ex(const void* q, const void* k, const void* v, void* o, float* lse, int B, int H, int N,
                     int d, int causal, float scale, void* stream) {
  int rc = check_shape(B, H, N, d);
  if (scale == 0.f) scale = 1.0f / std::sqrt((float)d);
  if (rc) return rc;
  if ((size_t)B * H * N == 0) return DASH_OK;
  if (!q || !k || !v || !o || !lse) return fail(DASH_ERR_INVALID_ARG, "null tensor pointer");
  if (!(scale > 0.f) || !std::isfinite(scale)) return fail(DASH_ERR_INVALID_ARG, "scale must be finite and > 0");
  DeviceInfo di;
  if ((rc = device_info(&di))) return rc;
  dash::FwdArgs a{q, k, v, o, lse, B * H, N, causal ? 1 : 0, scale};
  hipError_t e = dash::launch_attn_fwd(a, d, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "forward launch");
  return DASH_OK;
}

int dash_attn_fwd(const void* q, const void* k, const void* v, void* o, float* lse, int B, int H, int N, int d,
                  int causal) {
  if (d != 64 && d != 128 && d != 256) return fail(DASH_ERR_INVALID_ARG, "head dim d must be 64, 128 or 256");
  return dash_attn_fwd_ex(q, k, v, o, lse, B, H, N, d, causal, 1.0f / std::sqrt((float)d), nullptr);
}

}  // extern "C"

namespace {

int clear_flags(int* flag, int* status, void* stream) {
  if (!flag && !status) return DASH_OK;
  hipLaunchKernelGGL(clear_flags_kernel, dim3(1), dim3(64), 0, (hipStream_t)stream, flag, status);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? DASH_OK : hip_fail(e, "flag reset launch");
}

// The backward on `workspace` (dash_attn_bwd_ex's contract); `status`, if
// non-null, is a device int that bwd_pre zeroes and a wait timeout sets.
int bwd_launch(const void* q, const void* k, const void* v, const void* o, const void* dO, const float* lse,
               void* dq, void* dk, void* dv, int B, int H, int N, int d, int causal, int schedule,
               float scale, void* workspace, size_t ws_bytes, const dash_bwd_options_t* opts, int* status,
               void* stream) {
  if (scale == 0.f && d > 0) scale = 1.0f / std::sqrt((float)d);
  int rc = check_bwd(q, k, v, o, dO, lse, dq, dk, dv, B, H, N, d, causal, schedule, scale);
  if (rc) return rc;
  if ((size_t)B * H * N == 0) {
    // nothing to compute; the workspace's error flag and `status` still read "no timeout"
    int* flag = workspace && ws_bytes >= dash::kCtrlBytes ? (int*)workspace + dash::kCtrlError : nullptr;
    return clear_flags(flag, status, stream);
  }
  const Layout L = layout(B, H, N, d, resolve(schedule, d, causal));
  if (!workspace || ws_bytes < L.total)
    return fail(DASH_ERR_INVALID_ARG, "workspace missing or smaller than dash_bwd_workspace_size()");
  if (((uintptr_t)workspace & 255) != 0) return fail(DASH_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  if (opts && opts->spin_limit < 0) return fail(DASH_ERR_INVALID_ARG, "spin_limit must be >= 0");
  if (opts && opts->max_workgroups < 0) return fail(DASH_ERR_INVALID_ARG, "max_workgroups must be >= 0");
  const int tickets = opts ? opts->ticket_order : DASH_TICKETS_AUTO;
  if (tickets < DASH_TICKETS_AUTO || tickets > DASH_TICKETS_CHAIN_MAJOR)
    return fail(DASH_ERR_INVALID_ARG, "unknown ticket_order");
  const int placement = opts ? opts->placement : DASH_PLACEMENT_AUTO;
  if (placement < DASH_PLACEMENT_AUTO || placement > DASH_PLACEMENT_XCD)
    return fail(DASH_ERR_INVALID_ARG, "unknown placement");
  DeviceInfo di;
  if ((rc = device_info(&di, placement == DASH_PLACEMENT_XCD))) return rc;
  int sched = resolve(schedule, d, causal);
  if (schedule == DASH_SCHED_AUTO &&
      (rc = auto_pick(B, H, N, d, causal, (long)occupancy(di, d) * di.cus, &sched, nullptr)))
    return rc;
  if (tickets == DASH_TICKETS_CHAIN_MAJOR && (sched == DASH_SCHED_SHIFT || sched == DASH_SCHED_SYMSHIFT))
    return fail(DASH_ERR_INVALID_ARG, "Shift and Symmetric Shift take the chains of a head together (head-major tickets)");

  dash::Geom G = dash::make_geom(sched, causal, N, d, (long)B * H);
  bool xcd = false;
  if ((rc = choose_placement(di, sched, causal, N, d, (long)B * H, placement, &xcd)))
    return rc;
  if (xcd) dash::place_on_xcds(G);
  const int nq = xcd ? di.nxcd : 1;  // ticket queues; workgroup i serves queue i % nq
  // workgroups one queue keeps resident
  const long resident = (long)occupancy(di, d) * di.cus / nq;
  G.chain_major = tickets != DASH_TICKETS_AUTO ? tickets == DASH_TICKETS_CHAIN_MAJOR
                                                : auto_chain_major(sched, causal, d, G.chains, resident, xcd);
  // Shift-type chains wait on each other in a cycle: every chain of a Shift
  // group (Symmetric Shift: of a head) must be able to run at once.  Naive and
  // Descending chains only wait on chains with lower work tickets, which the
  // in-order ticket counter has already started, so any grid size works.
  const long coresident = sched == DASH_SCHED_SHIFT ? G.grp : sched == DASH_SCHED_SYMSHIFT ? G.chains : 1;
  if (coresident > resident)
    return fail(DASH_ERR_UNSUPPORTED, "too many KV tiles per head for the resident workgroups of this GPU");
  if ((long)(G.t_r + 1) * G.nsub > dash::kMaxChainSteps || N > 32768)
    return fail(DASH_ERR_UNSUPPORTED, "sequence too long for one workgroup chain (N <= 32768)");
  // per queue: its work items (XCD queues: the heads bh % nxcd == x, padded
  // to the largest such set) and at most `resident` workgroups
  const int xcd_cap = xcd ? ((B * H + nq - 1) / nq) * G.chains : 0;
  const long items = xcd ? (long)xcd_cap : (long)B * H * G.chains;
  long cap = resident;
  if (opts && opts->max_workgroups > 0) {
    if (opts->max_workgroups < coresident * nq)
      return fail(DASH_ERR_INVALID_ARG, "max_workgroups is below the chains that must run at once");
    if (opts->max_workgroups / nq < cap) cap = opts->max_workgroups / nq;
  }
  const int grid = (int)(items < cap ? items : cap) * nq;

  char* ws = (char*)workspace;
  dash::BwdArgs a;
  a.q = q;
  a.k = k;
  a.v = v;
  a.o = o;
  a.dO = dO;
  a.lse = lse;
  a.dq = dq;
  a.dk = dk;
  a.dv = dv;
  a.dqacc = (float*)(ws + L.dqacc);
  a.dvec = (float*)(ws + L.dvec);
  a.lse2 = (float*)(ws + L.lse2);
  a.counters = (int*)(ws + L.counters);
  a.ctrl = (int*)(ws + L.ctrl);
  a.steps = (unsigned*)(ws + L.steps);
  a.step_cap = L.step_cap;
  a.order = (int*)(ws + L.order);
  a.nxcd = xcd ? di.nxcd : 0;
  a.xcd_cap = xcd_cap;
  a.witness = opts ? opts->witness : nullptr;
  a.wait_stats = opts ? opts->wait_stats : nullptr;
  a.partials = opts ? opts->partials : nullptr;
  a.dq_accum = opts ? opts->dq_accum : nullptr;
  a.bh = B * H;
  a.n = N;
  a.nblk = (N + dash::kBlockRows - 1) / dash::kBlockRows;
  a.tc = (N + G.bc - 1) / G.bc;  // real KV tiles (before Symmetric Shift's padding)
  a.scale = scale;
  a.spin_limit = (opts && opts->spin_limit > 0) ? opts->spin_limit : (1 << 24);
  a.poison = (opts && (opts->flags & DASH_FLAG_POISON_COUNTERS)) ? 1 : 0;
  a.G = G;
  const bool timed = opts && opts->event_main_begin && opts->event_main_end;
  a.ev_begin = timed ? (hipEvent_t)opts->event_main_begin : nullptr;
  a.ev_end = timed ? (hipEvent_t)opts->event_main_end : nullptr;
  a.status = status;
  hipError_t e = dash::launch_bwd(a, d, grid, (hipStream_t)stream);
  if (e == hipErrorCooperativeLaunchTooLarge)
    return fail(DASH_ERR_UNSUPPORTED, "the device cannot keep every chain of a Shift group (Symmetric Shift: of a head) "
                                      "resident at once: cooperative launch refused");
  if (e != hipSuccess) return hip_fail(e, "backward launch");
  return DASH_OK;
}

// Device address of dash_scratch on each device, looked up once per device
// (in host code the array's name is a host-side stand-in, not a device
// address).
void* g_scratch[64];

int scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(DASH_ERR_NO_DEVICE, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= 64) return fail(DASH_ERR_NO_DEVICE, "device index out of range");
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(dash_scratch));
    if (e != hipSuccess || !p) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return DASH_OK;
}

}  // namespace

extern "C" {

int dash_attn_bwd_ex(const void* q, const void* k, const void* v, const void* o, const void* dO, const float* lse,
                     void* dq, void* dk, void* dv, int B, int H, int N, int d, int causal, int schedule,
                     float scale, void* workspace, size_t ws_bytes, const dash_bwd_options_t* opts,
                     void* stream) {
  return bwd_launch(q, k, v, o, dO, lse, dq, dk, dv, B, H, N, d, causal, schedule, scale, workspace, ws_bytes, opts,
                    nullptr, stream);
}

int dash_attn_bwd_noalloc(const void* q, const void* k, const void* v, const void* o, const void* dO,
                          const float* lse, void* dq, void* dk, void* dv, int B, int H, int N, int d, int causal,
                          int schedule, float scale, int* status, void* stream) {
  int rc = check_shape(B, H, N, d);
  if (rc) return rc;
  if ((size_t)B * H * N == 0) {
    if ((rc = check_schedule(schedule, causal))) return rc;
    return clear_flags(nullptr, status, stream);
  }
  const size_t need = dash_bwd_workspace_size(B, H, N, d, schedule);
  if (need == 0) return fail(DASH_ERR_INVALID_ARG, "unknown schedule");
  if (need > kScratchBytes)
    return fail(DASH_ERR_UNSUPPORTED, "problem needs " + std::to_string(need) + " bytes of scratch, more than the " +
                                          std::to_string(kScratchBytes) + " of dash_attn_bwd_noalloc");
  void* ws = nullptr;
  rc = scratch_address(&ws);
  if (rc) return rc;
  return bwd_launch(q, k, v, o, dO, lse, dq, dk, dv, B, H, N, d, causal, schedule, scale, ws, kScratchBytes, nullptr,
                    status, stream);
}

int dash_bwd_check(void* workspace, void* stream) {
  if (!workspace) return fail(DASH_ERR_INVALID_ARG, "null workspace");
  hipError_t e = hipStreamSynchronize((hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  int flag = 0;
  e = hipMemcpy(&flag, (char*)workspace + dash::kCtrlError * sizeof(int), sizeof(int), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "reading the error flag");
  if (flag) return fail(DASH_ERR_TIMEOUT, "an ordering wait exceeded its spin limit");
  return DASH_OK;
}

int dash_attn_bwd(const void* q, const void* k, const void* v, const void* o, const void* dO, const float* lse,
                  void* dq, void* dk, void* dv, int B, int H, int N, int d, int causal, int schedule) {
  if (d != 64 && d != 128 && d != 256) return fail(DASH_ERR_INVALID_ARG, "head dim d must be 64, 128 or 256");
  const float scale = 1.0f / std::sqrt((float)d);
  int rc = check_bwd(q, k, v, o, dO, lse, dq, dk, dv, B, H, N, d, causal, schedule, scale);
  if (rc) return rc;
  if ((size_t)B * H * N == 0) return DASH_OK;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(DASH_ERR_NO_DEVICE, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= 64) return fail(DASH_ERR_NO_DEVICE, "device index out of range");
  std::lock_guard<std::mutex> lk(g_ws_mu);
  CachedWorkspace& ws = g_ws[dev];
  const size_t need = layout(B, H, N, d, resolve(schedule, d, causal)).total;
  if (ws.bytes < need) {
    if (ws.p) (void)hipFree(ws.p);
    ws.p = nullptr;
    ws.bytes = 0;
    e = hipMalloc(&ws.p, need);
    if (e != hipSuccess) return hip_fail(e, "hipMalloc(workspace)");
    ws.bytes = need;
  }
  rc = dash_attn_bwd_ex(q, k, v, o, dO, lse, dq, dk, dv, B, H, N, d, causal, schedule, scale, ws.p, ws.bytes,
                        nullptr, nullptr);
  if (rc) return rc;
  return dash_bwd_check(ws.p, nullptr);
}

int dash_auto_schedule(int B, int H, int N, int d, int causal, int workers, int* schedule, double* predicted_ms) {
  int rc = check_shape(B, H, N, d);
  if (rc) return rc;
  if (!schedule) return fail(DASH_ERR_INVALID_ARG, "schedule is NULL");
  if (workers < 0) return fail(DASH_ERR_INVALID_ARG, "workers < 0");
  long resident = workers;
  if (workers == 0) {
    DeviceInfo di;
    if ((rc = device_info(&di))) return rc;
    resident = (long)occupancy(di, d) * di.cus;
  }
  return auto_pick(B, H, N, d, causal ? 1 : 0, resident, schedule, predicted_ms);
}

int dash_model_makespan(int schedule, int B, int H, int N, int d, int causal, int workers, int ticket_order,
                        int max_heads, double c, double r, double* makespan) {
  int rc = check_shape(B, H, N, d);
  if (rc) return rc;
  if ((rc = check_schedule(schedule, causal))) return rc;
  if (schedule != DASH_SCHED_NAIVE && schedule != DASH_SCHED_DESCENDING && schedule != DASH_SCHED_SHIFT &&
      schedule != DASH_SCHED_SYMSHIFT)
    return fail(DASH_ERR_INVALID_ARG, "the model covers the ordered schedules (naive, descending, shift, symshift)");
  if (!makespan) return fail(DASH_ERR_INVALID_ARG, "makespan is NULL");
  if (workers <= 0) return fail(DASH_ERR_INVALID_ARG, "workers must be > 0");
  if (ticket_order < DASH_TICKETS_AUTO || ticket_order > DASH_TICKETS_CHAIN_MAJOR)
    return fail(DASH_ERR_INVALID_ARG, "unknown ticket_order");
  if (max_heads < 0) return fail(DASH_ERR_INVALID_ARG, "max_heads < 0");
  if (!(c >= 0) || !(r >= 0) || !std::isfinite(c) || !std::isfinite(r))
    return fail(DASH_ERR_INVALID_ARG, "c and r must be finite and >= 0");
  const int sched = resolve(schedule, d, causal);
  const double m = model_makespan(sched, B, H, N, d, causal ? 1 : 0, workers, ticket_order, c, r, max_heads);
  if (m < 0) return fail(DASH_ERR_UNSUPPORTED, "the chains that must run together exceed the workgroups: no chain finishes");
  *makespan = m;
  return DASH_OK;
}

int dash_bwd_placement(int B, int H, int N, int d, int causal, int schedule) {
  int rc = check_shape(B, H, N, d);
  if (rc) return rc;
  if ((rc = check_schedule(schedule, causal))) return rc;
  DeviceInfo di;
  if ((rc = device_info(&di))) return rc;
  bool xcd = false;
  if ((rc = choose_placement(di, resolve(schedule, d, causal), causal, N, d, (long)B * H, DASH_PLACEMENT_AUTO, &xcd)))
    return rc;
  return xcd ? DASH_PLACEMENT_XCD : DASH_PLACEMENT_GLOBAL;
}

int dash_mfma_peak(int iters, double* tflops) {
  if (!tflops) return fail(DASH_ERR_INVALID_ARG, "tflops is NULL");
  if (iters < 0) return fail(DASH_ERR_INVALID_ARG, "iters < 0");
  if (iters == 0) iters = 20000;
  DeviceInfo di;
  int rc = device_info(&di);
  if (rc) return rc;
  const int grid = 2 * di.cus;  // two workgroups (8 waves) per CU
  float* sink = nullptr;
  hipError_t e = hipMalloc(&sink, (size_t)grid * 256 * sizeof(float));
  if (e != hipSuccess) return hip_fail(e, "hipMalloc");
  hipStream_t st = nullptr;
  hipEvent_t b = nullptr, en = nullptr;
  double best = 0.0;
  if ((e = hipStreamCreate(&st)) == hipSuccess && (e = hipEventCreate(&b)) == hipSuccess &&
      (e = hipEventCreate(&en)) == hipSuccess) {
    dash::launch_mfma_peak(grid, iters / 10 + 1, sink, st);  // warm-up (clocks up)
    for (int rep = 0; rep < 3 && e == hipSuccess; ++rep) {
      (void)hipEventRecord(b, st);
      dash::launch_mfma_peak(grid, iters, sink, st);
      (void)hipEventRecord(en, st);
      if ((e = hipEventSynchronize(en)) != hipSuccess) break;
      float ms = 0.f;
      if ((e = hipEventElapsedTime(&ms, b, en)) != hipSuccess) break;
      const double t = dash::mfma_peak_flops_per_launch(grid, iters) / (ms * 1e-3) / 1e12;
      best = t > best ? t : best;
    }
    if (e == hipSuccess) e = hipGetLastError();
  }
  if (en) (void)hipEventDestroy(en);
  if (b) (void)hipEventDestroy(b);
  if (st) (void)hipStreamDestroy(st);
  (void)hipFree(sink);
  if (e != hipSuccess) return hip_fail(e, "MFMA peak measurement");
  *tflops = best;
  return DASH_OK;
}

void dash_release_workspace(void) {
  std::lock_guard<std::mutex> lk(g_ws_mu);
  int cur = -1;
  const bool restore = hipGetDevice(&cur) == hipSuccess;
  for (int dev = 0; dev < 64; ++dev) {
    CachedWorkspace& ws = g_ws[dev];
    if (!ws.p) continue;
    if (hipSetDevice(dev) == hipSuccess) (void)hipFree(ws.p);
    ws.p = nullptr;
    ws.bytes = 0;
  }
  if (restore) (void)hipSetDevice(cur);
}

int dash_schedule_table(int schedule, int heads, int N, int d, int causal, int placement, int* geometry,
                        int* chain_len, int* task_kv, int* task_q, int* rank) {
  if (heads < 1) return fail(DASH_ERR_INVALID_ARG, "heads must be >= 1");
  int rc = check_shape(1, heads, N, d);
  if (rc) return rc;
  if ((rc = check_schedule(schedule, causal))) return rc;
  if (placement != DASH_PLACEMENT_GLOBAL && placement != DASH_PLACEMENT_XCD)
    return fail(DASH_ERR_INVALID_ARG, "placement must be DASH_PLACEMENT_GLOBAL or DASH_PLACEMENT_XCD");
  const int sched = resolve(schedule, d, causal);
  dash::Geom G = dash::make_geom(sched, causal, N, d, heads);
  if (placement == DASH_PLACEMENT_XCD) dash::place_on_xcds(G);
  if (geometry) {
    geometry[0] = G.t_r;
    geometry[1] = G.t_c;
    geometry[2] = G.br;
    geometry[3] = G.chains;
    geometry[4] = G.bc;
    geometry[5] = G.grp;
  }
  const int cap = G.t_r + 1;
  for (int w = 0; w < G.chains; ++w) {
    const int len = dash::chain_len(G, w);
    if (chain_len) chain_len[w] = len;
    for (int t = 0; t < len; ++t) {
      int j, i;
      dash::task(G, w, t, &j, &i);
      if (task_kv) task_kv[(size_t)w * cap + t] = j;
      if (task_q) task_q[(size_t)w * cap + t] = i;
    }
  }
  if (rank)
    for (int i = 0; i < G.t_r; ++i)
      for (int j = 0; j < G.t_c; ++j)
        rank[(size_t)i * G.t_c + j] = dash::interacts(G, i, j) ? dash::rank_of(G, i, j) : -1;
  return DASH_OK;
}

}  // extern "C"
