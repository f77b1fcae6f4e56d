// attn_bwd.hip -- deterministic attention backward for gfx950: the kernels
// around the main kernel, the d = 128 main kernel's instantiation, and the
// launch sequence of a backward call.
//
// bwd_pre  : D = rowsum(dO o O) per query row in fp32 (Algorithm 1, the
//            preprocessing kernel); resets the ordering counters, the work
//            ticket and the error flag (and dQacc for the atomic variant).
// bwd_main : the KV-tile kernels with the ordered dQ reduction: 128-row tiles
//            (bwd_main.h; d = 128 here, d = 64 in attn_bwd_d64.hip), 256-row
//            d = 64 tiles (attn_bwd64w.hip), d = 256 (attn_bwd256.hip).
// bwd_post : atomic variant only: dQ = bf16(s * dQacc).
// bwd_sum_partials : PARTIALS variant: the fixed-order sum of the partials.
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "bwd_common.h"
#include "bwd_main.h"

namespace dash {


// ---------------------------------------------------------------- bwd_pre
template <int D>
__global__ __launch_bounds__(256) void bwd_pre_kernel(BwdArgs a, int zero_acc) {
  constexpr int TPR = D / 8;  // threads per row, 8 elements each
  const long gtid = (long)blockIdx.x * 256 + threadIdx.x;
  const long rows = (long)a.bh * a.n;
  const long row = gtid / TPR;
  const int c = (int)(gtid % TPR);
  float acc = 0.f;
  if (row < rows) {
    const __bf16* pdo = (const __bf16*)a.dO + row * D + 8 * c;
    const __bf16* po = (const __bf16*)a.o + row * D + 8 * c;
    const u32x4 x = *(const u32x4*)pdo;
    const u32x4 y = *(const u32x4*)po;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float xf = bf16_to_f32((unsigned short)(x[e >> 1] >> (16 * (e & 1))));
      const float yf = bf16_to_f32((unsigned short)(y[e >> 1] >> (16 * (e & 1))));
      acc = __builtin_fmaf(xf, yf, acc);
    }
  }
  // butterfly over the TPR lanes of a row: a+b == b+a exactly, so every lane
  // ends with the same bits and the tree is fixed
#pragma unroll
  for (int off = 1; off < TPR; off <<= 1) acc += __shfl_xor(acc, off);
  if (row < rows && c == 0) {
    a.dvec[row] = acc;
    a.lse2[row] = a.lse[row] * kLog2e;
  }

  const long nthreads = (long)gridDim.x * 256;
  const long nctr = (long)a.bh * a.nblk;
  const int init = a.poison ? kPoison : 0;
  for (long i = gtid; i < nctr; i += nthreads) a.counters[i * kCtrStride] = init;
  if (gtid == 0) {
    a.ctrl[kCtrlTicket] = 0;
    a.ctrl[kCtrlError] = 0;
    if (a.status) *a.status = 0;
  }
  if (gtid < kMaxXcd) a.ctrl[kCtrlXcdTicket + gtid] = 0;
  // every chain's step table (the same for every head): entry 0 is the number
  // of steps; entry 1 + st is step st, i.e. 64-row block pb of Q tile i with
  // KV tile j, its rank in the block's summation order and whether it is the
  // last one (see pack_step)
  {
    const Geom& G = a.G;
    const int bc = G.bc;
    const long ntab = (long)G.chains * a.step_cap;
    for (long x = gtid; x < ntab; x += nthreads) {
      const int w = (int)(x / a.step_cap), e = (int)(x % a.step_cap);
      const int len = chain_len(G, w) * G.nsub;
      if (e == 0) {
        a.steps[x] = (unsigned)len;
        continue;
      }
      const int st = e - 1;
      if (st >= len) continue;
      int j, i;
      task(G, w, st / G.nsub, &j, &i);
      const int pb = i * G.nsub + st % G.nsub;
      const int rank = rank_of(G, i, j);
      a.steps[x] = (pb * kBlockRows < a.n && j * bc < a.n) ? pack_step(pb, j, rank, rank == contributors(G, i) - 1) : kNoStep;
    }
    // work ticket -> (head, chain); XCD-local placement: one segment of
    // xcd_cap tickets per XCD
    if (a.nxcd > 0) {
      const long nitems = (long)a.nxcd * a.xcd_cap;
      for (long x = gtid; x < nitems; x += nthreads) {
        const int q = (int)(x / a.xcd_cap), t = (int)(x % a.xcd_cap);
        if (t >= xcd_heads(a.bh, a.nxcd, q) * G.chains) continue;
        int bh, w;
        ticket_chain_xcd(G, a.bh, a.nxcd, q, t, &bh, &w);
        a.order[2 * x] = bh;
        a.order[2 * x + 1] = w;
      }
    } else {
      const long nitems = (long)a.bh * G.chains;
      for (long x = gtid; x < nitems; x += nthreads) {
        int bh, w;
        ticket_chain(G, a.bh, (int)x, &bh, &w);
        a.order[2 * x] = bh;
        a.order[2 * x + 1] = w;
      }
    }
  }
  if (zero_acc) {
    const long n4 = (long)a.bh * a.n * D / 4;
    for (long i = gtid; i < n4; i += nthreads) ((f32x4*)a.dqacc)[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
}

// ---------------------------------------------------------------- bwd_post
template <int D>
__global__ __launch_bounds__(256) void bwd_post_kernel(BwdArgs a) {
  const long n8 = (long)a.bh * a.n * D / 8;
  for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < n8; i += (long)gridDim.x * 256) {
    const f32x4 x = ((const f32x4*)a.dqacc)[2 * i];
    const f32x4 y = ((const f32x4*)a.dqacc)[2 * i + 1];
    const float s = a.scale;
    u32x4 r = {pack_bf16(x[0] * s, x[1] * s), pack_bf16(x[2] * s, x[3] * s), pack_bf16(y[0] * s, y[1] * s),
               pack_bf16(y[2] * s, y[3] * s)};
    ((u32x4*)a.dq)[i] = r;
  }
}

// ---------------------------------------------------------------- bwd_sum_partials
// PARTIALS variant: dQ = bf16(s * sum_j partial_j), the partials of each
// 64-row block added in ascending KV order (the order NAIVE's counters
// enforce, so the result is bitwise NAIVE's).  Partial j of block pb of head
// bh is the register-order block at ((bh * T_c + j) * nblk + pb) * 64 * D; one
// thread per 4 floats, consecutive threads on consecutive 16-byte pieces.
template <int D>
__global__ __launch_bounds__(256) void bwd_sum_partials_kernel(BwdArgs a) {
  constexpr int BM = kBlockRows;
  constexpr int PER = BM * D / 4;  // f32x4 pieces per block
  const long total = (long)a.bh * a.nblk * PER;
  const size_t stride_j = (size_t)a.nblk * BM * D;
  for (long idx = (long)blockIdx.x * 256 + threadIdx.x; idx < total; idx += (long)gridDim.x * 256) {
    const int e4 = (int)(idx % PER);
    const long bp = idx / PER;
    const int pb = (int)(bp % a.nblk), bh = (int)(bp / a.nblk);
    // register order: 32 x 32 tile T = 2 * (d block) + (query half) of 1024
    // floats, 1 KB chunk rb of 256 floats, lane l of 4 floats
    const int T = e4 >> 8, rb = (e4 >> 6) & 3, l = e4 & 63;
    const int q = pb * BM + 32 * (T & 1) + (l & 31);
    const int col = 32 * (T >> 1) + 8 * rb + 4 * (l >> 5);
    if (q >= a.n) continue;
    const int c = contributors(a.G, pb / a.G.nsub);
    const f32x4* p = (const f32x4*)(a.dqacc + ((size_t)bh * a.tc * a.nblk + pb) * BM * D) + e4;
    f32x4 s = p[0];
    for (int j = 1; j < c; ++j) s = s + p[j * stride_j / 4];
    const float sc = a.scale;
    u32x2 t = {pack_bf16(s[0] * sc, s[1] * sc), pack_bf16(s[2] * sc, s[3] * sc)};
    *(u32x2*)((__bf16*)a.dq + ((size_t)bh * a.n + q) * D + col) = t;
    if (a.dq_accum) *(f32x4*)(a.dq_accum + ((size_t)bh * a.n + q) * D + col) = s;
  }
}

template <int D>
hipError_t launch_all(const BwdArgs& a, long pre_blocks, int grid_main, hipStream_t stream) {
  const bool atomic = a.G.sched == S_ATOMIC;
  hipLaunchKernelGGL(bwd_pre_kernel<D>, dim3((unsigned)pre_blocks), dim3(256), 0, stream, a, (int)atomic);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.ev_begin) (void)hipEventRecord(a.ev_begin, stream);
  if constexpr (D == 256)
    e = launch_main256(a, grid_main, stream);
  else if constexpr (D == 64)
    e = a.G.bc == 256 ? launch_main64w(a, grid_main, stream) : launch_main64(a, grid_main, stream);
  else
    e = launch_main<D>(a, grid_main, stream);
  if (e != hipSuccess) return e;
  if (a.ev_end) (void)hipEventRecord(a.ev_end, stream);
  if (atomic) hipLaunchKernelGGL(bwd_post_kernel<D>, dim3(1024), dim3(256), 0, stream, a);
  if constexpr (D <= 128) {
    if (a.G.sched == S_PARTIALS) hipLaunchKernelGGL(bwd_sum_partials_kernel<D>, dim3(4096), dim3(256), 0, stream, a);
    if (a.G.sched == S_SPLIT) (void)launch_dq(a, D, stream);
  }
  return hipGetLastError();
}

hipError_t launch_bwd(const BwdArgs& a, int d, int grid_main, hipStream_t stream) {
  const long rows = (long)a.bh * a.n;
  const int tpr = d / 8;
  long pre_blocks = (rows * tpr + 255) / 256;
  if (pre_blocks < 1) pre_blocks = 1;
  if (pre_blocks > 65535L * 16) pre_blocks = 65535L * 16;
  if (d == 64) return launch_all<64>(a, pre_blocks, grid_main, stream);
  if (d == 128) return launch_all<128>(a, pre_blocks, grid_main, stream);
  return launch_all<256>(a, pre_blocks, grid_main, stream);
}

int bwd_main_occupancy(int d) {
  if (d == 64) {
    const int a = main64_occupancy(), b = bwd_main64w_occupancy();
    return a < b ? a : b;
  }
  return d == 128 ? main_occupancy<128>() : bwd_main256_occupancy();
}

}  // namespace dash
