// attn_bwd.hip -- deterministic attention backward for gfx950.
//
// bwd_pre  : D = rowsum(dO o O) per query row in fp32 (Algorithm 1, the
//            preprocessing kernel); resets the ordering counters, the work
//            ticket and the error flag (and dQacc for the atomic variant).
// bwd_main : one KV tile of d rows per work item, d/32 waves; wave w owns KV
//            rows [32w, 32w+32) of the tile and keeps K, V, K^T operands and the
//            dK, dV accumulators in registers for the whole chain.  For every
//            64-row Q block of the chain (Algorithm 1, the consumer loop):
//              S = Q K^T, dP = dO V^T            (bf16 MFMA 32x32x16)
//              P = exp(S - L), dS = P o (dP - D)  (fp32)
//              dV += P^T dO, dK += dS^T Q          (P^T, dS^T fed from registers)
//              dQ^T_loc = K^T dS^T                 (dS staged through LDS)
//            then the ordered reduction (Algorithm 1, the dQ writer): wait until
//            the block's counter equals this tile's rank, add the partial into
//            the fp32 dQ accumulator with device-coherent (SC1) loads/stores, make
//            the stores visible, bump the counter.  The last rank writes bf16
//            s*dQ directly.  No atomics touch the data; the order is fixed by the
//            schedule, so results are bitwise reproducible.
//            The grid is persistent: workgroups take work items from a ticket
//            counter in order, so every item a wait depends on has been started.
// bwd_post : atomic variant only: dQ = bf16(s * dQacc).
#include "common.h"
#include "kernels.h"

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
  if (row < rows && c == 0) a.dvec[row] = acc;

  const long nthreads = (long)gridDim.x * 256;
  const long nctr = (long)a.bh * a.nblk;
  const int init = a.poison ? kPoison : 0;
  for (long i = gtid; i < nctr; i += nthreads) a.counters[i * kCtrStride] = init;
  if (gtid == 0) {
    a.ctrl[kCtrlTicket] = 0;
    a.ctrl[kCtrlError] = 0;
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

// ---------------------------------------------------------------- ordering
// Spin until *ctr == want (relaxed, device-coherent loads).  Wave-uniform.
// Returns false after `limit` polls; the caller then skips its update.
__device__ inline bool wait_turn(const int* ctr, int want, int limit) {
  for (int n = 0;; ++n) {
    const int v = __builtin_amdgcn_readfirstlane(__hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
    if (v == want) break;
    if (n >= limit) return false;
    __builtin_amdgcn_s_sleep(2);
  }
  __atomic_signal_fence(__ATOMIC_SEQ_CST);  // keep the data loads after the wait
  return true;
}

// ---------------------------------------------------------------- bwd_main
template <int D>
struct MainSmem {
  static constexpr int BM = kBlockRows;  // 64 query rows per block
  static constexpr int QP = D + 8;       // padded row of Qs / dOs
  static constexpr int SP = D + 8;       // padded row of dSs (BC = D columns)
  __bf16 qs[BM * QP];
  __bf16 dos[BM * QP];
  __bf16 qts[D * BM];   // Q^T, chunk-swizzled
  __bf16 dots[D * BM];  // dO^T, chunk-swizzled
  __bf16 dss[BM * SP];  // dS (bf16), [q][kv]
  float ls[BM];         // L * log2(e)
  float ds[BM];         // D
  int item;
};

template <int D>
__global__ __launch_bounds__(2 * D) void bwd_main_kernel(BwdArgs a) {
  constexpr int NW = D / 32;   // waves
  constexpr int NT = 64 * NW;  // threads
  constexpr int BC = D;        // KV rows per tile
  constexpr int BM = kBlockRows;
  constexpr int KS = D / 16;   // k-steps over d
  constexpr int KSC = BC / 16; // k-steps over kv
  constexpr int NB = D / 32;   // 32-column blocks of d
  constexpr int QP = MainSmem<D>::QP, SP = MainSmem<D>::SP;
  constexpr int CPR = D / 8;   // 16-byte chunks per row
  static_assert(16 * CPR == NT, "one loader unit per thread");
  __shared__ __attribute__((aligned(16))) MainSmem<D> sm;

  const Geom G = a.G;
  const int N = a.n;
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, g = l >> 5, lc = l & 31;
  const int lu_c = tid % CPR, lu_rg = tid / CPR;  // loader unit: rows 4rg..4rg+3, cols 8c..8c+7
  const float c2 = a.scale * kLog2e;
  const uint32_t hbytes = (uint32_t)((size_t)N * D * 2);
  const int total = a.bh * G.chains;
  const bool ordered = G.sched != S_ATOMIC;
  bool failed = false;  // this wave hit a wait timeout: skip further waits

  for (;;) {
    if (tid == 0) sm.item = atomicAdd(&a.ctrl[kCtrlTicket], 1);
    __syncthreads();
    const int item = sm.item;
    if (item >= total) break;
    const int bh = item / G.chains, wch = item % G.chains;
    const size_t head = (size_t)bh * N * D;
    const auto rq = make_rsrc((const __bf16*)a.q + head, hbytes);
    const auto rk = make_rsrc((const __bf16*)a.k + head, hbytes);
    const auto rv = make_rsrc((const __bf16*)a.v + head, hbytes);
    const auto rdo = make_rsrc((const __bf16*)a.dO + head, hbytes);
    const auto rdq = make_rsrc((__bf16*)a.dq + head, hbytes);
    const auto rdk = make_rsrc((__bf16*)a.dk + head, hbytes);
    const auto rdv = make_rsrc((__bf16*)a.dv + head, hbytes);
    const auto racc = make_rsrc(a.dqacc + head, hbytes * 2);
    const auto rl = make_rsrc(a.lse + (size_t)bh * N, (uint32_t)N * 4);
    const auto rD = make_rsrc(a.dvec + (size_t)bh * N, (uint32_t)N * 4);
    int* ctr_head = a.counters + (size_t)bh * a.nblk * kCtrStride;

    const int nsteps = chain_len(G, wch) * G.nsub;
    int cur_j = -1;
    bf16x8 kreg[KS], vreg[KS], ktreg[KSC];
    f32x16 dkacc[NB], dvacc[NB];

    // prefetch registers for the next Q block
    u32x4 pq[4], pdo[4];
    float pl = 0.f, pd = 0.f;
    auto step_block = [&](int st, int* j, int* i, int* pb) {
      task(G, wch, st / G.nsub, j, i);
      *pb = *i * G.nsub + st % G.nsub;
    };
    auto prefetch = [&](int pb) {
      const int q0 = pb * BM;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const uint32_t off = (uint32_t)((q0 + 4 * lu_rg + r) * D + 8 * lu_c) * 2;
        pq[r] = ld16(rq, off);
        pdo[r] = ld16(rdo, off);
      }
      if (tid < BM) {
        pl = ld4f(rl, (uint32_t)(q0 + tid) * 4);
        pd = ld4f(rD, (uint32_t)(q0 + tid) * 4);
      }
    };
    auto store_dkdv = [&](int j) {
      const int kv0 = j * BC;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int kv = kv0 + 32 * w + 8 * (r >> 2) + 4 * g + (r & 3);
          const uint32_t off = (uint32_t)(kv * D + 32 * nb + lc) * 2;
          st2(rdv, off, to_bf16(dvacc[nb][r]));
          st2(rdk, off, to_bf16(dkacc[nb][r] * a.scale));
        }
    };

    // skip leading empty blocks (Q rows past N, or KV tiles past N)
    auto valid_step = [&](int st) {
      int j, i, pb;
      step_block(st, &j, &i, &pb);
      return pb * BM < N && j * BC < N;
    };
    int st = 0;
    while (st < nsteps && !valid_step(st)) ++st;
    if (st < nsteps) {
      int j0, i0, pb0;
      step_block(st, &j0, &i0, &pb0);
      prefetch(pb0);
    }

    for (; st < nsteps;) {
      int j, i, pb;
      step_block(st, &j, &i, &pb);
      const int q0 = pb * BM;

      if (j != cur_j) {  // new KV tile: flush the previous one, load operands
        if (cur_j >= 0) store_dkdv(cur_j);
        cur_j = j;
        const int kv0 = j * BC;
        const int kvr = kv0 + 32 * w + lc;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const uint32_t off = (uint32_t)(kvr * D + 16 * ks + 8 * g) * 2;
          kreg[ks] = as_bf16x8(ld16(rk, off));
          vreg[ks] = as_bf16x8(ld16(rv, off));
        }
#pragma unroll
        for (int ks = 0; ks < KSC; ++ks) {
          unsigned short t[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) t[e] = ld2(rk, (uint32_t)((kv0 + 16 * ks + 8 * g + e) * D + 32 * w + lc) * 2);
          u32x4 pk = {t[0] | ((unsigned)t[1] << 16), t[2] | ((unsigned)t[3] << 16), t[4] | ((unsigned)t[5] << 16),
                      t[6] | ((unsigned)t[7] << 16)};
          ktreg[ks] = as_bf16x8(pk);
        }
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            dkacc[nb][r] = 0.f;
            dvacc[nb][r] = 0.f;
          }
      }

      // ---- stage the prefetched Q / dO block into LDS
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        *(u32x4*)&sm.qs[(4 * lu_rg + r) * QP + 8 * lu_c] = pq[r];
        *(u32x4*)&sm.dos[(4 * lu_rg + r) * QP + 8 * lu_c] = pdo[r];
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int d = 8 * lu_c + e;
        const int at = d * BM + 4 * (lu_rg ^ tswz(d));
        u32x2 tq = {pick16(pq[0][e >> 1], pq[1][e >> 1], e & 1), pick16(pq[2][e >> 1], pq[3][e >> 1], e & 1)};
        u32x2 to = {pick16(pdo[0][e >> 1], pdo[1][e >> 1], e & 1), pick16(pdo[2][e >> 1], pdo[3][e >> 1], e & 1)};
        *(u32x2*)&sm.qts[at] = tq;
        *(u32x2*)&sm.dots[at] = to;
      }
      if (tid < BM) {
        sm.ls[tid] = pl * kLog2e;
        sm.ds[tid] = pd;
      }
      __syncthreads();

      // ---- prefetch the next valid block while this one computes
      int nst = st + 1;
      while (nst < nsteps && !valid_step(nst)) ++nst;
      if (nst < nsteps) {
        int jn, in_, pbn;
        step_block(nst, &jn, &in_, &pbn);
        prefetch(pbn);
      }

      // ---- S = Q K^T and dP = dO V^T for this wave's 32 KV columns
      f32x16 s[2], dp[2];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          s[qb][r] = 0.f;
          dp[qb][r] = 0.f;
        }
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8 aq = *(const bf16x8*)&sm.qs[(32 * qb + lc) * QP + 16 * ks + 8 * g];
          const bf16x8 ao = *(const bf16x8*)&sm.dos[(32 * qb + lc) * QP + 16 * ks + 8 * g];
          s[qb] = mfma32(aq, kreg[ks], s[qb]);
          dp[qb] = mfma32(ao, vreg[ks], dp[qb]);
        }
      }

      // ---- P = exp(S - L), dS = P (dP - D); element (qb, r) is query
      //      q0 + 32qb + 8(r/4) + 4g + r%4, key j*BC + 32w + lc
      const int kv = j * BC + 32 * w + lc;
      const bool need_mask = (j * BC + BC > N) || (G.causal && j * BC + BC - 1 > q0);
      bf16x8 pbf[2][2], dsbf[2][2];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) {
          const int ql = 32 * qb + 8 * rb + 4 * g;
          const f32x4 L4 = *(const f32x4*)&sm.ls[ql];
          const f32x4 D4 = *(const f32x4*)&sm.ds[ql];
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const int r = 4 * rb + c;
            float p = exp2f(s[qb][r] * c2 - L4[c]);
            if (need_mask) {
              const int qg = q0 + ql + c;
              if (kv >= N || (G.causal && kv > qg)) p = 0.f;
            }
            s[qb][r] = p;
            dp[qb][r] = p * (dp[qb][r] - D4[c]);
          }
        }
        pbf[qb][0] = pack8(s[qb], 0);
        pbf[qb][1] = pack8(s[qb], 8);
        dsbf[qb][0] = pack8(dp[qb], 0);
        dsbf[qb][1] = pack8(dp[qb], 8);
      }

      // ---- dV += P^T dO, dK += dS^T Q  (A operands straight from registers)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int d = 32 * nb + lc;
        const int sw = tswz(d);
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const int qb = kk >> 1, half = kk & 1;
          const int ch = (32 * qb + 16 * half + 4 * g) >> 2;
          const int a0 = d * BM + 4 * (ch ^ sw), a1 = d * BM + 4 * ((ch + 2) ^ sw);
          const bf16x8 bo = as_bf16x8(*(const u32x2*)&sm.dots[a0], *(const u32x2*)&sm.dots[a1]);
          const bf16x8 bq = as_bf16x8(*(const u32x2*)&sm.qts[a0], *(const u32x2*)&sm.qts[a1]);
          dvacc[nb] = mfma32(pbf[qb][half], bo, dvacc[nb]);
          dkacc[nb] = mfma32(dsbf[qb][half], bq, dkacc[nb]);
        }
      }

      // ---- dS -> LDS as [q][kv] for the dQ product
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int ql = 32 * qb + 8 * (r >> 2) + 4 * g + (r & 3);
          sm.dss[ql * SP + 32 * w + lc] = (__bf16)dp[qb][r];
        }
      __syncthreads();

      // ---- dQ^T_loc (rows d in [32w, 32w+32), all 64 queries) = K^T dS^T
      f32x16 dq[2];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) dq[qb][r] = 0.f;
#pragma unroll
        for (int ks = 0; ks < KSC; ++ks) {
          const bf16x8 bs = *(const bf16x8*)&sm.dss[(32 * qb + lc) * SP + 16 * ks + 8 * g];
          dq[qb] = mfma32(ktreg[ks], bs, dq[qb]);
        }
      }
      // dq[qb][r] <-> query q0 + 32qb + lc, column d = 32w + 8(r/4) + 4g + r%4

      if (a.partials) {
        const auto rp = make_rsrc(a.partials + ((size_t)bh * a.tc + j) * N * D, hbytes * 2);
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
#pragma unroll
          for (int rb = 0; rb < 4; ++rb) {
            const u32x4 v = __builtin_bit_cast(u32x4, f32x4{dq[qb][4 * rb], dq[qb][4 * rb + 1], dq[qb][4 * rb + 2],
                                                            dq[qb][4 * rb + 3]});
            st16(rp, (uint32_t)((q0 + 32 * qb + lc) * D + 32 * w + 8 * rb + 4 * g) * 4, v);
          }
      }

      if (!ordered) {
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
          const int q = q0 + 32 * qb + lc;
          if (q < N) {
            float* dst = a.dqacc + head + (size_t)q * D + 32 * w + 4 * g;
#pragma unroll
            for (int r = 0; r < 16; ++r) atomicAdd(dst + 8 * (r >> 2) + (r & 3), dq[qb][r]);
          }
        }
        __syncthreads();  // LDS reuse by the next block
      } else {
        // ---- ordered reduction into the fp32 accumulator
        const int rank = rank_of(G, i, j);
        const bool last = rank == contributors(G, i) - 1;
        int* ctr = ctr_head + (size_t)pb * kCtrStride;
        const bool turn = !failed && wait_turn(ctr, rank, a.spin_limit);
        if (!turn && !failed) {
          failed = true;
          __hip_atomic_store(&a.ctrl[kCtrlError], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        if (turn) {
#pragma unroll
          for (int qb = 0; qb < 2; ++qb) {
            const int q = q0 + 32 * qb + lc;
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) {
              const uint32_t off = (uint32_t)(q * D + 32 * w + 8 * rb + 4 * g);
              f32x4 v = {dq[qb][4 * rb], dq[qb][4 * rb + 1], dq[qb][4 * rb + 2], dq[qb][4 * rb + 3]};
              if (rank > 0) {
                const f32x4 old = __builtin_bit_cast(f32x4, ld16_coherent(racc, off * 4));
                v = old + v;
              }
              if (last) {
                u32x2 t = {pack_bf16(v[0] * a.scale, v[1] * a.scale), pack_bf16(v[2] * a.scale, v[3] * a.scale)};
                st8(rdq, off * 2, t);
                if (a.dq_accum) st16(make_rsrc(a.dq_accum + head, hbytes * 2), off * 4, __builtin_bit_cast(u32x4, v));
              } else {
                st16_coherent(racc, off * 4, __builtin_bit_cast(u32x4, v));
              }
            }
          }
        }
        // every wave's stores complete before the counter moves on
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (tid == 0) {
          if (a.witness && rank < a.tc) a.witness[((size_t)bh * a.nblk + pb) * a.tc + rank] = j;
          __hip_atomic_store(ctr, rank + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
      st = nst;
    }
    if (cur_j >= 0) store_dkdv(cur_j);
    __syncthreads();  // sm.item is rewritten by the next ticket
  }
}

hipError_t launch_bwd(const BwdArgs& a, int d, int grid_main, hipStream_t stream) {
  const bool atomic = a.G.sched == S_ATOMIC;
  const long rows = (long)a.bh * a.n;
  const int tpr = d / 8;
  long pre_blocks = (rows * tpr + 255) / 256;
  if (pre_blocks < 1) pre_blocks = 1;
  if (pre_blocks > 65535L * 16) pre_blocks = 65535L * 16;
  if (d == 64) {
    hipLaunchKernelGGL(bwd_pre_kernel<64>, dim3((unsigned)pre_blocks), dim3(256), 0, stream, a, (int)atomic);
    if (a.ev_begin) (void)hipEventRecord(a.ev_begin, stream);
    hipLaunchKernelGGL(bwd_main_kernel<64>, dim3(grid_main), dim3(128), 0, stream, a);
    if (a.ev_end) (void)hipEventRecord(a.ev_end, stream);
    if (atomic) hipLaunchKernelGGL(bwd_post_kernel<64>, dim3(1024), dim3(256), 0, stream, a);
  } else {
    hipLaunchKernelGGL(bwd_pre_kernel<128>, dim3((unsigned)pre_blocks), dim3(256), 0, stream, a, (int)atomic);
    if (a.ev_begin) (void)hipEventRecord(a.ev_begin, stream);
    hipLaunchKernelGGL(bwd_main_kernel<128>, dim3(grid_main), dim3(256), 0, stream, a);
    if (a.ev_end) (void)hipEventRecord(a.ev_end, stream);
    if (atomic) hipLaunchKernelGGL(bwd_post_kernel<128>, dim3(1024), dim3(256), 0, stream, a);
  }
  return hipGetLastError();
}

int bwd_main_occupancy(int d) {
  int blocks = 0;
  hipError_t e = d == 64
                     ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, bwd_main_kernel<64>, 128, 0)
                     : hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, bwd_main_kernel<128>, 256, 0);
  return e == hipSuccess ? blocks : 0;
}

}  // namespace dash
