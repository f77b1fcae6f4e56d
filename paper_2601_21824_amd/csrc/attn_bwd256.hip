// attn_bwd256.hip -- the backward main kernel for head dim 256.
//
// Same method as bwd_main_kernel (Algorithm 1: each KV-tile workgroup keeps
// dK_j, dV_j on chip; the dQ partials of a 64-row Q block are added into an
// fp32 accumulator in the schedule's fixed order, one counter per block), with
// a tiling sized for d = 256: at 32 KV rows per wave the fp32 dK/dV
// accumulators alone would fill the register file, so a KV tile has 64 rows,
// each of the 4 waves owns 16 of them and the contractions run on bf16 MFMA
// 16x16x32.  Per wave, for every 64-row Q block of its chain:
//   S = Q K^T, dP = dO V^T      16 x 64 per wave: A = Q / dO rows (LDS),
//                               B = K / V rows of the wave's keys (registers)
//   P = exp(S - L), dS = P o (dP - D)
//   dV += P^T dO, dK += dS^T Q  A = P^T, dS^T from registers, B = dO, Q by
//                               transposed LDS reads
//   dQ^T_loc = K^T dS^T         the wave's 64 columns of d, all 64 queries;
//                               A = K^T (registers), B = dS^T (LDS)
// then the ordered add into its 64-column slice of the block's accumulator.
// The Q / dO block is single-buffered (a 64 x 256 bf16 pair is 64 KB, and the
// accumulator slice landing pad another 64 KB): the next block is fetched
// while dQ^T runs.
//
// v_mfma_f32_16x16x32_bf16 operand layout (checked on the device): A lane l
// holds row l%16, k = 8(l/16) .. +7; B lane l holds column l%16, the same k;
// C lane l holds column l%16, rows 4(l/16) .. +3.
#include "common.h"
#include "kernels.h"
#include "bwd_common.h"
#include "lds_layout.h"

namespace dash {
namespace {

constexpr int D = 256;
constexpr int BC = 64;            // KV rows per tile
constexpr int BM = kBlockRows;    // Q rows per block
constexpr int NW = 4, NT = 256;   // waves, threads
constexpr int KS = D / 32;        // k-steps of 32 over d (S, dP)
constexpr int NDB = D / 16;       // 16-column blocks of d (dV, dK)
constexpr int CPR = D / 8;        // 16-byte chunks per bf16 row
constexpr int QLD = BM * CPR / NT;  // direct loads per thread for a Q (or dO) block
static_assert(QLD == 8, "tile shape");

__device__ inline f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// LDS layouts of the Q / dO blocks and the dS^T tile: lds_layout.h.

struct Smem256 {
  __bf16 qs[BM * D];     // Q block [q][d]
  __bf16 dos[BM * D];    // dO block [q][d]
  __bf16 dst[BC * BM];   // dS^T [kv][q]
  float acc[BM * D];     // accumulator slices as they arrive (wave w: 4096 floats at 4096 w)
  float ls[BM];          // L * log2(e) per query row
  float ds[BM];          // D per query row
  unsigned steps[kMaxChainSteps];
  int item;
};

template <bool CAUSAL, bool ORDERED, bool XCD, bool STATS = false>
__global__ __launch_bounds__(NT) void bwd_main256_kernel(BwdArgs a) {
  __shared__ __attribute__((aligned(16))) Smem256 sm;

  const Geom G = a.G;
  const int N = a.n;
  const int tid = threadIdx.x, l = tid & 63, gq = l >> 4, lr = l & 15;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const float c2 = a.scale * kLog2e;
  const uint32_t hbytes = (uint32_t)((size_t)N * D * 2);
  constexpr bool ordered = ORDERED;  // false: the atomic variant
  // XCD-local placement (ordered only): the heads of this XCD from its own
  // ticket queue; the accumulator stays device-coherent (SC1) as under global
  // placement, since an SC0 read may hit a stale line in this CU's L1
  constexpr bool xcd = XCD;
  const int xq = xcd ? xcc_id() : 0;
  const int total = xcd ? (xq < a.nxcd ? xcd_heads(a.bh, a.nxcd, xq) * G.chains : 0) : a.bh * G.chains;
  int* const ticket = &a.ctrl[xcd ? kCtrlXcdTicket + xq : kCtrlTicket];
  const int* const order = a.order + (xcd ? 2 * xq * a.xcd_cap : 0);
  // Shift-type orders are conflict-free: the next contributor to a block comes
  // at least one step later, so the counter release can wait until the next
  // step's dV/dK work has covered the store latency.
  const bool deferred = G.sched == S_SHIFT || G.sched == S_SYMSHIFT;
  bool failed = false;
  WaitStats wst;
  if constexpr (STATS) stats_wave_begin(wst);

  for (;;) {
    if (tid == 0) sm.item = atomicAdd(ticket, 1);
    __syncthreads();
    const int item = __builtin_amdgcn_readfirstlane(sm.item);  // wave-uniform (SGPR)
    if (item >= total) break;
    // (head, chain) of the ticket from bwd_pre's table; wave-uniform, so the
    // head's buffer descriptors stay in SGPRs
    const int bh = __builtin_amdgcn_readfirstlane(order[2 * item]);
    const int wch = __builtin_amdgcn_readfirstlane(order[2 * item + 1]);
    const size_t head = (size_t)bh * N * D;
    const auto rq = make_rsrc((const __bf16*)a.q + head, hbytes);
    const auto rk = make_rsrc((const __bf16*)a.k + head, hbytes);
    const auto rv = make_rsrc((const __bf16*)a.v + head, hbytes);
    const auto rdo = make_rsrc((const __bf16*)a.dO + head, hbytes);
    const auto racc = make_rsrc(a.dqacc + (size_t)bh * a.nblk * BM * D, (uint32_t)a.nblk * BM * D * 4);
    int* ctr_head = a.counters + (size_t)bh * a.nblk * kCtrStride;

    const unsigned* tab = a.steps + (size_t)wch * a.step_cap;
    const int nsteps = __builtin_amdgcn_readfirstlane((int)tab[0]);
    // the chain's schedule (computed by bwd_pre) into LDS
    for (int st = tid; st < nsteps; st += NT) sm.steps[st] = tab[1 + st];
    __syncthreads();

    int cur_j = -1;
    bf16x8 kreg[KS], vreg[KS];  // K, V rows of this wave's 16 keys (B of S, dP)
    bf16x8 ktreg[4][2];         // K^T of this wave's 64 columns of d (A of dQ^T), [d block][kv step]
    f32x4 dkacc[NDB], dvacc[NDB];
    int pend_ctr = -1, poll_v = -1;
    bool top_wait = true;

    auto step_at = [&](int st) -> unsigned { return __builtin_amdgcn_readfirstlane(sm.steps[st]); };
    auto next_valid = [&](int st) {
      while (st < nsteps && step_at(st) == kNoStep) ++st;
      return st;
    };
    auto load_block = [&](int pb) {  // Q, dO, L, D of block pb into LDS (vmcnt)
      // the thread index is recomputed here rather than kept live (the eight
      // per-part offsets would otherwise be hoisted out of the step loop)
      unsigned lane;
      asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(lane));
      const int t0 = 64 * w + (int)lane;
#pragma unroll
      for (int k = 0; k < QLD; ++k) {
        const int slot = k * NT + t0, r = slot / CPR, c = (slot % CPR) ^ q256_swz(r);
        const uint32_t off = (uint32_t)((pb * BM + r) * D + 8 * c) * 2;
        lds_load16(rq, &sm.qs[(k * NT + 64 * w) * 8], off);
        lds_load16(rdo, &sm.dos[(k * NT + 64 * w) * 8], off);
      }
      if (w == 0) lds_load4(make_rsrc(a.lse2 + (size_t)bh * N, (uint32_t)N * 4), &sm.ls[0], (uint32_t)(pb * BM + (int)lane) * 4);
      if (w == 1) lds_load4(make_rsrc(a.dvec + (size_t)bh * N, (uint32_t)N * 4), &sm.ds[0], (uint32_t)(pb * BM + (int)lane) * 4);
    };
    // The ordered variants keep dQacc in register order: block pb is BM*D
    // floats at pb*BM*D; wave w's slice (columns [64w, 64w+64)) is the 4096
    // floats at 4096 w; tile t = 4 db + qb of lane l at 256 t + 4 l holds
    // query 16 qb + l%16, columns 64w + 16db + 4(l/16) .. +3.
    float* acc_w = &sm.acc[w * 4096];
    auto acc_off = [&](int pb, int t) { return (uint32_t)(pb * BM * D + w * 4096 + t * 256 + 4 * l) * 4; };
    auto load_acc = [&](int pb) {
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        lds_load16_coherent(racc, &acc_w[t * 256], acc_off(pb, t));
      }
    };
    auto store_dkdv = [&](int j) {
      const auto rdk = make_rsrc((__bf16*)a.dk + head, hbytes);
      const auto rdv = make_rsrc((__bf16*)a.dv + head, hbytes);
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int kv = j * BC + 16 * w + 4 * gq + r;
          const uint32_t off = (uint32_t)(kv * D + 16 * db + lr) * 2;
          st2(rdv, off, to_bf16(dvacc[db][r]));
          st2(rdk, off, to_bf16(dkacc[db][r] * a.scale));
        }
    };
    auto release = [&]() {
      if (l == 0 && pend_ctr >= 0)
        __hip_atomic_fetch_add(ctr_head + (size_t)pend_ctr * kCtrStride, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      pend_ctr = -1;
    };

    int st = next_valid(0);
    if (st < nsteps) {
      const int pb0 = step_at(st) & 0xfff;
      load_block(pb0);
      if (ordered) poll_v = __hip_atomic_load(ctr_head + (size_t)pb0 * kCtrStride, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }

    for (; st < nsteps;) {
      const unsigned e = step_at(st);
      const int pb = e & 0xfff, j = (e >> 12) & 0x1ff, rank = (e >> 21) & 0x3ff;
      const bool last = (e >> 31) != 0;
      const int q0 = pb * BM;

      if (j != cur_j) {  // new KV tile: flush the previous one, load its operands
        if (cur_j >= 0) store_dkdv(cur_j);
        cur_j = j;
        const int kvr = j * BC + 16 * w + lr;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          kreg[ks] = as_bf16x8(ld16(rk, (uint32_t)(kvr * D + 32 * ks + 8 * gq) * 2));
          vreg[ks] = as_bf16x8(ld16(rv, (uint32_t)(kvr * D + 32 * ks + 8 * gq) * 2));
        }
        // K^T: lane holds column d = 64w + 16db + l%16 over keys 32kk + 8(l/16) .. +7
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
          for (int kk = 0; kk < 2; ++kk) {
            unsigned short t[8];
#pragma unroll
            for (int x = 0; x < 8; ++x)
              t[x] = ld2(rk, (uint32_t)((j * BC + 32 * kk + 8 * gq + x) * D + 64 * w + 16 * db + lr) * 2);
            ktreg[db][kk] = as_bf16x8(u32x4{t[0] | ((unsigned)t[1] << 16), t[2] | ((unsigned)t[3] << 16),
                                            t[4] | ((unsigned)t[5] << 16), t[6] | ((unsigned)t[7] << 16)});
          }
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          dkacc[db] = f32x4{0.f, 0.f, 0.f, 0.f};
          dvacc[db] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
      }

      // ---- this block's Q / dO / L / D are in LDS (each wave waited for its own
      //      loads at the end of the previous step, or here for the first one)
      if (top_wait) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      top_wait = false;
      __syncthreads();

      const int nst = next_valid(st + 1);
      const int pb_next = nst < nsteps ? (int)(step_at(nst) & 0xfff) : -1;
      // the chain moves to another KV tile after this step (Symmetric Shift,
      // between its two tiles)
      const bool tile_ends = nst < nsteps && (int)((step_at(nst) >> 12) & 0x1ff) != j;
      int* ctr = ctr_head + (size_t)pb * kCtrStride;
      bool have_turn = false;

      // ---- S = Q K^T, dP = dO V^T: 4 query blocks of 16 x this wave's 16 keys;
      //      k-step ks reads the 8 row operands of step ks + 1 first
      f32x4 s[4], dp[4];
#pragma unroll
      for (int qb = 0; qb < 4; ++qb) {
        s[qb] = f32x4{0.f, 0.f, 0.f, 0.f};
        dp[qb] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
      {
        auto rd = [&](int ks, bf16x8* op) {
#pragma unroll
          for (int qb = 0; qb < 4; ++qb) {
            const int at = q256_at(16 * qb + lr, 32 * ks + 8 * gq);
            op[qb] = *(const bf16x8*)&sm.qs[at];
            op[4 + qb] = *(const bf16x8*)&sm.dos[at];
          }
        };
        bf16x8 ring[2][8];
        rd(0, ring[0]);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          if (ks + 1 < KS) rd(ks + 1, ring[(ks + 1) & 1]);
          __builtin_amdgcn_sched_barrier(0);
          const bf16x8* op = ring[ks & 1];
#pragma unroll
          for (int qb = 0; qb < 4; ++qb) {
            s[qb] = mfma16(op[qb], kreg[ks], s[qb]);
            dp[qb] = mfma16(op[4 + qb], vreg[ks], dp[qb]);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }

      // ---- ordering: the counter was loaded at the end of the previous step;
      //      if the turn is ours, fetch the accumulator slice now
      if (ordered && !failed) {
        const int v0 = __builtin_amdgcn_readfirstlane(poll_v);
        if (v0 >= NW * rank) {
          have_turn = true;
          __atomic_signal_fence(__ATOMIC_SEQ_CST);
          if (rank > 0) load_acc(pb);
        }
      }

      // ---- P = exp(S - L), dS = P (dP - D).  Element (qb, r) is query
      //      16qb + 4(l/16) + r of the block and key 16w + l%16 of the tile.
      //      Keys past N need no mask: their K, V rows read as zero, P is at
      //      most 1 there (exp2_unit) and their dK, dV rows are not stored.
      const int kvl = 16 * w + lr;
      const int thr = j * BC + kvl - q0 - 4 * gq;  // causal: masked iff 16qb + r < thr
#pragma unroll
      for (int qb = 0; qb < 4; ++qb) {
        const f32x4 L4 = *(const f32x4*)&sm.ls[16 * qb + 4 * gq];
        const f32x4 D4 = *(const f32x4*)&sm.ds[16 * qb + 4 * gq];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float p = exp2_unit(__builtin_fmaf(s[qb][r], c2, -L4[r]));
          if (CAUSAL) p = (16 * qb + r < thr) ? 0.f : p;
          s[qb][r] = p;
          dp[qb][r] = p * (dp[qb][r] - D4[r]);
        }
      }
      // A operands of dV / dK (k = query): k-step kq covers queries
      // 32kq + 16(x/4) + 4(l/16) + x%4, x = 0..7
      bf16x8 pbf[2], dsbf[2];
#pragma unroll
      for (int kq = 0; kq < 2; ++kq) {
        pbf[kq] = as_bf16x8(u32x4{pack_bf16(s[2 * kq][0], s[2 * kq][1]), pack_bf16(s[2 * kq][2], s[2 * kq][3]),
                                  pack_bf16(s[2 * kq + 1][0], s[2 * kq + 1][1]), pack_bf16(s[2 * kq + 1][2], s[2 * kq + 1][3])});
        dsbf[kq] = as_bf16x8(u32x4{pack_bf16(dp[2 * kq][0], dp[2 * kq][1]), pack_bf16(dp[2 * kq][2], dp[2 * kq][3]),
                                   pack_bf16(dp[2 * kq + 1][0], dp[2 * kq + 1][1]), pack_bf16(dp[2 * kq + 1][2], dp[2 * kq + 1][3])});
      }
      // dS^T -> LDS: row = key, 4 queries per 8-byte write
#pragma unroll
      for (int qb = 0; qb < 4; ++qb)
        *(u32x2*)&sm.dst[ds256_at(kvl, 16 * qb + 4 * gq)] =
            u32x2{pack_bf16(dp[qb][0], dp[qb][1]), pack_bf16(dp[qb][2], dp[qb][3])};

      // ---- dV += P^T dO, dK += dS^T Q: B operand of d block db, k-step kq =
      //      two transposed reads (queries 32kq + 4(l/16) + 0..3 and +16)
      {
        auto rd = [&](int k, bf16x8* bo, bf16x8* bqv) {
          const int db = k >> 1, kq = k & 1;
          const int col = 16 * db + 4 * (lr & 3);
          const int row = 32 * kq + 4 * gq + (lr >> 2);
          *bo = as_bf16x8(tr_read(&sm.dos[q256_at(row, col)]), tr_read(&sm.dos[q256_at(row + 16, col)]));
          *bqv = as_bf16x8(tr_read(&sm.qs[q256_at(row, col)]), tr_read(&sm.qs[q256_at(row + 16, col)]));
        };
        constexpr int NP = 2 * NDB, RING = 3;
        bf16x8 ro[RING], rqv[RING];
#pragma unroll
        for (int k = 0; k < RING; ++k) rd(k, &ro[k], &rqv[k]);
#pragma unroll
        for (int k = 0; k < NP; ++k) {
          __builtin_amdgcn_sched_barrier(0);
          const int db = k >> 1, kq = k & 1;
          dvacc[db] = mfma16(pbf[kq], ro[k % RING], dvacc[db]);
          dkacc[db] = mfma16(dsbf[kq], rqv[k % RING], dkacc[db]);
          if (k + RING < NP) rd(k + RING, &ro[k % RING], &rqv[k % RING]);
        }
        __builtin_amdgcn_sched_barrier(0);
      }

      // deferred release of the previous block (its stores were issued a step ago)
      if (pend_ctr >= 0) {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        release();
      }
      // dS^T complete; every wave is done with this block's Q / dO / L / D
      __syncthreads();
      if (pb_next >= 0) load_block(pb_next);

      // ---- dQ^T_loc (columns d in [64w, 64w+64), all 64 queries) = K^T dS^T;
      //      tile t = 4 db + qb
      f32x4 dq[16];
#pragma unroll
      for (int t = 0; t < 16; ++t) dq[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        bf16x8 bds[4];
#pragma unroll
        for (int qb = 0; qb < 4; ++qb) {
          const int row = 32 * kk + 8 * gq + (lr >> 2);
          const int col = 16 * qb + 4 * (lr & 3);
          bds[qb] = as_bf16x8(tr_read(&sm.dst[ds256_at(row, col)]), tr_read(&sm.dst[ds256_at(row + 4, col)]));
        }
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
          for (int qb = 0; qb < 4; ++qb) dq[4 * db + qb] = mfma16(ktreg[db][kk], bds[qb], dq[4 * db + qb]);
      }
      // dq[4db + qb][r] <-> query 16qb + l%16, column d = 64w + 16db + 4(l/16) + r

      if (a.partials) {
        const auto rp = make_rsrc(a.partials + ((size_t)bh * a.tc + j) * N * D, hbytes * 2);
#pragma unroll
        for (int t = 0; t < 16; ++t)
          st16(rp, (uint32_t)((q0 + 16 * (t & 3) + lr) * D + 64 * w + 16 * (t >> 2) + 4 * gq) * 4,
               __builtin_bit_cast(u32x4, dq[t]));
      }

      bool add = false;
      if (ordered) {
        if (!have_turn && !failed) {
          if constexpr (STATS) vm_wait<0>();  // time the wait only, not this wave's own loads
          const unsigned long long t0 = STATS ? clock_now() : 0ull;
          have_turn = wait_turn(ctr, NW * rank, a.spin_limit);
          if constexpr (STATS) stats_wait(wst, t0);
          if (!have_turn) {
            failed = true;
            __hip_atomic_store(&a.ctrl[kCtrlError], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (a.status) __hip_atomic_store(a.status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          } else if (rank > 0) {
            load_acc(pb);  // late fetch: the turn came after the early poll
          }
        }
        add = have_turn && rank > 0;
      }
      // this wave's slice and the next block's Q / dO / L / D have landed
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      if (ordered && pb_next >= 0)
        poll_v = __hip_atomic_load(ctr_head + (size_t)pb_next * kCtrStride, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if constexpr (ordered) {
        // ---- add the partial into the slice straight from registers (one lane
        //      per element: the order is the schedule's), then store it
        if (have_turn) {
          const auto rdq = make_rsrc((__bf16*)a.dq + head, hbytes);
#pragma unroll
          for (int t = 0; t < 16; ++t) {
            f32x4 v = dq[t];
            const f32x4 old = *(const f32x4*)&acc_w[t * 256 + 4 * l];
            const f32x4 sum = old + v;
#pragma unroll
            for (int x = 0; x < 4; ++x) v[x] = add ? sum[x] : v[x];
            if (last) {
              const uint32_t off = (uint32_t)((q0 + 16 * (t & 3) + lr) * D + 64 * w + 16 * (t >> 2) + 4 * gq);
              st8(rdq, off * 2, u32x2{pack_bf16(v[0] * a.scale, v[1] * a.scale), pack_bf16(v[2] * a.scale, v[3] * a.scale)});
              if (a.dq_accum) st16(make_rsrc(a.dq_accum + head, hbytes * 2), off * 4, __builtin_bit_cast(u32x4, v));
            } else {
              st16_coherent(racc, acc_off(pb, t), __builtin_bit_cast(u32x4, v));
            }
          }
        }
        if (tid == 0 && a.witness && rank < a.tc) a.witness[((size_t)bh * a.nblk + pb) * a.tc + rank] = j;
        pend_ctr = pb;
        // at the end of the chain or of its KV tile the release comes now: the
        // tile switch (dK, dV stores, K, V loads) would hold it back, and under
        // Symmetric Shift every later contributor of the block, one task behind
        // the one before, would wait for its own predecessor's switch in turn
        if (!deferred || nst >= nsteps || tile_ends) {
          asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
          release();
        }
      } else {
        // ---- atomic variant: stage the partial row-major in LDS ([q][64 d],
        //      16-byte chunk c of row q at c ^ (q & 15)), then one fp32 atomic per
        //      element, each instruction covering one 256-byte row segment
#pragma unroll
        for (int t = 0; t < 16; ++t) {
          const int q = 16 * (t & 3) + lr, c = 4 * (t >> 2) + gq;
          *(f32x4*)&acc_w[q * 64 + 4 * (c ^ (q & 15))] = dq[t];
        }
        asm volatile("" ::: "memory");  // lanes read what other lanes wrote
#pragma unroll 8
        for (int q = 0; q < BM; ++q) {
          const float v = acc_w[q * 64 + 4 * ((l >> 2) ^ (q & 15)) + (l & 3)];
          if (q0 + q < N) atomicAdd(a.dqacc + head + (size_t)(q0 + q) * D + 64 * w + l, v);
        }
      }
      st = nst;
    }
    if (cur_j >= 0) store_dkdv(cur_j);
    __syncthreads();  // sm.item is rewritten by the next ticket
  }
  if constexpr (STATS) stats_wave_end(wst, a.wait_stats, l);
}

template <bool CAUSAL>
hipError_t launch_main256_mask(const BwdArgs& a, int grid, hipStream_t stream) {
  if (a.G.sched == S_ATOMIC) return launch_main_grid(bwd_main256_kernel<CAUSAL, false, false>, a, grid, NT, stream);
  if (a.nxcd > 0 && a.wait_stats) return launch_main_grid(bwd_main256_kernel<CAUSAL, true, true, true>, a, grid, NT, stream);
  if (a.nxcd > 0) return launch_main_grid(bwd_main256_kernel<CAUSAL, true, true>, a, grid, NT, stream);
  if (a.wait_stats) return launch_main_grid(bwd_main256_kernel<CAUSAL, true, false, true>, a, grid, NT, stream);
  return launch_main_grid(bwd_main256_kernel<CAUSAL, true, false>, a, grid, NT, stream);
}

}  // namespace

hipError_t launch_main256(const BwdArgs& a, int grid_main, hipStream_t stream) {
  return a.G.causal ? launch_main256_mask<true>(a, grid_main, stream) : launch_main256_mask<false>(a, grid_main, stream);
}

int bwd_main256_occupancy() {
  int lo = 1 << 30;
  const void* fns[10] = {(const void*)bwd_main256_kernel<false, false, false>, (const void*)bwd_main256_kernel<false, true, false>,
                         (const void*)bwd_main256_kernel<false, true, true>, (const void*)bwd_main256_kernel<true, false, false>,
                         (const void*)bwd_main256_kernel<true, true, false>, (const void*)bwd_main256_kernel<true, true, true>,
                         (const void*)bwd_main256_kernel<false, true, false, true>, (const void*)bwd_main256_kernel<false, true, true, true>,
                         (const void*)bwd_main256_kernel<true, true, false, true>, (const void*)bwd_main256_kernel<true, true, true, true>};
  for (const void* f : fns) {
    int blocks = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, f, NT, 0) != hipSuccess) return 0;
    lo = blocks < lo ? blocks : lo;
  }
  return lo;
}

}  // namespace dash
