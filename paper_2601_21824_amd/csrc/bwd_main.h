// bwd_main.h -- the backward main kernel with KV tiles of 128 rows (d = 128,
// and d = 64 where its tiles are 128 rows), its launch and its occupancy.
//
// One KV tile of 128 rows per work item, 4 waves; wave w owns KV rows
// [32w, 32w+32) of the tile and keeps K, V, K^T operands and the dK, dV
// accumulators in registers for the whole chain.  For every 64-row Q block
// of the chain (Algorithm 1, the consumer loop):
//   S = Q K^T, dP = dO V^T            (bf16 MFMA 32x32x16)
//   P = exp(S - L), dS = P o (dP - D)  (fp32)
//   dV += P^T dO, dK += dS^T Q          (P^T, dS^T fed from registers)
//   dQ^T_loc = K^T dS^T                 (dS staged through LDS)
// then the ordered reduction (Algorithm 1, the dQ writer): wait until the
// block's counter has reached this tile's rank, add the partial into the fp32
// dQ accumulator with device-coherent (SC1) loads/stores, make the stores
// visible, bump the counter.  The last rank writes bf16 s*dQ directly.  No
// atomics touch the data; the order is fixed by the schedule, so results are
// bitwise reproducible.  The grid is persistent: workgroups take work items
// from a ticket counter in order, so every item a wait depends on has been
// started.
//
// A template over the head dim, included by the translation unit of each
// head dim (attn_bwd.hip: d = 128; attn_bwd_d64.hip: d = 64), so that each
// is compiled with the flags that suit it.
#pragma once
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "bwd_common.h"
#include "lds_layout.h"

namespace dash {

// ---------------------------------------------------------------- bwd_main
// LDS layouts of the Q / dO blocks and the dS^T tile: lds_layout.h.

template <int D>
struct MainSmem {
  static constexpr int BM = kBlockRows;
  __bf16 qs[2][BM * D];    // Q block [q][d], double-buffered
  __bf16 dos[2][BM * D];   // dO block [q][d], double-buffered
  __bf16 dst[kTileKV * BM];  // dS^T (bf16) [kv][q], swizzled 8-byte slots (dst_at)
  float acc[BM * D];       // dQ accumulator block as it arrives, per-wave slices in register order
  float ls[2][BM];         // L * log2(e) per query row
  float ds[2][BM];         // D per query row
  unsigned steps[kMaxChainSteps];  // this chain's blocks, see pack_step
  int poll[kTileKV / 32][64];  // per wave: the coming block's counter (direct load, all lanes alike)
  int item;
};

template <int D, bool CAUSAL, int MODE, bool STATS = false>
__global__ __launch_bounds__(256) void bwd_main_kernel(BwdArgs a) {
  constexpr int BC = kTileKV;   // KV rows per tile (128 for d = 64 and 128)
  constexpr int NW = BC / 32;   // waves, 32 KV rows each
  constexpr int NT = 64 * NW;   // threads
  constexpr int BM = kBlockRows;
  constexpr int KS = D / 16;    // k-steps over d
  constexpr int KSC = BC / 16;  // k-steps over kv
  constexpr int NB = D / 32;    // 32-column blocks of d
  constexpr int CPR = D / 8;    // 16-byte bf16 chunks per row
  constexpr int QLD = BM * CPR / NT;   // direct loads per thread for a Q / dO block
  // dQ^T of a block is (D / 32) x 2 tiles of 32 x 32 (d block, query half),
  // tile T = 2 * (d block) + (query half); wave w computes tiles
  // [w * DQT, (w + 1) * DQT): one d block and one or both query halves
  constexpr int DQT = D / 64;
  constexpr int NACC = 4 * DQT;  // its accumulator slice in 1 KB chunks
  static_assert(NT == 256 && QLD * 32 == D && BM * D == NW * DQT * 1024, "thread/tile shape");
  __shared__ __attribute__((aligned(16))) MainSmem<D> sm;

  const Geom G = a.G;
  const int N = a.n;
  const int tid = threadIdx.x, l = tid & 63, g = l >> 5, lc = l & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int L16 = l & 15, nh = (l >> 4) & 1;  // transpose-read lane roles
  const int dblk = (w * DQT) >> 1, qh0 = (w * DQT) & 1;  // this wave's d block, first query half
  const float c2 = a.scale * kLog2e;
  const uint32_t hbytes = (uint32_t)((size_t)N * D * 2);
  constexpr bool ordered = MODE == kModeOrdered || MODE == kModeOrderedXcd;
  // XCD-local placement: this workgroup serves the heads of its own XCD from
  // that XCD's ticket queue (no other XCD touches those heads).  The
  // accumulator is still read and written device-coherently (SC1), as under
  // global placement: an L2-scope (SC0) read may hit this CU's L1, which keeps
  // lines that workgroups on other CUs have since overwritten in the L2.
  constexpr bool xcd = MODE == kModeOrderedXcd;
  const int xq = xcd ? xcc_id() : 0;
  const int total = xcd ? (xq < a.nxcd ? xcd_heads(a.bh, a.nxcd, xq) * G.chains : 0) : a.bh * G.chains;
  int* const ticket = &a.ctrl[xcd ? kCtrlXcdTicket + xq : kCtrlTicket];
  const int* const order = a.order + (xcd ? 2 * xq * a.xcd_cap : 0);
  // LDS byte addresses for the direct copies: the base once, offsets as
  // integers (no generic-to-LDS pointer conversion per copy)
  const uint32_t sm_lds = lds_base(&sm);
  auto lds_of = [&](const void* p) { return sm_lds + (uint32_t)((const char*)p - (const char*)&sm); };
  // Shift-type orders are conflict-free: the next contributor to a block reaches
  // it at least one step later, so the counter release can wait until the
  // second MFMA run of the next step, by which time the accumulator stores
  // have drained without a wait of their own.
  const bool deferred = G.sched == S_SHIFT || G.sched == S_SYMSHIFT;
  bool failed = false;  // this wave hit a wait timeout: skip further waits
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
    const auto rctr = make_rsrc(ctr_head, (uint32_t)a.nblk * kCtrStride * 4);
    // L * log2(e) and D of this head's N rows: the padded rows of a ragged
    // last block read 0, so P = 1 there, multiplied by Q and dO rows that
    // also read 0: those rows add exactly nothing to dK and dV
    const auto rls = make_rsrc(a.lse2 + (size_t)bh * N, (uint32_t)N * 4);
    const auto rds = make_rsrc(a.dvec + (size_t)bh * N, (uint32_t)N * 4);

    const unsigned* tab = a.steps + (size_t)wch * a.step_cap;
    const int nsteps = __builtin_amdgcn_readfirstlane((int)tab[0]);
    // the chain's schedule (computed by bwd_pre) into LDS; the previous
    // chain's readers all passed the barrier after the ticket
    for (int st = tid; st < nsteps; st += NT) sm.steps[st] = tab[1 + st];
    __syncthreads();
    int cur_j = -1;
    bf16x8 kreg[KS], vreg[KS], ktreg[KSC];  // K, V rows (B of S = Q K^T, dP = dO V^T), K^T (A of dQ^T = K^T dS^T)
    f32x16 dkacc[NB], dvacc[NB];
    int pend_ctr = -1;  // block whose counter this wave still has to advance
    // The coming block's counter is copied into sm.poll[w] one step early.
    // vm_poll counts this wave's vector memory operations issued since that
    // copy (a lower bound is safe: the wait before reading it only gets
    // longer), vm_rel those issued since the accumulator stores of the
    // previous block.
    int vm_poll = 63, vm_rel = 63;
    bool top_wait = true;  // first block of the chain: wait for this wave's LDS loads at the top

    auto step_at = [&](int st) -> unsigned { return __builtin_amdgcn_readfirstlane(sm.steps[st]); };
    auto next_valid = [&](int st) {
      while (st < nsteps && step_at(st) == kNoStep) ++st;
      return st;
    };
    // Q / dO / L / D of block pb into LDS buffer b (asynchronous, vmcnt)
    // Part k of a block is rows 16k (D = 128; 32k at D = 64) further down, i.e.
    // 4 KB further in both the global tile and the LDS tile, with the same
    // swizzle (tile_swz repeats every 16 / 32 rows).
    static_assert((NT / CPR) * D * 2 == 4096 && NT * 16 == 4096, "a part is 4 KB");
    auto load_part = [&](int pb, int b, int k) {  // part k < QLD of the Q and dO rows
      const int r = tid / CPR, c = (tid % CPR) ^ tile_swz<D>(r);
      const uint32_t off = (uint32_t)((pb * BM + r) * D + 8 * c) * 2;
      const uint32_t at = lds_of(&sm.qs[b][64 * w * 8]) + 4096u * k;
      dma16_pair(rq, rdo, at, at + (uint32_t)sizeof(sm.qs), off, 4096u * k);
    };
    auto load_ld = [&](int pb, int b) {  // L * log2(e) and D of the block's rows
      const uint32_t row = (uint32_t)(pb * BM + fresh_lane());
      if (w == 0) dma4(rls, lds_of(&sm.ls[b][0]), row * 4);
      if (w == 1) dma4(rds, lds_of(&sm.ds[b][0]), row * 4);
    };
    auto load_block = [&](int pb, int b) {
#pragma unroll
      for (int k = 0; k < QLD; ++k) load_part(pb, b, k);
      load_ld(pb, b);
    };
    constexpr int kBlockLoads = 2 * QLD;  // direct loads of one block by waves >= 2 (waves 0, 1: one more)
    // The ordered variants keep dQacc in register order: 64-row block pb is
    // BM*D floats at pb*BM*D, 32 x 32 tile T at T*1024; wave w's slice (its
    // DQT tiles) is at w*DQT*1024, and its chunk k (tile w*DQT + k/4, rb = k%4)
    // of lane l at k*256 + 4l holds row 32 (qh0 + k/4) + l%32, columns
    // 32 dblk + 8rb + 4(l/32) .. +3.
    float* acc_w = &sm.acc[w * DQT * 1024];
    auto acc_off = [&](int pb, int k) { return (uint32_t)(pb * BM * D + w * DQT * 1024 + k * 256 + 4 * l) * 4; };
    // block pb's counter into this wave's poll slot.  The counters stay
    // device-coherent under XCD-local placement too: the atomic adds are
    // performed past the L2, so an L2 read of a counter can stay stale.
    auto poll_copy = [&](int pb) { dma4_coherent(rctr, lds_of(&sm.poll[w][0]), (uint32_t)pb * kCtrStride * 4); };
    auto acc_copy = [&](int pb, int k4) {  // chunks 4 k4 .. 4 k4 + 3 of the slice into its landing pad
      dma16x4_coherent(racc, lds_of(&acc_w[k4 * 1024]), acc_off(pb, 0), 4096u * k4);
    };
    auto load_acc = [&](int pb) {
#pragma unroll
      for (int k4 = 0; k4 < NACC / 4; ++k4) acc_copy(pb, k4);
    };
    auto store_dkdv = [&](int j) {
      const auto rdk = make_rsrc((__bf16*)a.dk + head, hbytes);
      const auto rdv = make_rsrc((__bf16*)a.dv + head, hbytes);
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
    // this wave's accumulator stores are complete (caller waited on vmcnt):
    // add its share to the block's counter
    auto release = [&]() {
      if (l == 0 && pend_ctr >= 0)
        __hip_atomic_fetch_add(ctr_head + (size_t)pend_ctr * kCtrStride, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      pend_ctr = -1;
    };

    int st = next_valid(0);
    int buf = 0;
    if (st < nsteps) {
      const int pb0 = step_at(st) & 0xfff;
      load_block(pb0, buf);
      if (ordered) poll_copy(pb0);
    }

    for (; st < nsteps;) {
      const unsigned e = step_at(st);
      const int pb = e & 0xfff, j = (e >> 12) & 0x1ff, rank = (e >> 21) & 0x3ff;
      const bool last = (e >> 31) != 0;
      const int q0 = pb * BM;

      if (j != cur_j) {  // new KV tile: flush the previous one, load K/V operands
        if (cur_j >= 0) store_dkdv(cur_j);
        cur_j = j;
        const int kv0 = j * BC;
        const int kvr = kv0 + 32 * w + lc;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          kreg[ks] = as_bf16x8(ld16(rk, (uint32_t)(kvr * D + 16 * ks + 8 * g) * 2));
          vreg[ks] = as_bf16x8(ld16(rv, (uint32_t)(kvr * D + 16 * ks + 8 * g) * 2));
        }
        // K^T operand: lane holds column d = 32 dblk + lc of K over keys 16ks + 8g .. +7
#pragma unroll
        for (int ks = 0; ks < KSC; ++ks) {
          unsigned short t[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) t[e] = ld2(rk, (uint32_t)((kv0 + 16 * ks + 8 * g + e) * D + 32 * dblk + lc) * 2);
          ktreg[ks] = as_bf16x8(u32x4{t[0] | ((unsigned)t[1] << 16), t[2] | ((unsigned)t[3] << 16),
                                      t[4] | ((unsigned)t[5] << 16), t[6] | ((unsigned)t[7] << 16)});
        }
        // wait for the operands here, on this path only: otherwise the
        // compiler guards their first uses in every step with waits that also
        // drain the prefetch issued in between
        vm_wait<0>();
        vm_poll = vm_rel = 63;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            dkacc[nb][r] = 0.f;
            dvacc[nb][r] = 0.f;
          }
      }

      // ---- this block's Q / dO landed in LDS (each wave waited for its own
      //      loads at the end of the previous block; only a new chain or V tile
      //      waits here), so after the barrier all of it is visible and the other
      //      buffer is free
      if (top_wait) {
        vm_wait<0>();
        vm_poll = vm_rel = 63;
      }
      top_wait = false;
      __syncthreads();

      // ---- the next valid block (prefetched into the other buffer below)
      const int nst = next_valid(st + 1);
      const int pb_next = nst < nsteps ? (int)(step_at(nst) & 0xfff) : -1;
      // the chain moves to another KV tile after this step (Symmetric Shift,
      // between its two tiles)
      const bool tile_ends = nst < nsteps && (int)((step_at(nst) >> 12) & 0x1ff) != j;

      int* ctr = ctr_head + (size_t)pb * kCtrStride;
      bool have_turn = false;

      const __bf16* qs = sm.qs[buf];
      const __bf16* dos = sm.dos[buf];
      f32x16 s[2], dp[2];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          s[qb][r] = 0.f;
          dp[qb][r] = 0.f;
        }
      // The step is four runs of 16 MFMAs -- S/dP of query half 0, S/dP of
      // half 1, dV/dK of half 0, dV/dK of half 1 -- and the vector, LDS-store
      // and DMA work of the step is cut into pieces issued between them:
      // the next block's prefetch during the first run, softmax of half 0 and
      // the accumulator fetch during the second, softmax of half 1 during the
      // third, the dS^T stores during the fourth.  The sched_barrier fences
      // keep that interleaving.
      //
      // S = Q K^T, dP = dO V^T for query half qb and this wave's 32 keys:
      // A = Q / dO rows from LDS (RING - 1 k-steps ahead), B = K / V rows
      // from registers.
      auto sdp = [&](int qb, auto&& extra) {
        constexpr int RING = 4;
        bf16x8 rq[RING], ro[RING];
        auto rd = [&](int ks) {
          const int at = bf_at<D>(32 * qb + lc, 16 * ks + 8 * g);
          rq[ks % RING] = *(const bf16x8*)&qs[at];
          ro[ks % RING] = *(const bf16x8*)&dos[at];
        };
#pragma unroll
        for (int k = 0; k < RING - 1; ++k) rd(k);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          if (ks + RING - 1 < KS) rd(ks + RING - 1);
          __builtin_amdgcn_sched_barrier(0);
          s[qb] = mfma32(rq[ks % RING], kreg[ks], s[qb]);
          dp[qb] = mfma32(ro[ks % RING], vreg[ks], dp[qb]);
          extra(ks);
          __builtin_amdgcn_sched_barrier(0);
        }
      };

      // P = exp(S - L), dS = P (dP - D) in 8 pieces per query half: piece k
      // covers row group rb = k/2 (queries 32qb + 8rb + 4g + c) for c in
      // {2(k%2), 2(k%2)+1}; L and D of the next row group are read one piece
      // ahead.  Element (qb, r) is query 32qb + 8(r/4) + 4g + r%4 of the block
      // and key 32w + lc of the tile.  Keys past N need no mask: their K, V
      // rows read as zero, P is at most 1 there (exp2_unit) and their dK, dV
      // rows are not stored.
      const int kvl = 32 * w + lc;
      const int thr = j * BC + kvl - q0 - 4 * g;  // causal: masked iff 32qb+8rb+c < thr
      bf16x8 pbf[2][2], dsbf[2][2];
      f32x4 Lc, Dc, Ln, Dn;
      auto read_ld = [&](int qb, int rb) {
        const int ql = 32 * qb + 8 * rb + 4 * g;
        Ln = *(const f32x4*)&sm.ls[buf][ql];
        Dn = *(const f32x4*)&sm.ds[buf][ql];
      };
      auto softmax_piece = [&](int qb, int k) {
        const int rb = k >> 1;
        if ((k & 1) == 0) {
          Lc = Ln;
          Dc = Dn;
        } else if (rb < 3 || qb == 0) {
          read_ld(rb < 3 ? qb : qb + 1, rb < 3 ? rb + 1 : 0);
        }
#pragma unroll
        for (int cc = 0; cc < 2; ++cc) {
          const int c = 2 * (k & 1) + cc, r = 4 * rb + c;
          float p = exp2_unit(__builtin_fmaf(s[qb][r], c2, -Lc[c]));
          if (CAUSAL) p = (32 * qb + 8 * rb + c < thr) ? 0.f : p;
          s[qb][r] = p;
          dp[qb][r] = p * (dp[qb][r] - Dc[c]);
        }
        if (k == 3) {
          pbf[qb][0] = pack8(s[qb], 0);
          dsbf[qb][0] = pack8(dp[qb], 0);
        } else if (k == 7) {
          pbf[qb][1] = pack8(s[qb], 8);
          dsbf[qb][1] = pack8(dp[qb], 8);
        }
      };
      // dS^T -> LDS, piece k of 8: query half k/4, 8-byte slot k%4
      auto store_ds_piece = [&](int k) {
        const int qb = k >> 2, half = (k >> 1) & 1, part = k & 1;
        const u32x4 dv4 = __builtin_bit_cast(u32x4, dsbf[qb][half]);
        *(u32x2*)&sm.dst[dst_at(kvl, 32 * qb + 16 * half + 8 * part + 4 * g)] =
            part ? u32x2{dv4[2], dv4[3]} : u32x2{dv4[0], dv4[1]};
      };
      // dV += P^T dO and dK += dS^T Q for query half qb: A = P^T, dS^T from
      // registers, B = dO^T, Q^T by transposed reads of the row-major tiles
      // (RING - 1 operand pairs ahead)
      auto dvdk = [&](int qb, auto&& extra) {
        constexpr int NP = 2 * NB, RING = 3;
        auto rd = [&](int k, bf16x8* bo, bf16x8* bq) {
          const int nb = k >> 1, half = k & 1;
          const int col = 32 * nb + 16 * nh + 4 * (L16 & 3);
          const int row = 32 * qb + 16 * half + 4 * g + (L16 >> 2);
          *bo = as_bf16x8(tr_read(&dos[bf_at<D>(row, col)]), tr_read(&dos[bf_at<D>(row + 8, col)]));
          *bq = as_bf16x8(tr_read(&qs[bf_at<D>(row, col)]), tr_read(&qs[bf_at<D>(row + 8, col)]));
        };
        bf16x8 ro[RING], rq[RING];
#pragma unroll
        for (int k = 0; k < RING; ++k) rd(k, &ro[k], &rq[k]);
#pragma unroll
        for (int k = 0; k < NP; ++k) {
          __builtin_amdgcn_sched_barrier(0);
          const int nb = k >> 1, half = k & 1;
          dvacc[nb] = mfma32(pbf[qb][half], ro[k % RING], dvacc[nb]);
          dkacc[nb] = mfma32(dsbf[qb][half], rq[k % RING], dkacc[nb]);
          if (k + RING < NP) rd(k + RING, &ro[k % RING], &rq[k % RING]);
          extra(k);
        }
        __builtin_amdgcn_sched_barrier(0);
      };

      // run 1: S/dP of half 0, with the next block's Q / dO / L / D prefetch
      sdp(0, [&](int ks) {
        if (pb_next < 0) return;
        if (ks < QLD) load_part(pb_next, buf ^ 1, ks);
        if (ks == 0) load_ld(pb_next, buf ^ 1);
      });
      if (pb_next >= 0) {
        const int n = kBlockLoads + (w < 2 ? 1 : 0);
        vm_poll += n;
        vm_rel += n;
      }
      // ---- ordering: the counter of this block was copied at the end of the
      //      previous step; if the turn is ours, fetch the accumulator slice
      //      during the next run so its latency hides behind the MFMAs
      if (ordered && !failed) {
        vm_wait_le(vm_poll);  // the copy has landed (the prefetch need not have)
        const int v0 = __builtin_amdgcn_readfirstlane(sm.poll[w][0]);
        if (v0 >= NW * rank) {
          have_turn = true;
          __atomic_signal_fence(__ATOMIC_SEQ_CST);
        }
      }
      const bool early_acc = ordered && have_turn && rank > 0;
      read_ld(0, 0);
      // run 2: S/dP of half 1, with softmax of half 0 and the accumulator fetch
      sdp(1, [&](int ks) {
#pragma unroll
        for (int p = ks * 8 / KS; p < (ks + 1) * 8 / KS; ++p) {
          softmax_piece(0, p);
          if (early_acc && (p & 3) == 0 && p < NACC) acc_copy(pb, p >> 2);
        }
      });
      if (early_acc) vm_rel += NACC;
      // deferred release of the previous block, after the second run: its
      // accumulator stores were followed by vm_rel operations (this step's
      // prefetch and accumulator fetch), and vector memory operations
      // complete in issue order, so at most vm_rel in flight means the stores
      // are done.  Released this early, the block's next contributor (a step
      // or more behind under Shift and Symmetric Shift) finds its turn at its
      // early look instead of waiting at the end of its step.
      if (pend_ctr >= 0) {
        vm_wait_le(vm_rel);
        release();
      }
      // run 3: dV/dK of half 0, with softmax of half 1
      dvdk(0, [&](int k) {
#pragma unroll
        for (int p = k * 8 / (2 * NB); p < (k + 1) * 8 / (2 * NB); ++p) softmax_piece(1, p);
      });
      // run 4: dV/dK of half 1, with the dS^T stores
      dvdk(1, [&](int k) {
        if constexpr (MODE != kModeNoDq) {
#pragma unroll
          for (int p = k * 8 / (2 * NB); p < (k + 1) * 8 / (2 * NB); ++p) store_ds_piece(p);
        }
      });

      if constexpr (MODE == kModeNoDq) {
        // dK, dV only: the next block's Q / dO have landed before the barrier
        vm_wait<0>();
      } else {
        __syncthreads();

        // ---- dQ^T_loc (rows d in [32w, 32w+32), all 64 queries) = K^T dS^T,
        //      k-step ks reads A = K^T (shared by both query halves) and two B's
        f32x16 dq[DQT];
  #pragma unroll
        for (int t = 0; t < DQT; ++t)
  #pragma unroll
          for (int r = 0; r < 16; ++r) dq[t][r] = 0.f;
        {
          constexpr int RING = 3;
          auto rd = [&](int ks, bf16x8* bt) {
            const int krow = 16 * ks + 8 * g + (L16 >> 2);
  #pragma unroll
            for (int t = 0; t < DQT; ++t) {
              const int qc = 32 * (qh0 + t) + 16 * nh + 4 * (L16 & 3);
              bt[t] = as_bf16x8(tr_read(&sm.dst[dst_at(krow, qc)]), tr_read(&sm.dst[dst_at(krow + 4, qc)]));
            }
          };
          bf16x8 rb[RING][DQT];
  #pragma unroll
          for (int k = 0; k < RING; ++k) rd(k, rb[k]);
  #pragma unroll
          for (int ks = 0; ks < KSC; ++ks) {
            __builtin_amdgcn_sched_barrier(0);
  #pragma unroll
            for (int t = 0; t < DQT; ++t) dq[t] = mfma32(ktreg[ks], rb[ks % RING][t], dq[t]);
            if (ks + RING < KSC) rd(ks + RING, rb[ks % RING]);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
        // dq[t][r] <-> query 32 (qh0 + t) + lc, column d = 32 dblk + 8(r/4) + 4g + r%4

        if (a.partials) {
          const auto rp = make_rsrc(a.partials + ((size_t)bh * a.tc + j) * N * D, hbytes * 2);
  #pragma unroll
          for (int t = 0; t < DQT; ++t)
  #pragma unroll
            for (int rb = 0; rb < 4; ++rb)
              st16(rp, (uint32_t)((q0 + 32 * (qh0 + t) + lc) * D + 32 * dblk + 8 * rb + 4 * g) * 4,
                   __builtin_bit_cast(u32x4, f32x4{dq[t][4 * rb], dq[t][4 * rb + 1], dq[t][4 * rb + 2], dq[t][4 * rb + 3]}));
        }

        bool add = false;  // accumulate into the slice (else: the partial is stored as is)
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
        // this wave's slice (and the next block's Q / dO) have landed
        vm_wait<0>();
        vm_poll = vm_rel = 0;
        // copy the next block's counter now, ahead of the stores below
        if (ordered && pb_next >= 0) poll_copy(pb_next);
        if constexpr (ordered) {
          // ---- add this wave's partial into its slice straight from registers:
          //      the accumulator is stored in this wave's register order, so the
          //      slice arrives (LDS landing pad) and leaves in 1 KB coalesced rows.
          //      Each element is touched by exactly one lane: the sum order is the
          //      schedule's.
          // (`add` and `last` are wave-uniform: one straight path each)
          auto finish = [&](auto add_c, auto last_c) {
            constexpr bool kAdd = decltype(add_c)::value, kLast = decltype(last_c)::value;
            f32x4 old[NACC];
            if constexpr (kAdd) {
  #pragma unroll
              for (int k = 0; k < NACC; ++k) old[k] = *(const f32x4*)&acc_w[k * 256 + 4 * l];
            }
  #pragma unroll
            for (int k = 0; k < NACC; ++k) {
              const int t = k >> 2, rb = k & 3;
              f32x4 v = {dq[t][4 * rb], dq[t][4 * rb + 1], dq[t][4 * rb + 2], dq[t][4 * rb + 3]};
              if constexpr (kAdd) v = old[k] + v;
              if constexpr (kLast) {
                const auto rdq = make_rsrc((__bf16*)a.dq + head, hbytes);
                const uint32_t off = (uint32_t)((q0 + 32 * (qh0 + t) + lc) * D + 32 * dblk + 8 * rb + 4 * g);
                st8(rdq, off * 2, u32x2{pack_bf16(v[0] * a.scale, v[1] * a.scale), pack_bf16(v[2] * a.scale, v[3] * a.scale)});
                if (a.dq_accum) st16(make_rsrc(a.dq_accum + head, hbytes * 2), off * 4, __builtin_bit_cast(u32x4, v));
              } else {
                st16_coherent(racc, acc_off(pb, k), __builtin_bit_cast(u32x4, v));
              }
            }
          };
          using T_ = std::true_type;
          using F_ = std::false_type;
          if (have_turn) {
            if (!last) {
              if (add) finish(T_{}, F_{});
              else finish(F_{}, F_{});
            } else {
              if (add) finish(T_{}, T_{});
              else finish(F_{}, T_{});
            }
            vm_poll += last ? (a.dq_accum ? 2 * NACC : NACC) : NACC;
          }
        } else if constexpr (MODE == kModePartials) {
          // ---- partials variant: the partial goes to KV tile j's own buffer, in
          //      the same register order as the ordered accumulator
          const auto rpb = make_rsrc(a.dqacc + ((size_t)bh * a.tc + j) * a.nblk * BM * D, (uint32_t)a.nblk * BM * D * 4);
  #pragma unroll
          for (int k = 0; k < NACC; ++k) {
            const int t = k >> 2, rb = k & 3;
            st16(rpb, acc_off(pb, k), __builtin_bit_cast(u32x4, f32x4{dq[t][4 * rb], dq[t][4 * rb + 1], dq[t][4 * rb + 2], dq[t][4 * rb + 3]}));
          }
        } else {
          // ---- atomic variant: partial -> LDS (row-major slice), then one fp32
          //      atomic per element, each instruction covering two whole 128-byte
          //      row segments of the row-major dQacc.  Staging: 16-byte chunk
          //      c of row q at c ^ ((q >> 1) & 7), conflict-free for the chunk
          //      writes (16 rows per lane group) and the row reads (two rows per
          //      instruction); the read of rows 2k, 2k+1 XORs with k & 7, the
          //      same for every lane, so no per-row lane offsets stay live.
          //      Staged row rr of the wave's slice is block row 32 qh0 + rr.
  #pragma unroll
          for (int k = 0; k < NACC; ++k) {
            const int t = k >> 2, rb = k & 3, rr = 32 * t + lc;
            *(f32x4*)&acc_w[(rr * 8 + ((2 * rb + g) ^ ((rr >> 1) & 7))) * 4] =
                f32x4{dq[t][4 * rb], dq[t][4 * rb + 1], dq[t][4 * rb + 2], dq[t][4 * rb + 3]};
          }
          asm volatile("" ::: "memory");  // lanes read what other lanes wrote
          const int c = l & 31, hi = l >> 5;
          const int lane_off = hi * D + 32 * dblk + c;  // this lane's element of a two-row pair
          const int qr0 = q0 + 32 * qh0;
  #pragma unroll 8
          for (int k = 0; k < 16 * DQT; ++k) {
            const float v = acc_w[(2 * k + hi) * 32 + (((c >> 2) ^ (k & 7)) << 2) + (c & 3)];
            float* rows = a.dqacc + head + (size_t)(qr0 + 2 * k) * D;  // wave-uniform
            if (qr0 + 2 * k + hi < N) atomicAdd(rows + lane_off, v);
          }
        }
        if (ordered) {
          if (tid == 0 && a.witness && rank < a.tc) a.witness[((size_t)bh * a.nblk + pb) * a.tc + rank] = j;
          if (w == 0 && a.witness && rank < a.tc) vm_poll += 1;
          pend_ctr = pb;
          // at the end of the chain or of its KV tile the release comes now: the
          // tile switch (dK, dV stores, K, V loads) would hold it back, and under
          // Symmetric Shift every later contributor of the block, one task behind
          // the one before, would wait for its own predecessor's switch in turn
          if (!deferred || nst >= nsteps || tile_ends) {
            vm_wait<0>();  // the copy of the next counter has landed as well
            release();
            vm_poll = 63;
          }
          vm_rel = 0;  // (the witness store, if any, is not counted: the wait only gets longer)
        }
      }
      buf ^= 1;
      st = nst;
    }
    if (cur_j >= 0) store_dkdv(cur_j);
    __syncthreads();  // sm.item is rewritten by the next ticket
  }
  if constexpr (STATS) stats_wave_end(wst, a.wait_stats, l);
}

template <int D, bool CAUSAL>
hipError_t launch_main_mask(const BwdArgs& a, int grid, hipStream_t stream) {
  if (a.G.sched == S_ATOMIC) return launch_main_grid(bwd_main_kernel<D, CAUSAL, kModeAtomic>, a, grid, 256, stream);
  if (a.G.sched == S_PARTIALS) return launch_main_grid(bwd_main_kernel<D, CAUSAL, kModePartials>, a, grid, 256, stream);
  if (a.G.sched == S_SPLIT) return launch_main_grid(bwd_main_kernel<D, CAUSAL, kModeNoDq>, a, grid, 256, stream);
  if (a.nxcd > 0 && a.wait_stats)
    return launch_main_grid(bwd_main_kernel<D, CAUSAL, kModeOrderedXcd, true>, a, grid, 256, stream);
  if (a.nxcd > 0) return launch_main_grid(bwd_main_kernel<D, CAUSAL, kModeOrderedXcd>, a, grid, 256, stream);
  if (a.wait_stats) return launch_main_grid(bwd_main_kernel<D, CAUSAL, kModeOrdered, true>, a, grid, 256, stream);
  return launch_main_grid(bwd_main_kernel<D, CAUSAL, kModeOrdered>, a, grid, 256, stream);
}

template <int D>
hipError_t launch_main(const BwdArgs& a, int grid_main, hipStream_t stream) {
  return a.G.causal ? launch_main_mask<D, true>(a, grid_main, stream) : launch_main_mask<D, false>(a, grid_main, stream);
}

template <int D>
int main_occupancy() {
  int lo = 1 << 30;
  const void* fns[14] = {(const void*)bwd_main_kernel<D, false, kModeAtomic>, (const void*)bwd_main_kernel<D, false, kModeOrdered>,
                         (const void*)bwd_main_kernel<D, false, kModePartials>, (const void*)bwd_main_kernel<D, false, kModeNoDq>,
                         (const void*)bwd_main_kernel<D, false, kModeOrderedXcd>,
                         (const void*)bwd_main_kernel<D, false, kModeOrdered, true>,
                         (const void*)bwd_main_kernel<D, false, kModeOrderedXcd, true>,
                         (const void*)bwd_main_kernel<D, true, kModeAtomic>, (const void*)bwd_main_kernel<D, true, kModeOrdered>,
                         (const void*)bwd_main_kernel<D, true, kModePartials>, (const void*)bwd_main_kernel<D, true, kModeNoDq>,
                         (const void*)bwd_main_kernel<D, true, kModeOrderedXcd>,
                         (const void*)bwd_main_kernel<D, true, kModeOrdered, true>,
                         (const void*)bwd_main_kernel<D, true, kModeOrderedXcd, true>};
  for (const void* f : fns) {
    int blocks = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, f, 256, 0) != hipSuccess) return 0;
    lo = blocks < lo ? blocks : lo;
  }
  return lo;
}

}  // namespace dash
