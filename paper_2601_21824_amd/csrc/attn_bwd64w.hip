// attn_bwd64w.hip -- the backward main kernel for head dim 64: one KV tile of
// 256 rows per work item, 4 waves of 64 keys each.
//
// The work per 64-row Q block is that of the d = 128 kernel in attn_bwd.hip
// (Algorithm 1's consumer loop, then the ordered dQ reduction), with twice the
// keys per workgroup: the fp32 accumulator, the Q / dO blocks and every fixed
// cost of a step (barriers, counter traffic, the slice wait) are paid once per
// 64 x 256 block pair instead of per 64 x 128, half as often per FLOP.  Wave w
// owns keys [64w, 64w+64) as two 32-key blocks kb; it keeps their K and V rows
// and the dK, dV accumulators in registers, and reads K^T for dQ^T from a copy
// of the K tile in LDS.  Per key block, a step runs four MFMA runs of 8:
//   run 1: S, dP of query half 0 (key block 0: next block's prefetch)
//   run 2: S, dP of query half 1, softmax of half 0 (key block 0: accumulator
//          fetch)
//   run 3: dV, dK += (P, dS of half 0)^T (dO, Q), softmax of half 1
//   run 4: dV, dK of half 1, dS^T into LDS
// then dQ^T of this wave's 32 x 32 tile (one d block, one query half) over
// all 256 keys, and the ordered add of its 4 KB slice.
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "bwd_common.h"
#include "lds_layout.h"

namespace dash {

namespace {

constexpr int kW64Rows = 256;  // KV rows per tile

struct Smem64w {
  static constexpr int BM = kBlockRows, D = 64;
  __bf16 qs[2][BM * D];             // Q block [q][d], double-buffered (bf_at<64>)
  __bf16 dos[2][BM * D];            // dO block
  __bf16 kt[kW64Rows * D];          // K tile [kv][d] (bf_at<64>): K^T operand of dQ^T
  __bf16 dst[kW64Rows * BM];        // dS^T [kv][q] (dst_at)
  float acc[BM * D];                // dQ accumulator block landing pad, per-wave slices in register order
  float ls[2][BM];                  // L * log2(e) per query row
  float ds[2][BM];                  // D per query row
  unsigned steps[kMaxChainSteps];   // this chain's blocks (pack_step)
  int poll[4][64];                  // per wave: the coming block's counter
  int item;
};

template <bool CAUSAL, int MODE, bool STATS = false>
__global__ __launch_bounds__(256) void bwd_main64w_kernel(BwdArgs a) {
  constexpr int D = 64;
  constexpr int BC = kW64Rows;
  constexpr int NW = 4;          // waves
  constexpr int KB = 2;          // 32-key blocks per wave
  constexpr int NT = 256;
  constexpr int BM = kBlockRows;
  constexpr int KS = D / 16;     // k-steps over d
  constexpr int KSC = BC / 16;   // k-steps over the tile's keys
  constexpr int NB = D / 32;     // 32-column blocks of d
  constexpr int CPR = D / 8;     // 16-byte chunks per row
  constexpr int QLD = BM * CPR / NT;  // direct loads per thread for a Q / dO block
  constexpr int KLD = BC * CPR / NT;  // ... for the K tile
  constexpr int NACC = 4;        // the wave's 32 x 32 dQ^T tile: 4 chunks of 1 KB
  static_assert(QLD == 2 && KLD == 8 && BM * D == NW * NACC * 256, "thread/tile shape");
  __shared__ __attribute__((aligned(16))) Smem64w sm;

  const Geom G = a.G;
  const int N = a.n;
  const int tid = threadIdx.x, l = tid & 63, g = l >> 5, lc = l & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int L16 = l & 15, nh = (l >> 4) & 1;  // transposed-read lane roles
  const int dblk = w >> 1, qh0 = w & 1;       // this wave's dQ^T tile: d block, query half
  const float c2 = a.scale * kLog2e;
  const uint32_t hbytes = (uint32_t)((size_t)N * D * 2);
  constexpr bool ordered = MODE == kModeOrdered || MODE == kModeOrderedXcd;
  constexpr bool xcd = MODE == kModeOrderedXcd;
  const int xq = xcd ? xcc_id() : 0;
  const int total = xcd ? (xq < a.nxcd ? xcd_heads(a.bh, a.nxcd, xq) * G.chains : 0) : a.bh * G.chains;
  int* const ticket = &a.ctrl[xcd ? kCtrlXcdTicket + xq : kCtrlTicket];
  const int* const order = a.order + (xcd ? 2 * xq * a.xcd_cap : 0);
  const uint32_t sm_lds = lds_base(&sm);
  auto lds_of = [&](const void* p) { return sm_lds + (uint32_t)((const char*)p - (const char*)&sm); };
  // Shift-type orders: the next contributor to a block reaches it a step or
  // more later, so the counter release waits until the second run of the
  // next step, when the stores have drained without a wait of their own
  const bool deferred = G.sched == S_SHIFT || G.sched == S_SYMSHIFT;
  bool failed = false;
  WaitStats wst;
  if constexpr (STATS) stats_wave_begin(wst);

  for (;;) {
    if (tid == 0) sm.item = atomicAdd(ticket, 1);
    __syncthreads();
    const int item = __builtin_amdgcn_readfirstlane(sm.item);
    if (item >= total) break;
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
    // padded rows of a ragged last block read L = D = 0 (P = 1 there), and
    // their Q and dO rows read 0: they add nothing to dK and dV
    const auto rls = make_rsrc(a.lse2 + (size_t)bh * N, (uint32_t)N * 4);
    const auto rds = make_rsrc(a.dvec + (size_t)bh * N, (uint32_t)N * 4);

    const unsigned* tab = a.steps + (size_t)wch * a.step_cap;
    const int nsteps = __builtin_amdgcn_readfirstlane((int)tab[0]);
    for (int st = tid; st < nsteps; st += NT) sm.steps[st] = tab[1 + st];
    __syncthreads();
    int cur_j = -1;
    bf16x8 kreg[KB][KS], vreg[KB][KS];  // K, V rows of the wave's key blocks (B of S = Q K^T, dP = dO V^T)
    f32x16 dkacc[KB][NB], dvacc[KB][NB];
    int pend_ctr = -1;
    int vm_poll = 63, vm_rel = 63;  // as in the d = 128 kernel: operations since the poll copy / the stores
    bool top_wait = true;

    auto step_at = [&](int st) -> unsigned { return __builtin_amdgcn_readfirstlane(sm.steps[st]); };
    auto next_valid = [&](int st) {
      while (st < nsteps && step_at(st) == kNoStep) ++st;
      return st;
    };
    // part k of block pb's Q and dO rows (32 rows, 4 KB each) into buffer b
    static_assert((NT / CPR) * D * 2 == 4096, "a part is 4 KB");
    auto load_part = [&](int pb, int b, int k) {
      const int r = tid / CPR, c = (tid % CPR) ^ tile_swz<D>(r);
      const uint32_t off = (uint32_t)((pb * BM + r) * D + 8 * c) * 2;
      const uint32_t at = lds_of(&sm.qs[b][64 * w * 8]) + 4096u * k;
      dma16_pair(rq, rdo, at, at + (uint32_t)sizeof(sm.qs), off, 4096u * k);
    };
    auto load_ld = [&](int pb, int b) {
      const uint32_t row = (uint32_t)(pb * BM + fresh_lane());
      if (w == 0) dma4(rls, lds_of(&sm.ls[b][0]), row * 4);
      if (w == 1) dma4(rds, lds_of(&sm.ds[b][0]), row * 4);
    };
    auto load_block = [&](int pb, int b) {
#pragma unroll
      for (int k = 0; k < QLD; ++k) load_part(pb, b, k);
      load_ld(pb, b);
    };
    constexpr int kBlockLoads = 2 * QLD;
    // the ordered accumulator in register order: block pb is BM*D floats at
    // pb*BM*D, wave w's 32 x 32 tile at w*1024, its chunk k of lane l at k*256 + 4l
    // (row 32 qh0 + l%32 of the block, columns 32 dblk + 8k + 4(l/32) .. +3)
    float* acc_w = &sm.acc[w * 1024];
    auto acc_off = [&](int pb, int k) { return (uint32_t)(pb * BM * D + w * 1024 + k * 256 + 4 * l) * 4; };
    auto poll_copy = [&](int pb) { dma4_coherent(rctr, lds_of(&sm.poll[w][0]), (uint32_t)pb * kCtrStride * 4); };
    auto load_acc = [&](int pb) { dma16x4_coherent(racc, lds_of(acc_w), acc_off(pb, 0), 0u); };
    auto store_dkdv = [&](int j) {
      const auto rdk = make_rsrc((__bf16*)a.dk + head, hbytes);
      const auto rdv = make_rsrc((__bf16*)a.dv + head, hbytes);
      const int kv0 = j * BC;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int kv = kv0 + 64 * w + 32 * kb + 8 * (r >> 2) + 4 * g + (r & 3);
            const uint32_t off = (uint32_t)(kv * D + 32 * nb + lc) * 2;
            st2(rdv, off, to_bf16(dvacc[kb][nb][r]));
            st2(rdk, off, to_bf16(dkacc[kb][nb][r] * a.scale));
          }
    };
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

      if (j != cur_j) {  // new KV tile: flush the previous one, load K / V and the K tile
        if (cur_j >= 0) store_dkdv(cur_j);
        cur_j = j;
        const int kv0 = j * BC;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
          const int kvr = kv0 + 64 * w + 32 * kb + lc;
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            kreg[kb][ks] = as_bf16x8(ld16(rk, (uint32_t)(kvr * D + 16 * ks + 8 * g) * 2));
            vreg[kb][ks] = as_bf16x8(ld16(rv, (uint32_t)(kvr * D + 16 * ks + 8 * g) * 2));
          }
        }
        // every wave is past its last dQ^T reads of the previous tile's copy
        __syncthreads();
        {
          const int r = tid / CPR, c = (tid % CPR) ^ tile_swz<D>(r);
          const uint32_t at = lds_of(&sm.kt[64 * w * 8]);
#pragma unroll
          for (int k = 0; k < KLD; ++k)  // rows 32k + r (the swizzle repeats every 16 rows)
            dma16(rk, at + 4096u * k, (uint32_t)((kv0 + 32 * k + r) * D + 8 * c) * 2);
        }
        // wait for the operands here: the K tile is published by the
        // barrier at the top of the step
        vm_wait<0>();
        vm_poll = vm_rel = 63;
        top_wait = true;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              dkacc[kb][nb][r] = 0.f;
              dvacc[kb][nb][r] = 0.f;
            }
      }

      // ---- this block's Q / dO landed (each wave waited for its own loads at
      //      the end of the previous block), so after the barrier all of it is
      //      visible and the other buffer is free
      if (top_wait) {
        vm_wait<0>();
        vm_poll = vm_rel = 63;
      }
      top_wait = false;
      __syncthreads();

      const int nst = next_valid(st + 1);
      const int pb_next = nst < nsteps ? (int)(step_at(nst) & 0xfff) : -1;
      // the chain moves to another KV tile after this step (Symmetric Shift,
      // between its two tiles)
      const bool tile_ends = nst < nsteps && (int)((step_at(nst) >> 12) & 0x1ff) != j;
      int* ctr = ctr_head + (size_t)pb * kCtrStride;
      bool have_turn = false;
      const __bf16* qs = sm.qs[buf];
      const __bf16* dos = sm.dos[buf];
      // LDS reads below are per-lane byte offsets computed once per run from
      // a fresh lane index, plus compile-time offsets: each swizzle depends
      // only on row bits that the compile-time part leaves alone
      const int slf = fresh_lane() & 63;  // this step's lane index, for every LDS address below
      auto at16 = [](const void* base, uint32_t off) { return *(const bf16x8*)((const char*)base + off); };
      auto tr_at = [](const void* base, uint32_t off) { return tr_read((const __bf16*)((const char*)base + off)); };

      // The two key blocks run one after the other, each as the d = 128
      // kernel runs its 32 keys: S/dP of query half 0, S/dP of half 1 with
      // softmax of half 0, dV/dK of half 0 with softmax of half 1, dV/dK of
      // half 1 with its dS^T stores -- so only one key block's S and dP
      // (64 registers) are live at a time.
      //
      // S = Q K^T, dP = dO V^T of query half qb and key block kb: A = Q / dO
      // rows from LDS (all four k-steps read up front), B = K / V rows from
      // registers
      f32x16 s[2], dp[2];
      auto sdp = [&](int qb, int kb, auto&& extra) {
        bf16x8 rq[KS], ro[KS];
        const int lf = slf;
        // row 32qb + lc: rows 32 apart share the swizzle
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const uint32_t off = (uint32_t)bf_at<D>(lf & 31, 16 * ks + 8 * (lf >> 5)) * 2 + 32 * qb * D * 2;
          rq[ks] = at16(qs, off);
          ro[ks] = at16(dos, off);
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          s[qb][r] = 0.f;
          dp[qb][r] = 0.f;
        }
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          __builtin_amdgcn_sched_barrier(0);
          s[qb] = mfma32(rq[ks], kreg[kb][ks], s[qb]);
          dp[qb] = mfma32(ro[ks], vreg[kb][ks], dp[qb]);
          extra(ks);
          __builtin_amdgcn_sched_barrier(0);
        }
      };

      // P = exp(S - L), dS = P (dP - D) of query half qb in 8 pieces: piece k
      // covers row group rb = k/2 (queries 32qb + 8rb + 4g + c, c in {2(k%2),
      // 2(k%2)+1}); L and D of the next row group are read one piece ahead.
      // Element (qb, r) is query 32qb + 8(r/4) + 4g + r%4 and key
      // 64w + 32kb + lc of the tile.  Keys past N need no mask: their K, V
      // rows read as zero and P is at most 1 there.
      const int thr0 = j * BC + 64 * w + lc - q0 - 4 * g;  // causal: masked iff 32qb+8rb+c < thr0 + 32kb
      bf16x8 pbf[2][2], dsbf[2][2];
      f32x4 Lc, Dc, Ln, Dn;
      auto read_ld = [&](int qb, int rb) {
        const int ql = 32 * qb + 8 * rb + 4 * g;
        Ln = *(const f32x4*)&sm.ls[buf][ql];
        Dn = *(const f32x4*)&sm.ds[buf][ql];
      };
      auto softmax_piece = [&](int qb, int kb, int k) {
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
          if (CAUSAL) p = (32 * qb + 8 * rb + c < thr0 + 32 * kb) ? 0.f : p;
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
      // dS^T of key block kb -> LDS, piece k of 8: query half k/4, 16-query
      // half (k/2)%2, 8-byte slot k%2
      auto store_ds_piece = [&](int kb, int k) {
        const int qb = k >> 2, half = (k >> 1) & 1, part = k & 1;
        const u32x4 dv4 = __builtin_bit_cast(u32x4, dsbf[qb][half]);
        const int lf = slf;
        // rows 64w + 32kb + lc share lc's swizzle
        *(u32x2*)((char*)sm.dst + dst_at(lf & 31, 32 * qb + 16 * half + 8 * part + 4 * (lf >> 5)) * 2 +
                  (64 * w + 32 * kb) * BM * 2) =
            part ? u32x2{dv4[2], dv4[3]} : u32x2{dv4[0], dv4[1]};
      };
      // dV += P^T dO and dK += dS^T Q of key block kb, query half qb:
      // A = P^T, dS^T from registers, B = dO^T, Q^T by transposed reads;
      // iteration k = (d block, 16-query half)
      auto dvdk = [&](int qb, int kb, auto&& extra) {
        constexpr int NP = 2 * NB;
        const int lf = slf;
        // rows 32qb + 16half + x and x + 8 (x < 8): the swizzle of x and x + 8
        auto rd = [&](int k, bf16x8* bo, bf16x8* bq) {
          const int nb = k >> 1, half = k & 1;
          const int col = 32 * nb + 16 * ((lf >> 4) & 1) + 4 * (lf & 3);
          const int x = 4 * (lf >> 5) + ((lf & 15) >> 2);
          const uint32_t m = (uint32_t)(32 * qb + 16 * half) * D * 2;
          const uint32_t o0 = (uint32_t)bf_at<D>(x, col) * 2 + m, o1 = (uint32_t)bf_at<D>(x + 8, col) * 2 + m;
          *bo = as_bf16x8(tr_at(dos, o0), tr_at(dos, o1));
          *bq = as_bf16x8(tr_at(qs, o0), tr_at(qs, o1));
        };
        bf16x8 ro[NP], rq[NP];
#pragma unroll
        for (int k = 0; k < NP; ++k) rd(k, &ro[k], &rq[k]);
#pragma unroll
        for (int k = 0; k < NP; ++k) {
          __builtin_amdgcn_sched_barrier(0);
          const int nb = k >> 1, half = k & 1;
          dvacc[kb][nb] = mfma32(pbf[qb][half], ro[k], dvacc[kb][nb]);
          dkacc[kb][nb] = mfma32(dsbf[qb][half], rq[k], dkacc[kb][nb]);
          extra(k);
        }
        __builtin_amdgcn_sched_barrier(0);
      };

      bool early_acc = false;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        // run 1: S/dP of half 0 (key block 0: with the next block's Q / dO /
        // L / D prefetch)
        sdp(0, kb, [&](int ks) {
          if (kb > 0 || pb_next < 0) return;
          if (ks < QLD) load_part(pb_next, buf ^ 1, ks);
          if (ks == 0) load_ld(pb_next, buf ^ 1);
        });
        if (kb == 0) {
          if (pb_next >= 0) {
            const int n = kBlockLoads + (w < 2 ? 1 : 0);
            vm_poll += n;
            vm_rel += n;
          }
          // ---- ordering: this block's counter was copied at the end of the
          //      previous step; with the turn already ours, the slice is
          //      fetched during the next run
          if (ordered && !failed) {
            vm_wait_le(vm_poll);
            const int v0 = __builtin_amdgcn_readfirstlane(sm.poll[w][0]);
            if (v0 >= NW * rank) {
              have_turn = true;
              __atomic_signal_fence(__ATOMIC_SEQ_CST);
            }
          }
          early_acc = ordered && have_turn && rank > 0;
        }
        read_ld(0, 0);
        // run 2: S/dP of half 1, with softmax of half 0 (key block 0: and the
        // accumulator fetch)
        sdp(1, kb, [&](int ks) {
#pragma unroll
          for (int p = 2 * ks; p < 2 * ks + 2; ++p) softmax_piece(0, kb, p);
          if (kb == 0 && early_acc && ks == 0) load_acc(pb);
        });
        if (kb == 0) {
          if (early_acc) vm_rel += NACC;
          // deferred release of the previous block: its stores were followed
          // by vm_rel operations, and vector memory operations complete in order
          if (pend_ctr >= 0) {
            vm_wait_le(vm_rel);
            release();
          }
        }
        // run 3: dV/dK of half 0, with softmax of half 1
        dvdk(0, kb, [&](int k) {
#pragma unroll
          for (int p = 2 * k; p < 2 * k + 2; ++p) softmax_piece(1, kb, p);
        });
        // run 4: dV/dK of half 1, with the dS^T stores
        dvdk(1, kb, [&](int k) {
          if constexpr (MODE != kModeNoDq) {
#pragma unroll
            for (int p = 2 * k; p < 2 * k + 2; ++p) store_ds_piece(kb, p);
          }
        });
      }

      if constexpr (MODE == kModeNoDq) {
        vm_wait<0>();
      } else {
        __syncthreads();

        // ---- dQ^T of this wave's tile (d in [32 dblk, +32), queries
        //      [32 qh0, +32)) = K^T dS^T over the tile's 256 keys: A = K^T by
        //      transposed reads of the K tile, B = dS^T by transposed reads
        f32x16 dq;
#pragma unroll
        for (int r = 0; r < 16; ++r) dq[r] = 0.f;
        {
          constexpr int RING = 4;
          const int lf = slf;
          // keys 16ks + x and x + 4 (x < 12): the K tile's swizzle repeats
          // every 16 rows, dS^T's every 32 (two bases, even and odd ks)
          auto rd = [&](int ks, bf16x8* ka, bf16x8* db) {
            const int x = 8 * (lf >> 5) + ((lf & 15) >> 2), p = ks & 1;
            const int dc = 32 * dblk + 16 * ((lf >> 4) & 1) + 4 * (lf & 3);
            const int qc = 32 * qh0 + 16 * ((lf >> 4) & 1) + 4 * (lf & 3);
            const uint32_t mk = (uint32_t)(16 * ks) * D * 2, md = (uint32_t)(16 * (ks - p)) * BM * 2;
            *ka = as_bf16x8(tr_at(sm.kt, (uint32_t)bf_at<D>(x, dc) * 2 + mk),
                            tr_at(sm.kt, (uint32_t)bf_at<D>(x + 4, dc) * 2 + mk));
            *db = as_bf16x8(tr_at(sm.dst, (uint32_t)dst_at(x + 16 * p, qc) * 2 + md),
                            tr_at(sm.dst, (uint32_t)dst_at(x + 4 + 16 * p, qc) * 2 + md));
          };
          bf16x8 ka[RING], db[RING];
#pragma unroll
          for (int k = 0; k < RING; ++k) rd(k, &ka[k], &db[k]);
#pragma unroll
          for (int ks = 0; ks < KSC; ++ks) {
            __builtin_amdgcn_sched_barrier(0);
            dq = mfma32(ka[ks % RING], db[ks % RING], dq);
            if (ks + RING < KSC) rd(ks + RING, &ka[ks % RING], &db[ks % RING]);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
        // dq[r] <-> query 32 qh0 + lc, column d = 32 dblk + 8(r/4) + 4g + r%4

        if (a.partials) {
          const auto rp = make_rsrc(a.partials + ((size_t)bh * a.tc + j) * N * D, hbytes * 2);
#pragma unroll
          for (int rb = 0; rb < 4; ++rb)
            st16(rp, (uint32_t)((q0 + 32 * qh0 + lc) * D + 32 * dblk + 8 * rb + 4 * g) * 4,
                 __builtin_bit_cast(u32x4, f32x4{dq[4 * rb], dq[4 * rb + 1], dq[4 * rb + 2], dq[4 * rb + 3]}));
        }

        bool add = false;
        if (ordered) {
          if (!have_turn && !failed) {
            if constexpr (STATS) vm_wait<0>();
            const unsigned long long t0 = STATS ? clock_now() : 0ull;
            have_turn = wait_turn(ctr, NW * rank, a.spin_limit);
            if constexpr (STATS) stats_wait(wst, t0);
            if (!have_turn) {
              failed = true;
              __hip_atomic_store(&a.ctrl[kCtrlError], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              if (a.status) __hip_atomic_store(a.status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            } else if (rank > 0) {
              load_acc(pb);  // late fetch: the turn came after the early look
            }
          }
          add = have_turn && rank > 0;
        }
        // this wave's slice (and the next block's Q / dO) have landed
        vm_wait<0>();
        vm_poll = vm_rel = 0;
        if (ordered && pb_next >= 0) poll_copy(pb_next);
        if constexpr (ordered) {
          // ---- add the partial into the slice from registers, one lane per
          //      element: the sum order is the schedule's
          auto finish = [&](auto add_c, auto last_c) {
            constexpr bool kAdd = decltype(add_c)::value, kLast = decltype(last_c)::value;
            f32x4 old[NACC];
            if constexpr (kAdd) {
#pragma unroll
              for (int k = 0; k < NACC; ++k) old[k] = *(const f32x4*)&acc_w[k * 256 + 4 * l];
            }
#pragma unroll
            for (int k = 0; k < NACC; ++k) {
              f32x4 v = {dq[4 * k], dq[4 * k + 1], dq[4 * k + 2], dq[4 * k + 3]};
              if constexpr (kAdd) v = old[k] + v;
              if constexpr (kLast) {
                const auto rdq = make_rsrc((__bf16*)a.dq + head, hbytes);
                const uint32_t off = (uint32_t)((q0 + 32 * qh0 + lc) * D + 32 * dblk + 8 * k + 4 * g);
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
          // ---- the partial goes to KV tile j's own buffer, in the ordered
          //      accumulator's register order
          const auto rpb = make_rsrc(a.dqacc + ((size_t)bh * a.tc + j) * a.nblk * BM * D, (uint32_t)a.nblk * BM * D * 4);
#pragma unroll
          for (int k = 0; k < NACC; ++k)
            st16(rpb, acc_off(pb, k), __builtin_bit_cast(u32x4, f32x4{dq[4 * k], dq[4 * k + 1], dq[4 * k + 2], dq[4 * k + 3]}));
        } else {
          // ---- atomic variant: the tile -> LDS (row-major, 32 rows of 32
          //      floats), then one fp32 atomic per element, each instruction
          //      covering two whole 128-byte row segments of dQacc.  Chunk c
          //      of row rr is staged at c ^ ((rr >> 1) & 7): conflict-free for
          //      the chunk writes and the two-row reads.
#pragma unroll
          for (int k = 0; k < NACC; ++k) {
            const int rr = lc;
            *(f32x4*)&acc_w[(rr * 8 + ((2 * k + g) ^ ((rr >> 1) & 7))) * 4] =
                f32x4{dq[4 * k], dq[4 * k + 1], dq[4 * k + 2], dq[4 * k + 3]};
          }
          asm volatile("" ::: "memory");  // lanes read what other lanes wrote
          const int c = l & 31, hi = l >> 5;
          const int lane_off = hi * D + 32 * dblk + c;
          const int qr0 = q0 + 32 * qh0;
#pragma unroll 8
          for (int k = 0; k < 16; ++k) {
            const float v = acc_w[(2 * k + hi) * 32 + (((c >> 2) ^ (k & 7)) << 2) + (c & 3)];
            float* rows = a.dqacc + head + (size_t)(qr0 + 2 * k) * D;
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
            vm_wait<0>();
            release();
            vm_poll = 63;
          }
          vm_rel = 0;
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

template <bool CAUSAL>
hipError_t launch_mask(const BwdArgs& a, int grid, hipStream_t stream) {
  if (a.G.sched == S_ATOMIC) return launch_main_grid(bwd_main64w_kernel<CAUSAL, kModeAtomic>, a, grid, 256, stream);
  if (a.G.sched == S_PARTIALS) return launch_main_grid(bwd_main64w_kernel<CAUSAL, kModePartials>, a, grid, 256, stream);
  if (a.G.sched == S_SPLIT) return launch_main_grid(bwd_main64w_kernel<CAUSAL, kModeNoDq>, a, grid, 256, stream);
  if (a.nxcd > 0 && a.wait_stats)
    return launch_main_grid(bwd_main64w_kernel<CAUSAL, kModeOrderedXcd, true>, a, grid, 256, stream);
  if (a.nxcd > 0) return launch_main_grid(bwd_main64w_kernel<CAUSAL, kModeOrderedXcd>, a, grid, 256, stream);
  if (a.wait_stats) return launch_main_grid(bwd_main64w_kernel<CAUSAL, kModeOrdered, true>, a, grid, 256, stream);
  return launch_main_grid(bwd_main64w_kernel<CAUSAL, kModeOrdered>, a, grid, 256, stream);
}

}  // namespace

hipError_t launch_main64w(const BwdArgs& a, int grid_main, hipStream_t stream) {
  return a.G.causal ? launch_mask<true>(a, grid_main, stream) : launch_mask<false>(a, grid_main, stream);
}

int bwd_main64w_occupancy() {
  int lo = 1 << 30;
  const void* fns[14] = {
      (const void*)bwd_main64w_kernel<false, kModeAtomic>, (const void*)bwd_main64w_kernel<false, kModeOrdered>,
      (const void*)bwd_main64w_kernel<false, kModePartials>, (const void*)bwd_main64w_kernel<false, kModeNoDq>,
      (const void*)bwd_main64w_kernel<false, kModeOrderedXcd>, (const void*)bwd_main64w_kernel<false, kModeOrdered, true>,
      (const void*)bwd_main64w_kernel<false, kModeOrderedXcd, true>,
      (const void*)bwd_main64w_kernel<true, kModeAtomic>, (const void*)bwd_main64w_kernel<true, kModeOrdered>,
      (const void*)bwd_main64w_kernel<true, kModePartials>, (const void*)bwd_main64w_kernel<true, kModeNoDq>,
      (const void*)bwd_main64w_kernel<true, kModeOrderedXcd>, (const void*)bwd_main64w_kernel<true, kModeOrdered, true>,
      (const void*)bwd_main64w_kernel<true, kModeOrderedXcd, true>};
  for (const void* f : fns) {
    int blocks = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, f, 256, 0) != hipSuccess) return 0;
    lo = blocks < lo ? blocks : lo;
  }
  return lo;
}

}  // namespace dash
