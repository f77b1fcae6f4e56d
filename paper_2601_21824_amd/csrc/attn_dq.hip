// attn_dq.hip -- dQ as a pass of its own: the second pass of the SPLIT
// comparison variant (the related work's deterministic design that splits the
// dK, dV and dQ computations into different passes and reads K, V twice).
//
// One workgroup = 4 waves = 128 query rows; each wave owns 32 rows and loops
// over 64-row K/V blocks staged in LDS, like the forward.  Per wave and block:
//   S^T = K Q^T, dP^T = V dO^T      A = K / V rows (LDS), B = Q / dO of the
//                                   wave's queries (registers)
//   P^T = exp(S^T - L), dS^T = P^T o (dP^T - D)   one query per lane
//   dQ^T += K^T dS^T                A = K^T (LDS), B = dS^T (registers)
// Deterministic without any cross-workgroup reduction: every dQ row is summed
// by one wave in ascending KV order.
#include "common.h"
#include "kernels.h"

namespace dash {

template <int D, bool CAUSAL>
__global__ __launch_bounds__(256) void attn_dq_kernel(BwdArgs a) {
  constexpr int KB = 64;       // kv rows per block
  constexpr int KS = D / 16;   // k-steps over d
  constexpr int NDB = D / 32;  // 32-row blocks of d in dQ^T
  constexpr int KP = D + 8;    // padded bf16 row of Ks / Vs
  constexpr int CPR = D / 8;   // 16-byte chunks per row
  __shared__ __attribute__((aligned(16))) __bf16 Ks[KB * KP];
  __shared__ __attribute__((aligned(16))) __bf16 Vs[KB * KP];
  __shared__ __attribute__((aligned(16))) __bf16 KTs[D * KB];

  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, g = l >> 5, lc = l & 31;
  // one workgroup per (128-row query block, head), query-block major; with a
  // causal mask the longest blocks (last rows) of every head go first
  const int nqb = (a.n + 127) / 128;
  const int qb_i = (int)blockIdx.x / a.bh, bh = (int)blockIdx.x % a.bh;
  const int q0 = (CAUSAL ? nqb - 1 - qb_i : qb_i) * 128, N = a.n;
  const size_t head = (size_t)bh * N * D;
  const uint32_t hbytes = (uint32_t)((size_t)N * D * 2);
  const auto rq = make_rsrc((const __bf16*)a.q + head, hbytes);
  const auto rk = make_rsrc((const __bf16*)a.k + head, hbytes);
  const auto rv = make_rsrc((const __bf16*)a.v + head, hbytes);
  const auto rdo = make_rsrc((const __bf16*)a.dO + head, hbytes);
  const auto rdq = make_rsrc((__bf16*)a.dq + head, hbytes);
  const auto rvec = make_rsrc(a.dvec + (size_t)bh * N, (uint32_t)N * 4);
  const auto rl2 = make_rsrc(a.lse2 + (size_t)bh * N, (uint32_t)N * 4);
  const float c2 = a.scale * kLog2e;

  const int qrow = q0 + 32 * w + lc;
  bf16x8 qreg[KS], doreg[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    qreg[ks] = as_bf16x8(ld16(rq, (uint32_t)(qrow * D + 16 * ks + 8 * g) * 2));
    doreg[ks] = as_bf16x8(ld16(rdo, (uint32_t)(qrow * D + 16 * ks + 8 * g) * 2));
  }
  const float L2 = ld4f(rl2, (uint32_t)qrow * 4);  // L * log2(e) of this lane's query
  const float Dq = ld4f(rvec, (uint32_t)qrow * 4);

  f32x16 dacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) dacc[db][r] = 0.f;

  const int kv_end = CAUSAL ? min(N, q0 + 128) : N;
  for (int kv0 = 0; kv0 < kv_end; kv0 += KB) {
    __syncthreads();
    // K and V rows as they are (A operands of S^T, dP^T) and K transposed
    // (A operand of dQ^T; 4-row slots XOR-swizzled as in the forward's V^T)
#pragma unroll
    for (int unit = tid; unit < 16 * CPR; unit += 256) {
      const int lu_c = unit % CPR, lu_rg = unit / CPR;
      u32x4 kr[4], vr[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const uint32_t off = (uint32_t)((kv0 + 4 * lu_rg + r) * D + 8 * lu_c) * 2;
        kr[r] = ld16(rk, off);
        vr[r] = ld16(rv, off);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        *(u32x4*)&Ks[(4 * lu_rg + r) * KP + 8 * lu_c] = kr[r];
        *(u32x4*)&Vs[(4 * lu_rg + r) * KP + 8 * lu_c] = vr[r];
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int d = 8 * lu_c + e;
        u32x2 t = {pick16(kr[0][e >> 1], kr[1][e >> 1], e & 1), pick16(kr[2][e >> 1], kr[3][e >> 1], e & 1)};
        *(u32x2*)&KTs[d * KB + 4 * (lu_rg ^ tswz(d))] = t;
      }
    }
    __syncthreads();

    f32x16 s[2], dp[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[kb][r] = 0.f;
        dp[kb][r] = 0.f;
      }
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 ak = *(const bf16x8*)&Ks[(32 * kb + lc) * KP + 16 * ks + 8 * g];
        const bf16x8 av = *(const bf16x8*)&Vs[(32 * kb + lc) * KP + 16 * ks + 8 * g];
        s[kb] = mfma32(ak, qreg[ks], s[kb]);
        dp[kb] = mfma32(av, doreg[ks], dp[kb]);
      }
    }
    // s[kb][r], dp[kb][r] <-> key kv0 + 32kb + 8(r/4) + 4g + r%4, query qrow
    const bool need_mask = (kv0 + KB > N) || (CAUSAL && kv0 + KB - 1 > q0 + 32 * w);
    bf16x8 dsb[2][2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kb][r], c2, -L2));
        if (need_mask) {
          const int kv = kv0 + 32 * kb + 8 * (r >> 2) + 4 * g + (r & 3);
          if (kv >= N || (CAUSAL && kv > qrow)) p = 0.f;
        }
        dp[kb][r] = p * (dp[kb][r] - Dq);
      }
      dsb[kb][0] = pack8(dp[kb], 0);
      dsb[kb][1] = pack8(dp[kb], 8);
    }
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const int d = 32 * db + lc;
      const int sw = tswz(d);
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int kb = kk >> 1, half = kk & 1;
        const int ch = (32 * kb + 16 * half + 4 * g) >> 2;
        const u32x2 lo = *(const u32x2*)&KTs[d * KB + 4 * (ch ^ sw)];
        const u32x2 hi = *(const u32x2*)&KTs[d * KB + 4 * ((ch + 2) ^ sw)];
        dacc[db] = mfma32(as_bf16x8(lo, hi), dsb[kb][half], dacc[db]);
      }
    }
  }

  // dacc[db][r] <-> d = 32db + 8(r/4) + 4g + r%4, query qrow
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      const float sc = a.scale;
      u32x2 t = {pack_bf16(dacc[db][4 * rb] * sc, dacc[db][4 * rb + 1] * sc),
                 pack_bf16(dacc[db][4 * rb + 2] * sc, dacc[db][4 * rb + 3] * sc)};
      st8(rdq, (uint32_t)(qrow * D + 32 * db + 8 * rb + 4 * g) * 2, t);
    }
}

hipError_t launch_dq(const BwdArgs& a, int d, hipStream_t stream) {
  const dim3 grid((unsigned)(((a.n + 127) / 128) * a.bh));
  if (d == 64) {
    if (a.G.causal) hipLaunchKernelGGL((attn_dq_kernel<64, true>), grid, dim3(256), 0, stream, a);
    else hipLaunchKernelGGL((attn_dq_kernel<64, false>), grid, dim3(256), 0, stream, a);
  } else {
    if (a.G.causal) hipLaunchKernelGGL((attn_dq_kernel<128, true>), grid, dim3(256), 0, stream, a);
    else hipLaunchKernelGGL((attn_dq_kernel<128, false>), grid, dim3(256), 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace dash
