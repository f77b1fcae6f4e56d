// attn_fwd.hip -- attention forward producing O (bf16) and L = logsumexp (fp32),
// the inputs Algorithm 1 takes.  One workgroup = 4 waves = 128 query rows;
// each wave owns 32 rows and loops over 64-row K/V blocks staged in LDS.
//
// Per wave and KV block: S^T = K Q^T on bf16 MFMA 32x32x16 (the C layout then
// holds one query per lane, so the row max/sum are mostly in-lane), online
// softmax in the log2 domain, O^T += V^T P^T where P^T is fed to the next MFMA
// straight from registers.  Deterministic: every reduction is inside one wave
// in a fixed order.
#include "common.h"
#include "kernels.h"

namespace dash {

template <int D>
__global__ __launch_bounds__(256) void attn_fwd_kernel(FwdArgs a) {
  constexpr int KB = 64;       // kv rows per iteration
  constexpr int KS = D / 16;   // k-steps over d
  constexpr int NDB = D / 32;  // 32-row blocks of d in O^T
  constexpr int KP = D + 8;    // padded row (bf16) of Ks
  __shared__ __attribute__((aligned(16))) __bf16 Ks[KB * KP];
  __shared__ __attribute__((aligned(16))) __bf16 VTs[D * KB];

  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, g = l >> 5, lc = l & 31;
  // causal: the longest query blocks (last rows) are dispatched first
  const int bh = blockIdx.y, q0 = (a.causal ? gridDim.x - 1 - blockIdx.x : blockIdx.x) * 128, N = a.n;
  const size_t head = (size_t)bh * N * D;
  const uint32_t hbytes = (uint32_t)((size_t)N * D * 2);
  const auto rq = make_rsrc((const __bf16*)a.q + head, hbytes);
  const auto rk = make_rsrc((const __bf16*)a.k + head, hbytes);
  const auto rv = make_rsrc((const __bf16*)a.v + head, hbytes);
  const auto ro = make_rsrc((__bf16*)a.o + head, hbytes);
  const auto rl = make_rsrc(a.lse + (size_t)bh * N, (uint32_t)N * 4);
  const float c2 = a.scale * kLog2e;

  const int qrow = q0 + 32 * w + lc;
  bf16x8 qreg[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) qreg[ks] = as_bf16x8(ld16(rq, (uint32_t)(qrow * D + 16 * ks + 8 * g) * 2));

  f32x16 oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[db][r] = 0.f;
  float m = -INFINITY, lsum = 0.f;

  const int kv_end = a.causal ? min(N, q0 + 128) : N;
  // loader unit: 4 rows x 8 columns; 16 * CPR units per KV block
  constexpr int CPR = D / 8;

  for (int kv0 = 0; kv0 < kv_end; kv0 += KB) {
    __syncthreads();
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
      for (int r = 0; r < 4; ++r) *(u32x4*)&Ks[(4 * lu_rg + r) * KP + 8 * lu_c] = kr[r];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int d = 8 * lu_c + e;
        u32x2 t = {pick16(vr[0][e >> 1], vr[1][e >> 1], e & 1), pick16(vr[2][e >> 1], vr[3][e >> 1], e & 1)};
        *(u32x2*)&VTs[d * KB + 4 * (lu_rg ^ tswz(d))] = t;
      }
    }
    __syncthreads();

    f32x16 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kb][r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 ak = *(const bf16x8*)&Ks[(32 * kb + lc) * KP + 16 * ks + 8 * g];
        s[kb] = mfma32(ak, qreg[ks], s[kb]);
      }
    }
    // s[kb][r] <-> key kv0 + 32kb + 8(r/4) + 4g + r%4, query qrow
    const bool need_mask = (kv0 + KB > N) || (a.causal && kv0 + KB - 1 > q0 + 32 * w);
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float x = s[kb][r] * c2;
        if (need_mask) {
          const int kv = kv0 + 32 * kb + 8 * (r >> 2) + 4 * g + (r & 3);
          if (kv >= N || (a.causal && kv > qrow)) x = -INFINITY;
        }
        s[kb][r] = x;
        mx = fmaxf(mx, x);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float mnew = fmaxf(m, mx);
    const float alpha = exp2f(m - mnew);
    float rs = 0.f;
    bf16x8 pb[2][2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = exp2f(s[kb][r] - mnew);
        s[kb][r] = p;
        rs += p;
      }
      pb[kb][0] = pack8(s[kb], 0);
      pb[kb][1] = pack8(s[kb], 8);
    }
    rs += __shfl_xor(rs, 32);
    lsum = lsum * alpha + rs;
    m = mnew;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[db][r] *= alpha;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const int d = 32 * db + lc;
      const int sw = tswz(d);
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int kb = kk >> 1, half = kk & 1;
        const int ch = (32 * kb + 16 * half + 4 * g) >> 2;
        const u32x2 lo = *(const u32x2*)&VTs[d * KB + 4 * (ch ^ sw)];
        const u32x2 hi = *(const u32x2*)&VTs[d * KB + 4 * ((ch + 2) ^ sw)];
        oacc[db] = mfma32(as_bf16x8(lo, hi), pb[kb][half], oacc[db]);
      }
    }
  }

  // oacc[db][r] <-> d = 32db + 8(r/4) + 4g + r%4, query qrow
  const float inv = 1.f / lsum;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      const int d = 32 * db + 8 * rb + 4 * g;
      u32x2 t = {pack_bf16(oacc[db][4 * rb] * inv, oacc[db][4 * rb + 1] * inv),
                 pack_bf16(oacc[db][4 * rb + 2] * inv, oacc[db][4 * rb + 3] * inv)};
      st8(ro, (uint32_t)(qrow * D + d) * 2, t);
    }
  if (g == 0) st4f(rl, (uint32_t)qrow * 4, (m + __log2f(lsum)) * kLn2);
}

hipError_t launch_attn_fwd(const FwdArgs& a, int d, hipStream_t stream) {
  dim3 grid((a.n + 127) / 128, a.bh);
  if (d == 64)
    hipLaunchKernelGGL(attn_fwd_kernel<64>, grid, dim3(256), 0, stream, a);
  else if (d == 128)
    hipLaunchKernelGGL(attn_fwd_kernel<128>, grid, dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(attn_fwd_kernel<256>, grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace dash
