// Bank-conflict check of the backward kernels' LDS layouts (host build of
// paper_2601_21824_amd/csrc/lds_layout.h).
//
// Bank model of gfx950 (measured with the hardware bank-conflict counter on a
// one-wave probe): 64 banks of 4 bytes; 16-byte-per-lane accesses are served
// in lane groups of 16, 8-byte-per-lane accesses in groups of 32; a group
// costs (largest number of distinct dwords that share one bank) - 1 extra
// cycles.  The lane -> (row, column) mappings below are those of the kernels'
// LDS accesses.  Prints one line per pattern; exits 1 if any kernel pattern
// has a conflict or the model does not reproduce the probe's counts.
#include <cstdio>
#include <map>
#include <set>
#include <vector>
#include "lds_layout.h"

using namespace dash;

static int conflicts(const std::vector<long>& byte_addr, int nbytes) {
  const int per = nbytes == 16 ? 16 : nbytes == 8 ? 32 : 64;
  int total = 0;
  for (int g0 = 0; g0 < 64; g0 += per) {
    std::map<long, std::set<long>> bank;
    for (int l = g0; l < g0 + per; ++l)
      for (int b = 0; b < nbytes / 4; ++b) {
        const long dw = byte_addr[l] / 4 + b;
        bank[dw % 64].insert(dw);
      }
    size_t worst = 0;
    for (auto& kv : bank) worst = kv.second.size() > worst ? kv.second.size() : worst;
    total += (int)worst - 1;
  }
  return total;
}

static int failures = 0;
static void expect(const char* what, int got, int want) {
  std::printf("%-58s %4d (expected %d)\n", what, got, want);
  if (got != want) ++failures;
}

template <int D>
static void tile_patterns(const char* name) {
  const int KS = D / 16, NB = D / 32;
  int rows = 0, tr = 0, dma = 0;
  for (int h = 0; h < 2; ++h)
    for (int ks = 0; ks < KS; ++ks) {  // MFMA row operands
      std::vector<long> a(64);
      for (int l = 0; l < 64; ++l) a[l] = 2L * bf_at<D>(32 * h + (l & 31), 16 * ks + 8 * (l >> 5));
      rows += conflicts(a, 16);
    }
  for (int h = 0; h < 2; ++h)
    for (int k = 0; k < 2 * NB; ++k)  // transposed operands of dV, dK
      for (int dr = 0; dr < 16; dr += 8) {
        std::vector<long> a(64);
        for (int l = 0; l < 64; ++l) {
          const int L16 = l & 15, nh = (l >> 4) & 1, g = l >> 5, nb = k >> 1, half = k & 1;
          a[l] = 2L * bf_at<D>(32 * h + 16 * half + 4 * g + (L16 >> 2) + dr, 32 * nb + 16 * nh + 4 * (L16 & 3));
        }
        tr += conflicts(a, 8);
      }
  {  // the direct loads land row-major in LDS: each lane's 16 bytes at 16 * lane
    std::vector<long> a(64);
    for (int l = 0; l < 64; ++l) a[l] = 16L * l;
    dma += conflicts(a, 16);
  }
  char buf[96];
  std::snprintf(buf, sizeof buf, "%s row operands (per wave and step)", name);
  expect(buf, rows, 0);
  std::snprintf(buf, sizeof buf, "%s transposed operands (per wave and step)", name);
  expect(buf, tr, 0);
}

static void dst_patterns() {
  int wr = 0, rd = 0;
  for (int w = 0; w < 4; ++w)
    for (int p = 0; p < 8; ++p) {  // dS^T stores, piece p
      std::vector<long> a(64);
      const int qb = p >> 2, half = (p >> 1) & 1, part = p & 1;
      for (int l = 0; l < 64; ++l) a[l] = 2L * dst_at(32 * w + (l & 31), 32 * qb + 16 * half + 8 * part + 4 * (l >> 5));
      wr += conflicts(a, 8);
    }
  for (int ks = 0; ks < 8; ++ks)  // transposed reads for dQ^T
    for (int qc = 0; qc < 64; qc += 32)
      for (int dr = 0; dr < 8; dr += 4) {
        std::vector<long> a(64);
        for (int l = 0; l < 64; ++l) {
          const int L16 = l & 15, nh = (l >> 4) & 1, g = l >> 5;
          a[l] = 2L * dst_at(16 * ks + 8 * g + (L16 >> 2) + dr, qc + 16 * nh + 4 * (L16 & 3));
        }
        rd += conflicts(a, 8);
      }
  expect("d<=128 dS^T stores (all waves, per step)", wr, 0);
  expect("d<=128 dS^T transposed reads (per wave and step)", rd, 0);
}

// d = 64 kernel with 256-row KV tiles (attn_bwd64w.hip): the Q / dO patterns
// are tile_patterns<64>'s; new are the dS^T stores of 8 waves' worth of rows
// (64 keys per wave), the K tile's transposed reads (A = K^T of dQ^T) and the
// dS^T transposed reads over 256 keys
static void w64_patterns() {
  int wr = 0, rdk = 0, rdd = 0;
  for (int w = 0; w < 4; ++w)
    for (int kb = 0; kb < 2; ++kb)
      for (int p = 0; p < 8; ++p) {
        std::vector<long> a(64);
        const int qb = p >> 2, half = (p >> 1) & 1, part = p & 1;
        for (int l = 0; l < 64; ++l)
          a[l] = 2L * dst_at(64 * w + 32 * kb + (l & 31), 32 * qb + 16 * half + 8 * part + 4 * (l >> 5));
        wr += conflicts(a, 8);
      }
  for (int ks = 0; ks < 16; ++ks)
    for (int blk = 0; blk < 2; ++blk)  // d block of the K^T operand / query half of dS^T
      for (int dr = 0; dr < 8; dr += 4) {
        std::vector<long> k(64), d(64);
        for (int l = 0; l < 64; ++l) {
          const int L16 = l & 15, nh = (l >> 4) & 1, g = l >> 5;
          const int row = 16 * ks + 8 * g + (L16 >> 2) + dr, col = 32 * blk + 16 * nh + 4 * (L16 & 3);
          k[l] = 2L * bf_at<64>(row, col);
          d[l] = 2L * dst_at(row, col);
        }
        rdk += conflicts(k, 8);
        rdd += conflicts(d, 8);
      }
  expect("d=64 256-row dS^T stores (all waves, per step)", wr, 0);
  expect("d=64 256-row K^T transposed reads (per step, both d blocks)", rdk, 0);
  expect("d=64 256-row dS^T transposed reads (per step, both halves)", rdd, 0);
}

static void d256_patterns() {
  int rows = 0, tr = 0, wr = 0, rd = 0;
  for (int qb = 0; qb < 4; ++qb)
    for (int ks = 0; ks < 8; ++ks) {
      std::vector<long> a(64);
      for (int l = 0; l < 64; ++l) a[l] = 2L * q256_at(16 * qb + (l & 15), 32 * ks + 8 * (l >> 4));
      rows += conflicts(a, 16);
    }
  for (int k = 0; k < 32; ++k)
    for (int dr = 0; dr < 32; dr += 16) {
      std::vector<long> a(64);
      for (int l = 0; l < 64; ++l) {
        const int lr = l & 15, gq = l >> 4, db = k >> 1, kq = k & 1;
        a[l] = 2L * q256_at(32 * kq + 4 * gq + (lr >> 2) + dr, 16 * db + 4 * (lr & 3));
      }
      tr += conflicts(a, 8);
    }
  for (int w = 0; w < 4; ++w)
    for (int qb = 0; qb < 4; ++qb) {
      std::vector<long> a(64);
      for (int l = 0; l < 64; ++l) a[l] = 2L * ds256_at(16 * w + (l & 15), 16 * qb + 4 * (l >> 4));
      wr += conflicts(a, 8);
    }
  for (int kk = 0; kk < 2; ++kk)
    for (int qb = 0; qb < 4; ++qb)
      for (int dr = 0; dr < 8; dr += 4) {
        std::vector<long> a(64);
        for (int l = 0; l < 64; ++l)
          a[l] = 2L * ds256_at(32 * kk + 8 * (l >> 4) + ((l & 15) >> 2) + dr, 16 * qb + 4 * (l & 3));
        rd += conflicts(a, 8);
      }
  expect("d=256 Q/dO row operands (per wave and step)", rows, 0);
  expect("d=256 Q/dO transposed operands (per wave and step)", tr, 0);
  expect("d=256 dS^T stores (all waves, per step)", wr, 0);
  expect("d=256 dS^T transposed reads (per wave and step)", rd, 0);
}

static void probe_patterns() {
  // the probe's measured conflict cycles per instruction
  auto rows_at = [](int period) {
    std::vector<long> a(64);
    for (int l = 0; l < 64; ++l) a[l] = 256L * l + 16 * (period ? l % period : 0);
    return a;
  };
  std::vector<long> lin(64);
  for (int l = 0; l < 64; ++l) lin[l] = 16L * l;
  expect("probe: 16-byte reads, linear", conflicts(lin, 16), 0);
  expect("probe: 16-byte reads, 64 rows at one chunk", conflicts(rows_at(0), 16), 60);
  expect("probe: 16-byte reads, chunk = row % 4", conflicts(rows_at(4), 16), 12);
  expect("probe: 16-byte reads, chunk = row % 8", conflicts(rows_at(8), 16), 4);
  expect("probe: 16-byte reads, chunk = row % 16", conflicts(rows_at(16), 16), 0);
  std::vector<long> tr(64);
  for (int l = 0; l < 64; ++l) {  // transposed-read lane pattern without a swizzle
    const int L16 = l & 15, nh = (l >> 4) & 1, g = l >> 5;
    tr[l] = 256L * (4 * g + (L16 >> 2)) + 2 * (16 * nh + 4 * (L16 & 3));
  }
  expect("probe: 8-byte transposed reads, rows unswizzled", conflicts(tr, 8), 6);
}

int main() {
  probe_patterns();
  tile_patterns<128>("d=128 Q/dO");
  tile_patterns<64>("d=64 Q/dO");
  dst_patterns();
  w64_patterns();
  d256_patterns();
  std::printf(failures ? "FAIL\n" : "OK\n");
  return failures ? 1 : 0;
}
