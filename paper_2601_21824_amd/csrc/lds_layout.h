// lds_layout.h -- where the backward kernels keep bf16 tiles in LDS.
//
// The LDS of gfx950 has 64 banks of 4 bytes.  A read of 16 bytes per lane is
// served 16 lanes at a time (lanes 0-15, 16-31, 32-47, 48-63); a read or write
// of 8 bytes per lane (ds_read_b64, ds_read_b64_tr_b16, ds_write_b64) 32 lanes
// at a time.  Lanes of one group that touch different dwords in the same bank
// cost one extra cycle each.  (Measured with the hardware bank-conflict
// counter on a one-wave probe of fixed address patterns.)
//
// Each swizzle below puts the lanes of every group of every access the
// kernels make on distinct banks; a host test checks them against this model
// with the kernels' lane mappings.  Functions are usable on host and device.
#pragma once

#if defined(__HIPCC__)
#define DASH_LDS_HD __host__ __device__ inline
#else
#define DASH_LDS_HD inline
#endif

namespace dash {

// ---- d = 64 / 128 kernel: [rows][D] bf16 tiles (the Q and dO blocks)
// 16-byte chunk c of row r is stored at chunk c ^ tile_swz<D>(r).  Accesses:
//  * MFMA row operands: lane l reads row 32h + l%32, chunk 2k + l/32
//    (16 consecutive rows at one chunk per lane group);
//  * transposed operands (ds_read_b64_tr_b16): lanes 0-31 read rows
//    r0 .. r0+3 (r0 a multiple of 4), 4 chunks of 8-byte halves each.
// D = 128 (256-byte rows, one per bank cycle): rows r .. r+15 must map to 16
// distinct chunks, and rows r0 .. r0+3 to distinct chunk quads.
// D = 64 (128-byte rows, two per bank cycle): the same over row pairs.
template <int D>
DASH_LDS_HD int tile_swz(int r);
template <>
DASH_LDS_HD int tile_swz<128>(int r) {
  return ((r & 3) << 2) | ((r >> 2) & 3);
}
template <>
DASH_LDS_HD int tile_swz<64>(int r) {
  return ((r >> 1) & 1) | (((r >> 2) & 1) << 1) | ((((r >> 1) ^ (r >> 3)) & 1) << 2);
}
// element index of (row r, column col) in a [rows][D] bf16 tile
template <int D>
DASH_LDS_HD int bf_at(int r, int col) {
  return r * D + (((col >> 3) ^ tile_swz<D>(r)) << 3) + (col & 7);
}

// ---- d = 64 / 128 kernel: dS^T tile [kv][64 q] bf16
// 8-byte slot s (4 queries) of row r is stored at slot s ^ dst_swz(r).
// Writes: lane l of wave w writes row 32w + l%32 at slot 2p + l/32 for piece
// p (32 rows per lane group); transposed reads: rows r0 .. r0+3 x 4 slots per
// lane group.
DASH_LDS_HD int dst_swz(int r) {
  return ((r >> 1) & 7) | ((((r >> 1) ^ (r >> 4)) & 1) << 3);
}
// element index of (kv row r, query q), q a multiple of 4
DASH_LDS_HD int dst_at(int r, int q) {
  return r * 64 + (((q >> 2) ^ dst_swz(r)) << 2);
}

// ---- d = 256 kernel: [64][256] bf16 Q / dO tiles (512-byte rows)
// Row operands: lane l reads row 16h + l%16 at chunk 4k + l/16; transposed
// operands: lanes 0-31 read rows r0 .. r0+7 (r0 a multiple of 8), two chunks
// each.
DASH_LDS_HD int q256_swz(int r) {
  return (r & 7) | ((((r >> 3) ^ r) & 1) << 3);
}
DASH_LDS_HD int q256_at(int r, int col) {
  return r * 256 + (((col >> 3) ^ q256_swz(r)) << 3) + (col & 7);
}

// ---- d = 256 kernel: dS^T [64 kv][64 q] bf16, 8-byte slots
DASH_LDS_HD int ds256_swz(int r) {
  const int m = (r >> 1) & 7;
  return 2 * (((m & 1) << 2) | (m >> 1));
}
DASH_LDS_HD int ds256_at(int r, int q) {
  return r * 64 + (((q >> 2) ^ ds256_swz(r)) << 2) + (q & 3);
}

}  // namespace dash
