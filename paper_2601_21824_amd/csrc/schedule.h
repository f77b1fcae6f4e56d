// schedule.h -- closed-form dQ-reduction schedules, usable on host and device.
//
// One attention head of N rows is cut into KV tiles of BC rows (kv_tile_rows:
// one workgroup's resident K_j, V_j, dK_j, dV_j)
// and scheduling Q tiles of br rows;
// a scheduling Q tile is processed as br/64 physical 64-row blocks, each with
// its own ordering counter.  A workgroup runs a "chain" of tasks (KV tile j,
// Q tile i); the dQ partials of Q tile i are added in the order rank(i, j).
//
//  NAIVE       -- ascending Q tiles; dQ summed in ascending KV order
//                 (the deterministic baseline analysed in Section 3.2).
//  DESCENDING  -- Descending Q-Tile Iteration (Section 3.3): Q tiles from last
//                 to first, summation order unchanged (ascending KV).
//  SHIFT       -- Shift Scheduling (Section 3.4, full mask): workgroup j visits
//                 Q tiles (j*g + t) mod T_r, g = T_r / T_c; the summation order is
//                 the visiting order, so rank = (i/g - j) mod T_c.  A head with
//                 more than kMaxGroup KV tiles is split into groups of kMaxGroup
//                 consecutive tiles whose chains must run at the same time; the
//                 order is group-major and the visiting order within a group.
//  SYMSHIFT    -- Symmetric Shift (Section 3.4, causal): workgroup p owns KV tiles
//                 p and T-1-p (T even, h = T/2).  Phase 1 (steps 0..h-1): Q tile
//                 h + (p+t) mod h with KV p (dense lower-left rectangle).  Phase 2
//                 (steps h..2h): KV p over Q tiles p..h-1 top-down, then KV T-1-p
//                 over Q tiles T-1 down to T-1-p.  The summation order is the
//                 visiting order: rank = i-j for i < h; for i >= h,
//                 (i-h-j) mod h when j < h and j when j >= h.
//  ATOMIC      -- NAIVE's iteration order, unordered fp32 atomic adds.
//  PARTIALS    -- NAIVE's iteration order; each partial goes to its own
//                 buffer and a second kernel sums them in ascending KV order.
//
// Padding: with a causal mask every schedule uses br = BC; T_r = g*T_c always
// (Q tiles past N are empty and skipped); SYMSHIFT rounds T up to even with an
// empty KV/Q tile, which touches no real dQ tile.
#pragma once

#if defined(__HIPCC__)
#define DASH_HD __host__ __device__ inline
#else
#define DASH_HD inline
#endif

namespace dash {

// S_PARTIALS runs NAIVE's chains and writes every partial to its own buffer
// S_SPLIT runs NAIVE's chains for dK, dV only; dQ is a separate pass
enum Sched { S_ATOMIC = 0, S_NAIVE = 1, S_DESCENDING = 2, S_SHIFT = 3, S_SYMSHIFT = 4, S_PARTIALS = 6, S_SPLIT = 7 };

constexpr int kBlockRows = 64;  // rows of a physical Q block (one counter each)
constexpr int kTileKV = 128;    // KV rows per tile of the d = 128 kernel
constexpr int kMaxGroup = 256;  // Shift: KV-tile chains that must be co-resident
constexpr int kXcdGroup = 32;   // ... under XCD-local placement (one XCD's resident workgroups)

struct Geom {
  int sched;   // Sched
  int causal;  // 0/1
  int bc;      // rows per KV tile (kv_tile_rows)
  int br;      // rows per scheduling Q tile (64, or bc when causal)
  int g;       // bc / br
  int t_c;     // KV tiles per head (SYMSHIFT: rounded up to even)
  int t_r;     // scheduling Q tiles per head (= g * t_c)
  int nsub;    // physical 64-row blocks per scheduling Q tile (= br / 64)
  int chains;  // workgroup chains per head
  int grp;     // SHIFT: chains per group (others: = chains)
  int chain_major;  // work tickets chain-major (see ticket_chain), else head-major
};

// rows per KV tile: 128 at d = 128, 64 at d = 256.  At d = 64, 256 (the
// 256-row kernel, half the accumulator traffic per FLOP) when the call has
// KV tiles enough to keep a 256-CU GPU busy -- at least 256 of them over all
// `heads` heads for a full mask, 512 and N >= 1024 for a causal one (whose
// chains are uneven) -- else 128.  The tile size is part of the summation
// order, so it is a function of the problem (d, mask, N, heads) alone, never
// of the device.
DASH_HD int kv_tile_rows(int d, int causal, int N, long heads) {
  if (d == 64) {
    const long wide = heads * (long)((N + 255) / 256);
    return (causal ? (N >= 1024 && wide >= 512) : wide >= 256) ? 256 : 128;
  }
  return d == 128 ? 128 : 64;
}

DASH_HD Geom make_geom(int sched, int causal, int N, int d, long heads) {
  Geom G;
  G.sched = sched;
  G.causal = causal ? 1 : 0;
  G.bc = kv_tile_rows(d, causal, N, heads);
  G.br = causal ? G.bc : kBlockRows;
  G.g = G.bc / G.br;
  G.t_c = (N + G.bc - 1) / G.bc;
  if (sched == S_SYMSHIFT) G.t_c += G.t_c & 1;
  G.t_r = G.g * G.t_c;
  G.nsub = G.br / kBlockRows;
  G.chains = sched == S_SYMSHIFT ? G.t_c / 2 : G.t_c;
  G.grp = (sched == S_SHIFT && G.chains > kMaxGroup) ? kMaxGroup : G.chains;
  G.chain_major = 0;  // the library picks the ticket order per call (device-dependent)
  return G;
}

// first Q tile that interacts with KV tile j
DASH_HD int first_q(const Geom& G, int j) { return G.causal ? (j * G.bc) / G.br : 0; }

DASH_HD bool interacts(const Geom& G, int i, int j) {
  return !G.causal || (i + 1) * G.br - 1 >= j * G.bc;
}

// number of KV tiles whose partials are summed into Q tile i
DASH_HD int contributors(const Geom& G, int i) {
  if (!G.causal) return G.t_c;
  int c = ((i + 1) * G.br - 1) / G.bc + 1;
  return c < G.t_c ? c : G.t_c;
}

DASH_HD int chain_len(const Geom& G, int w) {
  if (G.sched == S_SYMSHIFT) return G.t_r + 1;
  if (G.sched == S_SHIFT) return G.t_r;
  return G.t_r - first_q(G, w);
}

DASH_HD int pmod(int a, int m) {
  int r = a % m;
  return r < 0 ? r + m : r;
}

// t-th task of chain w: KV tile *j, Q tile *i
DASH_HD void task(const Geom& G, int w, int t, int* j, int* i) {
  switch (G.sched) {
    case S_DESCENDING:
      *j = w;
      *i = G.t_r - 1 - t;
      return;
    case S_SHIFT:
      *j = w;
      *i = pmod(w * G.g + t, G.t_r);
      return;
    case S_SYMSHIFT: {
      const int h = G.t_r / 2;
      if (t < h) {
        *j = w;
        *i = h + pmod(w + t, h);
      } else if (t - h <= h - 1 - w) {
        *j = w;
        *i = w + (t - h);
      } else {
        *j = G.t_r - 1 - w;
        *i = 3 * h - 1 - (t - h) - w;
      }
      return;
    }
    default:  // NAIVE, ATOMIC
      *j = w;
      *i = first_q(G, w) + t;
      return;
  }
}

// XCD-local placement: every chain of head bh runs on XCD bh % nxcd, from
// that XCD's own ticket queue.  A Shift group must then fit one XCD's resident workgroups: groups of at most kXcdGroup
// chains, which the XCD runs one after another (the group-major order of
// rank_of).  The other schedules' orders do not depend on the placement.
DASH_HD void place_on_xcds(Geom& G) {
  if (G.sched == S_SHIFT && G.grp > kXcdGroup) G.grp = kXcdGroup;
}

// heads of XCD x (of nxcd) under XCD-local placement: x, x + nxcd, ...
DASH_HD int xcd_heads(int heads, int nxcd, int x) { return x < heads ? (heads - x + nxcd - 1) / nxcd : 0; }

// XCD x's work ticket t -> (head, chain), head-major or chain-major over the
// XCD's own heads as ticket_chain
DASH_HD void ticket_chain_xcd(const Geom& G, int heads, int nxcd, int x, int t, int* bh, int* w) {
  const int hx = xcd_heads(heads, nxcd, x);
  int k;
  if (G.chain_major) {
    *w = t / hx;
    k = t % hx;
  } else {
    k = t / G.chains;
    *w = t % G.chains;
  }
  *bh = x + nxcd * k;
}

// Work ticket -> (head, chain).  Head-major (all chains of a head in a row,
// as Shift and Symmetric Shift need them together) or, for the schedules whose
// waits only point to lower KV tiles, chain-major (G.chain_major): chain w of
// every head before chain w+1, i.e. the longest chains first across heads
// under a causal mask (longest-processing-time order).  Either way every chain
// a wait points to has a lower ticket.
DASH_HD void ticket_chain(const Geom& G, int heads, int item, int* bh, int* w) {
  if (G.chain_major) {
    *w = item / heads;
    *bh = item % heads;
  } else {
    *bh = item / G.chains;
    *w = item % G.chains;
  }
}

// position of KV tile j in Q tile i's summation order
DASH_HD int rank_of(const Geom& G, int i, int j) {
  switch (G.sched) {
    case S_SHIFT: {
      // group-major; inside a group (tiles j0 .. j0+s-1) the visiting order:
      // with a = i/g and u = (a - j0) mod T_c, tile j0+v visits Q tile i at
      // step ((a - j0 - v) mod T_c) * g + i % g, so it comes after the tiles
      // v' in (v, min(u, s-1)] when v <= u, else after all v' <= u and v' > v
      const int j0 = j - j % G.grp;
      const int sz = G.t_c - j0 < G.grp ? G.t_c - j0 : G.grp;
      const int v = j - j0, u = pmod(i / G.g - j0, G.t_c);
      const int top = u < sz - 1 ? u : sz - 1;
      return j0 + (v <= u ? top - v : u + sz - v);
    }
    case S_SYMSHIFT: {
      const int h = G.t_r / 2;
      if (i < h) return i - j;
      return j < h ? pmod(i - h - j, h) : j;
    }
    default:
      return j;
  }
}

}  // namespace dash
