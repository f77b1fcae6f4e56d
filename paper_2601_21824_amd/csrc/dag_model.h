// dag_model.h -- the DAG model of a backward call (Section 3.1), host side.
//
// Section 3.1 models the backward as a DAG over (KV tile, Q tile) tasks: a
// workgroup runs its chain of tasks back to back, every task computes for c
// and then reduces into its dQ tile for r, and a reduction may start only
// after the reduction of the tile's previous contributor in the summation
// order.  Chains are dealt to the workgroups in ticket order and a free
// workgroup takes the next ticket.  The makespan is the critical path of that
// DAG under this list scheduling.
//
// Here the tasks are the kernels' own steps: one 64-row Q block against one
// KV tile (a scheduling Q tile of br rows is br/64 steps, each with its own
// ordering counter), in the order of the step tables the kernels follow, with
// the steps past N left out, and tickets dealt as ticket_chain deals them.
// The library uses the model to pick DASH_SCHED_AUTO's schedule: every
// candidate is simulated with the step time calibrated for it on MI355X
// (model_calibration.h), and the shortest predicted makespan wins.
#pragma once

#include <algorithm>
#include <cmath>
#include <queue>
#include <vector>

#include "schedule.h"

namespace dash {

constexpr int kModelBlockRows = 64;  // rows of a physical Q block (kBlockRows)

// One head's steps: chain w's steps are [off[w], off[w+1]); pred[s] is the step
// whose reduction precedes step s's reduction on the same block (-1: none).
struct HeadDag {
  std::vector<int> off, pred;
};

inline HeadDag build_head_dag(const Geom& G, int N) {
  HeadDag h;
  h.off.assign(G.chains + 1, 0);
  std::vector<int> blk, rnk;
  for (int w = 0; w < G.chains; ++w) {
    const int len = chain_len(G, w);
    for (int t = 0; t < len; ++t) {
      int j, i;
      task(G, w, t, &j, &i);
      for (int s = 0; s < G.nsub; ++s) {
        const int pb = i * G.nsub + s;
        if ((long)pb * kModelBlockRows >= N || (long)j * G.bc >= N) continue;  // the kernels skip it
        blk.push_back(pb);
        rnk.push_back(rank_of(G, i, j));
      }
    }
    h.off[w + 1] = (int)blk.size();
  }
  // each block's contributions in rank order: the previous one is the
  // predecessor (a table over (block, rank): ranks are below T_c and every
  // (block, rank) pair occurs at most once)
  int nb = 0;
  for (int pb : blk) nb = pb + 1 > nb ? pb + 1 : nb;
  const size_t tc = (size_t)G.t_c;
  std::vector<int> at((size_t)nb * tc, -1);
  for (size_t s = 0; s < blk.size(); ++s) at[(size_t)blk[s] * tc + rnk[s]] = (int)s;
  h.pred.assign(blk.size(), -1);
  for (int pb = 0; pb < nb; ++pb) {
    int prev = -1;
    for (size_t r = 0; r < tc; ++r) {
      const int s = at[(size_t)pb * tc + r];
      if (s < 0) continue;
      h.pred[s] = prev;
      prev = s;
    }
  }
  return h;
}

// Makespan of `heads` heads on `workers` workgroups, every step computing for
// c and then reducing for r; tickets as ticket_chain deals them under G's
// chain_major.  Returns -1 if some chain never finishes (a Shift group larger
// than the workgroups: the library refuses such a launch).
inline double simulate_dag(const Geom& G, const HeadDag& hd, int heads, int workers, double c, double r) {
  const int chains = G.chains;
  const long items = (long)heads * chains;
  const int nsteps = (int)hd.pred.size();
  if (items == 0 || nsteps == 0) return 0.0;
  // per (head, step): reduction end time (< 0: not yet) and the chain waiting on it
  std::vector<double> done((size_t)heads * nsteps, -1.0);
  std::vector<long> waiter((size_t)heads * nsteps, -1);
  std::vector<int> at(items, 0);  // per chain instance (ticket): its next step, relative to the chain's first
  struct Ev {
    double t;
    long seq;
    int kind;   // 0: computed, 1: reduced
    long item;  // ticket
    bool operator>(const Ev& o) const { return t != o.t ? t > o.t : seq > o.seq; }
  };
  std::priority_queue<Ev, std::vector<Ev>, std::greater<Ev>> ev;
  long seq = 0, next_item = 0, finished = 0;
  double makespan = 0.0;
  auto chain_of = [&](long item, int* h, int* w) { ticket_chain(G, heads, (int)item, h, w); };
  std::vector<int> item_head(items), item_chain(items);
  for (long x = 0; x < items; ++x) chain_of(x, &item_head[x], &item_chain[x]);
  // a chain starting at time t: its first step, or at once the next ticket if it has none
  auto start = [&](double t) {
    while (next_item < items) {
      const long x = next_item++;
      const int w = item_chain[x];
      if (hd.off[w + 1] > hd.off[w]) {
        ev.push({t + c, seq++, 0, x});
        return;
      }
      ++finished;
    }
  };
  for (int k = 0; k < workers && next_item < items; ++k) start(0.0);
  auto reduce_from = [&](double t, long x) { ev.push({t + r, seq++, 1, x}); };
  while (!ev.empty()) {
    const Ev e = ev.top();
    ev.pop();
    const long x = e.item;
    const int h = item_head[x], w = item_chain[x];
    const int s = hd.off[w] + at[x];
    const size_t hs = (size_t)h * nsteps;
    if (e.kind == 0) {
      const int p = hd.pred[s];
      if (p < 0 || done[hs + p] >= 0.0)
        reduce_from(e.t, x);
      else
        waiter[hs + p] = x;
    } else {
      done[hs + s] = e.t;
      makespan = std::max(makespan, e.t);
      if (waiter[hs + s] >= 0) {
        reduce_from(e.t, waiter[hs + s]);
        waiter[hs + s] = -1;
      }
      if (s + 1 < hd.off[w + 1]) {
        ++at[x];
        ev.push({e.t + c, seq++, 0, x});
      } else {
        ++finished;
        start(e.t);
      }
    }
  }
  return finished == items ? makespan : -1.0;
}

}  // namespace dash
