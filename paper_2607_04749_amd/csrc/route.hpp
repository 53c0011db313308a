// route.hpp -- which source rank sends which part of a tensor to which target
// rank.  Used by the host planner (boxes, message layouts) and by the cost
// matrix kernel (byte counts), so both sides see one definition.
//
// A tensor's TP shards are ranges of its split dim: shard tp of TP covers
// [tp*E/TP, (tp+1)*E/TP) where E is the split dim's extent; a replicated
// tensor is the single range [0, 1) of "whole tensor" units.  Because every
// split is even, two shards of the same TP are equal or disjoint, and the
// intersection of a source shard with a target shard is one range (a whole
// number of LCM(TP_src, TP_dst) slices, Sec. III-C).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "etc_internal.hpp"

namespace etc {

struct Span {
  int64_t lo, hi;
  __host__ __device__ int64_t len() const { return hi > lo ? hi - lo : 0; }
};

__host__ __device__ inline int64_t split_extent(const RouteTensor& t) {
  return t.split == kRows ? t.rows : t.split == kCols ? t.cols : 1;
}

// elements per unit of the split-dim range
__host__ __device__ inline int64_t unit_elems(const RouteTensor& t) {
  return t.split == kRows ? t.cols : t.split == kCols ? t.rows : t.rows * t.cols;
}

__host__ __device__ inline Span shard_span(const RouteTensor& t, int tp, int TP) {
  if (t.split == kRepl) return Span{0, 1};
  const int64_t w = split_extent(t) / TP;
  return Span{tp * w, (tp + 1) * w};
}

// copy role of the tensor held on stage pp (a stage holds at most one role)
__host__ __device__ inline int role_on(const int32_t stage[2], int pp) {
  return stage[0] == pp ? 0 : (stage[1] == pp ? 1 : -1);
}

// Lexicographic key of a candidate sender: prefer the target's own copy role,
// then the TP rank congruent to the target's, then lower stage, lower TP rank.
__host__ __device__ inline bool key_less(int role, int tp, int pp, int best_role, int best_tp,
                                         int best_pp, int role_d, int tpd_mod) {
  const int a0 = role != role_d, b0 = best_role != role_d;
  if (a0 != b0) return a0 < b0;
  const int a1 = tp != tpd_mod, b1 = best_tp != tpd_mod;
  if (a1 != b1) return a1 < b1;
  if (pp != best_pp) return pp < best_pp;
  return tp < best_tp;
}

__host__ __device__ inline bool rank_dead(const RouteCtx& c, int s) {
  return c.failed != nullptr && ((c.failed[s >> 5] >> (s & 31)) & 1u);
}

// Range of the split dim that source s sends to target d for tensor t (empty
// when s sends nothing).  home is the source rank paired with d in the
// migration sketch (the same GPU), or -1.  Rules (Sec. III-D, Sec. III-C):
//  - data the paired source already holds stays with it (Refer);
//  - otherwise target replica j is served by source replica j mod DP_src (kept
//    replicas stay, scale-out replicas are fed round-robin), and within it by
//    the live holder with the smallest key_less key;
//  - if no live rank of that replica holds the data, the next replicas in
//    order stand in (fault tolerance through DP replicas).
// A failed rank sends nothing.  Data with no live holder is routed nowhere;
// the planner reports it as unrecoverable.
__host__ __device__ inline Span routed_span(const RouteTensor& t, int s, int d, int home,
                                            const RouteCtx& c) {
  const Span none{0, 0};
  const int rd = d % (c.tpd * c.ppd);
  const int pp_d = rd / c.tpd, tp_d = rd % c.tpd, rep_d = d / (c.tpd * c.ppd);
  const int role_d = role_on(t.dst_stage, pp_d);
  if (role_d < 0) return none;
  const int pt = c.tps * c.pps;
  const int pp_s = (s % pt) / c.tps, tp_s = s % c.tps;
  if (rank_dead(c, s) || role_on(t.src_stage, pp_s) < 0) return none;
  const Span need = shard_span(t, tp_d, c.tpd);
  const Span have = shard_span(t, tp_s, c.tps);
  const Span x{have.lo > need.lo ? have.lo : need.lo, have.hi < need.hi ? have.hi : need.hi};
  if (x.len() == 0) return none;
  if (s == home) return x;
  if (home >= 0) {  // does the paired source hold this range?  Then it keeps it.
    const int pp_x = (home % pt) / c.tps, tp_x = home % c.tps;
    if (role_on(t.src_stage, pp_x) >= 0) {
      const Span hx = shard_span(t, tp_x, c.tps);
      if (hx.lo == have.lo && hx.hi == have.hi) return none;
    }
  }
  // Holders of `have` in a replica: per copy role, the rank on that role's
  // stage (any TP rank for a replicated tensor); the first replica in serving
  // order with a live holder decides.
  const int tpd_mod = tp_d % c.tps;
  const int r0 = rep_d % c.dps;
  for (int step = 0; step < c.dps; ++step) {
    const int rep = (r0 + step) % c.dps;
    int best_role = -1, best_tp = 0, best_pp = 0;
    for (int r = 0; r < 2; ++r) {
      const int st = t.src_stage[r];
      if (st < 0) continue;
      const int tp_lo = t.split == kRepl ? 0 : tp_s;
      const int tp_hi = t.split == kRepl ? c.tps : tp_s + 1;
      for (int tp = tp_lo; tp < tp_hi; ++tp) {
        if (rank_dead(c, rep * pt + st * c.tps + tp)) continue;
        if (best_role < 0 || key_less(r, tp, st, best_role, best_tp, best_pp, role_d, tpd_mod)) {
          best_role = r;
          best_tp = tp;
          best_pp = st;
        }
      }
    }
    if (best_role >= 0) return (rep * pt + best_pp * c.tps + best_tp == s) ? x : none;
  }
  return none;
}

}  // namespace etc
