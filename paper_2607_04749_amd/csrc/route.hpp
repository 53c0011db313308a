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

// Range of the split dim that source s sends to target d for tensor t (empty
// when s sends nothing).  home is the source rank paired with d in the
// migration sketch (the same GPU), or -1.  Rules (Sec. III-D): data the
// paired source already holds stays with it (Refer); any other needed element
// comes from its holder with the smallest key_less key.
__host__ __device__ inline Span routed_span(const RouteTensor& t, int s, int d, int home, int TPs,
                                            int TPd) {
  const Span none{0, 0};
  const int pp_d = d / TPd, tp_d = d % TPd;
  const int role_d = role_on(t.dst_stage, pp_d);
  if (role_d < 0) return none;
  const int pp_s = s / TPs, tp_s = s % TPs;
  if (role_on(t.src_stage, pp_s) < 0) return none;
  const Span need = shard_span(t, tp_d, TPd);
  const Span have = shard_span(t, tp_s, TPs);
  const Span x{have.lo > need.lo ? have.lo : need.lo, have.hi < need.hi ? have.hi : need.hi};
  if (x.len() == 0) return none;
  if (s == home) return x;
  if (home >= 0) {  // does the paired source hold this range?  Then it keeps it.
    const int pp_x = home / TPs, tp_x = home % TPs;
    if (role_on(t.src_stage, pp_x) >= 0) {
      const Span hx = shard_span(t, tp_x, TPs);
      if (hx.lo == have.lo && hx.hi == have.hi) return none;
    }
  }
  // Holders of `have`: per copy role, the rank on that role's stage; for a
  // replicated tensor any TP rank holds it, and the best of them is the one
  // congruent to tp_d.
  const int tpd_mod = tp_d % TPs;
  int best_role = -1, best_tp = 0, best_pp = 0;
  for (int r = 0; r < 2; ++r) {
    const int st = t.src_stage[r];
    if (st < 0) continue;
    const int tp = t.split == kRepl ? tpd_mod : tp_s;
    if (best_role < 0 || key_less(r, tp, st, best_role, best_tp, best_pp, role_d, tpd_mod)) {
      best_role = r;
      best_tp = tp;
      best_pp = st;
    }
  }
  return (best_role >= 0 && best_pp * TPs + best_tp == s) ? x : none;
}

}  // namespace etc
