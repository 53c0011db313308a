// tilewalk.cpp -- host replay of the copy kernels' walks over the copy
// tables the planner builds (pack, unpack and Refer; all kinds at once, one
// sub-chunk of each kind per workgroup; one kind at a time, kind_group(es)
// sub-chunks of kind_sub_elems(es) elements per workgroup).  For every tile it checks that each row stays inside its arena,
// message section or source arena, that vector accesses are 16-byte aligned,
// that a sub-chunk needs no more lanes than a workgroup has, and that the
// writes of a launch cover the target bytes exactly once: each message
// (padding included) for a pack, each target piece for the unpack plus Refer
// of one target.
//
// Test code: it links the library's host planner and its tile geometry
// header; it computes no expected values.
//
// usage: tilewalk arch L h nh nkv ffn V max_pos tied flags  tp pp dp  tp pp dp
//                 refer pairing [failed ...]
//   refer: 1 builds the plan with ETC_PLAN_DIRECT_REFER
//   pairing: "identity", "sketch", or comma-separated pair[d] (-1 = none)
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <string>
#include <vector>
#include "copy_geom.hpp"
#include "plan.hpp"
using namespace etc;
struct Iv { uint64_t lo, hi; };
static int errors = 0;
#define FAIL(...) do { if (errors++ < 20) { fprintf(stderr, __VA_ARGS__); fputc('\n', stderr);} } while (0)

static void merge_equal(std::vector<Iv> w, std::vector<Iv> want, const std::string& what) {
  std::sort(w.begin(), w.end(), [](Iv a, Iv b) { return a.lo < b.lo; });
  for (size_t i = 1; i < w.size(); ++i)
    if (w[i].lo < w[i - 1].hi) { FAIL("%s: overlapping writes", what.c_str()); return; }
  std::vector<Iv> m;
  for (auto x : w) { if (!m.empty() && m.back().hi == x.lo) m.back().hi = x.hi; else m.push_back(x); }
  std::sort(want.begin(), want.end(), [](Iv a, Iv b) { return a.lo < b.lo; });
  std::vector<Iv> mw;
  for (auto x : want) { if (x.hi == x.lo) continue; if (!mw.empty() && mw.back().hi == x.lo) mw.back().hi = x.hi; else mw.push_back(x); }
  if (m.size() != mw.size()) { FAIL("%s: coverage pieces %zu vs %zu", what.c_str(), m.size(), mw.size()); return; }
  for (size_t i = 0; i < m.size(); ++i)
    if (m[i].lo != mw[i].lo || m[i].hi != mw[i].hi) { FAIL("%s: coverage differs", what.c_str()); return; }
}

// padded elements per kind section of message s -> d (0 when empty)
static uint64_t npad_of(const etc_plan_t& P, int s, int d) {
  const auto* m = P.find_msg(s, d);
  return m ? m->npad : 0;
}

// Sort and merge one tile's write intervals, failing on any overlap.
static std::vector<Iv> merge_tile(std::vector<Iv> w, const char* what) {
  std::sort(w.begin(), w.end(), [](Iv a, Iv b) { return a.lo < b.lo; });
  std::vector<Iv> m;
  for (auto x : w) {
    if (x.hi == x.lo) continue;
    if (!m.empty() && x.lo < m.back().hi) { FAIL("%s: sub-chunks of one tile overlap", what); continue; }
    if (!m.empty() && m.back().hi == x.lo) m.back().hi = x.hi; else m.push_back(x);
  }
  return m;
}

// Replay a launch as the kernels run it: for all four kinds, workgroup
// t * kSubPerTile + j copies sub-chunk j (kSubElems elements) of every kind
// of tile t; for one kind of es bytes, workgroup w of kind_grid(ntiles, es)
// copies, when kind_wg_tile(w) gives it tile t and group q, its sub-chunks
// [q * G, (q + 1) * G) of kind_sub_elems(es) elements, G = kind_group(es).
// Either way every sub-chunk of every tile must be copied once per kind in
// the launch.
static void replay_sub(const std::vector<CopyBox>& v, bool pack, bool sectioned, uint32_t kind_mask,
                       uint64_t arena_elems, const std::vector<uint64_t>& peer_bytes,
                       std::vector<std::vector<Iv>> W[4], std::vector<Iv> A[4], bool arenas) {
  const uint32_t nbox = uint32_t(v.size() - 1), ntiles = v.back().tile0;
  const bool all = kind_mask == 0xFu;
  const int kes = kind_mask == 1u ? 2 : 4;  // element size of a one-kind launch
  const uint32_t per_tile = kSubPerTile;  // all-kinds launches
  const uint32_t sub_elems = all ? kSubElems : kind_sub_elems(kes);
  const uint32_t subs_per_tile = kTileElems / sub_elems;
  // one-kind launches: the groups each tile receives, from the whole grid
  std::vector<std::vector<uint32_t>> groups_of;
  if (!all) {
    const uint64_t grid = kind_grid(ntiles, kes);
    if (grid > uint64_t(INT32_MAX)) { FAIL("grid over 2^31 - 1 workgroups"); return; }
    if (grid < uint64_t(ntiles) * kind_wg_per_tile(kes)) FAIL("one-kind grid smaller than the work");
    groups_of.resize(ntiles);
    for (uint64_t w = 0; w < grid; ++w) {
      uint32_t t, q;
      if (!kind_wg_tile(uint32_t(w), ntiles, kes, &t, &q)) continue;  // coverage below catches a wrong refusal
      if (t >= ntiles || q >= kind_wg_per_tile(kes)) { FAIL("workgroup %llu maps outside", (unsigned long long)w); continue; }
      groups_of[t].push_back(q);
    }
  }
  if (uint64_t(ntiles) * per_tile > uint64_t(INT32_MAX)) { FAIL("grid over 2^31 - 1 workgroups"); return; }
  for (uint32_t t = 0; t < ntiles; ++t) {
    const uint32_t bi = box_of_tile(v.data(), nbox, t);  // the same for every j of the tile
    if (bi >= nbox) { FAIL("tile past last box"); return; }
    const CopyBox& b = v[bi];
    const TileGeom g = tile_geom(b, t, v[bi + 1].tile0);
    if (g.nr == 0 || g.nc == 0 || g.r0 >= b.rows || g.c0 >= b.cols) FAIL("empty/outside tile");
    if (!arenas && b.peer >= peer_bytes.size()) { FAIL("peer slot %u out of range", b.peer); return; }
    for (int k = 0; k < 4; ++k) {
      if (!(kind_mask & (1u << k))) continue;
      const int es = k == 0 ? 2 : 4;
      const uint64_t ae = tile_arena_elem(b, g), me = tile_msg_elem(b, g);
      const uint64_t sec = (sectioned && !arenas) ? section_byte(b.msg_npad, k) : 0;
      const uint64_t sec_end = arenas ? peer_bytes[k] : sec + b.msg_npad * es;
      const uint64_t sp = (pack ? uint64_t(b.a_ld) : b.m_ld) * es, dp = (pack ? b.m_ld : uint64_t(b.a_ld)) * es;
      if (!arenas && b.m_ld != b.cols) FAIL("message box with a row stride");
      if (arenas && (b.pad || b.msg_npad)) FAIL("refer box with padding");
      if (std::max(sp, dp) * (g.nr - 1) + uint64_t(g.nc) * es >= (1ull << 31)) FAIL("tile extent over 2^31");
      const bool vk = sub_vectors(b, g, es);
      const uint32_t unit = vk ? 16u / uint32_t(es) : 1u;  // elements per item
      const uint32_t per = sub_elems / unit;               // items per sub-chunk
      const uint32_t ipr = g.nc / unit;                    // items per row
      if (vk && per > kSubThreads) FAIL("a vector sub-chunk needs more lanes than threads");
      if (!all && es != kes) FAIL("one-kind launch of another element size");
      if (vk && g.nc % unit) FAIL("vector rows not whole vectors");
      std::vector<Iv> tw;
      // the sub-chunks of tile t, in the order and with the index arithmetic
      // of the kernels' workgroups
      std::vector<uint32_t> subs;
      if (all) {
        for (uint32_t w = t * per_tile; w < (t + 1) * per_tile; ++w) {
          if (w / kSubPerTile != t) FAIL("workgroup %u maps to another tile", w);
          subs.push_back(w % kSubPerTile);
        }
      } else {
        const uint32_t grp = kind_group(kes);
        for (uint32_t q : groups_of[t])
          for (uint32_t i = 0; i < grp; ++i) subs.push_back(q * grp + i);
      }
      std::vector<char> seen(subs_per_tile, 0);
      for (uint32_t j : subs) {
        if (j >= subs_per_tile || seen[j]++) FAIL("sub-chunk %u of tile %u copied twice or out of range", j, t);
      }
      if (subs.size() != subs_per_tile) FAIL("tile %u: %zu sub-chunks copied, %u in the tile", t, subs.size(),
                                             subs_per_tile);
      for (uint32_t j : subs) {
        if (j >= subs_per_tile) continue;
        uint32_t lo, hi;
        sub_range(j, per, g.nr * ipr, &lo, &hi);
        for (uint32_t r = lo / (ipr ? ipr : 1); lo < hi && r <= (hi - 1) / ipr; ++r) {
          const uint32_t c0 = std::max(lo, r * ipr) - r * ipr, c1 = std::min(hi, (r + 1) * ipr) - r * ipr;
          const uint64_t abase = (ae + uint64_t(r) * b.a_ld) * es, mbase = sec + (me + uint64_t(r) * b.m_ld) * es;
          const uint64_t alo = abase + uint64_t(c0) * unit * es, ahi = abase + uint64_t(c1) * unit * es;
          const uint64_t mlo = mbase + uint64_t(c0) * unit * es, mhi = mbase + uint64_t(c1) * unit * es;
          if (ahi > arena_elems * es) FAIL("arena OOB kind %d", k);
          if ((!arenas && mhi > peer_bytes[b.peer]) || mhi > sec_end) FAIL("message OOB peer %u kind %d", b.peer, k);
          if (vk && (abase % 16 || mbase % 16)) FAIL("vector misaligned kind %d", k);
          tw.push_back(pack ? Iv{mlo, mhi} : Iv{alo, ahi});
        }
      }
      if (pack && g.last && b.pad) {
        const uint64_t plo = sec + (b.m_off + uint64_t(b.rows) * b.cols) * es, phi = plo + uint64_t(b.pad) * es;
        if (phi > sec_end) FAIL("pad overrun");
        tw.push_back({plo, phi});
      }
      for (auto x : merge_tile(tw, "sub-chunk walk")) {
        if (pack) W[k][b.peer].push_back(x); else A[k].push_back(x);
      }
    }
  }
}

// Replay one launch.  peer_bytes[p] = length of peer p's message; W[k][p]
// collects message writes (pack), A[k] arena writes.
static void replay(const std::vector<CopyBox>& v, bool pack, bool sectioned, uint32_t kind_mask,
                   uint64_t arena_elems, const std::vector<uint64_t>& peer_bytes,
                   std::vector<std::vector<Iv>> W[4], std::vector<Iv> A[4], bool arenas = false) {
  if (v.back().tile0 == 0) return;
  if (kind_mask != 0xFu && (kind_mask == 0 || (kind_mask & (kind_mask - 1)))) {
    FAIL("a launch of more than one kind but not all four");
    return;
  }
  replay_sub(v, pack, sectioned, kind_mask, arena_elems, peer_bytes, W, A, arenas);
}

static void check_plan(etc_plan_t& P, const char* name) {
  const int S = P.src.world(), D = P.dst.world();
  for (int sectioned = 1; sectioned >= 0; --sectioned) {
    for (int s = 0; s < S; ++s) {
      std::vector<int32_t> peers; uint64_t bytes;
      auto v = build_pack_boxes(P, s, &peers, &bytes);
      for (int k = 0; k < 4; ++k) {
        const uint32_t mask = sectioned ? 0xFu : (1u << k);
        if (sectioned && k) break;
        std::vector<uint64_t> pb;
        for (int d : peers) pb.push_back(npad_of(P, s, d) * (sectioned ? 14 : (k ? 4 : 2)));
        std::vector<std::vector<Iv>> W[4]; std::vector<Iv> A[4];
        for (int kk = 0; kk < 4; ++kk) W[kk].assign(peers.size(), {});
        replay(v, true, sectioned, mask, P.src_lay(s).elems, pb, W, A);
        for (int kk = 0; kk < 4; ++kk) {
          if (!(mask & (1u << kk))) continue;
          const int es = kk ? 4 : 2;
          for (size_t i = 0; i < peers.size(); ++i) {
            const uint64_t npad = npad_of(P, s, peers[i]);
            const uint64_t b0 = sectioned ? section_byte(npad, kk) : 0;
            merge_equal(W[kk][i], {{b0, b0 + npad * es}}, std::string(name) + " pack s" + std::to_string(s) + " peer " + std::to_string(i));
          }
        }
      }
    }
    for (int d = 0; d < D; ++d) {
      std::vector<int32_t> peers; uint64_t bytes;
      auto v = build_unpack_boxes(P, d, &peers, &bytes);
      for (int k = 0; k < 4; ++k) {
        const uint32_t mask = sectioned ? 0xFu : (1u << k);
        if (sectioned && k) break;
        std::vector<uint64_t> pb;
        for (int s : peers) pb.push_back(npad_of(P, s, d) * (sectioned ? 14 : (k ? 4 : 2)));
        std::vector<std::vector<Iv>> W[4]; std::vector<Iv> A[4];
        replay(v, false, sectioned, mask, P.dst_lay(d).elems, pb, W, A);
        if (P.flags & ETC_PLAN_DIRECT_REFER) {  // Refer writes complete the target
          uint64_t rb = 0;
          auto rv = build_refer_boxes(P, d, &rb);
          const int h = P.home[d];
          if (h < 0 && rv.size() > 1) FAIL("refer boxes without a paired source");
          if (h >= 0) {
            const uint64_t se = P.src_lay(h).elems;
            std::vector<uint64_t> sb = {se * 2, se * 4, se * 4, se * 4};
            std::vector<std::vector<Iv>> RW[4];
            replay(rv, false, false, mask, P.dst_lay(d).elems, sb, RW, A, true);
          }
        }
        for (int kk = 0; kk < 4; ++kk) {
          if (!(mask & (1u << kk))) continue;
          const int es = kk ? 4 : 2;
          std::vector<Iv> want;
          for (auto& q : P.dst_lay(d).pieces) want.push_back({q.off * es, (q.off + q.elems()) * es});
          merge_equal(A[kk], want, std::string(name) + " unpack d" + std::to_string(d));
        }
      }
    }
  }
}


int main(int argc, char** argv) {
  if (argc < 19) {
    fprintf(stderr, "usage: tilewalk arch L h nh nkv ffn V max_pos tied flags tp pp dp tp pp dp refer pairing [failed...]\n");
    return 2;
  }
  etc_model_desc m{};
  int i = 1;
  m.arch = atoi(argv[i++]); m.num_layers = atoi(argv[i++]); m.hidden = atoi(argv[i++]);
  m.num_heads = atoi(argv[i++]); m.num_kv_heads = atoi(argv[i++]); m.ffn_hidden = atoi(argv[i++]);
  m.vocab = atoi(argv[i++]); m.max_pos = atoi(argv[i++]); m.tied_embeddings = atoi(argv[i++]);
  m.flags = atoi(argv[i++]);
  etc_parallel_cfg a{atoi(argv[i]), atoi(argv[i + 1]), atoi(argv[i + 2])};
  etc_parallel_cfg b{atoi(argv[i + 3]), atoi(argv[i + 4]), atoi(argv[i + 5])};
  i += 6;
  const bool refer = atoi(argv[i++]) != 0;
  const std::string pairing = argv[i++];
  etc_plan_t P;
  P.model = m;
  P.src = Grid{a.tp, a.pp, a.dp};
  P.dst = Grid{b.tp, b.pp, b.dp};
  if (refer) P.flags |= ETC_PLAN_DIRECT_REFER;
  try {
    validate(m, a, b);
    const int S = P.src.world(), D = P.dst.world();
    std::vector<char> dead(S, 0);
    if (i < argc) {
      P.failed_bits.assign((S + 31) / 32, 0u);
      for (; i < argc; ++i) {
        const int f = atoi(argv[i]);
        dead[f] = 1;
        P.failed_bits[f >> 5] |= 1u << (f & 31);
      }
    }
    P.tensors = build_tensor_table(m);
    build_route_tensors(P);
    P.home.assign(D, -1);
    if (pairing == "sketch") {
      sketch_pairing(P, dead);
    } else if (pairing == "identity") {
      for (int d = 0; d < D && d < S; ++d)
        if (!dead[d] && P.src.replica(d) == P.dst.replica(d)) P.home[d] = d;
    } else {
      size_t pos = 0;
      for (int d = 0; d < D; ++d) {
        const size_t c = pairing.find(',', pos);
        P.home[d] = atoi(pairing.substr(pos, c == std::string::npos ? std::string::npos : c - pos).c_str());
        pos = c == std::string::npos ? pairing.size() : c + 1;
      }
    }
    build_host_plan(P);
    check_plan(P, "plan");
  } catch (PlanError& e) {
    fprintf(stderr, "plan error %d %s\n", e.code, e.what());
    return 1;
  }
  printf("%s\n", errors ? "ERRORS" : "ok");
  return errors ? 1 : 0;
}
