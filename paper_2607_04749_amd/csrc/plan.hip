// plan.hip -- host planner: tensor table, rank layouts, routing, message
// layouts and the tiled copy tables uploaded for the gfx950 kernels.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <numeric>
#include <stdexcept>
#include <string>

#include "etc_internal.hpp"
#include "plan.hpp"
#include "route.hpp"

namespace etc {

namespace {

int64_t round_up(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

// A layer tensor of an architecture: name, shape, how TP splits it.
struct LayerSpec {
  const char* name;
  int64_t rows, cols;
  Split split;
  bool fused;
};

std::vector<LayerSpec> layer_specs(const etc_model_desc& m) {
  const int64_t h = m.hidden, f = m.ffn_hidden;
  if (m.arch == ETC_ARCH_GPT) {
    // Megatron GPT block: column-parallel QKV and FC1 (weights and biases),
    // row-parallel projection and FC2 (their biases and the norms replicated).
    return {{"ln1.weight", h, 1, kRepl, false},  {"ln1.bias", h, 1, kRepl, false},
            {"qkv.weight", 3 * h, h, kRows, false}, {"qkv.bias", 3 * h, 1, kRows, false},
            {"proj.weight", h, h, kCols, false}, {"proj.bias", h, 1, kRepl, false},
            {"ln2.weight", h, 1, kRepl, false},  {"ln2.bias", h, 1, kRepl, false},
            {"fc1.weight", f, h, kRows, false},  {"fc1.bias", f, 1, kRows, false},
            {"fc2.weight", h, f, kCols, false},  {"fc2.bias", h, 1, kRepl, false}};
  }
  // Llama block: RMSNorms replicated; QKV rows grouped per KV head group;
  // SwiGLU gate and up column-parallel and stored fused; down row-parallel.
  const int64_t head_dim = h / m.num_heads;
  const int64_t qkv_rows = int64_t(m.num_heads + 2 * m.num_kv_heads) * head_dim;
  return {{"norm1.weight", h, 1, kRepl, false}, {"qkv.weight", qkv_rows, h, kRows, false},
          {"proj.weight", h, h, kCols, false},  {"norm2.weight", h, 1, kRepl, false},
          {"gate.weight", f, h, kRows, false},  {"up.weight", f, h, kRows, true},
          {"down.weight", h, f, kCols, false}};
}

}  // namespace

std::vector<LogicalTensor> build_tensor_table(const etc_model_desc& m) {
  std::vector<LogicalTensor> out;
  const bool whole_model = !(m.flags & ETC_F_LAYERS_ONLY);
  auto push = [&](std::string name, int64_t r, int64_t c, Split sp, Home home, int layer,
                  bool tied, bool fused) {
    LogicalTensor t;
    t.name = std::move(name);
    t.rows = r;
    t.cols = c;
    t.split = sp;
    t.home = home;
    t.layer = layer;
    t.tied_dup = tied;
    t.fused = fused;
    out.push_back(std::move(t));
  };
  const int64_t h = m.hidden, V = m.vocab;
  if (whole_model) {
    push("embed", V, h, kRows, kFirstStage, -1, m.tied_embeddings != 0, false);
    if (m.arch == ETC_ARCH_GPT && m.max_pos > 0)
      push("pos_embed", m.max_pos, h, kRepl, kFirstStage, -1, false, false);
  }
  const auto specs = layer_specs(m);
  for (int l = 0; l < m.num_layers; ++l)
    for (const auto& s : specs)
      push("layers." + std::to_string(l) + "." + s.name, s.rows, s.cols, s.split, kOwnLayer, l,
           false, s.fused);
  if (whole_model) {
    if (m.arch == ETC_ARCH_GPT) {
      push("final_ln.weight", h, 1, kRepl, kLastStage, -1, false, false);
      push("final_ln.bias", h, 1, kRepl, kLastStage, -1, false, false);
    } else {
      push("final_norm.weight", h, 1, kRepl, kLastStage, -1, false, false);
    }
    if (!m.tied_embeddings) push("output.weight", V, h, kRows, kLastStage, -1, false, false);
  }
  return out;
}

int stage_of(const LogicalTensor& t, int role, const Grid& g, int num_layers) {
  switch (t.home) {
    case kOwnLayer:
      return role == 0 ? t.layer / (num_layers / g.pp) : -1;
    case kFirstStage:
      if (role == 0) return 0;
      return (t.tied_dup && g.pp > 1) ? g.pp - 1 : -1;
    case kLastStage:
      return role == 0 ? g.pp - 1 : -1;
  }
  return -1;
}

RankLayout build_layout(const std::vector<LogicalTensor>& T, const Grid& g, int num_layers,
                        int rank) {
  RankLayout L;
  const int pp = g.pp_of(rank), tp = g.tp_of(rank);  // every replica has the same layout
  const int nt = int(T.size());
  L.piece_of_tensor[0].assign(nt, -1);
  L.piece_of_tensor[1].assign(nt, -1);
  uint64_t end = 0;
  int last_tensor = -1, last_role = -1;
  for (int role = 0; role < 2; ++role) {
    for (int i = 0; i < nt; ++i) {
      const LogicalTensor& t = T[i];
      if (stage_of(t, role, g, num_layers) != pp) continue;
      Piece p{};
      p.tensor = i;
      p.role = role;
      p.r0 = 0;
      p.r1 = t.rows;
      p.c0 = 0;
      p.c1 = t.cols;
      if (t.split == kRows) {
        p.r0 = tp * (t.rows / g.tp);
        p.r1 = p.r0 + t.rows / g.tp;
      } else if (t.split == kCols) {
        p.c0 = tp * (t.cols / g.tp);
        p.c1 = p.c0 + t.cols / g.tp;
      }
      const bool follows = t.fused && last_tensor == i - 1 && last_role == role;
      p.off = follows ? end : uint64_t(round_up(int64_t(end), 128));
      end = p.off + p.elems();
      L.piece_of_tensor[role][i] = int32_t(L.pieces.size());
      L.pieces.push_back(p);
      last_tensor = i;
      last_role = role;
    }
  }
  L.elems = uint64_t(round_up(int64_t(end), 128));
  return L;
}

// ---------------------------------------------------------------------------

namespace {

void fail(int code, const std::string& msg) { throw PlanError(code, msg); }

void check_inputs(const etc_model_desc& m, const Grid& g, const char* which) {
  if (g.tp < 1 || g.pp < 1 || g.dp < 1)
    fail(ETC_ERR_INVALID_ARG, std::string(which) + ": tp, pp and dp must be >= 1");
  if (int64_t(g.tp) * g.pp * g.dp > 65536) fail(ETC_ERR_UNSUPPORTED, std::string(which) + ": more than 65536 ranks");
  auto need = [&](bool ok, const std::string& what) {
    if (!ok)
      fail(ETC_ERR_INDIVISIBLE, std::string(which) + " (tp=" + std::to_string(g.tp) + ", pp=" +
                                    std::to_string(g.pp) + "): " + what);
  };
  need(m.num_layers % g.pp == 0, "num_layers must divide by pp");
  need(m.hidden % g.tp == 0, "hidden must divide by tp");
  need(m.ffn_hidden % g.tp == 0, "ffn_hidden must divide by tp");
  need(m.num_kv_heads % g.tp == 0, "num_kv_heads must divide by tp (whole KV groups per shard)");
  if (!(m.flags & ETC_F_LAYERS_ONLY)) need(m.vocab % g.tp == 0, "vocab must divide by tp");
}

void check_model(const etc_model_desc& m) {
  if (m.arch != ETC_ARCH_GPT && m.arch != ETC_ARCH_LLAMA) fail(ETC_ERR_INVALID_ARG, "unknown arch");
  if (m.num_layers < 1 || m.hidden < 1 || m.num_heads < 1 || m.num_kv_heads < 1 ||
      m.ffn_hidden < 1)
    fail(ETC_ERR_INVALID_ARG, "model sizes must be positive");
  if (!(m.flags & ETC_F_LAYERS_ONLY) && m.vocab < 1) fail(ETC_ERR_INVALID_ARG, "vocab must be positive");
  if (m.max_pos < 0) fail(ETC_ERR_INVALID_ARG, "max_pos must be >= 0");
  if (m.hidden % m.num_heads || m.num_heads % m.num_kv_heads)
    fail(ETC_ERR_INVALID_ARG, "hidden must divide by num_heads and num_heads by num_kv_heads");
  if (m.arch == ETC_ARCH_GPT && m.num_kv_heads != m.num_heads)
    fail(ETC_ERR_UNSUPPORTED, "GPT blocks have no grouped-query attention");
  if (m.flags & ~uint32_t(ETC_F_LAYERS_ONLY)) fail(ETC_ERR_INVALID_ARG, "unknown model flags");
}


// Source ranks that may send part of tensor t to target d, ascending: a
// superset of those for which routed_span is not empty.  They are the paired
// source, and the ranks on the tensor's stages whose TP shard overlaps d's in
// the replicas that may serve d: replica rep_d mod DP_src alone when no rank
// failed (it always holds the tensor), every replica otherwise (failover).
void candidate_senders(const RouteTensor& t, int d, int home, const RouteCtx& c,
                       std::vector<int>* out) {
  out->clear();
  const int rd = d % (c.tpd * c.ppd);
  const int tp_d = rd % c.tpd, rep_d = d / (c.tpd * c.ppd);
  int tp_lo = 0, tp_hi = c.tps;  // source TP ranks [tp_lo, tp_hi)
  if (t.split != kRepl) {
    const Span need = shard_span(t, tp_d, c.tpd);
    const int64_t w = split_extent(t) / c.tps;
    tp_lo = int(need.lo / w);
    tp_hi = int((need.hi + w - 1) / w);
  }
  const int pt = c.tps * c.pps;
  const int rep_lo = c.failed ? 0 : rep_d % c.dps, rep_hi = c.failed ? c.dps : rep_lo + 1;
  for (int rep = rep_lo; rep < rep_hi; ++rep)
    for (int r = 0; r < 2; ++r)
      if (t.src_stage[r] >= 0)
        for (int tp = tp_lo; tp < tp_hi; ++tp) out->push_back(rep * pt + t.src_stage[r] * c.tps + tp);
  if (home >= 0) out->push_back(home);
  std::sort(out->begin(), out->end());
  out->erase(std::unique(out->begin(), out->end()), out->end());
}

}  // namespace

PlanError::PlanError(int c, std::string m) : std::runtime_error(std::move(m)), code(c) {}

void build_host_plan(etc_plan_t& P) {
  const etc_model_desc& m = P.model;
  P.tensors = build_tensor_table(m);
  const int nt = int(P.tensors.size());
  const int S = P.src.world(), D = P.dst.world();
  if (int(P.home.size()) != D) fail(ETC_ERR_INVALID_ARG, "internal: pairing not set");
  const int Sr = P.src.replica_size(), Dr = P.dst.replica_size();
  P.src_layout.resize(Sr);
  P.dst_layout.resize(Dr);
  for (int s = 0; s < Sr; ++s) P.src_layout[s] = build_layout(P.tensors, P.src, m.num_layers, s);
  for (int d = 0; d < Dr; ++d) P.dst_layout[d] = build_layout(P.tensors, P.dst, m.num_layers, d);

  if (P.route_tensors.size() != size_t(nt)) build_route_tensors(P);

  const RouteCtx ctx = host_route_ctx(P);
  // Route every target piece: per target rank, per piece in arena order, the
  // sources that send part of it.  Messages list boxes in that order.
  P.msgs.clear();
  P.refer.assign(D, {});
  P.refer_elems.assign(D, 0);
  const bool direct_refer = (P.flags & ETC_PLAN_DIRECT_REFER) != 0;
  std::vector<int> cand;
  std::vector<etc_plan_s::Message> to_d;  // messages to the current target, by first box
  for (int d = 0; d < D; ++d) {
    to_d.clear();
    for (const Piece& q : P.dst_lay(d).pieces) {
      const RouteTensor& rt = P.route_tensors[q.tensor];
      uint64_t got = 0;
      candidate_senders(rt, d, P.home[d], ctx, &cand);
      for (const int s : cand) {
        const Span x = routed_span(rt, s, d, P.home[d], ctx);
        if (x.len() == 0) continue;
        etc_plan_s::MsgBox b{};
        b.tensor = q.tensor;
        b.role_d = q.role;
        b.r0 = 0;
        b.r1 = rt.rows;
        b.c0 = 0;
        b.c1 = rt.cols;
        if (rt.split == kRows) {
          b.r0 = x.lo;
          b.r1 = x.hi;
        } else if (rt.split == kCols) {
          b.c0 = x.lo;
          b.c1 = x.hi;
        }
        const uint64_t n = uint64_t((b.r1 - b.r0) * (b.c1 - b.c0));
        got += n;
        if (direct_refer && s == P.home[d]) {  // kept by the paired source: no message
          P.refer[d].push_back(b);
          P.refer_elems[d] += n;
          continue;
        }
        auto it = std::find_if(to_d.begin(), to_d.end(), [&](const etc_plan_s::Message& x) { return x.s == s; });
        if (it == to_d.end()) {
          to_d.emplace_back();
          it = to_d.end() - 1;
          it->s = s;
          it->d = d;
        }
        b.moff = it->npad;
        it->npad += uint64_t(round_up(int64_t(n), 8));
        it->elems += n;
        it->boxes.push_back(b);
      }
      if (got != q.elems())
        fail(ETC_ERR_UNRECOVERABLE, "no live source rank holds part of " + P.tensors[q.tensor].name +
                                        " needed by target rank " + std::to_string(d));
    }
    for (auto& x : to_d) P.msgs.push_back(std::move(x));
  }
  std::sort(P.msgs.begin(), P.msgs.end(), [](const etc_plan_s::Message& a, const etc_plan_s::Message& b) {
    return a.s != b.s ? a.s < b.s : a.d < b.d;
  });
  if (P.msgs.size() > size_t(UINT32_MAX)) fail(ETC_ERR_UNSUPPORTED, "too many messages");
  P.src_first.assign(size_t(S) + 1, 0);
  P.dst_first.assign(size_t(D) + 1, 0);
  for (const auto& x : P.msgs) {
    ++P.src_first[size_t(x.s) + 1];
    ++P.dst_first[size_t(x.d) + 1];
  }
  for (int s = 0; s < S; ++s) P.src_first[s + 1] += P.src_first[s];
  for (int d = 0; d < D; ++d) P.dst_first[d + 1] += P.dst_first[d];
  // a copy launch addresses its peers' messages through a fixed table
  for (int s = 0; s < S; ++s)
    if (P.src_first[s + 1] - P.src_first[s] > uint32_t(ETC_MAX_PEERS))
      fail(ETC_ERR_UNSUPPORTED, "source rank " + std::to_string(s) + " feeds more than ETC_MAX_PEERS targets");
  for (int d = 0; d < D; ++d)
    if (P.dst_first[d + 1] - P.dst_first[d] > uint32_t(ETC_MAX_PEERS))
      fail(ETC_ERR_UNSUPPORTED, "more than ETC_MAX_PEERS sources feed target rank " + std::to_string(d));
  {  // per target, by source: the messages are sorted by source, so a stable fill keeps that order
    std::vector<uint32_t> fill(P.dst_first.begin(), P.dst_first.end() - 1);
    P.dst_msgs.assign(P.msgs.size(), 0);
    for (uint32_t k = 0; k < uint32_t(P.msgs.size()); ++k) P.dst_msgs[fill[size_t(P.msgs[k].d)]++] = k;
  }
  // Send buffers: messages in target order, each at a multiple of 256 bytes;
  // chunk buffers the same, one kind section each.  An empty message takes no
  // room, so its (reported) offset is where the next one would start.
  P.sendbuf_bytes.assign(S, 0);
  for (int i = 0; i < 2; ++i) P.chunk_bytes[i].assign(S, 0);
  for (int s = 0; s < S; ++s) {
    uint64_t cur = 0, cur_k[2] = {0, 0};
    for (uint32_t k = P.src_first[s]; k < P.src_first[s + 1]; ++k) {
      etc_plan_s::Message& x = P.msgs[k];
      x.displ = uint64_t(round_up(int64_t(cur), 256));
      cur = x.displ + x.npad * 14;
      for (int i = 0; i < 2; ++i) {
        x.chunk_displ[i] = uint64_t(round_up(int64_t(cur_k[i]), 256));
        cur_k[i] = x.chunk_displ[i] + x.npad * (i == 0 ? 2 : 4);
      }
    }
    P.sendbuf_bytes[s] = uint64_t(round_up(int64_t(cur), 256));
    for (int i = 0; i < 2; ++i) P.chunk_bytes[i][s] = uint64_t(round_up(int64_t(cur_k[i]), 256));
  }
}

void build_route_tensors(etc_plan_t& P) {
  const int nt = int(P.tensors.size());
  P.route_tensors.resize(nt);
  for (int i = 0; i < nt; ++i) {
    const LogicalTensor& t = P.tensors[i];
    RouteTensor& r = P.route_tensors[i];
    r.rows = t.rows;
    r.cols = t.cols;
    r.split = t.split;
    int copies_src = 0, copies_dst = 0;  // copies within one data-parallel replica
    for (int role = 0; role < 2; ++role) {
      r.src_stage[role] = stage_of(t, role, P.src, P.model.num_layers);
      r.dst_stage[role] = stage_of(t, role, P.dst, P.model.num_layers);
      copies_src += r.src_stage[role] >= 0;
      copies_dst += r.dst_stage[role] >= 0;
    }
    if (t.split == kRepl) {
      copies_src *= P.src.tp;
      copies_dst *= P.dst.tp;
    }
    r.single_copy = copies_src == 1 && copies_dst == 1;
  }
}

RouteCtx host_route_ctx(const etc_plan_t& P) {
  return RouteCtx{P.src.tp, P.src.pp, P.src.dp, P.dst.tp, P.dst.pp, P.dst.dp,
                  P.failed_bits.empty() ? nullptr : P.failed_bits.data()};
}

// COST of one data-parallel replica pair (Sec. III-B, bytes): rows are the
// target ranks of a replica, columns the source ranks of one, COST[d][s] =
// bytes(d) - OVERLAP[s][d] with the interval arithmetic of the cost kernel.
// Every replica pair has this block, since a rank's workload depends only on
// its TP and PP coordinates.
std::vector<uint64_t> host_replica_cost(const etc_plan_t& P) {
  const int Sr = P.src.replica_size(), Dr = P.dst.replica_size();
  std::vector<uint64_t> cost(size_t(Dr) * Sr, 0);
  for (int d = 0; d < Dr; ++d) {
    const int pp_d = P.dst.pp_of(d), tp_d = P.dst.tp_of(d);
    for (int s = 0; s < Sr; ++s) {
      const int pp_s = P.src.pp_of(s), tp_s = P.src.tp_of(s);
      uint64_t need = 0, ov = 0;
      for (const RouteTensor& t : P.route_tensors) {
        if (role_on(t.dst_stage, pp_d) < 0) continue;
        const Span want = shard_span(t, tp_d, P.dst.tp);
        need += uint64_t(want.len() * unit_elems(t));
        if (role_on(t.src_stage, pp_s) < 0) continue;
        const Span have = shard_span(t, tp_s, P.src.tp);
        const Span x{std::max(have.lo, want.lo), std::min(have.hi, want.hi)};
        ov += uint64_t(x.len() * unit_elems(t));
      }
      cost[size_t(d) * Sr + s] = (need - ov) * 14;
    }
  }
  return cost;
}

// The migration sketch (Algorithm 1) with DP isolation (Sec. III-C).  COST is
// infinite across replicas and to failed ranks, so the zero-padded assignment
// over all ranks splits into one assignment per replica that both grids have
// (target replica r with source replica r).  Its pairs of finite cost are the
// pairs of finite cost of the assignment over the whole matrix: every
// cross-replica pair costs the same, and the number of them is forced.
// Replicas without failed ranks share one solution.  Pairs of infinite cost
// (a failed rank) are dropped; targets of replicas the source grid lacks stay
// unpaired.
void sketch_pairing(etc_plan_t& P, const std::vector<char>& dead) {
  const int Sr = P.src.replica_size(), Dr = P.dst.replica_size();
  const int reps = std::min(P.src.dp, P.dst.dp);
  P.home.assign(P.dst.world(), -1);
  const std::vector<uint64_t> base = host_replica_cost(P);
  std::vector<int32_t> base_pair, pair(Dr);
  std::vector<uint64_t> cost;
  for (int r = 0; r < reps; ++r) {
    bool any_dead = false;
    for (int j = 0; j < Sr; ++j) any_dead = any_dead || dead[size_t(r) * Sr + j];
    const uint64_t* C = base.data();
    const int32_t* pr = nullptr;
    if (any_dead) {
      cost = base;
      for (int i = 0; i < Dr; ++i)
        for (int j = 0; j < Sr; ++j)
          if (dead[size_t(r) * Sr + j]) cost[size_t(i) * Sr + j] = ETC_COST_INF;
      solve_sketch(cost.data(), Dr, Sr, pair.data());
      C = cost.data();
      pr = pair.data();
    } else {
      if (base_pair.empty()) {
        base_pair.resize(Dr);
        solve_sketch(base.data(), Dr, Sr, base_pair.data());
      }
      pr = base_pair.data();
    }
    for (int i = 0; i < Dr; ++i)
      if (pr[i] >= 0 && C[size_t(i) * Sr + pr[i]] < uint64_t(ETC_COST_INF)) P.home[r * Dr + i] = r * Sr + pr[i];
  }
}

void validate(const etc_model_desc& m, const etc_parallel_cfg& src, const etc_parallel_cfg& dst) {
  check_model(m);
  check_inputs(m, Grid{src.tp, src.pp, src.dp}, "source config");
  check_inputs(m, Grid{dst.tp, dst.pp, dst.dp}, "target config");
}

}  // namespace etc
