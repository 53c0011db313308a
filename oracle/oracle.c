/*
 * oracle.c -- CPU reference for checkpoint-free resharding of model states.
 *
 * TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.  Only the test suite, the
 * smoke check and the CPU-baseline leg of the benchmark load this library.
 * It shares no code, header, table or constant with the GPU library; the two
 * agree only because both follow the same paper and the same written
 * readings of it.  Plain, slow, single-threaded loops, chosen to be checked
 * by eye against the paper.
 *
 * What it computes (paper: "Direct Model State Migration for Elastic Training
 * of Large Language Models"):
 *  - Workloads (Sec. III-B, cost matrix paragraph): the list of logical tensor
 *    pieces each rank holds under a (TP, PP) configuration, derived locally
 *    from Megatron's even static partition rules (Sec. III-B, last paragraph
 *    before "Migration Sketch").
 *  - TP workloads at LCM(tp_prev, tp_curr) granularity, one item per slice
 *    (Sec. III-C, "Workload Abstraction and Cost Matrix of TP").
 *  - Cost c_ij = len(curr_i) - len(curr_i intersect prev_j) (Sec. III-B),
 *    counted in bytes over the four state kinds.
 *  - Send / Recv / Refer (Sec. III-D, "Migration Instructions"): a piece
 *    held by both sides of a pair stays (Refer); otherwise it is received
 *    from the source that the sender rule names.
 *  - States by workload type (Sec. III-D): bf16 parameter, fp32 master,
 *    fp32 Adam m, fp32 Adam v, packed when sent and unpacked after.
 *  - Placement-aware remapping of the virtual rank allocator (Sec. III-E,
 *    Algorithm 2).
 *  - The migration result itself: the plain definition.  Materialize each
 *    full logical tensor from the resident source shards (replicas must agree
 *    bit for bit), then cut every destination piece and every message box out
 *    of it.
 *
 * Readings where the paper is silent (rank order, stage split, per-tensor TP
 * split, arena layout, sender of a replicated element, wire format) are the
 * ones listed in the design notes; each is restated where it is used below.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#define ORC_ARCH_GPT 0
#define ORC_ARCH_LLAMA 1
#define ORC_LAYERS_ONLY 1

#define ORC_REPL 0 /* every TP rank of the stage holds the whole tensor */
#define ORC_ROWS 1 /* dim 0 split evenly over TP                      */
#define ORC_COLS 2 /* dim 1 split evenly over TP                      */

#define ORC_AT_FIRST 0 /* first pipeline stage (embeddings)          */
#define ORC_AT_LAYER 1 /* the stage owning the tensor's layer        */
#define ORC_AT_LAST 2  /* last pipeline stage (final norm, head)     */

#define ORC_OK 0
#define ORC_EINVAL -1
#define ORC_EINDIV -2
#define ORC_ERANK -3
#define ORC_EUNSUP -5
#define ORC_ENOMEM -6
#define ORC_EMISMATCH -10 /* replicas disagree                          */
#define ORC_EUNCOVERED -11 /* a needed element is held by no resident source */
#define ORC_EBOX -12 /* routed elements do not form one box          */
#define ORC_EUNRECOVERABLE -8 /* a needed element survives on no source rank */

/* cost between ranks of different data-parallel replicas (Sec. III-C: the
 * workload difference across DP ranks is taken as infinite) */
#define ORC_COST_INF ((uint64_t)1 << 50)

#define ORC_NKIND 4
#define ORC_ALIGN_ELEMS 128
#define ORC_MSG_ALIGN_BYTES 256
#define ORC_BOX_PAD_ELEMS 8

/* element size of each state kind: bf16 param, fp32 master, fp32 m, fp32 v */
static const int ESIZE[ORC_NKIND] = {2, 4, 4, 4};
#define BYTES_PER_ELEM 14

typedef struct {
  int32_t arch, num_layers, hidden, num_heads, num_kv_heads, ffn_hidden, vocab,
      max_pos, tied, flags;
} orc_model;

typedef struct {
  int32_t tp, pp, dp;
} orc_cfg;

/* Routing inputs beyond the two configurations: the migration sketch
 * (pair[d] = old rank paired with new rank d, or -1; NULL = identity), the
 * old ranks whose states are lost (failed[0..num_failed)), and direct_refer:
 * when non-zero, what a target's paired source keeps (Refer, Sec. III-D)
 * travels in no message (it stays on that GPU), so that message is empty. */
typedef struct {
  const int32_t* pair;
  const int32_t* failed;
  int32_t num_failed;
  int32_t direct_refer;
} orc_route;

typedef struct {
  char name[48];
  int64_t rows, cols;
  int32_t split;
  int32_t layer;      /* -1 for non-layer tensors            */
  int32_t where;      /* ORC_AT_*                             */
  int32_t tied_copy;  /* duplicate on the last stage if PP>1  */
  int32_t fused_prev; /* stored directly after the previous tensor */
} orc_tensor;

typedef struct {
  int32_t tensor, role;
  int64_t r0, r1, c0, c1; /* box in full-tensor coordinates          */
  uint64_t off;           /* arena element offset of its first element */
} orc_piece;

typedef struct {
  int32_t tensor, role_d; /* destination piece's tensor and copy role */
  int64_t r0, r1, c0, c1; /* routed box in full-tensor coordinates    */
  uint64_t moff;          /* element offset inside each kind section   */
} orc_mbox;

/* ------------------------------------------------------------------------ */
/* logical tensor table                                                      */
/* ------------------------------------------------------------------------ */

static int add_tensor(orc_tensor* out, int n, const char* name, int64_t rows,
                      int64_t cols, int split, int layer, int where,
                      int tied_copy, int fused_prev) {
  if (out) {
    orc_tensor* t = &out[n];
    memset(t, 0, sizeof *t);
    snprintf(t->name, sizeof t->name, "%s", name);
    t->rows = rows;
    t->cols = cols;
    t->split = split;
    t->layer = layer;
    t->where = where;
    t->tied_copy = tied_copy;
    t->fused_prev = fused_prev;
  }
  return n + 1;
}

/* The logical (TP=1, PP=1) tensors of the model, in the order they sit in a
 * rank's arena.  Vectors are stored as [n, 1].  Per-tensor TP split follows
 * Megatron: column-parallel weights and their biases split on dim 0,
 * row-parallel weights on dim 1, norms and row-parallel biases replicated.
 * Attention QKV rows are interleaved per KV group ([q heads of g; k_g; v_g]),
 * so a TP shard is a contiguous dim-0 chunk.  The SwiGLU first projection is
 * two logical tensors (gate, up), stored fused gate-shard then up-shard. */
static int build_tensors(const orc_model* m, orc_tensor* out) {
  int n = 0;
  const int64_t h = m->hidden, f = m->ffn_hidden, V = m->vocab;
  const int embed = !(m->flags & ORC_LAYERS_ONLY);
  char nm[48];
  if (embed) {
    n = add_tensor(out, n, "embed", V, h, ORC_ROWS, -1, ORC_AT_FIRST, m->tied, 0);
    if (m->arch == ORC_ARCH_GPT && m->max_pos > 0)
      n = add_tensor(out, n, "pos_embed", m->max_pos, h, ORC_REPL, -1,
                     ORC_AT_FIRST, 0, 0);
  }
  for (int l = 0; l < m->num_layers; ++l) {
#define T(suffix, r, c, sp, fu)                                     \
  do {                                                              \
    snprintf(nm, sizeof nm, "layers.%d.%s", l, suffix);             \
    n = add_tensor(out, n, nm, r, c, sp, l, ORC_AT_LAYER, 0, fu);   \
  } while (0)
    if (m->arch == ORC_ARCH_GPT) {
      T("ln1.weight", h, 1, ORC_REPL, 0);
      T("ln1.bias", h, 1, ORC_REPL, 0);
      T("qkv.weight", 3 * h, h, ORC_ROWS, 0);
      T("qkv.bias", 3 * h, 1, ORC_ROWS, 0);
      T("proj.weight", h, h, ORC_COLS, 0);
      T("proj.bias", h, 1, ORC_REPL, 0);
      T("ln2.weight", h, 1, ORC_REPL, 0);
      T("ln2.bias", h, 1, ORC_REPL, 0);
      T("fc1.weight", f, h, ORC_ROWS, 0);
      T("fc1.bias", f, 1, ORC_ROWS, 0);
      T("fc2.weight", h, f, ORC_COLS, 0);
      T("fc2.bias", h, 1, ORC_REPL, 0);
    } else {
      const int64_t hd = h / m->num_heads;
      const int64_t qkv_rows = (int64_t)(m->num_heads + 2 * m->num_kv_heads) * hd;
      T("norm1.weight", h, 1, ORC_REPL, 0);
      T("qkv.weight", qkv_rows, h, ORC_ROWS, 0);
      T("proj.weight", h, h, ORC_COLS, 0);
      T("norm2.weight", h, 1, ORC_REPL, 0);
      T("gate.weight", f, h, ORC_ROWS, 0);
      T("up.weight", f, h, ORC_ROWS, 1);
      T("down.weight", h, f, ORC_COLS, 0);
    }
#undef T
  }
  if (embed) {
    if (m->arch == ORC_ARCH_GPT) {
      n = add_tensor(out, n, "final_ln.weight", h, 1, ORC_REPL, -1, ORC_AT_LAST, 0, 0);
      n = add_tensor(out, n, "final_ln.bias", h, 1, ORC_REPL, -1, ORC_AT_LAST, 0, 0);
    } else {
      n = add_tensor(out, n, "final_norm.weight", h, 1, ORC_REPL, -1, ORC_AT_LAST, 0, 0);
    }
    if (!m->tied)
      n = add_tensor(out, n, "output.weight", V, h, ORC_ROWS, -1, ORC_AT_LAST, 0, 0);
  }
  return n;
}

/* ------------------------------------------------------------------------ */
/* configuration checks                                                      */
/* ------------------------------------------------------------------------ */

/* The paper requires the layer count to divide PP and the hidden size to
 * divide TP (Sec. IV-A, models paragraph).  Every other dim that TP splits
 * must divide too, and a QKV shard must hold whole KV groups. */
static int check_cfg(const orc_model* m, const orc_cfg* c) {
  if (c->tp < 1 || c->pp < 1 || c->dp < 1) return ORC_EINVAL;
  if (m->num_layers % c->pp) return ORC_EINDIV;
  if (m->hidden % c->tp || m->ffn_hidden % c->tp) return ORC_EINDIV;
  if (m->num_kv_heads % c->tp) return ORC_EINDIV;
  if (!(m->flags & ORC_LAYERS_ONLY) && m->vocab % c->tp) return ORC_EINDIV;
  return ORC_OK;
}

static int check_model(const orc_model* m) {
  if (m->arch != ORC_ARCH_GPT && m->arch != ORC_ARCH_LLAMA) return ORC_EINVAL;
  if (m->num_layers < 1 || m->hidden < 1 || m->num_heads < 1 ||
      m->num_kv_heads < 1 || m->ffn_hidden < 1)
    return ORC_EINVAL;
  if (!(m->flags & ORC_LAYERS_ONLY) && m->vocab < 1) return ORC_EINVAL;
  if (m->hidden % m->num_heads || m->num_heads % m->num_kv_heads) return ORC_EINVAL;
  if (m->arch == ORC_ARCH_GPT && m->num_kv_heads != m->num_heads) return ORC_EINVAL;
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* placement: which stage holds a tensor in a copy role, which box a TP rank */
/* holds                                                                     */
/* ------------------------------------------------------------------------ */

/* Stage holding (tensor, role), or -1.  Layers go to stages in contiguous
 * equal blocks; the embedding lives on the first stage and, when tied and
 * PP > 1, a duplicate (copy role 1) lives on the last stage. */
static int stage_of(const orc_model* m, const orc_cfg* c, const orc_tensor* t, int role) {
  if (t->where == ORC_AT_LAYER) return role == 0 ? t->layer / (m->num_layers / c->pp) : -1;
  if (t->where == ORC_AT_FIRST) {
    if (role == 0) return 0;
    return (t->tied_copy && c->pp > 1) ? c->pp - 1 : -1;
  }
  return role == 0 ? c->pp - 1 : -1;
}

static void box_of(const orc_tensor* t, int tp, int TP, int64_t* r0, int64_t* r1,
                   int64_t* c0, int64_t* c1) {
  *r0 = 0;
  *r1 = t->rows;
  *c0 = 0;
  *c1 = t->cols;
  if (t->split == ORC_ROWS) {
    *r0 = tp * (t->rows / TP);
    *r1 = *r0 + t->rows / TP;
  } else if (t->split == ORC_COLS) {
    *c0 = tp * (t->cols / TP);
    *c1 = *c0 + t->cols / TP;
  }
}

static int64_t align_up(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

/* Rank = dp * (PP * TP) + pp * TP + tp: TP fastest, then PP, each data-
 * parallel replica a contiguous block of ranks. */
static void coords(const orc_cfg* c, int rank, int* pp, int* tp) {
  const int in_replica = rank % (c->pp * c->tp);
  *pp = in_replica / c->tp;
  *tp = in_replica % c->tp;
}

static int replica_of(const orc_cfg* c, int rank) { return rank / (c->pp * c->tp); }

/* A rank's arena: role-0 pieces in tensor order, then role-1 pieces.  Each
 * local tensor starts at a multiple of 128 elements; a fused tensor (up after
 * gate) follows its predecessor with no gap.  Same element offsets for all
 * four kinds.  Returns the number of pieces; *arena_elems gets the arena
 * length (end rounded up to 128 elements). */
static int layout(const orc_model* m, const orc_cfg* c, const orc_tensor* T, int nt,
                  int rank, orc_piece* out, uint64_t* arena_elems) {
  int pp, tp, n = 0;
  coords(c, rank, &pp, &tp);
  int64_t cursor = 0;
  int prev_tensor = -2, prev_role = -1;
  for (int role = 0; role < 2; ++role) {
    for (int t = 0; t < nt; ++t) {
      if (stage_of(m, c, &T[t], role) != pp) continue;
      orc_piece p;
      p.tensor = t;
      p.role = role;
      box_of(&T[t], tp, c->tp, &p.r0, &p.r1, &p.c0, &p.c1);
      int64_t start = (T[t].fused_prev && prev_tensor == t - 1 && prev_role == role)
                          ? cursor
                          : align_up(cursor, ORC_ALIGN_ELEMS);
      p.off = (uint64_t)start;
      cursor = start + (p.r1 - p.r0) * (p.c1 - p.c0);
      if (out) out[n] = p;
      ++n;
      prev_tensor = t;
      prev_role = role;
    }
  }
  if (arena_elems) *arena_elems = (uint64_t)align_up(cursor, ORC_ALIGN_ELEMS);
  return n;
}

/* ------------------------------------------------------------------------ */
/* context                                                                   */
/* ------------------------------------------------------------------------ */

typedef struct {
  orc_model m;
  orc_cfg src, dst;
  int S, D, nt;
  int32_t* home;  /* home[d]: source rank paired with target d (the same GPU), or -1 */
  int direct_refer; /* Refer data travels in no message */
  char* failed;   /* failed[s]: source rank s lost its states */
  orc_tensor* T;
  int* ns;           /* pieces per source rank      */
  orc_piece** ps;    /* pieces of each source rank  */
  uint64_t* s_elems; /* arena length per source rank */
  int* nd;
  orc_piece** pd;
  uint64_t* d_elems;
} ctx_t;

static void ctx_free(ctx_t* x) {
  if (!x) return;
  for (int s = 0; x->ps && s < x->S; ++s) free(x->ps[s]);
  for (int d = 0; x->pd && d < x->D; ++d) free(x->pd[d]);
  free(x->ps);
  free(x->pd);
  free(x->ns);
  free(x->nd);
  free(x->s_elems);
  free(x->d_elems);
  free(x->T);
  free(x->home);
  free(x->failed);
  memset(x, 0, sizeof *x);
}

/* route: pairing and failed ranks (NULL = identity pairing, no failures).
 * Under the identity pairing target d pairs with source d when both exist
 * and source d is alive and in the same data-parallel replica.  A given
 * pairing never names a failed rank; it may join ranks of different replicas
 * (every replica holds the same states), which a coalesced pairing does
 * (Sec. III-E). */
static int ctx_init(ctx_t* x, const orc_model* m, const orc_cfg* src, const orc_cfg* dst,
                    const orc_route* route) {
  const int32_t* pair = route ? route->pair : NULL;
  memset(x, 0, sizeof *x);
  int rc = check_model(m);
  if (rc) return rc;
  if ((rc = check_cfg(m, src))) return rc;
  if ((rc = check_cfg(m, dst))) return rc;
  x->m = *m;
  x->src = *src;
  x->dst = *dst;
  x->S = src->tp * src->pp * src->dp;
  x->D = dst->tp * dst->pp * dst->dp;
  x->nt = build_tensors(m, NULL);
  x->T = calloc((size_t)x->nt, sizeof(orc_tensor));
  x->ns = calloc((size_t)x->S, sizeof(int));
  x->nd = calloc((size_t)x->D, sizeof(int));
  x->ps = calloc((size_t)x->S, sizeof(orc_piece*));
  x->pd = calloc((size_t)x->D, sizeof(orc_piece*));
  x->s_elems = calloc((size_t)x->S, sizeof(uint64_t));
  x->d_elems = calloc((size_t)x->D, sizeof(uint64_t));
  if (!x->T || !x->ns || !x->nd || !x->ps || !x->pd || !x->s_elems || !x->d_elems) {
    ctx_free(x);
    return ORC_ENOMEM;
  }
  build_tensors(m, x->T);
  x->home = calloc((size_t)x->D, sizeof(int32_t));
  x->failed = calloc((size_t)x->S, 1);
  if (!x->home || !x->failed) {
    ctx_free(x);
    return ORC_ENOMEM;
  }
  x->direct_refer = route ? route->direct_refer : 0;
  for (int i = 0; route && i < route->num_failed; ++i) {
    if (route->failed[i] < 0 || route->failed[i] >= x->S) {
      ctx_free(x);
      return ORC_EINVAL;
    }
    x->failed[route->failed[i]] = 1;
  }
  for (int d = 0; d < x->D; ++d) {
    if (pair) {
      x->home[d] = pair[d];
    } else {
      x->home[d] = -1;
      if (d < x->S && !x->failed[d] && replica_of(src, d) == replica_of(dst, d)) x->home[d] = d;
    }
    if (x->home[d] < -1 || x->home[d] >= x->S) {
      ctx_free(x);
      return ORC_EINVAL;
    }
    if (x->home[d] >= 0 && x->failed[x->home[d]]) {
      ctx_free(x);
      return ORC_EINVAL;
    }
    for (int e = 0; e < d; ++e)
      if (x->home[d] >= 0 && x->home[e] == x->home[d]) {
        ctx_free(x);
        return ORC_EINVAL; /* a source can be paired with one target at most */
      }
  }
  for (int s = 0; s < x->S; ++s) {
    x->ns[s] = layout(m, src, x->T, x->nt, s, NULL, NULL);
    x->ps[s] = calloc((size_t)x->ns[s] + 1, sizeof(orc_piece));
    if (!x->ps[s]) { ctx_free(x); return ORC_ENOMEM; }
    layout(m, src, x->T, x->nt, s, x->ps[s], &x->s_elems[s]);
  }
  for (int d = 0; d < x->D; ++d) {
    x->nd[d] = layout(m, dst, x->T, x->nt, d, NULL, NULL);
    x->pd[d] = calloc((size_t)x->nd[d] + 1, sizeof(orc_piece));
    if (!x->pd[d]) { ctx_free(x); return ORC_ENOMEM; }
    layout(m, dst, x->T, x->nt, d, x->pd[d], &x->d_elems[d]);
  }
  return ORC_OK;
}

static int64_t piece_elems(const orc_piece* p) { return (p->r1 - p->r0) * (p->c1 - p->c0); }

static int in_box(const orc_piece* p, int64_t r, int64_t c) {
  return r >= p->r0 && r < p->r1 && c >= p->c0 && c < p->c1;
}

/* ------------------------------------------------------------------------ */
/* the sender rule                                                           */
/* ------------------------------------------------------------------------ */

/* Which source rank sends element (r, c) of tensor t to destination d that
 * needs it in copy role role_d.  The paper pairs ranks and keeps what both
 * sides of a pair hold in place (Refer): the source paired with d keeps
 * whatever it already holds.  Any other element has several
 * possible senders only when it is replicated (TP-replicated tensors, the
 * tied embedding copy); the reading taken here picks the holder with the
 * smallest key (role differs from role_d, tp differs from tp_d mod TP_src,
 * pp, tp), which spreads replicas round-robin the way the paper spreads DP
 * scale-out sources.  Holders are found by scanning every source rank's
 * pieces.  Returns -1 if no source holds the element. */
static int sender_of_element(const ctx_t* x, int d, int role_d, int t, int64_t r, int64_t c) {
  const int h = x->home[d];
  if (h >= 0) {
    for (int i = 0; i < x->ns[h]; ++i) {
      const orc_piece* p = &x->ps[h][i];
      if (p->tensor == t && in_box(p, r, c)) return h;
    }
  }
  int pp_d, tp_d;
  coords(&x->dst, d, &pp_d, &tp_d);
  /* data-parallel isolation: target replica j is served by source replica
   * j mod DP_src (kept replicas stay, scale-out replicas round-robin); if no
   * live rank of that replica holds the element, the next replicas in order
   * stand in for it (fault tolerance through DP replicas, Sec. III-C) */
  const int r0 = replica_of(&x->dst, d) % x->src.dp;
  for (int step = 0; step < x->src.dp; ++step) {
    const int rep = (r0 + step) % x->src.dp;
    int best = -1;
    int bk[4] = {0, 0, 0, 0};
    for (int s = 0; s < x->S; ++s) {
      if (x->failed[s] || replica_of(&x->src, s) != rep) continue;
      for (int i = 0; i < x->ns[s]; ++i) {
        const orc_piece* p = &x->ps[s][i];
        if (p->tensor != t || !in_box(p, r, c)) continue;
        int pp_s, tp_s;
        coords(&x->src, s, &pp_s, &tp_s);
        int k[4] = {p->role != role_d, tp_s != tp_d % x->src.tp, pp_s, tp_s};
        int less = best < 0;
        for (int j = 0; j < 4 && !less; ++j) {
          if (k[j] != bk[j]) {
            less = k[j] < bk[j];
            break;
          }
        }
        if (less) {
          best = s;
          memcpy(bk, k, sizeof k);
        }
      }
    }
    if (best >= 0) return best;
  }
  return -1;
}

/* ------------------------------------------------------------------------ */
/* LCM workload items (Sec. III-C)                                           */
/* ------------------------------------------------------------------------ */

static int64_t gcd64(int64_t a, int64_t b) {
  while (b) {
    int64_t t = a % b;
    a = b;
    b = t;
  }
  return a;
}

/* Number of workload items a tensor has: LCM(TP_src, TP_dst) slices of the
 * split dim, or one item for a replicated tensor. */
static int64_t n_items(const ctx_t* x, const orc_tensor* t) {
  if (t->split == ORC_REPL) return 1;
  int64_t a = x->src.tp, b = x->dst.tp;
  return a / gcd64(a, b) * b;
}

/* Does (pp, tp) of config c hold item a of tensor t in copy role `role`? */
static int holds_item(const ctx_t* x, const orc_cfg* c, int pp, int tp, const orc_tensor* t,
                      int role, int64_t a) {
  if (stage_of(&x->m, c, t, role) != pp) return 0;
  if (t->split == ORC_REPL) return 1;
  int64_t per = n_items(x, t) / c->tp;
  return a >= tp * per && a < (tp + 1) * per;
}

/* The sender rule evaluated on a whole item (all its elements share holders). */
static int sender_of_item(const ctx_t* x, int d, int role_d, const orc_tensor* t, int64_t a) {
  const int h = x->home[d];
  if (h >= 0) {
    int pp, tp;
    coords(&x->src, h, &pp, &tp);
    if (holds_item(x, &x->src, pp, tp, t, 0, a) || holds_item(x, &x->src, pp, tp, t, 1, a))
      return h;
  }
  int pp_d, tp_d;
  coords(&x->dst, d, &pp_d, &tp_d);
  const int r0 = replica_of(&x->dst, d) % x->src.dp;
  for (int step = 0; step < x->src.dp; ++step) {
    const int rep = (r0 + step) % x->src.dp;
    int best = -1;
    int bk[4] = {0, 0, 0, 0};
    for (int s = 0; s < x->S; ++s) {
      if (x->failed[s] || replica_of(&x->src, s) != rep) continue;
      int pp_s, tp_s;
      coords(&x->src, s, &pp_s, &tp_s);
      for (int role = 0; role < 2; ++role) {
        if (!holds_item(x, &x->src, pp_s, tp_s, t, role, a)) continue;
        int k[4] = {role != role_d, tp_s != tp_d % x->src.tp, pp_s, tp_s};
        int less = best < 0;
        for (int j = 0; j < 4 && !less; ++j) {
          if (k[j] != bk[j]) {
            less = k[j] < bk[j];
            break;
          }
        }
        if (less) {
          best = s;
          memcpy(bk, k, sizeof k);
        }
      }
    }
    if (best >= 0) return best;
  }
  return -1;
}

/* Copies of a tensor inside one data-parallel replica of a configuration:
 * copy roles times TP ranks holding it. */
static int multiplicity(const ctx_t* x, const orc_cfg* c, const orc_tensor* t) {
  int roles = (stage_of(&x->m, c, t, 0) >= 0) + (stage_of(&x->m, c, t, 1) >= 0);
  return roles * (t->split == ORC_REPL ? c->tp : 1);
}

/* ------------------------------------------------------------------------ */
/* public: tables                                                            */
/* ------------------------------------------------------------------------ */

int orc_num_tensors(const orc_model* m) {
  if (check_model(m)) return -1;
  return build_tensors(m, NULL);
}

int orc_tensor_get(const orc_model* m, int t, orc_tensor* out) {
  int rc = check_model(m);
  if (rc) return rc;
  int nt = build_tensors(m, NULL);
  if (t < 0 || t >= nt) return ORC_EINVAL;
  orc_tensor* T = calloc((size_t)nt, sizeof *T);
  if (!T) return ORC_ENOMEM;
  build_tensors(m, T);
  *out = T[t];
  free(T);
  return ORC_OK;
}

/* Pieces of one rank of configuration c.  out may be NULL to count. */
int orc_layout(const orc_model* m, const orc_cfg* c, int rank, orc_piece* out, int cap,
               uint64_t* arena_elems) {
  int rc = check_model(m);
  if (rc) return rc;
  if ((rc = check_cfg(m, c))) return rc;
  if (rank < 0 || rank >= c->tp * c->pp * c->dp) return ORC_ERANK;
  int nt = build_tensors(m, NULL);
  orc_tensor* T = calloc((size_t)nt, sizeof *T);
  if (!T) return ORC_ENOMEM;
  build_tensors(m, T);
  int n = layout(m, c, T, nt, rank, NULL, arena_elems);
  if (out) {
    if (cap < n) {
      free(T);
      return ORC_EINVAL;
    }
    layout(m, c, T, nt, rank, out, arena_elems);
  }
  free(T);
  return n;
}

/* ------------------------------------------------------------------------ */
/* public: matrices                                                          */
/* ------------------------------------------------------------------------ */

/* ROUTE[s][d]: bytes source s sends to destination d under the sender rule.
 * OVERLAP[s][d]: bytes of (held by s) intersect (needed by d), intersecting
 *   logical identities (tensor, element), so a replica counts as held.
 * OVERLAP_SHARDED[s][d]: OVERLAP over tensors with exactly one copy per
 *   data-parallel replica in both configurations, counted only when s lies in
 *   the source replica serving d.
 * COST[d][s] = bytes(d) - OVERLAP[s][d]: the paper's c_ij with rows = the new
 *   (curr) ranks and columns = the old (prev) ranks (Sec. III-B), in bytes;
 *   ORC_COST_INF when s and d lie in different data-parallel replicas or s
 *   failed (Sec. III-C).  A failed rank holds nothing.
 * Computed over LCM workload items (Sec. III-C).  Any output may be NULL. */
int orc_matrices(const orc_model* m, const orc_cfg* src, const orc_cfg* dst, const orc_route* route,
                 uint64_t* route_m, uint64_t* overlap, uint64_t* overlap_sh, uint64_t* cost) {
  ctx_t x;
  int rc = ctx_init(&x, m, src, dst, route);
  if (rc) return rc;
  const int S = x.S, D = x.D;
  uint64_t* R = calloc((size_t)S * D, 8);
  uint64_t* O = calloc((size_t)S * D, 8);
  uint64_t* OS = calloc((size_t)S * D, 8);
  uint64_t* need = calloc((size_t)D, 8);
  if (!R || !O || !OS || !need) {
    free(R); free(O); free(OS); free(need);
    ctx_free(&x);
    return ORC_ENOMEM;
  }
  for (int ti = 0; ti < x.nt; ++ti) {
    const orc_tensor* t = &x.T[ti];
    const int64_t G = n_items(&x, t);
    const uint64_t item_bytes = (uint64_t)(t->rows * t->cols / G) * BYTES_PER_ELEM;
    const int sharded = multiplicity(&x, src, t) == 1 && multiplicity(&x, dst, t) == 1;
    for (int d = 0; d < D; ++d) {
      int pp_d, tp_d;
      coords(dst, d, &pp_d, &tp_d);
      const int serving = replica_of(dst, d) % src->dp; /* source replica serving d */
      for (int role_d = 0; role_d < 2; ++role_d) {
        for (int64_t a = 0; a < G; ++a) {
          if (!holds_item(&x, dst, pp_d, tp_d, t, role_d, a)) continue;
          need[d] += item_bytes;
          for (int s = 0; s < S; ++s) {
            if (x.failed[s]) continue; /* a failed rank holds nothing */
            int pp_s, tp_s;
            coords(src, s, &pp_s, &tp_s);
            if (holds_item(&x, src, pp_s, tp_s, t, 0, a) ||
                holds_item(&x, src, pp_s, tp_s, t, 1, a)) {
              O[(size_t)s * D + d] += item_bytes;
              if (sharded && replica_of(src, s) == serving) OS[(size_t)s * D + d] += item_bytes;
            }
          }
          int snd = sender_of_item(&x, d, role_d, t, a);
          if (snd < 0) {
            rc = ORC_EUNRECOVERABLE;
            goto out;
          }
          R[(size_t)snd * D + d] += item_bytes;
        }
      }
    }
  }
  if (route_m) memcpy(route_m, R, (size_t)S * D * 8);
  if (overlap) memcpy(overlap, O, (size_t)S * D * 8);
  if (overlap_sh) memcpy(overlap_sh, OS, (size_t)S * D * 8);
  if (cost)
    for (int d = 0; d < D; ++d)
      for (int s = 0; s < S; ++s)
        cost[(size_t)d * S + s] =
            (x.failed[s] || replica_of(src, s) != replica_of(dst, d))
                ? ORC_COST_INF
                : need[d] - O[(size_t)s * D + d];
out:
  free(R); free(O); free(OS); free(need);
  ctx_free(&x);
  return rc;
}

/* The same four matrices by enumerating every element of every tensor and
 * scanning every rank's pieces for it.  Tiny models only. */
int orc_matrices_bruteforce(const orc_model* m, const orc_cfg* src, const orc_cfg* dst,
                            const orc_route* route, uint64_t* route_m, uint64_t* overlap,
                            uint64_t* overlap_sh, uint64_t* cost) {
  ctx_t x;
  int rc = ctx_init(&x, m, src, dst, route);
  if (rc) return rc;
  const int S = x.S, D = x.D;
  uint64_t* R = calloc((size_t)S * D, 8);
  uint64_t* O = calloc((size_t)S * D, 8);
  uint64_t* OS = calloc((size_t)S * D, 8);
  uint64_t* need = calloc((size_t)D, 8);
  if (!R || !O || !OS || !need) {
    rc = ORC_ENOMEM;
    goto out;
  }
  /* a tensor's element is "sharded" when exactly one source piece and one
   * destination piece hold it. */
  for (int ti = 0; ti < x.nt; ++ti) {
    const orc_tensor* t = &x.T[ti];
    for (int64_t r = 0; r < t->rows; ++r) {
      for (int64_t c = 0; c < t->cols; ++c) {
        int cs = 0, cd = 0; /* copies of the element in the whole configurations */
        for (int s = 0; s < S; ++s)
          for (int i = 0; i < x.ns[s]; ++i)
            if (x.ps[s][i].tensor == ti && in_box(&x.ps[s][i], r, c)) ++cs;
        for (int d = 0; d < D; ++d)
          for (int i = 0; i < x.nd[d]; ++i)
            if (x.pd[d][i].tensor == ti && in_box(&x.pd[d][i], r, c)) ++cd;
        /* one copy per data-parallel replica on both sides */
        const int sharded = cs == src->dp && cd == dst->dp;
        for (int d = 0; d < D; ++d) {
          for (int i = 0; i < x.nd[d]; ++i) {
            const orc_piece* q = &x.pd[d][i];
            if (q->tensor != ti || !in_box(q, r, c)) continue;
            need[d] += BYTES_PER_ELEM;
            for (int s = 0; s < S; ++s) {
              if (x.failed[s]) continue;
              int held = 0;
              for (int j = 0; j < x.ns[s]; ++j)
                if (x.ps[s][j].tensor == ti && in_box(&x.ps[s][j], r, c)) held = 1;
              if (held) {
                O[(size_t)s * D + d] += BYTES_PER_ELEM;
                if (sharded && replica_of(src, s) == replica_of(dst, d) % src->dp)
                  OS[(size_t)s * D + d] += BYTES_PER_ELEM;
              }
            }
            int snd = sender_of_element(&x, d, q->role, ti, r, c);
            if (snd < 0) {
              rc = ORC_EUNRECOVERABLE;
              goto out;
            }
            R[(size_t)snd * D + d] += BYTES_PER_ELEM;
          }
        }
      }
    }
  }
  if (route_m) memcpy(route_m, R, (size_t)S * D * 8);
  if (overlap) memcpy(overlap, O, (size_t)S * D * 8);
  if (overlap_sh) memcpy(overlap_sh, OS, (size_t)S * D * 8);
  if (cost)
    for (int d = 0; d < D; ++d)
      for (int s = 0; s < S; ++s)
        cost[(size_t)d * S + s] =
            (x.failed[s] || replica_of(src, s) != replica_of(dst, d))
                ? ORC_COST_INF
                : need[d] - O[(size_t)s * D + d];
out:
  free(R); free(O); free(OS); free(need);
  ctx_free(&x);
  return rc;
}

/* ------------------------------------------------------------------------ */
/* messages                                                                  */
/* ------------------------------------------------------------------------ */

/* The boxes source s sends to destination d, in message order: d's pieces in
 * arena order, and for each piece the items whose sender is s.  Those items
 * must be one contiguous run (one box); otherwise ORC_EBOX.  Each box starts
 * at a multiple of 8 elements inside every kind section.  Returns the box
 * count; *npad gets the padded element count of one section. */
static int message_boxes(const ctx_t* x, int s, int d, orc_mbox* out, uint64_t* npad,
                         uint64_t* nelem) {
  int n = 0;
  uint64_t cur = 0, tot = 0;
  if (x->direct_refer && x->home[d] == s) { /* kept on the paired GPU: no message */
    if (npad) *npad = 0;
    if (nelem) *nelem = 0;
    return 0;
  }
  for (int i = 0; i < x->nd[d]; ++i) {
    const orc_piece* q = &x->pd[d][i];
    const orc_tensor* t = &x->T[q->tensor];
    const int64_t G = n_items(x, t);
    int64_t first = -1, last = -1;
    for (int64_t a = 0; a < G; ++a) {
      int pp, tp;
      coords(&x->dst, d, &pp, &tp);
      if (!holds_item(x, &x->dst, pp, tp, t, q->role, a)) continue;
      const int snd = sender_of_item(x, d, q->role, t, a);
      if (snd < 0) return ORC_EUNRECOVERABLE;
      if (snd != s) continue;
      if (first < 0) first = a;
      else if (a != last + 1) return ORC_EBOX;
      last = a;
    }
    if (first < 0) continue;
    orc_mbox b;
    b.tensor = q->tensor;
    b.role_d = q->role;
    b.r0 = 0;
    b.r1 = t->rows;
    b.c0 = 0;
    b.c1 = t->cols;
    if (t->split == ORC_ROWS) {
      b.r0 = first * (t->rows / G);
      b.r1 = (last + 1) * (t->rows / G);
    } else if (t->split == ORC_COLS) {
      b.c0 = first * (t->cols / G);
      b.c1 = (last + 1) * (t->cols / G);
    }
    b.moff = cur;
    const uint64_t ne = (uint64_t)((b.r1 - b.r0) * (b.c1 - b.c0));
    cur += (uint64_t)align_up((int64_t)ne, ORC_BOX_PAD_ELEMS);
    tot += ne;
    if (out) out[n] = b;
    ++n;
  }
  if (npad) *npad = cur;
  if (nelem) *nelem = tot;
  return n;
}

/* Send-buffer layout of source s: for each destination, the routed bytes
 * (unpadded, = ROUTE[s][d]), the padded message bytes, and the byte
 * displacement of the message (messages in destination order, each at a
 * multiple of 256 bytes).  *total = buffer length. */
int orc_send_layout(const orc_model* m, const orc_cfg* src, const orc_cfg* dst, const orc_route* route,
                    int s, uint64_t* count, uint64_t* padded, uint64_t* displ, uint64_t* total) {
  ctx_t x;
  int rc = ctx_init(&x, m, src, dst, route);
  if (rc) return rc;
  if (s < 0 || s >= x.S) {
    ctx_free(&x);
    return ORC_ERANK;
  }
  uint64_t cur = 0;
  for (int d = 0; d < x.D; ++d) {
    uint64_t np = 0, ne = 0;
    int nb = message_boxes(&x, s, d, NULL, &np, &ne);
    if (nb < 0) {
      ctx_free(&x);
      return nb;
    }
    if (count) count[d] = ne * BYTES_PER_ELEM;
    if (padded) padded[d] = np * BYTES_PER_ELEM;
    cur = (uint64_t)align_up((int64_t)cur, ORC_MSG_ALIGN_BYTES);
    if (displ) displ[d] = cur;
    cur += np * BYTES_PER_ELEM;
  }
  if (total) *total = (uint64_t)align_up((int64_t)cur, ORC_MSG_ALIGN_BYTES);
  ctx_free(&x);
  return ORC_OK;
}

/* Message s->d as a list of boxes (for tests and sampled checks). */
int orc_message(const orc_model* m, const orc_cfg* src, const orc_cfg* dst, const orc_route* route,
                int s, int d, orc_mbox* out, int cap, uint64_t* npad) {
  ctx_t x;
  int rc = ctx_init(&x, m, src, dst, route);
  if (rc) return rc;
  if (s < 0 || s >= x.S || d < 0 || d >= x.D) {
    ctx_free(&x);
    return ORC_ERANK;
  }
  int n = message_boxes(&x, s, d, NULL, npad, NULL);
  if (n >= 0 && out) {
    if (cap < n) n = ORC_EINVAL;
    else message_boxes(&x, s, d, out, npad, NULL);
  }
  ctx_free(&x);
  return n;
}

/* ------------------------------------------------------------------------ */
/* the migration itself: materialize then re-slice                          */
/* ------------------------------------------------------------------------ */

/* Migrate tensors [t_lo, t_hi).  src_arenas[s*4+k] is source rank s's arena
 * of kind k (NULL when that rank is not resident).  Every non-NULL
 * dst_arenas[d*4+k] receives destination d's pieces; every non-NULL
 * send_bufs[s] receives the part of source s's messages that belongs to these
 * tensors, zero padding included.  Gap bytes are never written.
 * Full tensors are materialized from all resident sources (replicas compared
 * bit for bit), then cut.  A needed element that no resident source covers
 * is an error. */
int orc_migrate(const orc_model* m, const orc_cfg* src, const orc_cfg* dst, const orc_route* route,
                const void* const* src_arenas, void* const* dst_arenas,
                void* const* send_bufs, int t_lo, int t_hi) {
  ctx_t x;
  int rc = ctx_init(&x, m, src, dst, route);
  if (rc) return rc;
  if (t_lo < 0) t_lo = 0;
  if (t_hi > x.nt || t_hi < 0) t_hi = x.nt;
  const int S = x.S, D = x.D;

  /* message layouts of every resident sender */
  orc_mbox** mb = calloc((size_t)S * D, sizeof(orc_mbox*));
  int* nmb = calloc((size_t)S * D, sizeof(int));
  uint64_t* mnpad = calloc((size_t)S * D, 8);
  uint64_t* mdispl = calloc((size_t)S * D, 8);
  uint8_t* full[ORC_NKIND] = {0};
  uint8_t* covered = NULL;
  if (!mb || !nmb || !mnpad || !mdispl) {
    rc = ORC_ENOMEM;
    goto out;
  }
  for (int s = 0; s < S; ++s) {
    if (!send_bufs || !send_bufs[s]) continue;
    uint64_t cur = 0;
    for (int d = 0; d < D; ++d) {
      int n = message_boxes(&x, s, d, NULL, NULL, NULL);
      if (n < 0) {
        rc = n;
        goto out;
      }
      mb[(size_t)s * D + d] = calloc((size_t)n + 1, sizeof(orc_mbox));
      if (!mb[(size_t)s * D + d]) {
        rc = ORC_ENOMEM;
        goto out;
      }
      nmb[(size_t)s * D + d] = message_boxes(&x, s, d, mb[(size_t)s * D + d],
                                             &mnpad[(size_t)s * D + d], NULL);
      cur = (uint64_t)align_up((int64_t)cur, ORC_MSG_ALIGN_BYTES);
      mdispl[(size_t)s * D + d] = cur;
      cur += mnpad[(size_t)s * D + d] * BYTES_PER_ELEM;
    }
  }

  for (int ti = t_lo; ti < t_hi; ++ti) {
    const orc_tensor* t = &x.T[ti];
    const size_t ne = (size_t)(t->rows * t->cols);
    for (int k = 0; k < ORC_NKIND; ++k) {
      full[k] = malloc(ne * (size_t)ESIZE[k]);
      if (!full[k]) {
        rc = ORC_ENOMEM;
        goto out;
      }
    }
    covered = calloc(ne, 1);
    if (!covered) {
      rc = ORC_ENOMEM;
      goto out;
    }
    /* 1. materialize from every resident source shard */
    for (int s = 0; s < S; ++s) {
      if (!src_arenas || !src_arenas[(size_t)s * 4] || x.failed[s]) continue;
      for (int i = 0; i < x.ns[s]; ++i) {
        const orc_piece* p = &x.ps[s][i];
        if (p->tensor != ti) continue;
        const int64_t ld = p->c1 - p->c0;
        for (int64_t r = p->r0; r < p->r1; ++r) {
          for (int64_t c = p->c0; c < p->c1; ++c) {
            const size_t g = (size_t)(r * t->cols + c);
            const uint64_t l = p->off + (uint64_t)((r - p->r0) * ld + (c - p->c0));
            for (int k = 0; k < ORC_NKIND; ++k) {
              const uint8_t* a = (const uint8_t*)src_arenas[(size_t)s * 4 + k] + l * ESIZE[k];
              uint8_t* f = full[k] + g * ESIZE[k];
              if (covered[g]) {
                if (memcmp(a, f, (size_t)ESIZE[k])) {
                  rc = ORC_EMISMATCH;
                  goto out;
                }
              } else {
                memcpy(f, a, (size_t)ESIZE[k]);
              }
            }
            covered[g] = 1;
          }
        }
      }
    }
    /* 2. cut every destination piece */
    for (int d = 0; d < D; ++d) {
      if (!dst_arenas || !dst_arenas[(size_t)d * 4]) continue;
      for (int i = 0; i < x.nd[d]; ++i) {
        const orc_piece* q = &x.pd[d][i];
        if (q->tensor != ti) continue;
        const int64_t ld = q->c1 - q->c0;
        for (int64_t r = q->r0; r < q->r1; ++r) {
          for (int64_t c = q->c0; c < q->c1; ++c) {
            const size_t g = (size_t)(r * t->cols + c);
            if (!covered[g]) {
              rc = ORC_EUNCOVERED;
              goto out;
            }
            const uint64_t l = q->off + (uint64_t)((r - q->r0) * ld + (c - q->c0));
            for (int k = 0; k < ORC_NKIND; ++k)
              memcpy((uint8_t*)dst_arenas[(size_t)d * 4 + k] + l * ESIZE[k],
                     full[k] + g * ESIZE[k], (size_t)ESIZE[k]);
          }
        }
      }
    }
    /* 3. cut every message box, row-major in full-tensor coordinates */
    for (int s = 0; s < S; ++s) {
      if (!send_bufs || !send_bufs[s]) continue;
      for (int d = 0; d < D; ++d) {
        const size_t sd = (size_t)s * D + d;
        for (int i = 0; i < nmb[sd]; ++i) {
          const orc_mbox* b = &mb[sd][i];
          if (b->tensor != ti) continue;
          const uint64_t ne_box = (uint64_t)((b->r1 - b->r0) * (b->c1 - b->c0));
          const uint64_t pad = (uint64_t)align_up((int64_t)ne_box, ORC_BOX_PAD_ELEMS) - ne_box;
          uint64_t sec = 0; /* byte offset of kind section k inside the message */
          for (int k = 0; k < ORC_NKIND; ++k) {
            uint8_t* base = (uint8_t*)send_bufs[s] + mdispl[sd] + sec;
            uint64_t e = b->moff;
            for (int64_t r = b->r0; r < b->r1; ++r) {
              for (int64_t c = b->c0; c < b->c1; ++c) {
                const size_t g = (size_t)(r * t->cols + c);
                if (!covered[g]) {
                  rc = ORC_EUNCOVERED;
                  goto out;
                }
                memcpy(base + e * ESIZE[k], full[k] + g * ESIZE[k], (size_t)ESIZE[k]);
                ++e;
              }
            }
            memset(base + e * ESIZE[k], 0, pad * (size_t)ESIZE[k]);
            sec += mnpad[sd] * (uint64_t)ESIZE[k];
          }
        }
      }
    }
    for (int k = 0; k < ORC_NKIND; ++k) {
      free(full[k]);
      full[k] = NULL;
    }
    free(covered);
    covered = NULL;
  }
out:
  for (int k = 0; k < ORC_NKIND; ++k) free(full[k]);
  free(covered);
  if (mb)
    for (size_t i = 0; i < (size_t)S * D; ++i) free(mb[i]);
  free(mb);
  free(nmb);
  free(mnpad);
  free(mdispl);
  ctx_free(&x);
  return rc;
}

/* ------------------------------------------------------------------------ */
/* element origins, for sampled checks at full size                          */
/* ------------------------------------------------------------------------ */

/* Source piece of rank s holding element (r, c) of tensor t; -1 if none. */
static int find_src_piece(const ctx_t* x, int s, int t, int64_t r, int64_t c) {
  for (int i = 0; i < x->ns[s]; ++i)
    if (x->ps[s][i].tensor == t && in_box(&x->ps[s][i], r, c)) return i;
  return -1;
}

/* For destination d and arena element offsets offs[0..n): the source rank
 * whose element ends up there (by the sender rule) and that element's offset
 * in the source arena.  Gap offsets get src_rank -1. */
int orc_dst_origin(const orc_model* m, const orc_cfg* src, const orc_cfg* dst, const orc_route* route,
                   int d, const uint64_t* offs, int64_t n, int32_t* src_rank, uint64_t* src_off) {
  ctx_t x;
  int rc = ctx_init(&x, m, src, dst, route);
  if (rc) return rc;
  if (d < 0 || d >= x.D) {
    ctx_free(&x);
    return ORC_ERANK;
  }
  for (int64_t j = 0; j < n; ++j) {
    src_rank[j] = -1;
    src_off[j] = 0;
    for (int i = 0; i < x.nd[d]; ++i) {
      const orc_piece* q = &x.pd[d][i];
      const uint64_t ne = (uint64_t)piece_elems(q);
      if (offs[j] < q->off || offs[j] >= q->off + ne) continue;
      const uint64_t l = offs[j] - q->off;
      const int64_t ld = q->c1 - q->c0;
      const int64_t r = q->r0 + (int64_t)(l / (uint64_t)ld);
      const int64_t c = q->c0 + (int64_t)(l % (uint64_t)ld);
      const int s = sender_of_element(&x, d, q->role, q->tensor, r, c);
      if (s < 0) {
        ctx_free(&x);
        return ORC_EUNCOVERED;
      }
      const int pi = find_src_piece(&x, s, q->tensor, r, c);
      const orc_piece* p = &x.ps[s][pi];
      src_rank[j] = s;
      src_off[j] = p->off + (uint64_t)((r - p->r0) * (p->c1 - p->c0) + (c - p->c0));
      break;
    }
  }
  ctx_free(&x);
  return ORC_OK;
}

/* For message s->d and element positions pos[0..n) inside a kind section:
 * the offset in source s's arena of the element stored there, or
 * UINT64_MAX for zero padding / past the end. */
int orc_msg_origin(const orc_model* m, const orc_cfg* src, const orc_cfg* dst, const orc_route* route,
                   int s, int d, const uint64_t* pos, int64_t n, uint64_t* src_off) {
  ctx_t x;
  int rc = ctx_init(&x, m, src, dst, route);
  if (rc) return rc;
  if (s < 0 || s >= x.S || d < 0 || d >= x.D) {
    ctx_free(&x);
    return ORC_ERANK;
  }
  int nb = message_boxes(&x, s, d, NULL, NULL, NULL);
  orc_mbox* B = calloc((size_t)nb + 1, sizeof *B);
  if (nb < 0 || !B) {
    free(B);
    ctx_free(&x);
    return nb < 0 ? nb : ORC_ENOMEM;
  }
  message_boxes(&x, s, d, B, NULL, NULL);
  for (int64_t j = 0; j < n; ++j) {
    src_off[j] = UINT64_MAX;
    for (int i = 0; i < nb; ++i) {
      const orc_mbox* b = &B[i];
      const int64_t w = b->c1 - b->c0;
      const uint64_t ne = (uint64_t)((b->r1 - b->r0) * w);
      if (pos[j] < b->moff || pos[j] >= b->moff + ne) continue;
      const uint64_t l = pos[j] - b->moff;
      const int64_t r = b->r0 + (int64_t)(l / (uint64_t)w);
      const int64_t c = b->c0 + (int64_t)(l % (uint64_t)w);
      const int pi = find_src_piece(&x, s, b->tensor, r, c);
      if (pi < 0) {
        free(B);
        ctx_free(&x);
        return ORC_EUNCOVERED;
      }
      const orc_piece* p = &x.ps[s][pi];
      src_off[j] = p->off + (uint64_t)((r - p->r0) * (p->c1 - p->c0) + (c - p->c0));
      break;
    }
  }
  free(B);
  ctx_free(&x);
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* migration sketch (Sec. III-B: indicator Eq. (1), objective Eq. (2),      */
/* constraints Eq. (3) for M > N and Eq. (4) for M <= N, Algorithm 1)        */
/* ------------------------------------------------------------------------ */

/* Pair the M new ranks (rows of cost) with the N old ranks (columns) so the
 * total cost of the pairs is minimal.  As Algorithm 1 does: pad the matrix
 * with zeros to k x k, k = max(M, N), solve the square assignment problem,
 * and drop every pair that involves a padded row or column.  The square
 * problem is solved here as a minimum-cost flow (source -> row -> column ->
 * sink, unit capacities) by k successive shortest augmenting paths, each
 * found with Bellman-Ford over the residual graph.  pair[i] = the old rank
 * paired with new rank i, or -1; *total = the kept pairs' cost. */
int orc_sketch(const uint64_t* cost, int M, int N, int32_t* pair, uint64_t* total) {
  if (!cost || !pair || M < 1 || N < 1) return ORC_EINVAL;
  const int k = M > N ? M : N;
  const int V = 2 * k + 2, SRC = 0, SNK = 2 * k + 1;
  const int E = 2 * (k * k + 2 * k);
  int* from = calloc((size_t)E, sizeof(int));
  int* to = calloc((size_t)E, sizeof(int));
  int* cap = calloc((size_t)E, sizeof(int));
  int64_t* w = calloc((size_t)E, sizeof(int64_t));
  int64_t* dist = calloc((size_t)V, sizeof(int64_t));
  int* via = calloc((size_t)V, sizeof(int));
  if (!from || !to || !cap || !w || !dist || !via) {
    free(from); free(to); free(cap); free(w); free(dist); free(via);
    return ORC_ENOMEM;
  }
  int ne = 0;
#define EDGE(a, b, c)                                          \
  do {                                                         \
    from[ne] = (a); to[ne] = (b); cap[ne] = 1; w[ne] = (c); ++ne;  \
    from[ne] = (b); to[ne] = (a); cap[ne] = 0; w[ne] = -(c); ++ne; \
  } while (0)
  for (int i = 0; i < k; ++i) EDGE(SRC, 1 + i, 0);
  for (int i = 0; i < k; ++i)
    for (int j = 0; j < k; ++j) {
      const int64_t c = (i < M && j < N) ? (int64_t)cost[(size_t)i * N + j] : 0; /* zero padding */
      EDGE(1 + i, 1 + k + j, c);
    }
  for (int j = 0; j < k; ++j) EDGE(1 + k + j, SNK, 0);
#undef EDGE
  const int64_t INF = INT64_MAX / 4;
  for (int round = 0; round < k; ++round) {
    for (int v = 0; v < V; ++v) {
      dist[v] = INF;
      via[v] = -1;
    }
    dist[SRC] = 0;
    for (int it = 0; it < V - 1; ++it) {
      int changed = 0;
      for (int e = 0; e < ne; ++e) {
        if (!cap[e] || dist[from[e]] == INF) continue;
        if (dist[from[e]] + w[e] < dist[to[e]]) {
          dist[to[e]] = dist[from[e]] + w[e];
          via[to[e]] = e;
          changed = 1;
        }
      }
      if (!changed) break;
    }
    if (dist[SNK] == INF) break; /* cannot happen on a complete bipartite graph */
    for (int v = SNK; v != SRC; v = from[via[v]]) {
      cap[via[v]] -= 1;
      cap[via[v] ^ 1] += 1;
    }
  }
  uint64_t tot = 0;
  for (int i = 0; i < M; ++i) {
    pair[i] = -1;
    for (int j = 0; j < k; ++j) {
      const int e = 2 * (k + i * k + j); /* the row i -> column j edge */
      if (cap[e] == 0) {
        if (j < N) {
          pair[i] = j;
          tot += cost[(size_t)i * N + j];
        }
        break;
      }
    }
  }
  if (total) *total = tot;
  free(from); free(to); free(cap); free(w); free(dist); free(via);
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* virtual rank allocator (Sec. III-E, Algorithm 2)                          */
/* ------------------------------------------------------------------------ */

/* Placement-aware remapping after a migration with pairing pair[d] (the old
 * rank whose device becomes new rank d, or -1).  Devices are grouped n to a
 * node.  The devices in play, in this order: the live old devices (ids
 * 0..S-1 without the failed ranks), then one fresh device per new rank that
 * the pairing leaves unpaired (ids S, S+1, ... in rank order).  p2c[i] is the
 * new rank hosted by the i-th device after the migration, or -1 (idle).
 *  mode 1, occupancy: walk the idle devices in order and the occupied devices
 *    in reverse order, node by node, and pair them until the two walks meet;
 *    each pair hands the occupied device's process to the idle device.
 *  mode 2, efficiency: the target placement puts ranks 0..D-1 node by node on
 *    the devices; a node whose target differs from its loads is fragmented,
 *    and at every position of it where they differ the target rank is moved
 *    onto that device.
 *  mode 0: no remapping.
 * Out: placement[d] (D) = device finally hosting new rank d; ops (3 entries
 * per operator: rank, from device, to device; may be NULL), *nops.  The node
 * size groups the devices only; the result does not depend on it. */
int orc_defrag(int S, int D, const int32_t* pair, const int32_t* failed, int num_failed, int n,
               int mode, int32_t* placement, int32_t* ops, int* nops) {
  if (S < 1 || D < 1 || n < 1 || !pair || !placement || !nops || num_failed < 0) return ORC_EINVAL;
  if (mode < 0 || mode > 2) return ORC_EINVAL;
  char* dead = calloc((size_t)S, 1);
  int32_t* dev = malloc(sizeof(int32_t) * (size_t)(S + D));
  int32_t* p2c = malloc(sizeof(int32_t) * (size_t)(S + D));
  int32_t* loc = malloc(sizeof(int32_t) * (size_t)D);
  int rc = ORC_OK;
  if (!dead || !dev || !p2c || !loc) { rc = ORC_ENOMEM; goto out; }
  for (int i = 0; i < num_failed; ++i) {
    if (failed[i] < 0 || failed[i] >= S) { rc = ORC_EINVAL; goto out; }
    dead[failed[i]] = 1;
  }
  for (int d = 0; d < D; ++d) {
    if (pair[d] < -1 || pair[d] >= S || (pair[d] >= 0 && dead[pair[d]])) { rc = ORC_EINVAL; goto out; }
    for (int e = 0; e < d; ++e)
      if (pair[d] >= 0 && pair[e] == pair[d]) { rc = ORC_EINVAL; goto out; }
  }
  /* the device list and what each device hosts after the migration */
  int nd = 0;
  for (int v = 0; v < S; ++v) {
    if (dead[v]) continue;
    dev[nd] = v;
    p2c[nd] = -1;
    for (int d = 0; d < D; ++d)
      if (pair[d] == v) p2c[nd] = d;
    ++nd;
  }
  int fresh = S;
  for (int d = 0; d < D; ++d)
    if (pair[d] < 0) {
      dev[nd] = fresh++;
      p2c[nd] = d;
      ++nd;
    }
  for (int i = 0; i < nd; ++i)
    if (p2c[i] >= 0) loc[p2c[i]] = dev[i];
  for (int d = 0; d < D; ++d) placement[d] = loc[d];
  int k = 0;
#define EMIT(rank, from, to)                   \
  do {                                         \
    if (ops) {                                 \
      ops[3 * k] = (rank);                     \
      ops[3 * k + 1] = (from);                 \
      ops[3 * k + 2] = (to);                   \
    }                                          \
    placement[(rank)] = (to);                  \
    ++k;                                       \
  } while (0)
  if (mode == 1) {
    int i = 0, j = nd - 1;
    for (;;) {
      while (i < nd && p2c[i] >= 0) ++i;  /* next idle device, in order */
      while (j >= 0 && p2c[j] < 0) --j;   /* next occupied device, in reverse */
      if (i >= nd || j < 0 || i > j) break; /* the walks have met */
      EMIT(p2c[j], dev[j], dev[i]);
      ++i;
      --j;
    }
  } else if (mode == 2) {
    const int nodes = (nd + n - 1) / n;
    for (int node = 0; node < nodes; ++node) {
      int fragmented = 0;
      for (int i = node * n; i < node * n + n && i < nd; ++i) {
        const int target = i < D ? i : -1;
        if (target != p2c[i]) fragmented = 1;
      }
      if (!fragmented) continue;
      for (int i = node * n; i < node * n + n && i < nd; ++i) {
        const int target = i < D ? i : -1;
        if (target >= 0 && target != p2c[i]) EMIT(target, loc[target], dev[i]);
      }
    }
  }
#undef EMIT
  *nops = k;
out:
  free(dead); free(dev); free(p2c); free(loc);
  return rc;
}
