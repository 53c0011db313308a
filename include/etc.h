/*
 * etc.h -- libetc: checkpoint-free resharding of GPU-resident model states
 * between two hybrid-parallel (TP, PP) configurations, for AMD Instinct
 * MI355X (gfx950).
 *
 * The operation (paper: "Direct Model State Migration for Elastic Training of
 * Large Language Models", Sec. III):
 *   - A rank's *workload* is the list of logical tensor pieces it holds under
 *     Megatron's even static partition rules; every rank can derive every
 *     other rank's workload locally (Sec. III-B).
 *   - TP-split dims are compared at LCM(tp_prev, tp_curr) granularity
 *     (Sec. III-C).
 *   - The cost matrix counts, for every (new rank, old rank) pair, the data the
 *     new rank lacks if it reuses the old one: c_ij = len(curr_i) -
 *     len(curr_i intersect prev_j) (Sec. III-B).
 *   - Pieces held by both sides of a pair stay (Refer); others are sent by
 *     one holder and received by the new owner (Send / Recv, Sec. III-D).  The
 *     states of every workload type move together: bf16 parameter, fp32
 *     master, fp32 Adam m, fp32 Adam v (Sec. III-D).
 * This library is the data-parallel hot path of that migration on one GPU:
 *   etc_sketch       host: the migration sketch (pairing of new and old ranks)
 *   etc_plan         host: layouts, routing, message layout, tile tables
 *   etc_plan_static  the same, device tables in a static array (no device
 *                    allocation)
 *   etc_plan_defrag  host: virtual rank allocator and the coalesced pairing
 *   etc_plan_message, etc_plan_refer   host: the instruction lists
 *   etc_cost_matrix  device: byte matrices over every (source, target) pair
 *   etc_pack         device: a source rank's shards -> one message per peer
 *   etc_unpack       device: received messages -> the target rank's shards
 *   etc_pack_kind,   device: the same, one state kind at a time (state
 *   etc_unpack_kind          chunking)
 *   etc_refer,       device: what a target's paired source keeps, arena to
 *   etc_refer_kind           arena (Refer), all kinds or one
 *   etc_plan_* queries      host: dimensions, pieces, arena sizes, send and
 *                            chunk layouts, receive counts, pairing, roles
 * Moving messages between GPUs is the caller's business (a grouped
 * send/recv or all-to-all-v with the counts from etc_plan_send_layout).
 *
 * Conventions shared by all calls
 *   Ranks.   rank = dp * (PP * TP) + pp * TP + tp: TP fastest, then PP; each
 *            data-parallel replica is a contiguous block of ranks.  Target
 *            replica j is served by source replica j mod DP_src (replicas that
 *            are kept stay, new replicas are fed round-robin; Sec. III-C), and
 *            a failed source's data comes from the next live replica.
 *   Layers.  Stage p holds layers [p*L/PP, (p+1)*L/PP); the embedding (and a
 *            GPT position table) sits on the first stage; the final norm and
 *            the output head on the last.  A tied embedding also has a
 *            duplicate on the last stage when PP > 1 ("copy role" 1).
 *   TP split. Column-parallel weights and biases split dim 0 (QKV rows are
 *            interleaved per KV group, so a shard is a contiguous row range),
 *            row-parallel weights split dim 1, norms and row-parallel biases
 *            are replicated, the vocab-parallel embedding and head split
 *            dim 0.  SwiGLU gate and up are separate logical tensors stored
 *            fused (gate shard, then up shard).
 *   Arenas.  Each rank keeps one arena per state kind (kind 0 bf16 param,
 *            1 fp32 master, 2 fp32 Adam m, 3 fp32 Adam v).  Local tensors
 *            are laid out in tensor order (role-1 copies last), each starting
 *            at a multiple of 128 elements (the up half of gate/up directly
 *            after gate); element offsets are the same in all four arenas.
 *            Bytes between tensors are never read or written.
 *   Messages. Message s->d holds four kind sections (param, master, m, v),
 *            each the routed boxes in d's arena order, every box row-major
 *            in full-tensor coordinates and starting at a multiple of 8
 *            elements (zero padded).  A send buffer holds the messages in
 *            target order, each at a multiple of 256 bytes.
 *   Memory.  The caller owns every arena, send buffer, message and output
 *            buffer.  All device pointers must be 256-byte aligned.  On
 *            MI355X a copy whose read and write addresses differ modulo
 *            1 KB runs 2-4 % slower.  With every arena and send-buffer base
 *            a multiple of 1 KB, the layouts above keep the two congruent
 *            wherever tensor pieces and box rows span whole multiples of
 *            1 KB, as in model shapes with power-of-two widths.
 *   Streams. Device calls only enqueue work on `stream` (a hipStream_t;
 *            NULL is the null stream) and return; they never allocate,
 *            free or synchronize.  Arguments are checked before anything is
 *            enqueued; a non-zero status means nothing was enqueued.
 *   Threads. A plan is immutable after etc_plan returns: any number of
 *            threads may use it at once, on any streams of its device.
 *   Errors.  Status 0 is success, negative values are ETC_ERR_*; the text
 *            of the last error of the calling thread is etc_last_error().
 */
#ifndef ETC_H
#define ETC_H

#include <stdint.h>

/* exported from libetc.so (the library is built with hidden visibility) */
#define ETC_API __attribute__((visibility("default")))

#ifdef __cplusplus
extern "C" {
#endif

enum { ETC_ARCH_GPT = 0,   /* LayerNorm w+b, linear biases, learned positions, GeLU MLP */
       ETC_ARCH_LLAMA = 1  /* RMSNorm, no biases, SwiGLU gate/up + down, GQA            */ };

enum { ETC_F_LAYERS_ONLY = 1 /* model flag: transformer layers only (no embeddings,
                                final norm or head) */ };

enum { ETC_KIND_PARAM_BF16 = 0, ETC_KIND_MASTER_F32 = 1, ETC_KIND_ADAM_M_F32 = 2,
       ETC_KIND_ADAM_V_F32 = 3, ETC_NUM_KINDS = 4 };

/* Matrix selectors for etc_cost_matrix (all values in bytes, over the four
 * state kinds = 14 bytes per element):
 *  ROUTE            S x D: bytes source s sends to target d.  Each target
 *                   element is sent once.  Target d keeps what its paired
 *                   source (the same GPU in the migration sketch; source d
 *                   under the identity pairing) already holds (Refer).  Any
 *                   other element comes from the holder with the smallest
 *                   key (copy role differs, tp_s != tp_d mod TP_src, pp_s,
 *                   tp_s).
 *  OVERLAP          S x D: bytes of (held by s) intersect (needed by d), by
 *                   logical identity (a replica counts as held).
 *  OVERLAP_SHARDED  S x D: OVERLAP over tensors with exactly one copy in both
 *                   configurations.
 *  COST             D x S: the paper's cost matrix c_ij (rows are the new
 *                   ranks, columns the old ranks, Sec. III-B):
 *                   bytes(d) - OVERLAP[s][d]; ETC_COST_INF between
 *                   different data-parallel replicas and towards failed
 *                   ranks.  A failed rank holds nothing.  OVERLAP_SHARDED
 *                   counts tensors with one copy per replica, and only when
 *                   s lies in the replica serving d. */
enum { ETC_CM_ROUTE = 0, ETC_CM_OVERLAP = 1, ETC_CM_OVERLAP_SHARDED = 2, ETC_CM_COST = 3 };

enum { ETC_ALL_RANKS = -1 };

enum { ETC_SIDE_SRC = 0, ETC_SIDE_DST = 1 };

/* etc_plan flags */
enum { ETC_PLAN_HOST_ONLY = 1, /* build host tables only: no device memory, no
                                  device calls allowed on this plan */
       ETC_PLAN_SKETCH = 2,    /* pair new and old ranks with the optimal
                                  migration sketch (etc_sketch on COST) */
       ETC_PLAN_DIRECT_REFER = 4 /* the data a target's paired source keeps
                                  (Refer, Sec. III-D) goes arena to arena
                                  with etc_refer instead of through a
                                  message: that message is empty */ };

enum {
  ETC_OK = 0,
  ETC_ERR_INVALID_ARG = -1, /* NULL or out-of-range argument                      */
  ETC_ERR_INDIVISIBLE = -2, /* a dim the configuration splits does not divide     */
  ETC_ERR_RANK = -3,        /* rank out of range, or not built into this plan     */
  ETC_ERR_ALIGN = -4,       /* a device pointer is not 256-byte aligned           */
  ETC_ERR_UNSUPPORTED = -5, /* a case outside the model family, too many peers or ranks, or a size limit */
  ETC_ERR_NOMEM = -6,       /* host or device allocation failed (etc_plan only)   */
  ETC_ERR_HIP = -7,         /* a HIP runtime call failed; see etc_last_error()    */
  ETC_ERR_UNRECOVERABLE = -8 /* needed data survives on no live source rank      */
};

/* COST between ranks of different data-parallel replicas, or towards a
 * failed rank: the paper's "infinite" workload difference (Sec. III-C). */
#define ETC_COST_INF (1ull << 50)

typedef struct {
  int32_t arch;            /* ETC_ARCH_*                                  */
  int32_t num_layers;      /* transformer layers L                        */
  int32_t hidden;          /* hidden size h                               */
  int32_t num_heads;       /* attention (query) heads                     */
  int32_t num_kv_heads;    /* KV heads (== num_heads without GQA)         */
  int32_t ffn_hidden;      /* MLP inner size f                            */
  int32_t vocab;           /* padded vocabulary size V                    */
  int32_t max_pos;         /* learned position table rows (GPT), 0 = none */
  int32_t tied_embeddings; /* 1: output head is the input embedding       */
  int32_t flags;           /* ETC_F_*                                     */
} etc_model_desc;

typedef struct {
  int32_t tp, pp, dp;
} etc_parallel_cfg;

typedef struct etc_plan_s etc_plan_t;

/* One local piece of a logical tensor on a rank. */
typedef struct {
  char name[48];           /* e.g. "layers.3.qkv.weight"                  */
  int32_t tensor;          /* logical tensor id (arena order)             */
  int32_t role;            /* copy role: 0, or 1 for the tied duplicate   */
  int64_t full_rows, full_cols; /* logical (TP = 1) shape; vectors [n, 1] */
  int64_t r0, r1, c0, c1;  /* the piece's box in full-tensor coordinates  */
  uint64_t elem_offset;    /* element offset in each of the four arenas;
                              the piece is stored row-major, row length
                              c1 - c0                                      */
} etc_piece_info;

/* Migration sketch (Sec. III-B, objective Eq. (2), constraints Eq. (3) for
 * M > N and Eq. (4) for M <= N, Algorithm 1): given an M x N cost matrix
 * (host memory, row-major, rows = new ranks, columns = old ranks, as COST
 * from etc_cost_matrix), pair rows with columns so the summed cost is
 * minimal: pad to k x k with zeros (k = max(M, N)), solve the square
 * assignment problem, drop pairs in the padding.  Output pair[i] (M entries,
 * host) = the column paired with row i, or -1; *total (may be NULL) = the
 * kept pairs' summed cost.  Several optimal pairings may exist; any one is
 * returned.  Host only, O(k^3), exact (integer arithmetic).
 * Errors: INVALID_ARG (NULL, M or N outside 1..65536), UNSUPPORTED (an entry
 * above 2^52, or min(M, N) times the largest entry above 2^64 - 1, the most a
 * pairing's total could reach), NOMEM. */
ETC_API int etc_sketch(const uint64_t* cost, int M, int N, int32_t* pair, uint64_t* total);

/* Options of etc_plan (NULL = all defaults: identity pairing, no failures,
 * every rank, no flags). */
typedef struct {
  const int32_t* pair;   /* D entries, host: pair[d] = the old rank whose GPU
                            becomes new rank d, or -1 for a new GPU; each old
                            rank at most once, never a failed rank.  It may
                            cross data-parallel replicas (all replicas hold
                            the same states), as a coalesced pairing does;
                            the sketch never does.  NULL: identity
                            pairing (d with d, where both lie in the same
                            replica and d is alive), or the optimal sketch
                            with ETC_PLAN_SKETCH */
  const int32_t* failed; /* old ranks whose states are lost (host), or NULL */
  int32_t num_failed;
  int32_t rank;          /* process to build device tables for, or ETC_ALL_RANKS */
  uint32_t flags;        /* ETC_PLAN_* */
} etc_plan_options;

/* Build a migration plan from `model`, the old configuration `src` and the new
 * configuration `dst` (Sec. III: the primitive's inputs are the two parallel
 * configurations and the model), with new ranks paired to old ranks as
 * opt->pair says.  Host work: the logical tensor table, every rank's layout,
 * the routing of every target element, every message layout.
 * opt->rank names a process: process p < S holds old rank p and becomes the
 * new rank paired with it (if any); processes S, S+1, ... are new GPUs and
 * take the unpaired new ranks in ascending order (etc_plan_process reports
 * both roles).  Device tables (routed boxes cut into uniform tiles, the tensor
 * table, the pairing and the failed ranks for etc_cost_matrix) are built for
 * that process's pack and unpack, or for every rank with ETC_ALL_RANKS, and
 * copied to the current device, which the plan is then bound to.  With
 * ETC_PLAN_HOST_ONLY no device memory is touched.
 * A routed run of contiguous elements may exceed 2^32 elements (it is copied
 * in pieces of 2^31); no tensor size limit applies beyond the int32 fields of
 * etc_model_desc and the workgroup limit below.
 * On success *out owns host and device memory until etc_plan_free.
 * Errors: INVALID_ARG (also a bad pairing or failed list), INDIVISIBLE,
 * UNSUPPORTED (GPT with GQA, more than 65536 ranks, a rank exchanging messages
 * with more than ETC_MAX_PEERS peers; with device tables, a rank's copy that
 * needs more than 2^31 - 1 GPU workgroups, i.e. about 5.5e11 routed
 * elements), UNRECOVERABLE (every replica of some needed data failed), RANK,
 * NOMEM, HIP. */
ETC_API int etc_plan(const etc_model_desc* model, const etc_parallel_cfg* src,
                     const etc_parallel_cfg* dst, const etc_plan_options* opt, etc_plan_t** out);

/* Size of the library's static device table array (per GPU), bytes. */
enum { ETC_STATIC_TABLE_BYTES = 4 << 20 };

/* etc_plan for callers that cannot allocate device memory (code that runs
 * while hipMalloc is forbidden: a serving loop, a harness that owns all of
 * HBM).  Same arguments, plan and results as etc_plan, but the device tables
 * are written into a static array of ETC_STATIC_TABLE_BYTES bytes that the
 * library holds on each GPU until the process ends, instead of memory of
 * their own: no hipMalloc, hipFree or other device allocation is made (host
 * memory for the plan itself is still allocated).  Every device call
 * (etc_cost_matrix, etc_pack, etc_unpack, the one-kind calls, etc_refer)
 * then reads the tables from that array.
 * One array per GPU, shared by every call: each etc_plan_static call on a
 * device first waits until the device is idle (hipDeviceSynchronize), then
 * replaces the tables; from then on device calls with a static plan built
 * earlier on that device fail with INVALID_ARG (the plan's host queries
 * still work; free it as usual).  Device calls of the live static plan may
 * run from any threads and streams.  Do not call it while a stream of the
 * device is being captured, and do not replay a graph captured with an
 * earlier static plan after a later call: its launches would read the new
 * tables.
 * Errors: as etc_plan; INVALID_ARG also for ETC_PLAN_HOST_ONLY; UNSUPPORTED
 * when the tables need more than ETC_STATIC_TABLE_BYTES (a plan with
 * ETC_ALL_RANKS for Llama-70B TP8xPP8 -> TP8xPP4 needs about 0.6 MB; a
 * per-process plan far less). */
ETC_API int etc_plan_static(const etc_model_desc* model, const etc_parallel_cfg* src,
                            const etc_parallel_cfg* dst, const etc_plan_options* opt,
                            etc_plan_t** out);

/* Virtual rank allocator (Sec. III-E, Algorithm 2): de-fragment the devices
 * after the plan's migration.  The migration leaves new rank d on the device
 * of its paired old rank; unpaired new ranks start on fresh devices numbered
 * S, S+1, ... in order of d (S = old world size).  Devices of failed old
 * ranks are gone and take part in nothing.  mode:
 *  ETC_DEFRAG_OCCUPANCY: idle live devices, in ascending order, take over the
 *    processes of occupied devices, in descending order, while the idle device
 *    precedes the occupied one, so the occupied devices end up first and whole
 *    nodes at the end are freed (whatever the node size);
 *  ETC_DEFRAG_EFFICIENCY: the k-th live device (old ones ascending, then fresh
 *    ones) hosts new rank k, so a TP group (consecutive ranks) shares a node
 *    whenever TP divides the node size;
 *  ETC_DEFRAG_NONE: no remapping.
 * Out (host arrays): placement[d] (D entries) = final device of new rank d;
 * ops (optional, 3 * D entries) = remap operators (rank, from device, to
 * device), *nops of them; coalesced (optional, D entries) = the coalesced
 * pairing (Sec. III-E): placement[d] where that is an old device (< S), else
 * -1.  A plan built with it migrates straight to the final devices, in place
 * of the migration followed by the remap, and yields the same target states.
 * Host only.  Errors: INVALID_ARG. */
enum { ETC_DEFRAG_NONE = 0, ETC_DEFRAG_OCCUPANCY = 1, ETC_DEFRAG_EFFICIENCY = 2 };
ETC_API int etc_plan_defrag(const etc_plan_t* plan, int mode, int32_t* placement, int32_t* ops,
                            int* nops, int32_t* coalesced);

/* The plan's pairing: pair[d] (D entries) = old rank paired with new rank d, or -1. */
ETC_API int etc_plan_pairing(const etc_plan_t* plan, int32_t* pair);

/* Roles of process `process` (see etc_plan): the old rank it holds and the
 * new rank it becomes, each -1 if none.  Errors: INVALID_ARG, RANK. */
ETC_API int etc_plan_process(const etc_plan_t* plan, int process, int* src_rank, int* dst_rank);

/* Release a plan (NULL is a no-op).  Device work using it must be complete. */
ETC_API void etc_plan_free(etc_plan_t* plan);

/* S = source world size, D = target world size. */
ETC_API int etc_plan_dims(const etc_plan_t* plan, int* S, int* D);

/* Number of logical tensors. */
ETC_API int etc_plan_num_tensors(const etc_plan_t* plan, int* n);

/* Arena length of a rank, in elements (multiply by 2 for kind 0, 4 for
 * kinds 1..3 to get bytes).  side: ETC_SIDE_SRC or ETC_SIDE_DST. */
ETC_API int etc_plan_arena_elems(const etc_plan_t* plan, int side, int rank, uint64_t* elems);

/* Pieces of a rank, in arena order. */
ETC_API int etc_plan_num_pieces(const etc_plan_t* plan, int side, int rank, int* n);
ETC_API int etc_plan_piece(const etc_plan_t* plan, int side, int rank, int index, etc_piece_info* out);

/* Send layout of source rank s (any rank, whatever the plan's `rank`):
 * counts[d] = routed bytes to target d (= ROUTE[s][d]); msg_bytes[d] = bytes
 * of message s->d including box padding (0 when nothing is routed);
 * displs[d] = byte offset of message s->d in s's send buffer; *total = send
 * buffer length.  Any output pointer may be NULL.  Arrays have D entries. */
ETC_API int etc_plan_send_layout(const etc_plan_t* plan, int src_rank, uint64_t* counts,
                         uint64_t* msg_bytes, uint64_t* displs, uint64_t* total);

/* counts[s] = bytes target d receives from source s (= ROUTE[s][d]); S entries. */
ETC_API int etc_plan_recv_counts(const etc_plan_t* plan, int dst_rank, uint64_t* counts);

/* One migration instruction (Sec. III-D: source, target, workload; all four
 * state kinds move together): a box of a logical tensor, row-major in
 * full-tensor coordinates, copied from the source rank's arenas to the target
 * rank's.  Offsets are in elements and the same in the four arenas of a rank
 * (and in the four kind sections of a message). */
typedef struct {
  int32_t tensor;          /* logical tensor (as etc_piece_info.tensor)           */
  int32_t role;            /* copy role of the target's piece (1: tied duplicate) */
  int64_t r0, r1, c0, c1;  /* the box: rows [r0, r1), columns [c0, c1)            */
  uint64_t src_offset;     /* element offset of the box's first element, source  */
  uint64_t src_ld;         /* row stride of the source piece, elements           */
  uint64_t dst_offset;     /* element offset of the box's first element, target  */
  uint64_t dst_ld;         /* row stride of the target piece, elements           */
  uint64_t msg_offset;     /* element offset inside each kind section of the
                              message; ETC_NO_MESSAGE for a Refer instruction   */
} etc_instruction;
#define ETC_NO_MESSAGE UINT64_MAX

/* The instruction list of message src_rank -> dst_rank (Send on the source,
 * Recv on the target), in message order; empty when nothing is routed.
 * *count = number of instructions; out (host, may be NULL) receives the first
 * min(cap, *count) of them.  Host only.  Errors: INVALID_ARG, RANK. */
ETC_API int etc_plan_message(const etc_plan_t* plan, int src_rank, int dst_rank, etc_instruction* out,
                             int cap, int* count);

/* The Refer instructions of dst_rank: what its paired source keeps, which
 * etc_refer copies arena to arena when the plan has ETC_PLAN_DIRECT_REFER
 * (source offsets are in the paired source's arenas); empty otherwise (the
 * kept part then travels in the paired source's message).  Same conventions
 * as etc_plan_message. */
ETC_API int etc_plan_refer(const etc_plan_t* plan, int dst_rank, etc_instruction* out, int cap,
                           int* count);

/* Compute one S x D (or D x S for ETC_CM_COST) uint64 matrix, row-major, into
 * device memory d_out, with one GPU kernel over every (source, target) pair
 * and every logical tensor (Sec. III-B, cost matrix; Sec. III-C, LCM items).
 * d_out must be 8-byte aligned.
 * Errors: INVALID_ARG (bad `which`, NULL, host-only plan), ALIGN,
 * UNSUPPORTED (S * D above 2^31 - 1), HIP. */
ETC_API int etc_cost_matrix(const etc_plan_t* plan, int which, uint64_t* d_out, void* stream);

/* Pack: copy source rank src_rank's shards (src_arena[k] = its arena of kind
 * k, device memory, read only) into send_buf (device, etc_plan_send_layout
 * total bytes): one contiguous message per target peer, the Send side of
 * Sec. III-D.  Every message byte is written (box padding is zero); other
 * bytes of send_buf are not touched.  A source that routes nothing (a failed
 * rank) returns ETC_OK at once, without reading any argument.
 * Errors: INVALID_ARG, RANK (src_rank's tables not built into the plan), ALIGN, HIP. */
ETC_API int etc_pack(const etc_plan_t* plan, int src_rank, const void* const src_arena[4],
             void* send_buf, void* stream);

/* Unpack: scatter the messages target dst_rank receives into its arenas
 * (dst_arena[k], device memory), the Recv / Refer side of Sec. III-D.  msg[s]
 * (S entries, device memory, read only) is the start of message s->dst_rank,
 * laid out as etc_pack writes it; it may be NULL when ROUTE[s][dst_rank] is 0.
 * Every payload element of the target arenas is written exactly once; bytes
 * between tensors are not touched.
 * Errors: INVALID_ARG (a needed msg[s] is NULL), RANK, ALIGN, HIP. */
ETC_API int etc_unpack(const etc_plan_t* plan, int dst_rank, const void* const* msg,
               void* const dst_arena[4], void* stream);

enum { ETC_MAX_PEERS = 256 };

/* State chunking (Sec. III-D; Sec. IV-G: one optimizer component at a time):
 * migrate one state kind at a time through a chunk buffer that holds only
 * that kind, so its memory can be allocated per chunk and each source arena
 * released as soon as its kind has been packed.  Message s->d of kind k in a
 * chunk buffer is byte for byte section k of the full message s->d.
 * Routing is per element, and the four arenas share one element layout, so
 * in the one-kind calls `kind` only selects the element size: 2 bytes for
 * ETC_KIND_PARAM_BF16, 4 for the other kinds.  Any further per-element
 * state in that layout (the paper's "other states", e.g. an fp32 gradient)
 * migrates through the same calls, passed as a kind of its element size.
 * etc_plan_chunk_layout: counts[d] = bytes of message s->d for this kind
 * (padded, 0 if nothing is routed), displs[d] = its byte offset in the chunk
 * buffer (multiple of 256), *total = chunk buffer length.  D entries each;
 * any output may be NULL. */
ETC_API int etc_plan_chunk_layout(const etc_plan_t* plan, int src_rank, int kind, uint64_t* counts,
                                  uint64_t* displs, uint64_t* total);

/* Refer (Sec. III-D): data that target dst_rank's paired source already
 * holds stays on that GPU.  With ETC_PLAN_DIRECT_REFER it is copied straight
 * from the paired source's arenas (src_arena[k], read only) into dst_rank's
 * (dst_arena[k]), all four kinds in one launch; the paired source's message
 * to dst_rank is then empty, and etc_unpack writes the rest.  etc_refer and
 * etc_unpack of one target write disjoint bytes, so they may run in either
 * order or concurrently.  A target with no paired source, or a plan without
 * the flag, has nothing to refer: ETC_OK at once.
 * Errors: INVALID_ARG, RANK (dst_rank's tables not built into the plan), ALIGN, HIP. */
ETC_API int etc_refer(const etc_plan_t* plan, int dst_rank, const void* const src_arena[4],
                      void* const dst_arena[4], void* stream);

/* etc_refer for one state kind (state chunking): src_arena and dst_arena are
 * that kind's arenas.  Errors as etc_refer, and INVALID_ARG for a bad kind. */
ETC_API int etc_refer_kind(const etc_plan_t* plan, int dst_rank, int kind, const void* src_arena,
                           void* dst_arena, void* stream);

/* Bytes (all four kinds) that etc_refer copies for dst_rank; 0 without
 * ETC_PLAN_DIRECT_REFER or without a paired source. */
ETC_API int etc_plan_refer_bytes(const etc_plan_t* plan, int dst_rank, uint64_t* bytes);

/* Pack kind `kind` of source rank src_rank (src_arena: that kind's arena,
 * device, read only) into chunk_buf (device, chunk layout).  A source that
 * routes nothing returns ETC_OK at once, as etc_pack does.  Errors as
 * etc_pack, and INVALID_ARG for a bad kind. */
ETC_API int etc_pack_kind(const etc_plan_t* plan, int src_rank, int kind, const void* src_arena,
                          void* chunk_buf, void* stream);

/* Unpack kind `kind` into target rank dst_rank's arena of that kind; msg[s]
 * (S entries) = message s->dst_rank in the sender's chunk layout, or NULL when
 * nothing is routed.  Errors as etc_unpack, and INVALID_ARG for a bad kind. */
ETC_API int etc_unpack_kind(const etc_plan_t* plan, int dst_rank, int kind, const void* const* msg,
                            void* dst_arena, void* stream);

/* Text of the calling thread's last error ("" if none).  Valid until the
 * thread's next failing call. */
ETC_API const char* etc_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ETC_H */
