// capi.hip -- the C ABI of libetc (include/etc.h): argument checks, error
// reporting, device table upload and kernel dispatch.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <memory>
#include <mutex>
#include <new>
#include <shared_mutex>
#include <string>
#include <vector>

#include "copy_geom.hpp"
#include "etc.h"
#include "etc_internal.hpp"
#include "plan.hpp"
#include "route.hpp"

namespace {

thread_local std::string g_last_error;

int fail(int code, const std::string& msg) {
  g_last_error = msg;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(ETC_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// ---------------------------------------------------------------------------
// Static device tables (etc_plan_static): a file-scope device array that the
// library never allocates or frees.  Each GPU holds its own copy at its own
// address, looked up once per device with that device current; host code
// uses only that address (the array's name is a host-side stand-in).  One
// static plan per device is live at a time: g_static_gen counts the calls
// per device, and a plan built by an earlier call is refused.  Device calls
// of a static plan hold the lock shared from the check to the launch, and
// etc_plan_static holds it exclusively while it waits for the device and
// rewrites the array, so no launch ever reads a half-written table.

__device__ __align__(256) unsigned char scratch[ETC_STATIC_TABLE_BYTES];

struct StaticSlot {
  void* ptr = nullptr;  // device address of `scratch` on this device
  uint64_t gen = 0;     // etc_plan_static calls on this device so far
};
std::shared_mutex g_static_mu;
std::vector<StaticSlot> g_static;  // by device ordinal; guarded by g_static_mu

// The array's address on `dev` (current device), looked up on first use.
// Caller holds g_static_mu exclusively.
hipError_t static_slot(int dev, StaticSlot** out) {
  if (size_t(dev) >= g_static.size()) g_static.resize(size_t(dev) + 1);
  StaticSlot& s = g_static[size_t(dev)];
  if (!s.ptr) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    s.ptr = p;
  }
  *out = &s;
  return hipSuccess;
}

void release_device(etc_plan_t* P) {
  if (P->device < 0) return;
  if (P->static_gen) {  // tables in the static array: nothing to free
    P->d_boxes = nullptr;
    P->d_route_tensors = nullptr;
    P->d_home = nullptr;
    P->d_failed = nullptr;
    return;
  }
  int prev = -1;
  const bool have_prev = hipGetDevice(&prev) == hipSuccess;
  if (prev != P->device) (void)hipSetDevice(P->device);
  if (P->d_boxes) (void)hipFree(P->d_boxes);
  if (P->d_route_tensors) (void)hipFree(P->d_route_tensors);
  if (P->d_home) (void)hipFree(P->d_home);
  if (P->d_failed) (void)hipFree(P->d_failed);
  if (have_prev && prev != P->device) (void)hipSetDevice(prev);
  P->d_boxes = nullptr;
  P->d_route_tensors = nullptr;
  P->d_home = nullptr;
  P->d_failed = nullptr;
}

int check_device_plan(const etc_plan_t* P) {
  if (!P) return fail(ETC_ERR_INVALID_ARG, "plan is NULL");
  if (P->device < 0 || !P->d_route_tensors || !P->d_home)
    return fail(ETC_ERR_INVALID_ARG, "plan was built with ETC_PLAN_HOST_ONLY");
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev != P->device)
    return fail(ETC_ERR_INVALID_ARG, "current device " + std::to_string(dev) +
                                         " is not the plan's device " + std::to_string(P->device));
  return ETC_OK;
}

// Held by every device call from its checks to its launch: shared for a
// static plan (whose tables must still be the live ones), nothing otherwise.
class DeviceCallGuard {
 public:
  explicit DeviceCallGuard(const etc_plan_t* P) {
    if (P && P->static_gen) lock_ = std::shared_lock<std::shared_mutex>(g_static_mu);
  }
  // ETC_OK, or the error of a static plan replaced by a later etc_plan_static
  int check(const etc_plan_t* P) const {
    if (!P || !P->static_gen) return ETC_OK;
    const uint64_t live = size_t(P->device) < g_static.size() ? g_static[size_t(P->device)].gen : 0;
    if (live != P->static_gen)
      return fail(ETC_ERR_INVALID_ARG, "the static device tables of this plan were replaced by a later "
                                       "etc_plan_static on device " + std::to_string(P->device));
    return ETC_OK;
  }

 private:
  std::shared_lock<std::shared_mutex> lock_;
};

// Roles of process p: it holds old rank p (p < S) and becomes the new rank
// paired with it; processes S, S+1, ... take the unpaired new ranks in order.
void process_roles(const etc_plan_t* P, int p, int* src_rank, int* dst_rank) {
  const int S = P->src.world(), D = P->dst.world();
  *src_rank = p < S ? p : -1;
  *dst_rank = -1;
  if (p < S) {
    for (int d = 0; d < D; ++d)
      if (P->home[d] == p) *dst_rank = d;
    return;
  }
  int fresh = p - S;
  for (int d = 0; d < D; ++d)
    if (P->home[d] < 0 && fresh-- == 0) *dst_rank = d;
}

int num_processes(const etc_plan_t* P) {
  int unpaired = 0;
  for (int32_t h : P->home) unpaired += h < 0;
  return P->src.world() + unpaired;
}

// Host side of the device tables: cut the routed boxes of the process's
// launches (every launch with ETC_ALL_RANKS) into tiles, in launch order.
int build_copy_tables(etc_plan_t* P, int rank, std::vector<etc::CopyBox>* all) {
  using namespace etc;
  const int S = P->src.world(), D = P->dst.world();
  int my_src = -1, my_dst = -1;
  if (rank != ETC_ALL_RANKS) process_roles(P, rank, &my_src, &my_dst);
  for (int s = 0; s < S; ++s) {
    if (rank != ETC_ALL_RANKS && my_src != s) continue;
    CopyTable& t = P->pack_tab[s];
    auto v = build_pack_boxes(*P, s, &t.peers, &t.bytes);
    t.first = uint32_t(all->size());
    t.nbox = uint32_t(v.size() - 1);
    t.ntiles = v.back().tile0;
    t.built = true;
    all->insert(all->end(), v.begin(), v.end());
  }
  for (int d = 0; d < D; ++d) {
    if (rank != ETC_ALL_RANKS && my_dst != d) continue;
    CopyTable& t = P->refer_tab[d];
    auto v = build_refer_boxes(*P, d, &t.bytes);
    t.first = uint32_t(all->size());
    t.nbox = uint32_t(v.size() - 1);
    t.ntiles = v.back().tile0;
    t.built = true;
    all->insert(all->end(), v.begin(), v.end());
  }
  for (int d = 0; d < D; ++d) {
    if (rank != ETC_ALL_RANKS && my_dst != d) continue;
    CopyTable& t = P->unpack_tab[d];
    auto v = build_unpack_boxes(*P, d, &t.peers, &t.bytes);
    t.first = uint32_t(all->size());
    t.nbox = uint32_t(v.size() - 1);
    t.ntiles = v.back().tile0;
    t.built = true;
    all->insert(all->end(), v.begin(), v.end());
  }
  // the copy kernels launch one workgroup per sub-chunk of every tile
  for (const auto* tabs : {&P->pack_tab, &P->unpack_tab, &P->refer_tab})
    for (const CopyTable& t : *tabs)
      if (uint64_t(t.ntiles) * kSubPerTile > uint64_t(INT32_MAX))
        return fail(ETC_ERR_UNSUPPORTED, "a rank's copy needs more than 2^31 - 1 GPU workgroups");
  return ETC_OK;
}

int upload(etc_plan_t* P, int rank) {
  using namespace etc;
  hipError_t e = hipGetDevice(&P->device);
  if (e != hipSuccess) {
    P->device = -1;
    return hip_fail(e, "hipGetDevice");
  }
  std::vector<CopyBox> all;
  int rc = build_copy_tables(P, rank, &all);
  if (rc) return rc;
  if (!all.empty()) {
    e = hipMalloc(&P->d_boxes, all.size() * sizeof(CopyBox));
    if (e != hipSuccess) return fail(ETC_ERR_NOMEM, std::string("hipMalloc: ") + hipGetErrorString(e));
    e = hipMemcpy(P->d_boxes, all.data(), all.size() * sizeof(CopyBox), hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy (copy tables)");
  }
  const size_t rt_bytes = std::max<size_t>(1, P->route_tensors.size()) * sizeof(RouteTensor);
  e = hipMalloc(&P->d_route_tensors, rt_bytes);
  if (e != hipSuccess) return fail(ETC_ERR_NOMEM, std::string("hipMalloc: ") + hipGetErrorString(e));
  if (!P->route_tensors.empty()) {
    e = hipMemcpy(P->d_route_tensors, P->route_tensors.data(),
                  P->route_tensors.size() * sizeof(RouteTensor), hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy (tensor table)");
  }
  e = hipMalloc(&P->d_home, std::max<size_t>(1, P->home.size()) * sizeof(int32_t));
  if (e != hipSuccess) return fail(ETC_ERR_NOMEM, std::string("hipMalloc: ") + hipGetErrorString(e));
  e = hipMemcpy(P->d_home, P->home.data(), P->home.size() * sizeof(int32_t), hipMemcpyHostToDevice);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpy (pairing)");
  if (!P->failed_bits.empty()) {
    e = hipMalloc(&P->d_failed, P->failed_bits.size() * sizeof(uint32_t));
    if (e != hipSuccess) return fail(ETC_ERR_NOMEM, std::string("hipMalloc: ") + hipGetErrorString(e));
    e = hipMemcpy(P->d_failed, P->failed_bits.data(), P->failed_bits.size() * sizeof(uint32_t),
                  hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy (failed ranks)");
  }
  return ETC_OK;
}

// The same device tables written into the current device's static array:
// copy boxes, tensor table, pairing, failed ranks, each at a multiple of 256
// bytes.  No device memory is allocated.
int upload_static(etc_plan_t* P, int rank) {
  using namespace etc;
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  std::vector<CopyBox> all;
  int rc = build_copy_tables(P, rank, &all);
  if (rc) return rc;
  auto up = [](size_t n) { return (n + 255) / 256 * 256; };
  const size_t o_rt = up(all.size() * sizeof(CopyBox));
  const size_t o_home = o_rt + up(P->route_tensors.size() * sizeof(RouteTensor));
  const size_t o_failed = o_home + up(P->home.size() * sizeof(int32_t));
  const size_t total = o_failed + P->failed_bits.size() * sizeof(uint32_t);
  if (total > size_t(ETC_STATIC_TABLE_BYTES))
    return fail(ETC_ERR_UNSUPPORTED, "the plan's device tables need " + std::to_string(total) +
                                         " bytes; etc_plan_static holds at most " +
                                         std::to_string(int(ETC_STATIC_TABLE_BYTES)) +
                                         " (ETC_STATIC_TABLE_BYTES); use etc_plan, or a plan per process");
  std::vector<unsigned char> img(std::max<size_t>(total, 1), 0);
  std::memcpy(img.data(), all.data(), all.size() * sizeof(CopyBox));
  std::memcpy(img.data() + o_rt, P->route_tensors.data(), P->route_tensors.size() * sizeof(RouteTensor));
  std::memcpy(img.data() + o_home, P->home.data(), P->home.size() * sizeof(int32_t));
  std::memcpy(img.data() + o_failed, P->failed_bits.data(), P->failed_bits.size() * sizeof(uint32_t));
  std::unique_lock<std::shared_mutex> lock(g_static_mu);
  StaticSlot* slot = nullptr;
  if ((e = static_slot(dev, &slot)) != hipSuccess) return hip_fail(e, "hipGetSymbolAddress (static tables)");
  // the previous static plan's launches may still read the array
  if ((e = hipDeviceSynchronize()) != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
  ++slot->gen;  // from here on, earlier static plans of this device are refused
  if ((e = hipMemcpy(slot->ptr, img.data(), img.size(), hipMemcpyHostToDevice)) != hipSuccess)
    return hip_fail(e, "hipMemcpy (static tables)");
  unsigned char* base = static_cast<unsigned char*>(slot->ptr);
  P->device = dev;
  P->static_gen = slot->gen;
  P->d_boxes = all.empty() ? nullptr : reinterpret_cast<CopyBox*>(base);
  P->d_route_tensors = reinterpret_cast<RouteTensor*>(base + o_rt);
  P->d_home = reinterpret_cast<int32_t*>(base + o_home);
  P->d_failed = P->failed_bits.empty() ? nullptr : reinterpret_cast<uint32_t*>(base + o_failed);
  return ETC_OK;
}

int check_side_rank(const etc_plan_t* P, int side, int rank) {
  if (!P) return fail(ETC_ERR_INVALID_ARG, "plan is NULL");
  if (side != ETC_SIDE_SRC && side != ETC_SIDE_DST) return fail(ETC_ERR_INVALID_ARG, "bad side");
  const int n = side == ETC_SIDE_SRC ? P->src.world() : P->dst.world();
  if (rank < 0 || rank >= n) return fail(ETC_ERR_RANK, "rank " + std::to_string(rank) + " out of range");
  return ETC_OK;
}

int check_arenas(const void* const* arenas, const char* what) {
  if (!arenas) return fail(ETC_ERR_INVALID_ARG, std::string(what) + " is NULL");
  for (int k = 0; k < 4; ++k) {
    if (!arenas[k]) return fail(ETC_ERR_INVALID_ARG, std::string(what) + "[" + std::to_string(k) + "] is NULL");
    if (!aligned(arenas[k], 256))
      return fail(ETC_ERR_ALIGN, std::string(what) + "[" + std::to_string(k) + "] is not 256-byte aligned");
  }
  return ETC_OK;
}

// The instruction of box b routed from source rank s (its arenas) to target
// rank d; msg_offset as given.
etc_instruction make_instruction(const etc_plan_t* P, int s, int d, const etc_plan_s::MsgBox& b,
                                 uint64_t msg_offset) {
  using namespace etc;
  const int role_s = role_on(P->route_tensors[size_t(b.tensor)].src_stage, P->src.pp_of(s));
  const RankLayout& Ls = P->src_lay(s);
  const RankLayout& Ld = P->dst_lay(d);
  const Piece& p = Ls.pieces[size_t(Ls.piece_of_tensor[role_s][size_t(b.tensor)])];
  const Piece& q = Ld.pieces[size_t(Ld.piece_of_tensor[b.role_d][size_t(b.tensor)])];
  etc_instruction x{};
  x.tensor = b.tensor;
  x.role = b.role_d;
  x.r0 = b.r0;
  x.r1 = b.r1;
  x.c0 = b.c0;
  x.c1 = b.c1;
  x.src_offset = p.off + uint64_t((b.r0 - p.r0) * p.ld() + (b.c0 - p.c0));
  x.src_ld = uint64_t(p.ld());
  x.dst_offset = q.off + uint64_t((b.r0 - q.r0) * q.ld() + (b.c0 - q.c0));
  x.dst_ld = uint64_t(q.ld());
  x.msg_offset = msg_offset;
  return x;
}

}  // namespace

extern "C" {

int etc_sketch(const uint64_t* cost, int M, int N, int32_t* pair, uint64_t* total) {
  if (!cost || !pair) return fail(ETC_ERR_INVALID_ARG, "cost and pair must not be NULL");
  if (M < 1 || N < 1 || M > 65536 || N > 65536) return fail(ETC_ERR_INVALID_ARG, "bad matrix shape");
  uint64_t top = 0;
  for (size_t i = 0; i < size_t(M) * N; ++i) top = std::max(top, cost[i]);
  if (top > (uint64_t(1) << 52)) return fail(ETC_ERR_UNSUPPORTED, "cost entries must not exceed 2^52");
  // at most min(M, N) pairs: their total must fit the 64-bit result
  if (top > 0 && uint64_t(std::min(M, N)) > UINT64_MAX / top)
    return fail(ETC_ERR_UNSUPPORTED, "the total cost of a pairing could exceed 2^64 - 1");
  try {
    const uint64_t t = etc::solve_sketch(cost, M, N, pair);
    if (total) *total = t;
  } catch (const std::bad_alloc&) {
    return fail(ETC_ERR_NOMEM, "host allocation failed");
  }
  return ETC_OK;
}

}  // extern "C"

namespace {

// etc_plan and etc_plan_static: the same plan, with its device tables in
// memory of their own (hipMalloc) or in the device's static array.
int make_plan(const etc_model_desc* model, const etc_parallel_cfg* src, const etc_parallel_cfg* dst,
              const etc_plan_options* opt, etc_plan_t** out, bool in_static) {
  if (!out) return fail(ETC_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (!model || !src || !dst) return fail(ETC_ERR_INVALID_ARG, "model, src and dst must not be NULL");
  const etc_plan_options defaults{nullptr, nullptr, 0, ETC_ALL_RANKS, 0};
  if (!opt) opt = &defaults;
  const int32_t* pair = opt->pair;
  const int rank = opt->rank;
  const uint32_t flags = opt->flags;
  if (flags & ~uint32_t(ETC_PLAN_HOST_ONLY | ETC_PLAN_SKETCH | ETC_PLAN_DIRECT_REFER))
    return fail(ETC_ERR_INVALID_ARG, "unknown plan flags");
  if (pair && (flags & ETC_PLAN_SKETCH)) return fail(ETC_ERR_INVALID_ARG, "pass a pairing or ETC_PLAN_SKETCH, not both");
  if (opt->num_failed < 0 || (opt->num_failed > 0 && !opt->failed))
    return fail(ETC_ERR_INVALID_ARG, "bad failed-rank list");
  std::unique_ptr<etc_plan_t> P;
  try {
    etc::validate(*model, *src, *dst);
    P.reset(new etc_plan_t());
    P->model = *model;
    P->src = etc::Grid{src->tp, src->pp, src->dp};
    P->dst = etc::Grid{dst->tp, dst->pp, dst->dp};
    P->rank = rank;
    P->flags = flags;
    const int S = P->src.world(), D = P->dst.world();
    std::vector<char> dead(S, 0);
    if (opt->num_failed > 0) {
      P->failed_bits.assign((S + 31) / 32, 0u);
      for (int i = 0; i < opt->num_failed; ++i) {
        const int f = opt->failed[i];
        if (f < 0 || f >= S) return fail(ETC_ERR_INVALID_ARG, "failed rank " + std::to_string(f) + " out of range");
        dead[f] = 1;
        P->failed_bits[f >> 5] |= 1u << (f & 31);
      }
    }
    P->tensors = etc::build_tensor_table(P->model);
    etc::build_route_tensors(*P);
    P->home.assign(D, -1);
    if (flags & ETC_PLAN_SKETCH) {
      etc::sketch_pairing(*P, dead);
    } else if (pair) {
      std::vector<char> taken(S, 0);
      for (int d = 0; d < D; ++d) {
        if (pair[d] < -1 || pair[d] >= S)
          return fail(ETC_ERR_INVALID_ARG, "pair[" + std::to_string(d) + "] is not a source rank or -1");
        if (pair[d] >= 0 && taken[pair[d]]++)
          return fail(ETC_ERR_INVALID_ARG, "source rank " + std::to_string(pair[d]) + " is paired twice");
        if (pair[d] >= 0 && dead[pair[d]])
          return fail(ETC_ERR_INVALID_ARG, "pair[" + std::to_string(d) + "] is a failed rank");
        P->home[d] = pair[d];
      }
    } else {  // identity pairing, where it stays inside one live replica
      for (int d = 0; d < D && d < S; ++d)
        if (!dead[d] && P->src.replica(d) == P->dst.replica(d)) P->home[d] = d;
    }
    if (rank != ETC_ALL_RANKS && (rank < 0 || rank >= num_processes(P.get())))
      return fail(ETC_ERR_RANK, "process " + std::to_string(rank) + " is out of range");
    etc::build_host_plan(*P);
    P->pack_tab.resize(S);
    P->unpack_tab.resize(D);
    P->refer_tab.resize(D);
    if (in_static && (flags & ETC_PLAN_HOST_ONLY))
      return fail(ETC_ERR_INVALID_ARG, "etc_plan_static builds device tables: ETC_PLAN_HOST_ONLY is not allowed");
    if (!(flags & ETC_PLAN_HOST_ONLY)) {
      const int rc = in_static ? upload_static(P.get(), rank) : upload(P.get(), rank);
      if (rc != ETC_OK) {
        release_device(P.get());
        return rc;
      }
    }
  } catch (const etc::PlanError& e) {
    if (P) release_device(P.get());
    return fail(e.code, e.what());
  } catch (const std::bad_alloc&) {
    if (P) release_device(P.get());
    return fail(ETC_ERR_NOMEM, "host allocation failed");
  }
  *out = P.release();
  g_last_error.clear();
  return ETC_OK;
}

}  // namespace

extern "C" {

int etc_plan(const etc_model_desc* model, const etc_parallel_cfg* src, const etc_parallel_cfg* dst,
             const etc_plan_options* opt, etc_plan_t** out) {
  return make_plan(model, src, dst, opt, out, false);
}

int etc_plan_static(const etc_model_desc* model, const etc_parallel_cfg* src, const etc_parallel_cfg* dst,
                    const etc_plan_options* opt, etc_plan_t** out) {
  return make_plan(model, src, dst, opt, out, true);
}

int etc_plan_defrag(const etc_plan_t* P, int mode, int32_t* placement, int32_t* ops, int* nops,
                    int32_t* coalesced) {
  if (!P || !placement || !nops) return fail(ETC_ERR_INVALID_ARG, "NULL argument");
  try {
    const int S = P->src.world(), D = P->dst.world();
    std::vector<char> dead(S, 0);
    for (int s = 0; s < S; ++s)
      dead[s] = !P->failed_bits.empty() && ((P->failed_bits[s >> 5] >> (s & 31)) & 1u);
    const int rc = etc::defrag(S, D, P->home.data(), dead, mode, placement, ops, nops);
    if (rc) return fail(rc, "unknown de-fragmentation mode " + std::to_string(mode));
    for (int d = 0; coalesced && d < D; ++d) coalesced[d] = placement[d] < S ? placement[d] : -1;
  } catch (const std::bad_alloc&) {
    return fail(ETC_ERR_NOMEM, "host allocation failed");
  }
  return ETC_OK;
}

int etc_plan_pairing(const etc_plan_t* P, int32_t* pair) {
  if (!P || !pair) return fail(ETC_ERR_INVALID_ARG, "NULL argument");
  for (size_t d = 0; d < P->home.size(); ++d) pair[d] = P->home[d];
  return ETC_OK;
}

int etc_plan_process(const etc_plan_t* P, int process, int* src_rank, int* dst_rank) {
  if (!P || !src_rank || !dst_rank) return fail(ETC_ERR_INVALID_ARG, "NULL argument");
  if (process < 0 || process >= num_processes(P))
    return fail(ETC_ERR_RANK, "process " + std::to_string(process) + " is out of range");
  process_roles(P, process, src_rank, dst_rank);
  return ETC_OK;
}

void etc_plan_free(etc_plan_t* plan) {
  if (!plan) return;
  release_device(plan);
  delete plan;
}

int etc_plan_dims(const etc_plan_t* P, int* S, int* D) {
  if (!P) return fail(ETC_ERR_INVALID_ARG, "plan is NULL");
  if (S) *S = P->src.world();
  if (D) *D = P->dst.world();
  return ETC_OK;
}

int etc_plan_num_tensors(const etc_plan_t* P, int* n) {
  if (!P || !n) return fail(ETC_ERR_INVALID_ARG, "NULL argument");
  *n = int(P->tensors.size());
  return ETC_OK;
}

int etc_plan_arena_elems(const etc_plan_t* P, int side, int rank, uint64_t* elems) {
  int rc = check_side_rank(P, side, rank);
  if (rc) return rc;
  if (!elems) return fail(ETC_ERR_INVALID_ARG, "elems is NULL");
  *elems = (side == ETC_SIDE_SRC ? P->src_lay(rank) : P->dst_lay(rank)).elems;
  return ETC_OK;
}

int etc_plan_num_pieces(const etc_plan_t* P, int side, int rank, int* n) {
  int rc = check_side_rank(P, side, rank);
  if (rc) return rc;
  if (!n) return fail(ETC_ERR_INVALID_ARG, "n is NULL");
  *n = int((side == ETC_SIDE_SRC ? P->src_lay(rank) : P->dst_lay(rank)).pieces.size());
  return ETC_OK;
}

int etc_plan_piece(const etc_plan_t* P, int side, int rank, int index, etc_piece_info* out) {
  int rc = check_side_rank(P, side, rank);
  if (rc) return rc;
  const auto& L = side == ETC_SIDE_SRC ? P->src_lay(rank) : P->dst_lay(rank);
  if (!out || index < 0 || index >= int(L.pieces.size()))
    return fail(ETC_ERR_INVALID_ARG, "bad piece index");
  const etc::Piece& p = L.pieces[index];
  const etc::LogicalTensor& t = P->tensors[p.tensor];
  std::memset(out, 0, sizeof *out);
  std::strncpy(out->name, t.name.c_str(), sizeof(out->name) - 1);
  out->tensor = p.tensor;
  out->role = p.role;
  out->full_rows = t.rows;
  out->full_cols = t.cols;
  out->r0 = p.r0;
  out->r1 = p.r1;
  out->c0 = p.c0;
  out->c1 = p.c1;
  out->elem_offset = p.off;
  return ETC_OK;
}

int etc_plan_send_layout(const etc_plan_t* P, int s, uint64_t* counts, uint64_t* msg_bytes,
                         uint64_t* displs, uint64_t* total) {
  int rc = check_side_rank(P, ETC_SIDE_SRC, s);
  if (rc) return rc;
  const int D = P->dst.world();
  // an empty message is reported where the next one would start
  uint32_t k = P->src_first[s];
  uint64_t cur = 0;
  for (int d = 0; d < D; ++d) {
    const bool has = k < P->src_first[s + 1] && P->msgs[k].d == d;
    const etc_plan_s::Message* m = has ? &P->msgs[k++] : nullptr;
    if (counts) counts[d] = m ? m->elems * 14 : 0;
    if (msg_bytes) msg_bytes[d] = m ? m->npad * 14 : 0;
    if (displs) displs[d] = m ? m->displ : (cur + 255) / 256 * 256;
    if (m) cur = m->displ + m->npad * 14;
  }
  if (total) *total = P->sendbuf_bytes[s];
  return ETC_OK;
}

int etc_plan_recv_counts(const etc_plan_t* P, int d, uint64_t* counts) {
  int rc = check_side_rank(P, ETC_SIDE_DST, d);
  if (rc) return rc;
  if (!counts) return fail(ETC_ERR_INVALID_ARG, "counts is NULL");
  const int S = P->src.world();
  for (int s = 0; s < S; ++s) counts[s] = 0;
  for (uint32_t k = P->dst_first[d]; k < P->dst_first[d + 1]; ++k) {
    const etc_plan_s::Message& m = P->msgs[P->dst_msgs[k]];
    counts[m.s] = m.elems * 14;
  }
  return ETC_OK;
}

int etc_plan_message(const etc_plan_t* P, int s, int d, etc_instruction* out, int cap, int* count) {
  int rc = check_side_rank(P, ETC_SIDE_SRC, s);
  if (rc) return rc;
  if ((rc = check_side_rank(P, ETC_SIDE_DST, d))) return rc;
  if (!count || cap < 0) return fail(ETC_ERR_INVALID_ARG, "count is NULL or cap is negative");
  const etc_plan_s::Message* m = P->find_msg(s, d);
  const size_t n = m ? m->boxes.size() : 0;
  *count = int(n);
  for (size_t i = 0; out && i < n && i < size_t(cap); ++i)
    out[i] = make_instruction(P, s, d, m->boxes[i], m->boxes[i].moff);
  return ETC_OK;
}

int etc_plan_refer(const etc_plan_t* P, int d, etc_instruction* out, int cap, int* count) {
  int rc = check_side_rank(P, ETC_SIDE_DST, d);
  if (rc) return rc;
  if (!count || cap < 0) return fail(ETC_ERR_INVALID_ARG, "count is NULL or cap is negative");
  const auto& boxes = P->refer[size_t(d)];
  *count = int(boxes.size());
  for (size_t i = 0; out && i < boxes.size() && i < size_t(cap); ++i)
    out[i] = make_instruction(P, P->home[size_t(d)], d, boxes[i], ETC_NO_MESSAGE);
  return ETC_OK;
}

int etc_cost_matrix(const etc_plan_t* P, int which, uint64_t* d_out, void* stream) {
  int rc = check_device_plan(P);
  if (rc) return rc;
  const DeviceCallGuard guard(P);
  if ((rc = guard.check(P))) return rc;
  if (which < ETC_CM_ROUTE || which > ETC_CM_COST) return fail(ETC_ERR_INVALID_ARG, "bad matrix selector");
  if (!d_out) return fail(ETC_ERR_INVALID_ARG, "d_out is NULL");
  if (!aligned(d_out, 8)) return fail(ETC_ERR_ALIGN, "d_out is not 8-byte aligned");
  // one matrix cell per (source, target) pair, indexed in 32 bits by the kernel
  if (uint64_t(P->src.world()) * uint64_t(P->dst.world()) > uint64_t(INT32_MAX))
    return fail(ETC_ERR_UNSUPPORTED, "a cost matrix is limited to 2^31 - 1 cells");
  const etc::RouteCtx ctx{P->src.tp, P->src.pp, P->src.dp, P->dst.tp, P->dst.pp, P->dst.dp,
                         P->d_failed};
  hipError_t e = etc::launch_cost(P->d_route_tensors, int(P->route_tensors.size()), P->d_home, ctx,
                                  which, d_out, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "cost matrix launch");
  return ETC_OK;
}

int etc_pack(const etc_plan_t* P, int s, const void* const src_arena[4], void* send_buf, void* stream) {
  int rc = check_device_plan(P);
  if (rc) return rc;
  const DeviceCallGuard guard(P);
  if ((rc = guard.check(P))) return rc;
  if (s < 0 || s >= P->src.world()) return fail(ETC_ERR_RANK, "source rank out of range");
  const etc::CopyTable& t = P->pack_tab[s];
  if (!t.built) return fail(ETC_ERR_RANK, "source rank " + std::to_string(s) + " is not built into this plan");
  if (t.ntiles == 0) return ETC_OK;  // routes nothing (e.g. a failed rank): nothing is read
  if ((rc = check_arenas(src_arena, "src_arena"))) return rc;
  if (!send_buf) return fail(ETC_ERR_INVALID_ARG, "send_buf is NULL");
  if (!aligned(send_buf, 256)) return fail(ETC_ERR_ALIGN, "send_buf is not 256-byte aligned");
  void* arenas[4];
  for (int k = 0; k < 4; ++k) arenas[k] = const_cast<void*>(src_arena[k]);
  void* peers[ETC_MAX_PEERS];
  for (size_t i = 0; i < t.peers.size(); ++i)  // the pack's peers are s's messages, in order
    peers[i] = static_cast<char*>(send_buf) + P->msgs[P->src_first[s] + i].displ;
  hipError_t e = etc::launch_copy(true, P->d_boxes + t.first, t.nbox, t.ntiles, 0xFu, etc::kMsgSections,
                                  arenas, peers, int(t.peers.size()), static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "pack launch");
  return ETC_OK;
}

int etc_unpack(const etc_plan_t* P, int d, const void* const* msg, void* const dst_arena[4], void* stream) {
  int rc = check_device_plan(P);
  if (rc) return rc;
  const DeviceCallGuard guard(P);
  if ((rc = guard.check(P))) return rc;
  if (d < 0 || d >= P->dst.world()) return fail(ETC_ERR_RANK, "target rank out of range");
  const etc::CopyTable& t = P->unpack_tab[d];
  if (!t.built) return fail(ETC_ERR_RANK, "target rank " + std::to_string(d) + " is not built into this plan");
  if ((rc = check_arenas(const_cast<const void* const*>(dst_arena), "dst_arena"))) return rc;
  if (!msg && !t.peers.empty()) return fail(ETC_ERR_INVALID_ARG, "msg is NULL");
  void* peers[ETC_MAX_PEERS];
  for (size_t i = 0; i < t.peers.size(); ++i) {
    const void* p = msg[t.peers[i]];
    if (!p) return fail(ETC_ERR_INVALID_ARG, "msg[" + std::to_string(t.peers[i]) + "] is NULL but source " +
                                                 std::to_string(t.peers[i]) + " sends to this target");
    if (!aligned(p, 256)) return fail(ETC_ERR_ALIGN, "msg[" + std::to_string(t.peers[i]) + "] is not 256-byte aligned");
    peers[i] = const_cast<void*>(p);
  }
  hipError_t e = etc::launch_copy(false, P->d_boxes + t.first, t.nbox, t.ntiles, 0xFu, etc::kMsgSections,
                                  dst_arena, peers, int(t.peers.size()), static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "unpack launch");
  return ETC_OK;
}

int etc_plan_chunk_layout(const etc_plan_t* P, int s, int kind, uint64_t* counts, uint64_t* displs,
                          uint64_t* total) {
  int rc = check_side_rank(P, ETC_SIDE_SRC, s);
  if (rc) return rc;
  if (kind < 0 || kind >= ETC_NUM_KINDS) return fail(ETC_ERR_INVALID_ARG, "bad kind");
  const int i = kind == ETC_KIND_PARAM_BF16 ? 0 : 1;
  const uint64_t es = i == 0 ? 2 : 4;
  const int D = P->dst.world();
  uint32_t k = P->src_first[s];
  uint64_t cur = 0;
  for (int d = 0; d < D; ++d) {
    const bool has = k < P->src_first[s + 1] && P->msgs[k].d == d;
    const etc_plan_s::Message* m = has ? &P->msgs[k++] : nullptr;
    if (counts) counts[d] = m ? m->npad * es : 0;
    if (displs) displs[d] = m ? m->chunk_displ[i] : (cur + 255) / 256 * 256;
    if (m) cur = m->chunk_displ[i] + m->npad * es;
  }
  if (total) *total = P->chunk_bytes[i][s];
  return ETC_OK;
}

int etc_pack_kind(const etc_plan_t* P, int s, int kind, const void* src_arena, void* chunk_buf,
                  void* stream) {
  int rc = check_device_plan(P);
  if (rc) return rc;
  const DeviceCallGuard guard(P);
  if ((rc = guard.check(P))) return rc;
  if (kind < 0 || kind >= ETC_NUM_KINDS) return fail(ETC_ERR_INVALID_ARG, "bad kind");
  if (s < 0 || s >= P->src.world()) return fail(ETC_ERR_RANK, "source rank out of range");
  const etc::CopyTable& t = P->pack_tab[s];
  if (!t.built) return fail(ETC_ERR_RANK, "source rank " + std::to_string(s) + " is not built into this plan");
  if (t.ntiles == 0) return ETC_OK;  // routes nothing (e.g. a failed rank): nothing is read
  if (!src_arena || !chunk_buf) return fail(ETC_ERR_INVALID_ARG, "src_arena and chunk_buf must not be NULL");
  if (!aligned(src_arena, 256) || !aligned(chunk_buf, 256))
    return fail(ETC_ERR_ALIGN, "src_arena and chunk_buf must be 256-byte aligned");
  void* arenas[4] = {nullptr, nullptr, nullptr, nullptr};
  arenas[kind] = const_cast<void*>(src_arena);
  const int i = kind == ETC_KIND_PARAM_BF16 ? 0 : 1;
  void* peers[ETC_MAX_PEERS];
  for (size_t j = 0; j < t.peers.size(); ++j)
    peers[j] = static_cast<char*>(chunk_buf) + P->msgs[P->src_first[s] + j].chunk_displ[i];
  hipError_t e = etc::launch_copy(true, P->d_boxes + t.first, t.nbox, t.ntiles, 1u << kind, etc::kMsgOneKind,
                                  arenas, peers, int(t.peers.size()), static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "pack launch");
  return ETC_OK;
}

int etc_unpack_kind(const etc_plan_t* P, int d, int kind, const void* const* msg, void* dst_arena,
                    void* stream) {
  int rc = check_device_plan(P);
  if (rc) return rc;
  const DeviceCallGuard guard(P);
  if ((rc = guard.check(P))) return rc;
  if (kind < 0 || kind >= ETC_NUM_KINDS) return fail(ETC_ERR_INVALID_ARG, "bad kind");
  if (d < 0 || d >= P->dst.world()) return fail(ETC_ERR_RANK, "target rank out of range");
  const etc::CopyTable& t = P->unpack_tab[d];
  if (!t.built) return fail(ETC_ERR_RANK, "target rank " + std::to_string(d) + " is not built into this plan");
  if (!dst_arena) return fail(ETC_ERR_INVALID_ARG, "dst_arena is NULL");
  if (!aligned(dst_arena, 256)) return fail(ETC_ERR_ALIGN, "dst_arena is not 256-byte aligned");
  if (!msg && !t.peers.empty()) return fail(ETC_ERR_INVALID_ARG, "msg is NULL");
  void* peers[ETC_MAX_PEERS];
  for (size_t j = 0; j < t.peers.size(); ++j) {
    const void* p = msg[t.peers[j]];
    if (!p) return fail(ETC_ERR_INVALID_ARG, "msg[" + std::to_string(t.peers[j]) + "] is NULL but source " +
                                                 std::to_string(t.peers[j]) + " sends to this target");
    if (!aligned(p, 256)) return fail(ETC_ERR_ALIGN, "msg[" + std::to_string(t.peers[j]) + "] is not 256-byte aligned");
    peers[j] = const_cast<void*>(p);
  }
  void* arenas[4] = {nullptr, nullptr, nullptr, nullptr};
  arenas[kind] = dst_arena;
  hipError_t e = etc::launch_copy(false, P->d_boxes + t.first, t.nbox, t.ntiles, 1u << kind, etc::kMsgOneKind,
                                  arenas, peers, int(t.peers.size()), static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "unpack launch");
  return ETC_OK;
}

int etc_refer(const etc_plan_t* P, int d, const void* const src_arena[4], void* const dst_arena[4],
              void* stream) {
  int rc = check_device_plan(P);
  if (rc) return rc;
  const DeviceCallGuard guard(P);
  if ((rc = guard.check(P))) return rc;
  if (d < 0 || d >= P->dst.world()) return fail(ETC_ERR_RANK, "target rank out of range");
  const etc::CopyTable& t = P->refer_tab[d];
  if (!t.built) return fail(ETC_ERR_RANK, "target rank " + std::to_string(d) + " is not built into this plan");
  if (t.ntiles == 0) return ETC_OK;  // nothing kept by a paired source
  if ((rc = check_arenas(src_arena, "src_arena"))) return rc;
  if ((rc = check_arenas(const_cast<const void* const*>(dst_arena), "dst_arena"))) return rc;
  void* sources[4];
  for (int k = 0; k < 4; ++k) sources[k] = const_cast<void*>(src_arena[k]);
  hipError_t e = etc::launch_copy(false, P->d_boxes + t.first, t.nbox, t.ntiles, 0xFu, etc::kMsgArenas,
                                  dst_arena, sources, 4, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "refer launch");
  return ETC_OK;
}

int etc_refer_kind(const etc_plan_t* P, int d, int kind, const void* src_arena, void* dst_arena,
                   void* stream) {
  int rc = check_device_plan(P);
  if (rc) return rc;
  const DeviceCallGuard guard(P);
  if ((rc = guard.check(P))) return rc;
  if (kind < 0 || kind >= ETC_NUM_KINDS) return fail(ETC_ERR_INVALID_ARG, "bad kind");
  if (d < 0 || d >= P->dst.world()) return fail(ETC_ERR_RANK, "target rank out of range");
  const etc::CopyTable& t = P->refer_tab[d];
  if (!t.built) return fail(ETC_ERR_RANK, "target rank " + std::to_string(d) + " is not built into this plan");
  if (t.ntiles == 0) return ETC_OK;
  if (!src_arena || !dst_arena) return fail(ETC_ERR_INVALID_ARG, "src_arena and dst_arena must not be NULL");
  if (!aligned(src_arena, 256) || !aligned(dst_arena, 256))
    return fail(ETC_ERR_ALIGN, "src_arena and dst_arena must be 256-byte aligned");
  void* arenas[4] = {nullptr, nullptr, nullptr, nullptr};
  void* sources[4] = {nullptr, nullptr, nullptr, nullptr};
  arenas[kind] = dst_arena;
  sources[kind] = const_cast<void*>(src_arena);
  hipError_t e = etc::launch_copy(false, P->d_boxes + t.first, t.nbox, t.ntiles, 1u << kind, etc::kMsgArenas,
                                  arenas, sources, 4, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "refer launch");
  return ETC_OK;
}

int etc_plan_refer_bytes(const etc_plan_t* P, int d, uint64_t* bytes) {
  int rc = check_side_rank(P, ETC_SIDE_DST, d);
  if (rc) return rc;
  if (!bytes) return fail(ETC_ERR_INVALID_ARG, "bytes is NULL");
  *bytes = P->refer_elems[size_t(d)] * 14;
  return ETC_OK;
}

const char* etc_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
