// copy.hip -- the pack / unpack copy engine for gfx950 (MI355X).
//
// Pure data movement, HBM bound: each launch copies a list of routed boxes
// between a rank's four state arenas (strided rows) and message sections
// (contiguous rows), for all four state kinds, or (Refer) straight from a
// source rank's arenas into a target rank's.  Boxes are pre-cut on the host
// into uniform tiles of kTileElems elements per kind.
//
// Two launch shapes, chosen by what a launch copies:
//
// All four kinds (pack, unpack, Refer): one short-lived one-wavefront
// workgroup per sub-chunk of a tile, kSubPerTile per tile and kSubElems
// elements of each kind per sub-chunk (1 KB of each fp32 kind, one 16-byte
// vector per lane; 512 B of bf16), the kinds copied one after another.  The
// hardware dispatches the workgroups in index order, so the whole GPU
// advances through each buffer as one compact front.  On MI355X this ran
// 5-14 % faster than a persistent grid on every share measured, and it holds
// its rate where the persistent kernel loses about 10 % to an unfavourable
// relative placement of the source and target buffers.
//
// One kind (state chunking): a persistent grid of one 256-thread workgroup
// per CU (the launcher reserves just over half of a CU's LDS per workgroup,
// so no second workgroup can become resident), walking tiles interleaved
// round by round over the grid, each XCD taking a contiguous run of every
// round (first_tile).  Within a tile each thread moves 16-byte vectors in
// batches: 16 loads in flight, then the 16 stores, for contiguous rows
// (8 deep for the shorter bf16 rows); 8, predicated, for strided rows.
//
// A tile's descriptor is uniform across the workgroup (scalar loads).  Loads
// and stores are non-temporal since nothing is reused.
#include <hip/hip_runtime.h>

#include "copy_geom.hpp"
#include "etc_internal.hpp"

namespace etc {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

struct CopyArgs {
  const CopyBox* boxes;  // nbox boxes + 1 sentinel (tile0 = ntiles)
  uint32_t nbox;
  uint32_t ntiles;
  uint32_t kind_mask;  // kinds to copy (bit k)
  uint32_t mode;       // MsgMode: what peer[] points at
  char* arena[4];
  char* peer[ETC_MAX_PEERS];  // start of each peer's message (kMsgArenas: source arena of kind k)
};

// One kind of one tile: where the copy reads and writes, and the row pitches.
template <bool kPack, int kKind>
struct KindTile {
  static constexpr int es = kKind == 0 ? 2 : 4;
  using E = typename std::conditional<es == 2, uint16_t, uint32_t>::type;
  char* Mb;  // this kind's section of the message, or (Refer) the source arena of this kind
  const char* src;
  char* dst;
  uint64_t sld, dld;  // row pitches in bytes
  __device__ __forceinline__ KindTile(const CopyArgs& a, const CopyBox& b, char* mbase, const TileGeom& g) {
    char* A = a.arena[kKind] + tile_arena_elem(b, g) * es;
    Mb = a.mode == kMsgArenas ? a.peer[kKind]
                              : mbase + (a.mode == kMsgSections ? section_byte(b.msg_npad, kKind) : 0);
    char* M = Mb + tile_msg_elem(b, g) * es;
    src = kPack ? A : M;
    dst = kPack ? M : A;
    sld = (kPack ? uint64_t(b.a_ld) : b.m_ld) * es;
    dld = (kPack ? b.m_ld : uint64_t(b.a_ld)) * es;
  }
  // zero the padding that rounds the box up to a multiple of 8 elements
  __device__ __forceinline__ void zero_pad(const CopyBox& b) const {
    E* tail = reinterpret_cast<E*>(Mb + (b.m_off + uint64_t(b.rows) * b.cols) * es);
    if (threadIdx.x < b.pad) tail[threadIdx.x] = 0;
  }
};

// ---------------------------------------------------------------------------
// All four kinds: one workgroup per sub-chunk.

template <bool kPack, int kKind>
__device__ __forceinline__ void copy_sub_kind(const CopyArgs& a, const CopyBox& b, char* mbase,
                                              const TileGeom& g, uint32_t j) {
  using KT = KindTile<kPack, kKind>;
  using E = typename KT::E;
  constexpr int es = KT::es;
  const KT k(a, b, mbase, g);
  uint32_t lo, hi;
  if (sub_vectors(b, g, es)) {
    constexpr uint32_t vw = 16 / es;
    const uint32_t vpr = g.nc / vw;
    sub_range(j, kSubElems / vw, g.nr * vpr, &lo, &hi);
    const uint32_t i = lo + threadIdx.x;  // at most one vector per lane
    if (i < hi) {
      const uint32_t r = g.nr == 1 ? 0 : i / vpr;
      const uint32_t c = i - r * vpr;
      __builtin_nontemporal_store(
          __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(k.src + r * k.sld + uint64_t(c) * 16)),
          reinterpret_cast<u32x4*>(k.dst + r * k.dld + uint64_t(c) * 16));
    }
  } else {
    sub_range(j, kSubElems, g.nr * g.nc, &lo, &hi);
    const E* S = reinterpret_cast<const E*>(k.src);
    E* D = reinterpret_cast<E*>(k.dst);
    for (uint32_t i = lo + threadIdx.x; i < hi; i += kSubThreads) {
      const uint32_t r = i / g.nc, c = i - r * g.nc;
      D[r * (k.dld / es) + c] = S[r * (k.sld / es) + c];
    }
  }
  if (kPack && j == 0 && g.last && b.pad) k.zero_pad(b);
}

template <bool kPack>
__global__ __launch_bounds__(kSubThreads) void copy_sub_kernel(CopyArgs a) {
  const uint32_t t = blockIdx.x / kSubPerTile, j = blockIdx.x % kSubPerTile;
  const uint32_t bi = box_of_tile(a.boxes, a.nbox, t);
  const CopyBox b = a.boxes[bi];
  const TileGeom g = tile_geom(b, t, a.boxes[bi + 1].tile0);
  char* mbase = a.peer[b.peer];
  copy_sub_kind<kPack, 0>(a, b, mbase, g, j);
  copy_sub_kind<kPack, 1>(a, b, mbase, g, j);
  copy_sub_kind<kPack, 2>(a, b, mbase, g, j);
  copy_sub_kind<kPack, 3>(a, b, mbase, g, j);
}

// ---------------------------------------------------------------------------
// One kind: a persistent grid.

constexpr int kRowBatch = 16;  // vectors in flight per thread, contiguous rows
constexpr int kRowBatch2 = 8;  // then the rest of a contiguous row (a bf16 tile is 8 vectors per thread)
constexpr int kBatch2D = 8;    // vectors in flight per thread, strided rows (predicated)

// Copy nr rows of row_bytes bytes (16-byte aligned starts, row_bytes a
// multiple of 16 when nr > 1) from src (row pitch sld bytes) to dst (pitch dld).
__device__ __forceinline__ void copy_vec_2d(const char* __restrict__ src, uint64_t sld,
                                            char* __restrict__ dst, uint64_t dld, uint32_t nr,
                                            uint32_t row_bytes) {
  const uint32_t vpr = row_bytes >> 4;
  const uint32_t nv = nr * vpr;
  uint32_t i = threadIdx.x;
  if (nr == 1) {
    for (; i + (kRowBatch - 1) * kCopyThreads < nv; i += kRowBatch * kCopyThreads) {
      u32x4 v[kRowBatch];
#pragma unroll
      for (int u = 0; u < kRowBatch; ++u)
        v[u] = __builtin_nontemporal_load(
            reinterpret_cast<const u32x4*>(src + uint64_t(i + u * kCopyThreads) * 16));
#pragma unroll
      for (int u = 0; u < kRowBatch; ++u)
        __builtin_nontemporal_store(
            v[u], reinterpret_cast<u32x4*>(dst + uint64_t(i + u * kCopyThreads) * 16));
    }
    for (; i + (kRowBatch2 - 1) * kCopyThreads < nv; i += kRowBatch2 * kCopyThreads) {
      u32x4 v[kRowBatch2];
#pragma unroll
      for (int u = 0; u < kRowBatch2; ++u)
        v[u] = __builtin_nontemporal_load(
            reinterpret_cast<const u32x4*>(src + uint64_t(i + u * kCopyThreads) * 16));
#pragma unroll
      for (int u = 0; u < kRowBatch2; ++u)
        __builtin_nontemporal_store(
            v[u], reinterpret_cast<u32x4*>(dst + uint64_t(i + u * kCopyThreads) * 16));
    }
    for (; i < nv; i += kCopyThreads)
      __builtin_nontemporal_store(
          __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src + uint64_t(i) * 16)),
          reinterpret_cast<u32x4*>(dst + uint64_t(i) * 16));
    return;
  }
  // Strided rows: a tile holds a few thousand vectors, not a multiple of the
  // batch, so the last batch is predicated rather than finished one vector at
  // a time.
  for (; i < nv; i += kBatch2D * kCopyThreads) {
    u32x4 v[kBatch2D];
    uint32_t r[kBatch2D], c[kBatch2D];
#pragma unroll
    for (int u = 0; u < kBatch2D; ++u) {
      const uint32_t idx = i + u * kCopyThreads;
      r[u] = idx / vpr;
      c[u] = idx - r[u] * vpr;
      if (idx < nv)
        v[u] = __builtin_nontemporal_load(
            reinterpret_cast<const u32x4*>(src + r[u] * sld + uint64_t(c[u]) * 16));
    }
#pragma unroll
    for (int u = 0; u < kBatch2D; ++u)
      if (i + u * kCopyThreads < nv)
        __builtin_nontemporal_store(
            v[u], reinterpret_cast<u32x4*>(dst + r[u] * dld + uint64_t(c[u]) * 16));
  }
}

// Element-wise copy of columns [c_begin, nc) of nr rows (any alignment).
template <typename E>
__device__ __forceinline__ void copy_elems_2d(const E* __restrict__ src, uint64_t sld,
                                              E* __restrict__ dst, uint64_t dld, uint32_t nr,
                                              uint32_t c_begin, uint32_t nc) {
  const uint32_t w = nc - c_begin;
  const uint32_t n = nr * w;
  for (uint32_t i = threadIdx.x; i < n; i += kCopyThreads) {
    const uint32_t r = i / w, c = c_begin + (i - r * w);
    dst[r * dld + c] = src[r * sld + c];
  }
}

template <bool kPack, int kKind>
__device__ __forceinline__ void copy_tile_kind(const CopyArgs& a, const CopyBox& b, char* mbase,
                                               const TileGeom& g) {
  using KT = KindTile<kPack, kKind>;
  using E = typename KT::E;
  constexpr int es = KT::es;
  const KT k(a, b, mbase, g);
  const bool vec = (b.vec >> (es == 2 ? 0 : 1)) & 1;
  if (vec) {
    constexpr uint32_t vw = 16 / es;
    const uint32_t nvc = g.nr == 1 ? (g.nc / vw) * vw : g.nc;  // vector part of each row
    copy_vec_2d(k.src, k.sld, k.dst, k.dld, g.nr, nvc * es);
    if (nvc < g.nc)
      copy_elems_2d<E>(reinterpret_cast<const E*>(k.src), k.sld / es, reinterpret_cast<E*>(k.dst),
                       k.dld / es, g.nr, nvc, g.nc);
  } else {
    copy_elems_2d<E>(reinterpret_cast<const E*>(k.src), k.sld / es, reinterpret_cast<E*>(k.dst),
                     k.dld / es, g.nr, 0, g.nc);
  }
  if (kPack && g.last && b.pad) k.zero_pad(b);
}

template <bool kPack, int kKind>
__device__ __forceinline__ void copy_walk(const CopyArgs& a) {
  uint32_t t = first_tile(blockIdx.x, gridDim.x);
  if (t >= a.ntiles) return;
  uint32_t bi = box_of_tile(a.boxes, a.nbox, t);
  CopyBox b = a.boxes[bi];
  uint32_t next0 = a.boxes[bi + 1].tile0;
  for (; t < a.ntiles; t += gridDim.x) {
    while (t >= next0) {
      ++bi;
      b = a.boxes[bi];
      next0 = a.boxes[bi + 1].tile0;
    }
    copy_tile_kind<kPack, kKind>(a, b, a.peer[b.peer], tile_geom(b, t, next0));
  }
}

template <bool kPack>
__global__ __launch_bounds__(kCopyThreads) void copy_kernel(CopyArgs a) {
  switch (a.kind_mask) {
    case 1: copy_walk<kPack, 0>(a); break;
    case 2: copy_walk<kPack, 1>(a); break;
    case 4: copy_walk<kPack, 2>(a); break;
    case 8: copy_walk<kPack, 3>(a); break;
    default: break;
  }
}

}  // namespace

hipError_t launch_copy(bool pack, const CopyBox* boxes, uint32_t nbox, uint32_t ntiles,
                       uint32_t grid, uint32_t lds_reserve, uint32_t kind_mask, MsgMode mode,
                       void* const arena[4], void* const* peers, int npeers, hipStream_t stream) {
  if (ntiles == 0 || kind_mask == 0) return hipSuccess;
  const bool all = kind_mask == 0xFu;
  const bool single = kind_mask < 16 && (kind_mask & (kind_mask - 1)) == 0;
  if (!all && !single) return hipErrorInvalidValue;  // a launch copies all four kinds or one
  CopyArgs a{};
  a.boxes = boxes;
  a.nbox = nbox;
  a.ntiles = ntiles;
  a.kind_mask = kind_mask;
  a.mode = mode;
  for (int k = 0; k < 4; ++k) a.arena[k] = static_cast<char*>(arena[k]);
  for (int p = 0; p < npeers; ++p) a.peer[p] = static_cast<char*>(peers[p]);
  if (all) {
    const uint64_t nwg = uint64_t(ntiles) * kSubPerTile;
    if (nwg > uint64_t(INT32_MAX)) return hipErrorInvalidValue;
    if (pack)
      hipLaunchKernelGGL((copy_sub_kernel<true>), dim3(uint32_t(nwg)), dim3(kSubThreads), 0, stream, a);
    else
      hipLaunchKernelGGL((copy_sub_kernel<false>), dim3(uint32_t(nwg)), dim3(kSubThreads), 0, stream, a);
    return hipGetLastError();
  }
  const uint32_t g = grid < ntiles ? grid : ntiles;
  // the dynamic LDS is not used by the kernel: it caps residency at one
  // workgroup per CU
  if (pack)
    hipLaunchKernelGGL((copy_kernel<true>), dim3(g), dim3(kCopyThreads), lds_reserve, stream, a);
  else
    hipLaunchKernelGGL((copy_kernel<false>), dim3(g), dim3(kCopyThreads), lds_reserve, stream, a);
  return hipGetLastError();
}

}  // namespace etc
