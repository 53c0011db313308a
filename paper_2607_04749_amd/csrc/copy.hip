// copy.hip -- the pack / unpack copy engine for gfx950 (MI355X).
//
// Pure data movement, HBM bound: each launch copies a list of routed boxes
// between a rank's four state arenas (strided rows) and message sections
// (contiguous rows), for all four state kinds, or (Refer) straight from a
// source rank's arenas into a target rank's.  Boxes are pre-cut on the host
// into uniform tiles of kTileElems elements per kind.
//
// Launch shape: a persistent grid of one 256-thread workgroup per CU (the
// launcher reserves just over half of a CU's LDS per workgroup, so no second
// workgroup can become resident), walking tiles interleaved round by round
// over the grid, each XCD taking a contiguous run of every round
// (first_tile), so the whole GPU sweeps the buffers front to back.
// A tile's descriptor is uniform across the workgroup (scalar loads).
// Within a tile, each thread moves 16-byte vectors in batches: 16 loads in
// flight, then the 16 stores, for contiguous rows (a workgroup streams 64 KB
// per batch); 8, predicated, for strided rows.  Loads and stores are non-temporal since
// nothing is reused.  On MI355X this shape measured best of the ones tried
// (deeper batches at low occupancy beat more resident waves with shallow
// batches: the memory system is saturated and fewer, larger contiguous
// request streams per CU use it better).  A launch of a single state kind
// (state chunking) also batches the shorter 2-byte rows 8 deep; a launch of
// all four kinds does not, which measured faster there.
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

constexpr int kRowBatch = 16;  // vectors in flight per thread, contiguous rows
constexpr int kBatch2D = 8;    // vectors in flight per thread, strided rows (predicated)

// Copy nr rows of row_bytes bytes (16-byte aligned starts, row_bytes a
// multiple of 16 when nr > 1) from src (row pitch sld bytes) to dst (pitch dld).
// kSingle: the launch copies one state kind only.
template <bool kSingle>
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
    if (kSingle) {
      for (; i + 7 * kCopyThreads < nv; i += 8 * kCopyThreads) {
        u32x4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          v[u] = __builtin_nontemporal_load(
              reinterpret_cast<const u32x4*>(src + uint64_t(i + u * kCopyThreads) * 16));
#pragma unroll
        for (int u = 0; u < 8; ++u)
          __builtin_nontemporal_store(
              v[u], reinterpret_cast<u32x4*>(dst + uint64_t(i + u * kCopyThreads) * 16));
      }
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

template <bool kPack, int kKind, bool kSingle>
__device__ __forceinline__ void copy_tile_kind(const CopyArgs& a, const CopyBox& b, char* mbase,
                                               const TileGeom& g) {
  constexpr int es = kKind == 0 ? 2 : 4;
  using E = typename std::conditional<es == 2, uint16_t, uint32_t>::type;
  char* A = a.arena[kKind] + tile_arena_elem(b, g) * es;
  // this kind's section of the message, or (Refer) the source arena of this kind
  char* Mb = a.mode == kMsgArenas ? a.peer[kKind]
                                  : mbase + (a.mode == kMsgSections ? section_byte(b.msg_npad, kKind) : 0);
  char* M = Mb + tile_msg_elem(b, g) * es;
  const char* src = kPack ? A : M;
  char* dst = kPack ? M : A;
  const uint64_t sld = (kPack ? uint64_t(b.a_ld) : b.m_ld) * es;
  const uint64_t dld = (kPack ? b.m_ld : uint64_t(b.a_ld)) * es;
  const bool vec = (b.vec >> (es == 2 ? 0 : 1)) & 1;
  if (vec) {
    constexpr uint32_t vw = 16 / es;
    const uint32_t nvc = g.nr == 1 ? (g.nc / vw) * vw : g.nc;  // vector part of each row
    copy_vec_2d<kSingle>(src, sld, dst, dld, g.nr, nvc * es);
    if (nvc < g.nc)
      copy_elems_2d<E>(reinterpret_cast<const E*>(src), sld / es, reinterpret_cast<E*>(dst),
                       dld / es, g.nr, nvc, g.nc);
  } else {
    copy_elems_2d<E>(reinterpret_cast<const E*>(src), sld / es, reinterpret_cast<E*>(dst),
                     dld / es, g.nr, 0, g.nc);
  }
  if (kPack && g.last && b.pad) {
    // zero the padding that rounds the box up to a multiple of 8 elements
    E* tail = reinterpret_cast<E*>(Mb + (b.m_off + uint64_t(b.rows) * b.cols) * es);
    if (threadIdx.x < b.pad) tail[threadIdx.x] = 0;
  }
}

template <bool kPack, bool kSingle>
__global__ __launch_bounds__(kCopyThreads) void copy_kernel(CopyArgs a) {
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
    const TileGeom g = tile_geom(b, t, next0);
    char* mbase = a.peer[b.peer];
    if (a.kind_mask & 1) copy_tile_kind<kPack, 0, kSingle>(a, b, mbase, g);
    if (a.kind_mask & 2) copy_tile_kind<kPack, 1, kSingle>(a, b, mbase, g);
    if (a.kind_mask & 4) copy_tile_kind<kPack, 2, kSingle>(a, b, mbase, g);
    if (a.kind_mask & 8) copy_tile_kind<kPack, 3, kSingle>(a, b, mbase, g);
  }
}

}  // namespace

hipError_t launch_copy(bool pack, const CopyBox* boxes, uint32_t nbox, uint32_t ntiles,
                       uint32_t grid, uint32_t lds_reserve, uint32_t kind_mask, MsgMode mode,
                       void* const arena[4], void* const* peers, int npeers, hipStream_t stream) {
  if (ntiles == 0 || kind_mask == 0) return hipSuccess;
  CopyArgs a{};
  a.boxes = boxes;
  a.nbox = nbox;
  a.ntiles = ntiles;
  a.kind_mask = kind_mask;
  a.mode = mode;
  for (int k = 0; k < 4; ++k) a.arena[k] = static_cast<char*>(arena[k]);
  for (int p = 0; p < npeers; ++p) a.peer[p] = static_cast<char*>(peers[p]);
  const uint32_t g = grid < ntiles ? grid : ntiles;
  // the dynamic LDS is not used by the kernel: it caps residency at one
  // workgroup per CU
  const bool single = (kind_mask & (kind_mask - 1)) == 0;
  if (pack && single)
    hipLaunchKernelGGL((copy_kernel<true, true>), dim3(g), dim3(kCopyThreads), lds_reserve, stream, a);
  else if (pack)
    hipLaunchKernelGGL((copy_kernel<true, false>), dim3(g), dim3(kCopyThreads), lds_reserve, stream, a);
  else if (single)
    hipLaunchKernelGGL((copy_kernel<false, true>), dim3(g), dim3(kCopyThreads), lds_reserve, stream, a);
  else
    hipLaunchKernelGGL((copy_kernel<false, false>), dim3(g), dim3(kCopyThreads), lds_reserve, stream, a);
  return hipGetLastError();
}

}  // namespace etc
