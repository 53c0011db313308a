// copy.hip -- the pack / unpack copy engine for gfx950 (MI355X).
//
// Pure data movement, HBM bound: each launch copies a list of routed boxes
// between a rank's four state arenas (strided rows) and message sections
// (contiguous rows), for all four state kinds, or (Refer) straight from a
// source rank's arenas into a target rank's.  Boxes are pre-cut on the host
// into uniform tiles of kTileElems elements per kind.
//
// Launch shape: short-lived one-wavefront workgroups (kSubThreads threads)
// over sub-chunks of the tiles, kSubElems elements of a kind each (1 KB of an
// fp32 kind, one 16-byte vector per lane; 512 B of bf16).  A launch of all
// four kinds (pack, unpack, Refer) gives each workgroup one sub-chunk of
// every kind, copied kind after kind; a launch of one kind (state chunking)
// gives each workgroup kind_group consecutive sub-chunks of that kind, each a
// full wavefront of vectors (kind_sub_elems: 1 KB, 512 bf16 elements or 256
// fp32 ones), 8 KB per workgroup, and walks the tiles in one window per XCD
// at a time (kind_wg_tile).
// Either way a workgroup finds its tile's descriptor once (a binary search of
// the tile table, scalar loads) and then moves a few KB.  The hardware
// dispatches the workgroups in index order, so the whole GPU advances
// through each buffer as one compact front; an all-kinds launch reserves
// LDS so that at most 25 of its workgroups share a CU (kSubLdsBytes).  On MI355X this ran 5-14 %
// faster than a persistent grid of one deep-batched workgroup per CU for all
// four kinds, and up to 9 % faster for one kind, and it holds its rate where
// the persistent grid lost about 10 % to an unfavourable relative placement
// of the source and target buffers.  Loads and stores are non-temporal since
// nothing is reused.
#include <hip/hip_runtime.h>

#include "copy_desc.hpp"
#include "copy_geom.hpp"
#include "etc.h"

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
// All four kinds: one sub-chunk of each kind per workgroup.

// Sub-chunk j (kSub elements) of one kind of a tile.
template <bool kPack, int kKind, uint32_t kSub>
__device__ __forceinline__ void copy_sub_kind(const CopyArgs& a, const CopyBox& b, char* mbase,
                                              const TileGeom& g, uint32_t j) {
  using KT = KindTile<kPack, kKind>;
  using E = typename KT::E;
  constexpr int es = KT::es;
  static_assert(kSub * es / 16 <= kSubThreads, "at most one vector per lane");
  const KT k(a, b, mbase, g);
  uint32_t lo, hi;
  if (sub_vectors(b, g, es)) {
    constexpr uint32_t vw = 16 / es;
    const uint32_t vpr = g.nc / vw;
    sub_range(j, kSub / vw, g.nr * vpr, &lo, &hi);
    const uint32_t i = lo + threadIdx.x;  // at most one vector per lane
    if (i < hi) {
      const uint32_t r = g.nr == 1 ? 0 : i / vpr;
      const uint32_t c = i - r * vpr;
      __builtin_nontemporal_store(
          __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(k.src + r * k.sld + uint64_t(c) * 16)),
          reinterpret_cast<u32x4*>(k.dst + r * k.dld + uint64_t(c) * 16));
    }
  } else {
    sub_range(j, kSub, g.nr * g.nc, &lo, &hi);
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
  copy_sub_kind<kPack, 0, kSubElems>(a, b, mbase, g, j);
  copy_sub_kind<kPack, 1, kSubElems>(a, b, mbase, g, j);
  copy_sub_kind<kPack, 2, kSubElems>(a, b, mbase, g, j);
  copy_sub_kind<kPack, 3, kSubElems>(a, b, mbase, g, j);
}

// ---------------------------------------------------------------------------
// One kind: kind_group(es) consecutive sub-chunks of kind_sub_elems(es)
// elements of one tile per workgroup.

template <bool kPack, int kKind>
__device__ __forceinline__ void copy_kind_group(const CopyArgs& a) {
  constexpr int es = kKind == 0 ? 2 : 4;
  constexpr uint32_t sub = kind_sub_elems(es), grp = kind_group(es);
  uint32_t t, q;
  if (!kind_wg_tile(blockIdx.x, a.ntiles, es, &t, &q)) return;  // past the last tile
  const uint32_t bi = box_of_tile(a.boxes, a.nbox, t);
  const CopyBox b = a.boxes[bi];
  const TileGeom g = tile_geom(b, t, a.boxes[bi + 1].tile0);
  char* mbase = a.peer[b.peer];
#pragma unroll
  for (uint32_t i = 0; i < grp; ++i) copy_sub_kind<kPack, kKind, sub>(a, b, mbase, g, q * grp + i);
}

template <bool kPack>
__global__ __launch_bounds__(kSubThreads) void copy_kind_kernel(CopyArgs a) {
  switch (a.kind_mask) {
    case 1: copy_kind_group<kPack, 0>(a); break;
    case 2: copy_kind_group<kPack, 1>(a); break;
    case 4: copy_kind_group<kPack, 2>(a); break;
    case 8: copy_kind_group<kPack, 3>(a); break;
    default: break;
  }
}

// LDS reserved per workgroup of an all-kinds launch and never touched: with
// 160 KB of LDS per CU it lets at most 25 of these one-wave workgroups share
// a CU, where they would otherwise fill its 32 wave slots.  The copy keeps
// HBM's queues full either way.  With fewer requests queued, MI355X ran the
// 70B and 7B shares 2-3 % faster in their slower buffer placements, and
// every other all-kinds launch measured within -1 to +1.6 %.  A cap of 21
// workgroups ran 1-3.5 % below the cap of 25.  One-kind launches, whose
// workgroups move 8 KB each, lost with any cap and keep all 32 slots.
constexpr unsigned kSubLdsBytes = 6400;

}  // namespace

hipError_t launch_copy(bool pack, const CopyBox* boxes, uint32_t nbox, uint32_t ntiles, uint32_t kind_mask,
                       MsgMode mode, void* const arena[4], void* const* peers, int npeers, hipStream_t stream) {
  if (ntiles == 0 || kind_mask == 0) return hipSuccess;
  const bool all = kind_mask == 0xFu;
  const bool single = kind_mask < 16 && (kind_mask & (kind_mask - 1)) == 0;
  if (!all && !single) return hipErrorInvalidValue;  // a launch copies all four kinds or one
  const uint64_t nwg = all ? uint64_t(ntiles) * kSubPerTile : kind_grid(ntiles, kind_mask == 1 ? 2 : 4);
  if (nwg > uint64_t(INT32_MAX)) return hipErrorInvalidValue;
  CopyArgs a{};
  a.boxes = boxes;
  a.nbox = nbox;
  a.ntiles = ntiles;
  a.kind_mask = kind_mask;
  a.mode = mode;
  for (int k = 0; k < 4; ++k) a.arena[k] = static_cast<char*>(arena[k]);
  for (int p = 0; p < npeers; ++p) a.peer[p] = static_cast<char*>(peers[p]);
  const dim3 grid = dim3(uint32_t(nwg)), block = dim3(kSubThreads);
  if (all && pack)
    hipLaunchKernelGGL((copy_sub_kernel<true>), grid, block, kSubLdsBytes, stream, a);
  else if (all)
    hipLaunchKernelGGL((copy_sub_kernel<false>), grid, block, kSubLdsBytes, stream, a);
  else if (pack)
    hipLaunchKernelGGL((copy_kind_kernel<true>), grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL((copy_kind_kernel<false>), grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace etc
