// copy_geom.hpp -- tile geometry of the copy engine: which box a tile belongs
// to, and the rows and columns of a tile.
// Host and device share it, so the planner's bounds checks and the kernel
// walk the same tiles.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "copy_desc.hpp"

namespace etc {

// Index of the box holding tile t: the last box with tile0 <= t.
__host__ __device__ inline uint32_t box_of_tile(const CopyBox* boxes, uint32_t nbox, uint32_t t) {
  uint32_t lo = 0, hi = nbox;
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) >> 1;
    if (boxes[mid].tile0 <= t) lo = mid;
    else hi = mid;
  }
  return lo;
}

struct TileGeom {
  uint32_t r0, c0, nr, nc;  // tile rows [r0, r0+nr), columns [c0, c0+nc) of the box
  bool last;                // last tile of its box
};

// Geometry of tile t of box b (next0 = first tile of the next box).
__host__ __device__ inline TileGeom tile_geom(const CopyBox& b, uint32_t t, uint32_t next0) {
  TileGeom g;
  const uint32_t j = t - b.tile0;
  const uint32_t band = j / b.ntc, tcol = j - band * b.ntc;
  g.r0 = band * b.tr;
  g.c0 = tcol * b.tc;
  g.nr = b.tr < b.rows - g.r0 ? b.tr : b.rows - g.r0;
  g.nc = b.tc < b.cols - g.c0 ? b.tc : b.cols - g.c0;
  g.last = t + 1 == next0;
  return g;
}

// Element offsets of a tile's first element on each side.
__host__ __device__ inline uint64_t tile_arena_elem(const CopyBox& b, const TileGeom& g) {
  return b.a_off + uint64_t(g.r0) * b.a_ld + g.c0;
}
__host__ __device__ inline uint64_t tile_msg_elem(const CopyBox& b, const TileGeom& g) {
  return b.m_off + uint64_t(g.r0) * b.m_ld + g.c0;
}

// Sub-chunks: a tile splits into kSubPerTile sub-chunks, copied by
// workgroups of kSubThreads threads (one wavefront); a launch of all four
// kinds gives workgroup kSubPerTile * t + j sub-chunk j of tile t.  For each
// kind, sub-chunk j covers the tile's vectors [j * kSubElems / vw,
// (j + 1) * kSubElems / vw) when the kind moves in 16-byte vectors of vw
// elements (one vector per lane at most), else its elements
// [j * kSubElems, (j + 1) * kSubElems), both in row-major order over the
// tile and clipped to the tile's size.
// A launch of one kind cuts a tile of that kind into kind_sub_elems(es)-element
// sub-chunks instead and gives each workgroup kind_group(es) consecutive
// ones of one tile.
constexpr uint32_t kSubThreads = 64;
constexpr uint32_t kSubPerTile = 64;
constexpr uint32_t kSubElems = kTileElems / kSubPerTile;  // 256
static_assert(kSubElems / 4 <= kSubThreads, "a 4-byte kind's sub-chunk must fit one vector per lane");

// One-kind launches, for a kind of es bytes per element: elements per
// sub-chunk (one 16-byte vector per lane of the wavefront: 256 of a 4-byte
// kind, 512 of bf16), sub-chunks per workgroup (8 KB per workgroup for
// every kind), and workgroups per tile.
__host__ __device__ constexpr uint32_t kind_sub_elems(int es) { return kSubThreads * 16u / uint32_t(es); }
__host__ __device__ constexpr uint32_t kind_group(int /*es*/) { return 8u; }
__host__ __device__ constexpr uint32_t kind_wg_per_tile(int es) {
  return kTileElems / kind_sub_elems(es) / kind_group(es);
}
static_assert(kTileElems % (kind_sub_elems(2) * kind_group(2)) == 0 &&
                  kTileElems % (kind_sub_elems(4) * kind_group(4)) == 0,
              "whole groups per tile");
static_assert(kind_sub_elems(2) / 8 <= kSubThreads && kind_sub_elems(4) / 4 <= kSubThreads,
              "a one-kind sub-chunk must fit one vector per lane");

// The workgroups of a one-kind launch walk the tile list in windows, one
// per XCD at a time: the list is cut into kXcds * kKindWindows equal windows
// of consecutive tiles, and the workgroups of XCD x (the hardware deals
// workgroup w to XCD w % kXcds) copy window x, then window x + kXcds, ...,
// each in tile order.  A launch of one kind has one read and one write
// stream; eight fronts far apart in each, every one fed by one XCD, kept
// them faster than one compact front on MI355X (the all-kinds launches,
// with four streams each way, stay compact).  Two windows per XCD rather
// than one keep the XCDs' shares of strided and contiguous tiles even.
constexpr uint32_t kXcds = 8;
constexpr uint32_t kKindWindows = 2;
__host__ __device__ inline uint32_t kind_window_tiles(uint32_t ntiles) {
  return (ntiles + kXcds * kKindWindows - 1) / (kXcds * kKindWindows);
}
// workgroups in a one-kind launch over ntiles tiles (a few past the last
// tile, when the windows overhang it, find no tile)
__host__ __device__ inline uint64_t kind_grid(uint32_t ntiles, int es) {
  return uint64_t(kXcds) * kKindWindows * kind_window_tiles(ntiles) * kind_wg_per_tile(es);
}
// Tile t and group q (sub-chunks [q * kind_group, (q + 1) * kind_group)) of
// workgroup w of a one-kind launch; false for a workgroup past the last tile.
__host__ __device__ inline bool kind_wg_tile(uint32_t w, uint32_t ntiles, int es, uint32_t* t, uint32_t* q) {
  const uint32_t gpt = kind_wg_per_tile(es), per = kind_window_tiles(ntiles);
  const uint32_t x = w % kXcds, k = w / kXcds, s = k / gpt, m = s / per;
  *t = (m * kXcds + x) * per + s % per;
  *q = k % gpt;
  return m < kKindWindows && *t < ntiles;
}

// Whether the kind of element size es moves a tile in 16-byte vectors: the
// box is vector-aligned for that size and every row of the tile is whole
// vectors (a ragged single-row tile goes element by element).
__host__ __device__ inline bool sub_vectors(const CopyBox& b, const TileGeom& g, int es) {
  return ((b.vec >> (es == 2 ? 0 : 1)) & 1) && g.nc % (16u / uint32_t(es)) == 0;
}

// Index range [lo, hi) of sub-chunk j over n items, per items per sub-chunk.
__host__ __device__ inline void sub_range(uint32_t j, uint32_t per, uint32_t n, uint32_t* lo, uint32_t* hi) {
  const uint32_t a = j * per;
  *lo = a < n ? a : n;
  *hi = a + per < n ? a + per : n;
}

// Byte offset of kind k's section inside a message of npad elements per section.
__host__ __device__ inline uint64_t section_byte(uint64_t npad, int k) {
  return npad * (k == 0 ? 0 : (k == 1 ? 2 : (k == 2 ? 6 : 10)));
}

}  // namespace etc
