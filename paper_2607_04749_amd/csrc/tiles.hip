// tiles.hip -- the copy engine's work tables: every routed box of a rank's
// pack or unpack as a copy descriptor, cut into uniform tiles (host only).
// The planner decides what moves (plan.hip); this file decides how the copy
// kernel walks it.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <string>

#include "etc_internal.hpp"
#include "plan.hpp"
#include "route.hpp"

namespace etc {

namespace {

void fail(int code, const std::string& msg) { throw PlanError(code, msg); }

// Longest row of a copy descriptor: a contiguous run longer than 2^32 - 1
// elements is cut into rows of this many elements plus a one-row remainder.
// A multiple of 8 and of kTileElems, so vector alignment and tile boundaries
// carry over to the pieces.
constexpr int64_t kMaxRunElems = int64_t(1) << 31;

// Fill the copy descriptor of one box with its tiles starting at tile0.
// m_ld: row stride on the message side (cols for a message, whose boxes are
// row-major; a source arena's row stride for a Refer box).
CopyBox make_box(uint64_t a_off, int64_t a_ld, int64_t rows, int64_t cols, uint64_t m_off,
                 uint64_t msg_npad, int peer, bool pack, uint32_t tile0, int64_t m_ld) {
  if (cols > int64_t(UINT32_MAX) || rows > int64_t(UINT32_MAX) || a_ld > int64_t(UINT32_MAX))
    fail(ETC_ERR_UNSUPPORTED, "a strided routed box exceeds 2^32 - 1 rows or elements per row");
  CopyBox b{};
  b.a_off = a_off;
  b.m_off = m_off;
  b.msg_npad = msg_npad;
  b.m_ld = uint64_t(m_ld);
  b.a_ld = uint32_t(a_ld);
  b.rows = uint32_t(rows);
  b.cols = uint32_t(cols);
  if (cols >= int64_t(kTileElems)) {
    b.tc = kTileElems;
    b.tr = 1;
  } else {
    b.tc = uint32_t(cols);
    b.tr = uint32_t(std::max<int64_t>(1, std::min<int64_t>(rows, kTileElems / cols)));
  }
  b.ntc = uint32_t((cols + b.tc - 1) / b.tc);
  b.tile0 = tile0;
  b.peer = uint16_t(peer);
  const uint64_t n = uint64_t(rows) * uint64_t(cols);
  b.pad = pack ? uint8_t((8 - n % 8) % 8) : 0;
  // 16-byte vectors: 8 elements of a 2-byte kind, 4 of a 4-byte kind.  The
  // message side starts every box at a multiple of 8 elements.
  auto ok = [&](uint64_t w) {
    if (a_off % w || m_off % w) return false;
    if (rows > 1 && (uint64_t(a_ld) % w || uint64_t(cols) % w || uint64_t(m_ld) % w)) return false;
    return true;
  };
  b.vec = uint8_t((ok(8) ? 1 : 0) | (ok(4) ? 2 : 0));
  return b;
}

uint32_t box_tiles(const CopyBox& b) {
  const uint64_t ntr = (uint64_t(b.rows) + b.tr - 1) / b.tr;
  return uint32_t(ntr * b.ntc);
}

// Append the descriptors of one routed box (rows x cols elements, arena row
// stride a_ld, message-side row stride m_ld) to a launch of `tiles` tiles so far.
// A box whose rows are adjacent on both sides is one contiguous run and is
// copied as such: as one row, or, beyond kMaxRunElems, as full rows of
// kMaxRunElems elements and a remainder row (the pack pads only after the last).
void add_box(std::vector<CopyBox>& v, uint32_t& tiles, uint64_t a_off, int64_t a_ld, int64_t rows,
             int64_t cols, uint64_t m_off, uint64_t msg_npad, int peer, bool pack, int64_t m_ld) {
  auto push = [&](const CopyBox& c) {
    const uint64_t nt = uint64_t(tiles) + box_tiles(c);
    if (nt > UINT32_MAX) fail(ETC_ERR_UNSUPPORTED, "too many tiles for one launch");
    tiles = uint32_t(nt);
    v.push_back(c);
  };
  if (rows == 1 || (cols == a_ld && cols == m_ld)) {
    const int64_t n = rows * cols;
    const int64_t full = n > int64_t(UINT32_MAX) ? n / kMaxRunElems : 0;
    if (full > 0)
      push(make_box(a_off, kMaxRunElems, full, kMaxRunElems, m_off, msg_npad, peer, false, tiles,
                    kMaxRunElems));
    const int64_t done = full * kMaxRunElems, rest = n - done;
    if (rest > 0)
      push(make_box(a_off + uint64_t(done), rest, 1, rest, m_off + uint64_t(done), msg_npad, peer, pack,
                    tiles, rest));
    return;
  }
  push(make_box(a_off, a_ld, rows, cols, m_off, msg_npad, peer, pack, tiles, m_ld));
}

}  // namespace

std::vector<CopyBox> build_pack_boxes(const etc_plan_t& P, int s, std::vector<int32_t>* peers,
                                      uint64_t* bytes) {
  std::vector<CopyBox> v;
  uint32_t tiles = 0;
  uint64_t moved = 0;
  const RankLayout& L = P.src_lay(s);
  peers->clear();
  for (uint32_t k = P.src_first[s]; k < P.src_first[s + 1]; ++k) {  // targets ascending
    const etc_plan_s::Message& m = P.msgs[k];
    const int slot = int(peers->size());
    if (slot >= ETC_MAX_PEERS) fail(ETC_ERR_UNSUPPORTED, "one source feeds more than ETC_MAX_PEERS targets");
    peers->push_back(m.d);
    for (const auto& b : m.boxes) {
      const int role_s = role_on(P.route_tensors[b.tensor].src_stage, P.src.pp_of(s));
      const Piece& p = L.pieces[L.piece_of_tensor[role_s][b.tensor]];
      const uint64_t a_off = p.off + uint64_t((b.r0 - p.r0) * p.ld() + (b.c0 - p.c0));
      add_box(v, tiles, a_off, p.ld(), b.r1 - b.r0, b.c1 - b.c0, b.moff, m.npad, slot, true,
              b.c1 - b.c0);
      moved += uint64_t((b.r1 - b.r0) * (b.c1 - b.c0)) * 14;
    }
  }
  CopyBox sentinel{};
  sentinel.tile0 = tiles;
  v.push_back(sentinel);
  if (bytes) *bytes = moved;
  return v;
}

std::vector<CopyBox> build_unpack_boxes(const etc_plan_t& P, int d, std::vector<int32_t>* peers,
                                        uint64_t* bytes) {
  std::vector<CopyBox> v;
  uint32_t tiles = 0;
  uint64_t moved = 0;
  const RankLayout& L = P.dst_lay(d);
  peers->clear();
  for (uint32_t k = P.dst_first[d]; k < P.dst_first[d + 1]; ++k) {  // sources ascending
    const etc_plan_s::Message& m = P.msgs[P.dst_msgs[k]];
    const int slot = int(peers->size());
    if (slot >= ETC_MAX_PEERS) fail(ETC_ERR_UNSUPPORTED, "more than ETC_MAX_PEERS sources feed one target");
    peers->push_back(m.s);
    for (const auto& b : m.boxes) {
      const Piece& q = L.pieces[L.piece_of_tensor[b.role_d][b.tensor]];
      const uint64_t a_off = q.off + uint64_t((b.r0 - q.r0) * q.ld() + (b.c0 - q.c0));
      add_box(v, tiles, a_off, q.ld(), b.r1 - b.r0, b.c1 - b.c0, b.moff, m.npad, slot, false,
              b.c1 - b.c0);
      moved += uint64_t((b.r1 - b.r0) * (b.c1 - b.c0)) * 14;
    }
  }
  CopyBox sentinel{};
  sentinel.tile0 = tiles;
  v.push_back(sentinel);
  if (bytes) *bytes = moved;
  return v;
}

std::vector<CopyBox> build_refer_boxes(const etc_plan_t& P, int d, uint64_t* bytes) {
  std::vector<CopyBox> v;
  uint32_t tiles = 0;
  uint64_t moved = 0;
  const int h = P.home[d];
  if (h >= 0) {
    const RankLayout& L = P.dst_lay(d);
    const RankLayout& H = P.src_lay(h);
    for (const auto& b : P.refer[d]) {
      const int role_s = role_on(P.route_tensors[b.tensor].src_stage, P.src.pp_of(h));
      const Piece& p = H.pieces[H.piece_of_tensor[role_s][b.tensor]];
      const Piece& q = L.pieces[L.piece_of_tensor[b.role_d][b.tensor]];
      const uint64_t a_off = q.off + uint64_t((b.r0 - q.r0) * q.ld() + (b.c0 - q.c0));
      const uint64_t s_off = p.off + uint64_t((b.r0 - p.r0) * p.ld() + (b.c0 - p.c0));
      add_box(v, tiles, a_off, q.ld(), b.r1 - b.r0, b.c1 - b.c0, s_off, 0, 0, false, p.ld());
      moved += uint64_t((b.r1 - b.r0) * (b.c1 - b.c0)) * 14;
    }
  }
  CopyBox sentinel{};
  sentinel.tile0 = tiles;
  v.push_back(sentinel);
  if (bytes) *bytes = moved;
  return v;
}

}  // namespace etc
