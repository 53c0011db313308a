// etc_internal.hpp -- internal types of libetc (host planner + gfx950 kernels).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "copy_desc.hpp"
#include "etc.h"

namespace etc {

// ---------------------------------------------------------------------------
// Logical tensors and rank layouts (host)
// ---------------------------------------------------------------------------

enum Split : int32_t { kRepl = 0, kRows = 1, kCols = 2 };
enum Home : int32_t { kFirstStage = 0, kOwnLayer = 1, kLastStage = 2 };

struct LogicalTensor {
  std::string name;
  int64_t rows = 0, cols = 0;  // full (TP = 1) shape; vectors are [n, 1]
  Split split = kRepl;
  Home home = kOwnLayer;
  int32_t layer = -1;
  bool tied_dup = false;  // duplicate (copy role 1) on the last stage when PP > 1
  bool fused = false;     // stored right after the previous tensor (up after gate)
};

// A parallel configuration.  rank = dp * (pp * tp) + pp_i * tp + tp_i: TP
// fastest, then PP, each data-parallel replica a contiguous block of ranks.
struct Grid {
  int tp = 1, pp = 1, dp = 1;
  int world() const { return tp * pp * dp; }
  int replica_size() const { return tp * pp; }
  int replica(int rank) const { return rank / (tp * pp); }
  int pp_of(int rank) const { return (rank % (tp * pp)) / tp; }
  int tp_of(int rank) const { return rank % tp; }
};

struct Piece {
  int32_t tensor, role;
  int64_t r0, r1, c0, c1;  // full-tensor box
  uint64_t off;            // arena element offset
  int64_t ld() const { return c1 - c0; }
  uint64_t elems() const { return uint64_t((r1 - r0) * (c1 - c0)); }
};

struct RankLayout {
  std::vector<Piece> pieces;
  std::vector<int32_t> piece_of_tensor[2];  // [role][tensor] -> piece index or -1
  uint64_t elems = 0;
};

// ---------------------------------------------------------------------------
// Per-tensor routing record, shared by the host planner and the cost kernel
// ---------------------------------------------------------------------------

struct RouteTensor {
  int64_t rows, cols;
  int32_t split;         // Split
  int32_t src_stage[2];  // stage holding copy role 0 / 1 in the source grid, -1 none
  int32_t dst_stage[2];  // same in the target grid
  int32_t single_copy;   // exactly one copy in both grids
};

// Launch table of one rank's pack or unpack.
struct CopyTable {
  bool built = false;
  uint32_t first = 0;   // index of the first box in the plan's device box array
  uint32_t nbox = 0;    // boxes (the array holds one more sentinel box)
  uint32_t ntiles = 0;
  uint64_t bytes = 0;   // payload bytes moved (all four kinds)
  std::vector<int32_t> peers;  // rank of each peer slot (pack: targets, unpack: sources)
};

constexpr int kCmThreads = 256;

// Routing context of a plan: both grids and the failed source ranks (bitmap,
// nullptr when none).  Device copies point at device memory.
struct RouteCtx {
  int tps, pps, dps, tpd, ppd, dpd;
  const uint32_t* failed;
};

hipError_t launch_cost(const RouteTensor* rt, int nt, const int32_t* home, RouteCtx ctx,
                       int which, uint64_t* out, hipStream_t stream);

}  // namespace etc

// The opaque plan.
struct etc_plan_s {
  etc_model_desc model{};
  etc::Grid src, dst;
  int rank = ETC_ALL_RANKS;
  uint32_t flags = 0;
  std::vector<etc::LogicalTensor> tensors;
  std::vector<etc::RouteTensor> route_tensors;
  // layouts of the ranks of one data-parallel replica: every replica has the
  // same (rank r's layout is that of r mod replica size)
  std::vector<etc::RankLayout> src_layout, dst_layout;
  const etc::RankLayout& src_lay(int s) const { return src_layout[size_t(s % src.replica_size())]; }
  const etc::RankLayout& dst_lay(int d) const { return dst_layout[size_t(d % dst.replica_size())]; }
  std::vector<int32_t> home;  // [d]: source rank paired with target d (migration sketch), or -1
  std::vector<uint32_t> failed_bits;  // bitmap of source ranks whose states are lost

  struct MsgBox {
    int32_t tensor, role_d;
    int64_t r0, r1, c0, c1;
    uint64_t moff;
  };
  // One non-empty message s -> d: its boxes in d's arena order.
  struct Message {
    int32_t s = 0, d = 0;
    std::vector<MsgBox> boxes;
    uint64_t elems = 0;  // routed elements
    uint64_t npad = 0;   // padded elements per kind section
    uint64_t displ = 0;  // byte offset in s's send buffer
    // byte offset in s's chunk buffer of a 2-byte (index 0) or 4-byte (1) kind
    uint64_t chunk_displ[2] = {0, 0};
  };
  // Every non-empty message, ordered by source, then target.  Only these are
  // stored (a target hears from a few sources), so a plan's host tables grow
  // with the number of ranks, not with its square.
  std::vector<Message> msgs;
  std::vector<uint32_t> src_first;  // [S + 1]: msgs[src_first[s] .. src_first[s + 1]) are s's
  std::vector<uint32_t> dst_msgs;   // indices into msgs, by target, then source
  std::vector<uint32_t> dst_first;  // [D + 1]: dst_msgs[dst_first[d] .. dst_first[d + 1]) are d's
  // the message s -> d, or nullptr when nothing is routed from s to d
  const Message* find_msg(int s, int d) const {
    size_t lo = src_first[size_t(s)], hi = src_first[size_t(s) + 1];
    while (lo < hi) {
      const size_t mid = (lo + hi) / 2;
      if (msgs[mid].d < d) lo = mid + 1;
      else hi = mid;
    }
    return lo < src_first[size_t(s) + 1] && msgs[lo].d == d ? &msgs[lo] : nullptr;
  }
  // [d]: boxes that d's paired source keeps (Refer), copied arena to arena by
  // etc_refer when the plan has ETC_PLAN_DIRECT_REFER; no message carries them
  std::vector<std::vector<MsgBox>> refer;
  std::vector<uint64_t> refer_elems;
  std::vector<uint64_t> sendbuf_bytes;   // [S]: send buffer length
  std::vector<uint64_t> chunk_bytes[2];  // [S]: chunk buffer length of a 2-byte / 4-byte kind

  // device side
  int device = -1;
  // non-zero: the device tables live in the library's static array of that
  // device (etc_plan_static), written by its static_gen-th call there
  uint64_t static_gen = 0;
  etc::RouteTensor* d_route_tensors = nullptr;
  int32_t* d_home = nullptr;  // device copy of home (D entries)
  uint32_t* d_failed = nullptr;  // device copy of failed_bits
  etc::CopyBox* d_boxes = nullptr;
  std::vector<etc::CopyTable> pack_tab, unpack_tab, refer_tab;
};
