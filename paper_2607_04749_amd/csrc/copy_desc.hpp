// copy_desc.hpp -- what the copy engine's kernels read: the routed-box
// descriptor, the nominal tile size, the message modes and the launcher.
// Host planner and kernels share it.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace etc {

// One routed box between an arena (strided rows) and a message section
// (contiguous, row-major).  Element offsets are kind-independent; the kernel
// scales them by each kind's element size.  The message itself is found
// through the launch's per-peer pointer table.  64 bytes.
struct CopyBox {
  uint64_t a_off;     // arena element offset of the box's first element
  uint64_t m_off;     // element offset inside each kind section of the message
  uint64_t msg_npad;  // elements per kind section of that message
  uint64_t m_ld;      // message-side row stride (elements): cols, or a source arena's row stride
  uint32_t a_ld;      // arena row stride, elements
  uint32_t rows, cols;  // box shape; contiguous boxes are collapsed to one row
  uint32_t tr, tc;    // tile shape (rows x cols)
  uint32_t ntc;       // tiles per row band
  uint32_t tile0;     // first tile of this box in its launch
  uint16_t peer;      // peer slot
  uint8_t pad;        // zero elements after the box in the message (pack)
  uint8_t vec;        // bit0: 16-byte vectors valid for 2-byte kinds, bit1: for 4-byte kinds
};
static_assert(sizeof(CopyBox) == 64, "CopyBox layout");

constexpr uint32_t kTileElems = 16384;  // nominal tile: 16384 elements per kind

// What the message side of a copy launch is.
enum MsgMode : uint32_t {
  kMsgOneKind = 0,   // one kind per message (chunk format)
  kMsgSections = 1,  // four kind sections per message (full format)
  kMsgArenas = 2,    // no message: peers[k] is a source arena of kind k (Refer)
};

// kernel launcher (copy.hip)
// kind_mask: kinds to copy (bit k): all four (one sub-chunk of each kind per
// workgroup) or one (kind_group sub-chunks per workgroup); any other mask is
// hipErrorInvalidValue, and so is a grid over 2^31 - 1 workgroups
hipError_t launch_copy(bool pack, const CopyBox* boxes, uint32_t nbox, uint32_t ntiles, uint32_t kind_mask,
                       MsgMode mode, void* const arena[4], void* const* peers, int npeers, hipStream_t stream);

}  // namespace etc
