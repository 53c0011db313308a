// defrag.hip -- the virtual rank allocator (Sec. III-E, Algorithm 2): which
// device finally hosts each new rank once devices are de-fragmented, and the
// remap operators that move processes there.  Host only.
//
// Devices: the S old devices keep their ids; every new rank with no paired
// old rank is started on a fresh device, numbered S, S+1, ... in order of the
// rank.  Devices of failed old ranks are gone and take part in nothing.
//  - occupancy: idle live devices in ascending order take over the processes
//    of occupied devices in descending order, for as long as the idle device
//    precedes the occupied one; the occupied devices end up being the first
//    ones, so whole nodes at the end are freed;
//  - efficiency: the k-th live device (old ones ascending, then fresh ones)
//    finally hosts new rank k, so consecutive ranks -- a TP group, TP being
//    the fastest coordinate -- share a node.
// Coalescing (Sec. III-E) then migrates each new rank straight to its final
// device: the migration whose pairing is the final placement.
#include <cstdint>
#include <vector>

#include "etc.h"
#include "plan.hpp"

namespace etc {

int defrag(int S, int D, const int32_t* home, const std::vector<char>& dead, int mode,
           int32_t* placement, int32_t* ops, int* nops) {
  std::vector<int32_t> where(D);  // device of new rank d right after the migration
  int fresh = S;
  for (int d = 0; d < D; ++d) where[d] = home[d] >= 0 ? home[d] : fresh++;
  const int ndev = fresh;
  std::vector<int32_t> rank_on(ndev, -1);
  for (int d = 0; d < D; ++d) rank_on[where[d]] = d;
  for (int d = 0; d < D; ++d) placement[d] = where[d];
  if (mode == ETC_DEFRAG_OCCUPANCY) {
    std::vector<int> idle, busy;
    for (int v = 0; v < ndev; ++v) {
      if (v < S && dead[v]) continue;
      (rank_on[v] < 0 ? idle : busy).push_back(v);
    }
    for (size_t i = 0, j = busy.size(); i < idle.size() && j > 0 && idle[i] < busy[j - 1]; ++i, --j)
      placement[rank_on[busy[j - 1]]] = idle[i];
  } else if (mode == ETC_DEFRAG_EFFICIENCY) {
    int d = 0;
    for (int v = 0; v < S && d < D; ++v)
      if (!dead[v]) placement[d++] = v;
    for (int v = S; d < D; ++v) placement[d++] = v;
  } else if (mode != ETC_DEFRAG_NONE) {
    return ETC_ERR_INVALID_ARG;
  }
  int k = 0;
  for (int d = 0; d < D; ++d) {
    if (placement[d] == where[d]) continue;
    if (ops) {
      ops[3 * k] = d;
      ops[3 * k + 1] = where[d];
      ops[3 * k + 2] = placement[d];
    }
    ++k;
  }
  *nops = k;
  return ETC_OK;
}

}  // namespace etc
