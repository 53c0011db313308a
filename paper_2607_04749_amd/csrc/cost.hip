// cost.hip -- byte-overlap / routing / cost matrices over every (source,
// target) rank pair, on the GPU (Sec. III-B cost matrix, Sec. III-C LCM
// workload items).  One workgroup per matrix cell; its threads stride over
// the logical tensors, each evaluating the interval form of the routing rule
// (route.hpp) for one tensor; 64-bit partial sums are reduced in LDS.
// Integer work on a few KB of tables: latency bound, microseconds.
#include <hip/hip_runtime.h>

#include "etc_internal.hpp"
#include "route.hpp"

namespace etc {

namespace {

__global__ __launch_bounds__(kCmThreads) void cost_kernel(const RouteTensor* __restrict__ T,
                                                          int nt, const int32_t* __restrict__ home,
                                                          int S, int D, int TPs, int TPd,
                                                          int which, uint64_t* __restrict__ out) {
  __shared__ uint64_t red_val[kCmThreads];
  __shared__ uint64_t red_need[kCmThreads];
  const int s = blockIdx.x / D, d = blockIdx.x % D;
  const int pp_d = d / TPd, tp_d = d % TPd;
  const int pp_s = s / TPs, tp_s = s % TPs;
  const int home_d = home[d];
  uint64_t val = 0, need = 0;
  for (int i = threadIdx.x; i < nt; i += kCmThreads) {
    const RouteTensor t = T[i];
    if (role_on(t.dst_stage, pp_d) < 0) continue;
    const int64_t unit = unit_elems(t);
    const Span want = shard_span(t, tp_d, TPd);
    need += uint64_t(want.len() * unit);
    if (which == ETC_CM_ROUTE) {
      val += uint64_t(routed_span(t, s, d, home_d, TPs, TPd).len() * unit);
    } else {
      if (role_on(t.src_stage, pp_s) < 0) continue;
      if (which == ETC_CM_OVERLAP_SHARDED && !t.single_copy) continue;
      const Span have = shard_span(t, tp_s, TPs);
      const Span x{have.lo > want.lo ? have.lo : want.lo, have.hi < want.hi ? have.hi : want.hi};
      val += uint64_t(x.len() * unit);
    }
  }
  red_val[threadIdx.x] = val;
  red_need[threadIdx.x] = need;
  __syncthreads();
  for (int w = kCmThreads / 2; w > 0; w >>= 1) {
    if (int(threadIdx.x) < w) {
      red_val[threadIdx.x] += red_val[threadIdx.x + w];
      red_need[threadIdx.x] += red_need[threadIdx.x + w];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    constexpr uint64_t kBytesPerElem = 14;  // 2 (bf16) + 4 + 4 + 4 (fp32)
    if (which == ETC_CM_COST)
      out[size_t(d) * S + s] = (red_need[0] - red_val[0]) * kBytesPerElem;
    else
      out[size_t(s) * D + d] = red_val[0] * kBytesPerElem;
  }
}

}  // namespace

hipError_t launch_cost(const RouteTensor* rt, int nt, const int32_t* home, int S, int D, int tps,
                       int tpd, int which, uint64_t* out, hipStream_t stream) {
  hipLaunchKernelGGL(cost_kernel, dim3(unsigned(S) * unsigned(D)), dim3(kCmThreads), 0, stream,
                     rt, nt, home, S, D, tps, tpd, which, out);
  return hipGetLastError();
}

}  // namespace etc
