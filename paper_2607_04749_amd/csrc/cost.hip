// cost.hip -- byte-overlap / routing / cost matrices over every (source,
// target) rank pair, on the GPU (Sec. III-B cost matrix, Sec. III-C LCM
// workload items).  One workgroup per matrix cell; its threads stride over
// the logical tensors, each evaluating the interval form of the routing rule
// (route.hpp) for one tensor; 64-bit partial sums are reduced in LDS.
// Integer work on a few KB of tables: latency bound, microseconds.
// COST is ETC_COST_INF between ranks of different data-parallel replicas and
// towards failed ranks (Sec. III-C); a failed rank holds and sends nothing.
#include <hip/hip_runtime.h>

#include "etc_internal.hpp"
#include "route.hpp"

namespace etc {

namespace {

__global__ __launch_bounds__(kCmThreads) void cost_kernel(const RouteTensor* __restrict__ T,
                                                          int nt, const int32_t* __restrict__ home,
                                                          RouteCtx c, int which,
                                                          uint64_t* __restrict__ out) {
  __shared__ uint64_t red_val[kCmThreads];
  __shared__ uint64_t red_need[kCmThreads];
  const int S = c.tps * c.pps * c.dps, D = c.tpd * c.ppd * c.dpd;
  const int s = blockIdx.x / D, d = blockIdx.x % D;
  const int pp_d = (d % (c.tpd * c.ppd)) / c.tpd, tp_d = d % c.tpd;
  const int pp_s = (s % (c.tps * c.pps)) / c.tps, tp_s = s % c.tps;
  const int rep_s = s / (c.tps * c.pps), rep_d = d / (c.tpd * c.ppd);
  const bool dead = rank_dead(c, s);
  const int home_d = home[d];
  uint64_t val = 0, need = 0;
  for (int i = threadIdx.x; i < nt; i += kCmThreads) {
    const RouteTensor t = T[i];
    if (role_on(t.dst_stage, pp_d) < 0) continue;
    const int64_t unit = unit_elems(t);
    const Span want = shard_span(t, tp_d, c.tpd);
    need += uint64_t(want.len() * unit);
    if (which == ETC_CM_ROUTE) {
      val += uint64_t(routed_span(t, s, d, home_d, c).len() * unit);
    } else {
      if (dead || role_on(t.src_stage, pp_s) < 0) continue;  // a failed rank holds nothing
      if (which == ETC_CM_OVERLAP_SHARDED && (!t.single_copy || rep_s != rep_d % c.dps)) continue;
      const Span have = shard_span(t, tp_s, c.tps);
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
      out[size_t(d) * S + s] = (dead || rep_s != rep_d) ? uint64_t(ETC_COST_INF)
                                                        : (red_need[0] - red_val[0]) * kBytesPerElem;
    else
      out[size_t(s) * D + d] = red_val[0] * kBytesPerElem;
  }
}

}  // namespace

hipError_t launch_cost(const RouteTensor* rt, int nt, const int32_t* home, RouteCtx ctx,
                       int which, uint64_t* out, hipStream_t stream) {
  const unsigned cells = unsigned(ctx.tps * ctx.pps * ctx.dps) * unsigned(ctx.tpd * ctx.ppd * ctx.dpd);
  hipLaunchKernelGGL(cost_kernel, dim3(cells), dim3(kCmThreads), 0, stream, rt, nt, home, ctx,
                     which, out);
  return hipGetLastError();
}

}  // namespace etc
