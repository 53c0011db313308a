// cost.hip -- byte-overlap / routing / cost matrices over every (source,
// target) rank pair, on the GPU (Sec. III-B cost matrix, Sec. III-C LCM
// workload items).  Two or four 64-wide wavefronts per matrix cell; their
// lanes stride over the logical tensors, each evaluating the interval form of
// the routing rule (route.hpp) for one tensor; the 64-bit partial sums are
// reduced with lane shuffles, then across the cell's wavefronts in LDS.
// Integer work on a few KB of tables: latency bound, microseconds.
// COST is ETC_COST_INF between ranks of different data-parallel replicas and
// towards failed ranks (Sec. III-C); a failed rank holds and sends nothing.
#include <hip/hip_runtime.h>

#include "etc_internal.hpp"
#include "route.hpp"

namespace etc {

namespace {

constexpr int kWave = 64;  // wavefront width on CDNA

// Sum of v over the 64 lanes of a wavefront (every lane gets the total).
__device__ __forceinline__ uint64_t wave_sum(uint64_t v) {
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// kWaves wavefronts per matrix cell, kCmThreads / (64 * kWaves) cells per
// workgroup.  Each wavefront reduces with lane shuffles; the wavefronts of a
// cell then add up in LDS after one barrier.
template <int kWaves>
__global__ __launch_bounds__(kCmThreads) void cost_kernel(const RouteTensor* __restrict__ T,
                                                          int nt, const int32_t* __restrict__ home,
                                                          RouteCtx c, int which,
                                                          uint64_t* __restrict__ out) {
  constexpr int kCellThreads = kWave * kWaves;
  constexpr int kCellsPerBlock = kCmThreads / kCellThreads;
  __shared__ uint64_t part[2][kCmThreads / kWave];
  const int S = c.tps * c.pps * c.dps, D = c.tpd * c.ppd * c.dpd;
  const int ct = int(threadIdx.x) % kCellThreads;
  const int cell = int(blockIdx.x) * kCellsPerBlock + int(threadIdx.x) / kCellThreads;
  const bool live = cell < S * D;  // every thread reaches the barrier below
  const int cc = live ? cell : 0;
  const int s = cc / D, d = cc % D;
  const int pp_d = (d % (c.tpd * c.ppd)) / c.tpd, tp_d = d % c.tpd;
  const int pp_s = (s % (c.tps * c.pps)) / c.tps, tp_s = s % c.tps;
  const int rep_s = s / (c.tps * c.pps), rep_d = d / (c.tpd * c.ppd);
  const bool dead = rank_dead(c, s);
  const int home_d = home[d];
  uint64_t val = 0, need = 0;
  for (int i = ct; live && i < nt; i += kCellThreads) {
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
  val = wave_sum(val);
  need = wave_sum(need);
  const int w = int(threadIdx.x) / kWave;
  if (int(threadIdx.x) % kWave == 0) {
    part[0][w] = val;
    part[1][w] = need;
  }
  __syncthreads();
  if (live && ct == 0) {
    val = 0;
    need = 0;
    for (int j = 0; j < kWaves; ++j) {
      val += part[0][w + j];
      need += part[1][w + j];
    }
    constexpr uint64_t kBytesPerElem = 14;  // 2 (bf16) + 4 + 4 + 4 (fp32)
    if (which == ETC_CM_COST)
      out[size_t(d) * S + s] = (dead || rep_s != rep_d) ? uint64_t(ETC_COST_INF)
                                                        : (need - val) * kBytesPerElem;
    else
      out[size_t(s) * D + d] = val * kBytesPerElem;
  }
}

}  // namespace

hipError_t launch_cost(const RouteTensor* rt, int nt, const int32_t* home, RouteCtx ctx,
                       int which, uint64_t* out, hipStream_t stream) {
  const unsigned cells = unsigned(ctx.tps * ctx.pps * ctx.dps) * unsigned(ctx.tpd * ctx.ppd * ctx.dpd);
  // few cells: 4 wavefronts each, so the tensor loop is short; many cells:
  // 2 each, which measured faster on MI355X at 2048 cells
  if (cells <= 1024) {
    hipLaunchKernelGGL(cost_kernel<4>, dim3(cells), dim3(kCmThreads), 0, stream, rt, nt, home,
                       ctx, which, out);
  } else {
    hipLaunchKernelGGL(cost_kernel<2>, dim3((cells + 1) / 2), dim3(kCmThreads), 0, stream, rt, nt,
                       home, ctx, which, out);
  }
  return hipGetLastError();
}

}  // namespace etc
