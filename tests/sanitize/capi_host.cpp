// capi_host.cpp -- host-only exercise of the C ABI, built with the host
// sanitizers by tests/test_sanitizers.py: plans built with ETC_PLAN_HOST_ONLY
// (GPT and Llama micro models over TP, PP in {1, 2, 4}, data parallelism with a
// failed rank, the Llama-70B shape), every query, the sketch, the rank
// allocator and error paths.  Test code: it computes no expected values.
#include <cstdio>
#include <cstdlib>
#include <vector>
#include "etc.h"
static int bad = 0;
#define CHECK(c) do { if (!(c)) { printf("FAIL line %d: %s (%s)\n", __LINE__, #c, etc_last_error()); ++bad; } } while (0)
static void exercise(const etc_model_desc& m, etc_parallel_cfg a, etc_parallel_cfg b, uint32_t flags,
                     const int32_t* failed, int nf) {
  etc_plan_options o{nullptr, failed, nf, ETC_ALL_RANKS, flags | ETC_PLAN_HOST_ONLY};
  etc_plan_t* p = nullptr;
  int rc = etc_plan(&m, &a, &b, &o, &p);
  if (rc == ETC_ERR_UNRECOVERABLE) return;
  CHECK(rc == ETC_OK);
  if (rc) return;
  int S = 0, D = 0;
  CHECK(etc_plan_dims(p, &S, &D) == ETC_OK);
  std::vector<uint64_t> c(D), mb(D), ds(D), rc2(S);
  uint64_t tot = 0;
  for (int s = 0; s < S; ++s) CHECK(etc_plan_send_layout(p, s, c.data(), mb.data(), ds.data(), &tot) == ETC_OK);
  for (int d = 0; d < D; ++d) {
    CHECK(etc_plan_recv_counts(p, d, rc2.data()) == ETC_OK);
    uint64_t rb = 0;
    CHECK(etc_plan_refer_bytes(p, d, &rb) == ETC_OK);
  }
  for (int side = 0; side < 2; ++side)
    for (int r = 0; r < (side ? D : S); ++r) {
      int n = 0;
      uint64_t el = 0;
      CHECK(etc_plan_num_pieces(p, side, r, &n) == ETC_OK);
      CHECK(etc_plan_arena_elems(p, side, r, &el) == ETC_OK);
      for (int i = 0; i < n; ++i) {
        etc_piece_info info;
        CHECK(etc_plan_piece(p, side, r, i, &info) == ETC_OK);
      }
    }
  for (int s = 0; s < S; ++s)
    for (int k = 0; k < 4; ++k) CHECK(etc_plan_chunk_layout(p, s, k, c.data(), ds.data(), &tot) == ETC_OK);
  std::vector<int32_t> pair(D), pl(D), ops(3 * D), co(D);
  CHECK(etc_plan_pairing(p, pair.data()) == ETC_OK);
  for (int mode = 0; mode < 3; ++mode) {
    int nops = 0;
    CHECK(etc_plan_defrag(p, mode, pl.data(), ops.data(), &nops, co.data()) == ETC_OK);
  }
  int nproc = 0, sr, dr;
  while (etc_plan_process(p, nproc, &sr, &dr) == ETC_OK) ++nproc;
  CHECK(nproc >= S);
  // error paths
  CHECK(etc_plan_send_layout(p, S, c.data(), mb.data(), ds.data(), &tot) == ETC_ERR_RANK);
  CHECK(etc_plan_piece(p, 0, 0, 1 << 20, nullptr) != ETC_OK);
  CHECK(etc_cost_matrix(p, ETC_CM_ROUTE, nullptr, nullptr) == ETC_ERR_INVALID_ARG);
  etc_plan_free(p);
}
int main() {
  etc_model_desc gpt{ETC_ARCH_GPT, 4, 16, 4, 4, 32, 16, 8, 1, 0};
  etc_model_desc llama{ETC_ARCH_LLAMA, 4, 16, 8, 4, 32, 16, 0, 0, 0};
  etc_model_desc l70{ETC_ARCH_LLAMA, 80, 8192, 64, 8, 28672, 32000, 0, 0, 0};
  const int32_t f1[] = {1};
  for (uint32_t flags : {0u, (uint32_t)ETC_PLAN_SKETCH, (uint32_t)(ETC_PLAN_SKETCH | ETC_PLAN_DIRECT_REFER), (uint32_t)ETC_PLAN_DIRECT_REFER}) {
    for (int ta : {1, 2, 4}) for (int pa : {1, 2, 4}) for (int tb : {1, 2, 4}) for (int pb : {1, 2, 4}) {
      exercise(gpt, {ta, pa, 1}, {tb, pb, 1}, flags, nullptr, 0);
      exercise(llama, {ta, pa, 2}, {tb, pb, 1}, flags, f1, 1);
    }
    exercise(l70, {8, 8, 1}, {8, 4, 1}, flags, nullptr, 0);
  }
  // sketch on its own
  std::vector<uint64_t> cost(6 * 4);
  for (size_t i = 0; i < cost.size(); ++i) cost[i] = (i * 7919) % 13;
  std::vector<int32_t> pr(6);
  uint64_t t = 0;
  CHECK(etc_sketch(cost.data(), 6, 4, pr.data(), &t) == ETC_OK);
  CHECK(etc_sketch(nullptr, 6, 4, pr.data(), &t) == ETC_ERR_INVALID_ARG);
  etc_plan_t* p = nullptr;
  etc_parallel_cfg a{3, 1, 1}, b{1, 1, 1};
  CHECK(etc_plan(&gpt, &a, &b, nullptr, &p) == ETC_ERR_INDIVISIBLE && p == nullptr);
  printf("capi host exercise: %s\n", bad ? "FAILURES" : "ok");
  return bad ? 1 : 0;
}
