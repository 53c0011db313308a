// sketch.hip -- the migration sketch (Sec. III-B): pair the new ranks with the
// old ranks so the total cost is minimal (objective Eq. (2); constraints
// Eq. (3) when M > N, Eq. (4) when M <= N).  As in Algorithm 1 the M x N cost
// matrix is padded with zeros to k x k, the square assignment problem is
// solved, and pairs involving padding are dropped.  The square problem is
// solved with the Kuhn-Munkres (Hungarian) method in its shortest-augmenting-
// path form with row and column potentials: O(k^3), microseconds for the
// k <= 128 of a PP x TP grid.  The potentials drift while rows are added (on
// some matrices to k times the largest entry), so they are 128-bit: entries
// below 2^53 and k <= 65536 keep them under 2^70.
#include <algorithm>
#include <cstdint>
#include <vector>

#include "plan.hpp"

namespace etc {

uint64_t solve_sketch(const uint64_t* cost, int M, int N, int32_t* pair) {
  const int k = std::max(M, N);
  using Pot = __int128;
  auto c = [&](int i, int j) -> Pot {  // 1-based rows / columns, zero padding
    return (i <= M && j <= N) ? Pot(cost[size_t(i - 1) * N + (j - 1)]) : 0;
  };
  const Pot INF = Pot(1) << 100;
  std::vector<Pot> u(k + 1, 0), v(k + 1, 0), slack(k + 1);
  std::vector<int> row_of(k + 1, 0), prev(k + 1, 0);  // row_of[j]: row matched to column j
  std::vector<char> visited(k + 1);
  for (int i = 1; i <= k; ++i) {
    // grow an alternating tree from free row i until it reaches a free column
    row_of[0] = i;
    int j0 = 0;
    std::fill(slack.begin(), slack.end(), INF);
    std::fill(visited.begin(), visited.end(), 0);
    do {
      visited[j0] = 1;
      const int i0 = row_of[j0];
      Pot delta = INF;
      int j1 = 0;
      for (int j = 1; j <= k; ++j) {
        if (visited[j]) continue;
        const Pot reduced = c(i0, j) - u[i0] - v[j];
        if (reduced < slack[j]) {
          slack[j] = reduced;
          prev[j] = j0;
        }
        if (slack[j] < delta) {
          delta = slack[j];
          j1 = j;
        }
      }
      for (int j = 0; j <= k; ++j) {
        if (visited[j]) {
          u[row_of[j]] += delta;
          v[j] -= delta;
        } else {
          slack[j] -= delta;
        }
      }
      j0 = j1;
    } while (row_of[j0] != 0);
    // flip the augmenting path
    do {
      const int j1 = prev[j0];
      row_of[j0] = row_of[j1];
      j0 = j1;
    } while (j0 != 0);
  }
  uint64_t total = 0;
  for (int i = 0; i < M; ++i) pair[i] = -1;
  for (int j = 1; j <= k; ++j) {
    const int i = row_of[j];
    if (i >= 1 && i <= M && j <= N) {
      pair[i - 1] = j - 1;
      total += cost[size_t(i - 1) * N + (j - 1)];
    }
  }
  return total;
}

}  // namespace etc
