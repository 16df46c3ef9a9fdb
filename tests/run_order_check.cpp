// Host check of run_at (the run -> (slice, table, run) decoding shared by the
// pooling, consumer, backward and delivery kernels): every decoding is a
// bijection onto slices x tables x runs, slice-major order has the table
// position fastest, and table-major order keeps run q in table group q mod G
// with each group's tables (and the slices inside a table) in order.
#include <cstdio>
#include <vector>

#include "common.h"

int main() {
  using namespace ebag;
  int bad = 0, cases = 0;
  for (int G : {0, 1, 2, 8})
    for (int T : {1, 3, 8, 16, 24, 64})
      for (int J : {1, 2, 5})
        for (int n : {1, 2, 7, 64}) {
          if (G > 1 && T % G) continue;
          ++cases;
          SliceOrder o{n, 1, 0, 0, G};
          const int64_t total = (int64_t)n * T * J;
          std::vector<int> seen((size_t)total, 0);
          std::vector<int64_t> last(G > 0 ? G : 1, -1);
          for (int64_t q = 0; q < total; ++q) {
            int64_t gs;
            int32_t tp, j;
            run_at(o, T, J, q, &gs, &tp, &j);
            if (gs < 0 || gs >= n || tp < 0 || tp >= T || j < 0 || j >= J) {
              ++bad;
              continue;
            }
            seen[((size_t)gs * T + tp) * J + j]++;
            if (G == 0) {
              if (tp != q % T || gs != q / ((int64_t)T * J)) ++bad;
            } else {
              if (tp % G != q % G) ++bad;
              const int64_t key = ((int64_t)tp * n + gs) * J + j;  // table, then slice, then run
              if (key <= last[q % G]) ++bad;
              last[q % G] = key;
            }
          }
          for (int c : seen)
            if (c != 1) ++bad;
        }
  std::printf("cases=%d bad=%d\n", cases, bad);
  return bad != 0;
}
