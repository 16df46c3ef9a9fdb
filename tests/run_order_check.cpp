// Host check of run_at (the run -> (slice, table, run) decoding shared by the
// pooling, consumer, backward and delivery kernels): every decoding is a
// bijection onto slices x tables x runs, slice-major order has the table
// position fastest, and table-major order keeps run q in table group q mod G
// with each group's tables (and the slices inside a table) in order.  Also
// the table order that balances row bytes over the XCDs (table_order).
#include <algorithm>
#include <cstdio>
#include <vector>

#include "common.h"
#include "table_order.h"

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
  // table_order: a permutation of the tables; with T a multiple of the XCD
  // count the row bytes per XCD (positions p, p + n_xcd, ...) differ by at
  // most the widest row; equal widths keep table t at position t; mixed's
  // cycle of 64/128/256/512-byte rows over 48 tables reaches the best
  // balance there is (11,520 bytes are 22.5 units of 64 per XCD: a 64-byte gap).
  {
    const int64_t widths4[4] = {64, 128, 256, 512};
    unsigned seed = 12345;
    for (int T = 1; T <= 96; ++T)
      for (int kind = 0; kind < 3; ++kind) {
        ++cases;
        std::vector<int64_t> rb(T);
        for (int t = 0; t < T; ++t) {
          seed = seed * 1103515245u + 12345u;
          rb[t] = kind == 0 ? 256 : kind == 1 ? widths4[t % 4] : widths4[(seed >> 16) % 4];
        }
        const int n_xcd = 8;
        std::vector<int32_t> perm(T), work(T);
        std::vector<int64_t> load(kMaxXcd);
        table_order(rb.data(), T, n_xcd, perm.data(), work.data(), load.data());
        std::vector<int> hit(T, 0);
        for (int32_t p : perm) {
          if (p < 0 || p >= T) ++bad;
          else ++hit[p];
        }
        for (int h : hit)
          if (h != 1) ++bad;
        if (kind == 0)
          for (int t = 0; t < T; ++t)
            if (perm[t] != t) ++bad;
        if (T % n_xcd == 0) {
          std::vector<int64_t> per(n_xcd, 0);
          for (int p = 0; p < T; ++p) per[p % n_xcd] += rb[perm[p]];
          const int64_t gap = *std::max_element(per.begin(), per.end()) - *std::min_element(per.begin(), per.end());
          if (gap > 512) ++bad;
          if (kind == 1 && T == 48 && gap != 64) ++bad;
        }
      }
  }
  std::printf("cases=%d bad=%d\n", cases, bad);
  return bad != 0;
}
