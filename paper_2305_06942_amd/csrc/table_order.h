// The table order of a plan (declared in common.h; used by the plan and by
// the plan-free forward).  Its one definition lives here, apart from the
// kernels, so that host tests can build it with a plain C++ compiler: the
// library includes this file from plan.hip only.
#pragma once

#include <algorithm>
#include <cstdint>
#include <cstdlib>
#include <utility>

#include "common.h"

// Table order inside a slice.  The dispatcher hands workgroups to the XCDs
// round-robin (workgroup i to XCD i mod n_xcd), and runs are numbered with
// the table position fastest, so when T is a multiple of n_xcd the runs at
// positions p, p + n_xcd, ... all land on XCD p mod n_xcd.  Assign tables to
// XCDs so that every XCD gets T / n_xcd tables with about the same expected
// bytes (row width; bag lengths are unknown here): widest first, each to the
// least-loaded XCD with room.  Tables of equal width keep t mod n_xcd, so an
// XCD's L2 sees the hot rows of only its own tables.  Any order is correct;
// this only balances work.  Writes perm[T]; work[T] and load[n_xcd] are
// caller-provided workspace (nothing is allocated).
void ebag::table_order(const int64_t* row_bytes, int32_t T, int n_xcd, int32_t* perm, int32_t* work,
                       int64_t* load) {
  for (int32_t t = 0; t < T; ++t) perm[t] = t;
  if (n_xcd <= 1 || n_xcd > kMaxXcd || T % n_xcd != 0) return;
  // perm holds the tables widest first (ties in table order) until the end.
  std::sort(perm, perm + T, [&](int32_t x, int32_t y) {
    return row_bytes[x] != row_bytes[y] ? row_bytes[x] > row_bytes[y] : x < y;
  });
  const int cap = T / n_xcd;
  int count[kMaxXcd];
  for (int x = 0; x < n_xcd; ++x) {
    count[x] = 0;
    load[x] = 0;
  }
  int32_t* bins = work;  // bin x: bins[x * cap .. x * cap + count[x])
  for (int32_t i = 0; i < T; ++i) {
    const int32_t t = perm[i];
    int best = -1;
    for (int x = 0; x < n_xcd; ++x)
      if (count[x] < cap && (best < 0 || load[x] < load[best])) best = x;
    bins[best * cap + count[best]++] = t;
    load[best] += row_bytes[t];
  }
  // Refine: swap a wider table of the most loaded XCD with a narrower one of
  // the least loaded while that narrows their gap (each swap strictly lowers
  // the sum of squared loads, so this ends).
  for (int it = 0; it < 2 * T; ++it) {
    const int hi = (int)(std::max_element(load, load + n_xcd) - load);
    const int lo = (int)(std::min_element(load, load + n_xcd) - load);
    const int64_t gap = load[hi] - load[lo];
    int bi = -1, bj = -1;
    int64_t bd = 0;
    for (int i = 0; i < cap; ++i)
      for (int j = 0; j < cap; ++j) {
        const int64_t d = row_bytes[bins[hi * cap + i]] - row_bytes[bins[lo * cap + j]];
        if (d > 0 && d < gap && (bi < 0 || std::llabs(gap - 2 * d) < std::llabs(gap - 2 * bd))) {
          bi = i;
          bj = j;
          bd = d;
        }
      }
    if (bi < 0) break;
    std::swap(bins[hi * cap + bi], bins[lo * cap + bj]);
    load[hi] -= bd;
    load[lo] += bd;
  }
  for (int x = 0; x < n_xcd; ++x) {
    std::sort(bins + x * cap, bins + (x + 1) * cap);
    for (int k = 0; k < cap; ++k) perm[x + n_xcd * k] = bins[x * cap + k];
  }
}

