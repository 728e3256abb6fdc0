// Host-side Pareto front and box decomposition of the non-dominated region.
//
// The acquisition (paper, "Constrained qNEHVI" paragraph) measures the
// hypervolume a candidate adds to the front of the observations. Both the
// front and the region it does not dominate are small (P up to a few
// hundred) and change once per model / reference point, so they are built
// here on the host and shipped to the device as a flat box list.
//
// Front: maximisation; y_j dominates y_i when y_j >= y_i everywhere and
// y_j != y_i; exact duplicates keep the lowest index; sorted by objective 0
// ascending, ties by index.
//
// Boxes: disjoint [lo, hi) with hi possibly +inf, covering
// {z > ref : no f in F with f >= z}.
//   m = 2: staircase under the sorted front, P + 1 boxes.
//   m = 3: sweep over objective 2 from the top. The active points (those at
//   or above the current level) cast a 2-D staircase kept in an ordered map
//   (x ascending, y descending). Inserting a point closes the boxes of the
//   staircase steps it removes and of its right neighbour, and opens its own
//   step and the neighbour's narrowed step; boxes that survive an insertion
//   keep growing downwards. Every box therefore spans the z-range during
//   which its (x, y) footprint was unchanged, and the count stays O(P).
#include <algorithm>
#include <cmath>
#include <cstring>
#include <limits>
#include <map>
#include <numeric>
#include <vector>

#include "bo_internal.h"

namespace bo {

template <typename T>
void host_front(const T* Y, int64_t n, int m, const T* ref, std::vector<int32_t>& out) {
  // Visit the rows in decreasing lexicographic order (objective 0, 1, ...,
  // then increasing index). A row can only be dominated, or duplicated with a
  // lower index, by a row visited before it, and if it is, some row already
  // kept dominates or duplicates it too (dominance is transitive), so each
  // row is checked against the kept rows only: O(n log n + n P).
  out.clear();
  std::vector<int32_t> order;
  order.reserve(static_cast<size_t>(n));
  for (int64_t i = 0; i < n; ++i) {
    const T* yi = Y + i * m;
    if (ref) {
      bool above = true;
      for (int k = 0; k < m; ++k) above = above && (yi[k] > ref[k]);
      if (!above) continue;
    }
    order.push_back(static_cast<int32_t>(i));
  }
  std::sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {
    const T* ya = Y + static_cast<int64_t>(a) * m;
    const T* yb = Y + static_cast<int64_t>(b) * m;
    for (int k = 0; k < m; ++k)
      if (ya[k] != yb[k]) return ya[k] > yb[k];
    return a < b;
  });
  if (m == 2) {
    // two objectives: kept iff objective 1 beats every row visited before
    T best = -std::numeric_limits<T>::infinity();
    for (int32_t i : order) {
      const T y1 = Y[static_cast<int64_t>(i) * 2 + 1];
      if (out.empty() || y1 > best) {
        out.push_back(i);
        best = y1;
      }
    }
  } else {
    for (int32_t i : order) {
      const T* yi = Y + static_cast<int64_t>(i) * m;
      bool keep = true;
      for (int32_t j : out) {
        const T* yj = Y + static_cast<int64_t>(j) * m;
        bool ge = true;
        for (int k = 0; k < m; ++k) ge = ge && (yj[k] >= yi[k]);
        if (ge) {            // dominated, or an exact duplicate of a lower index
          keep = false;
          break;
        }
      }
      if (keep) out.push_back(i);
    }
  }
  std::stable_sort(out.begin(), out.end(), [&](int32_t a, int32_t b) {
    const T ya = Y[static_cast<int64_t>(a) * m], yb = Y[static_cast<int64_t>(b) * m];
    return ya < yb || (ya == yb && a < b);
  });
}

namespace {

template <typename T>
void push_box(std::vector<T>& lo, std::vector<T>& hi, T l0, T l1, T l2, T h0, T h1, T h2, int m) {
  lo.push_back(l0); lo.push_back(l1);
  hi.push_back(h0); hi.push_back(h1);
  if (m == 3) { lo.push_back(l2); hi.push_back(h2); }
}

}  // namespace

template <typename T>
void host_boxes(const T* F, int P, int m, const T* ref, std::vector<T>& lo, std::vector<T>& hi) {
  constexpr T kInf = std::numeric_limits<T>::infinity();
  lo.clear();
  hi.clear();
  if (m == 2) {
    // F sorted by objective 0 ascending: box i covers objective 0 in
    // [x_{i-1}, x_i) (x_0 = ref_0) and objective 1 above y_i; the last box
    // covers [x_P, inf) above ref_1.
    T xlo = ref[0];
    for (int i = 0; i < P; ++i) {
      push_box<T>(lo, hi, xlo, F[2 * i + 1], T(0), F[2 * i], kInf, T(0), 2);
      xlo = F[2 * i];
    }
    push_box<T>(lo, hi, xlo, ref[1], T(0), kInf, kInf, T(0), 2);
    return;
  }
  // m == 3
  std::vector<int> order(P);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(),
                   [&](int a, int b) { return F[3 * a + 2] > F[3 * b + 2]; });
  struct Step { T y; T ztop; };          // box (prev.x, x) x [y, inf)
  std::map<T, Step> stair;                    // keyed by x ascending
  T tail_ztop = kInf;                         // box [last.x, inf) x [ref1, inf)
  auto close = [&](T xl, T xh, T yl, T zl, T zt) {
    if (zt > zl) push_box<T>(lo, hi, xl, yl, zl, xh, kInf, zt, 3);
  };
  for (int idx : order) {
    const T px = F[3 * idx], py = F[3 * idx + 1], zb = F[3 * idx + 2];
    // dominated in 2-D by an active point (x >= px and y >= py)?
    auto it = stair.lower_bound(px);              // first x >= px
    if (it != stair.end() && it->second.y >= py) continue;
    // predecessor chain: active points with x <= px and y <= py are removed
    // (only those with x < px can remain here, since it->x >= px has y < py
    // when it exists; an equal-x point with lower y is removed too)
    auto first_rm = it;
    if (it != stair.end() && it->first == px) {
      // equal x, lower y: removed below together with the predecessor run
      ++first_rm;
    }
    // walk left over predecessors with y <= py
    auto left = it;
    while (left != stair.begin()) {
      auto prev = std::prev(left);
      if (prev->second.y <= py) left = prev; else break;
    }
    // range [left, first_rm) is removed; compute the x just before it
    T pred_x = (left == stair.begin()) ? ref[0] : std::prev(left)->first;
    // close removed steps
    T xl = pred_x;
    for (auto r = left; r != first_rm; ++r) {
      close(xl, r->first, r->second.y, zb, r->second.ztop);
      xl = r->first;
    }
    // right neighbour (or the tail box) narrows from xl to px
    if (first_rm != stair.end()) {
      Step& s = first_rm->second;
      close(xl, first_rm->first, s.y, zb, s.ztop);
      s.ztop = zb;
    } else {
      close(xl, kInf, ref[1], zb, tail_ztop);
      tail_ztop = zb;
    }
    stair.erase(left, first_rm);
    stair[px] = Step{py, zb};
  }
  // close everything at ref_2
  T xl = ref[0];
  for (auto& kv : stair) {
    close(xl, kv.first, kv.second.y, ref[2], kv.second.ztop);
    xl = kv.first;
  }
  close(xl, kInf, ref[1], ref[2], tail_ztop);
}

template void host_front<float>(const float*, int64_t, int, const float*, std::vector<int32_t>&);
template void host_front<double>(const double*, int64_t, int, const double*, std::vector<int32_t>&);
template void host_boxes<float>(const float*, int, int, const float*, std::vector<float>&,
                                std::vector<float>&);
template void host_boxes<double>(const double*, int, int, const double*, std::vector<double>&,
                                 std::vector<double>&);

}  // namespace bo
