// Host-side check of the Pareto front and box decomposition routines, built
// with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_host_sanitized.py (host compiler only, no device code).
//
// For random point sets (continuous, and integer-valued with many ties and
// duplicates), in float and double, m = 2 and 3:
//   * the front equals an O(n^2) brute-force dominance scan (strictly above
//     the reference point, duplicates keep the lowest index, sorted by
//     objective 0 then index);
//   * the boxes are disjoint and cover exactly the part of the region above
//     the reference point that no front point weakly dominates: random probe
//     points lie in exactly one box iff they are not dominated, else in none.
// Prints one line per failure and exits non-zero if there was any.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <limits>
#include <random>
#include <vector>

#include "../paper_2602_10729_amd/csrc/bo_internal.h"

namespace {

int failures = 0;

template <typename T>
std::vector<int32_t> brute_front(const std::vector<T>& Y, int n, int m, const T* ref) {
  std::vector<int32_t> keep;
  for (int i = 0; i < n; ++i) {
    bool above = true;
    for (int k = 0; k < m; ++k) above = above && Y[i * m + k] > ref[k];
    if (!above) continue;
    bool drop = false;
    for (int j = 0; j < n && !drop; ++j) {
      if (j == i) continue;
      bool ge = true, gt = false, eq = true;
      for (int k = 0; k < m; ++k) {
        ge = ge && Y[j * m + k] >= Y[i * m + k];
        gt = gt || Y[j * m + k] > Y[i * m + k];
        eq = eq && Y[j * m + k] == Y[i * m + k];
      }
      drop = (ge && gt) || (eq && j < i);
    }
    if (!drop) keep.push_back(i);
  }
  // sort by objective 0, then index (insertion sort: small sets)
  for (size_t a = 1; a < keep.size(); ++a)
    for (size_t b = a; b > 0; --b) {
      const T ya = Y[keep[b - 1] * m], yb = Y[keep[b] * m];
      if (ya > yb || (ya == yb && keep[b - 1] > keep[b])) std::swap(keep[b - 1], keep[b]);
    }
  return keep;
}

template <typename T>
void check_case(std::mt19937_64& rng, int n, int m, bool integer, const char* tname, int id) {
  std::normal_distribution<double> nd(0.0, 1.0);
  std::uniform_int_distribution<int> ud(0, 5);
  std::vector<T> Y((size_t)n * m);
  for (auto& v : Y) v = integer ? static_cast<T>(ud(rng)) : static_cast<T>(nd(rng));
  T ref[3];
  for (int k = 0; k < m; ++k) {
    T lo = Y[k];
    for (int i = 0; i < n; ++i) lo = std::min(lo, Y[i * m + k]);
    ref[k] = integer ? lo : static_cast<T>(lo - 0.1);
  }
  std::vector<int32_t> got;
  bo::host_front<T>(Y.data(), n, m, ref, got);
  const std::vector<int32_t> want = brute_front<T>(Y, n, m, ref);
  if (got != want) {
    std::printf("FAIL front %s case %d (n=%d m=%d int=%d): %zu vs %zu points\n", tname, id, n, m,
                integer ? 1 : 0, got.size(), want.size());
    ++failures;
    return;
  }
  std::vector<T> F;
  for (int32_t i : got)
    for (int k = 0; k < m; ++k) F.push_back(Y[(size_t)i * m + k]);
  std::vector<T> lo, hi;
  bo::host_boxes<T>(F.data(), static_cast<int>(got.size()), m, ref, lo, hi);
  const size_t nb = lo.size() / m;
  if (hi.size() != lo.size() || nb == 0) {
    std::printf("FAIL boxes %s case %d: %zu boxes\n", tname, id, nb);
    ++failures;
    return;
  }
  // probes above ref: non-dominated probes lie in exactly one box, dominated
  // ones in none
  std::uniform_real_distribution<double> pu(-0.5, 6.5);
  for (int t = 0; t < 2000; ++t) {
    T z[3];
    for (int k = 0; k < m; ++k) {
      const double v = integer ? pu(rng) : nd(rng) * 1.5;
      z[k] = static_cast<T>(v);
    }
    bool above = true;
    for (int k = 0; k < m; ++k) above = above && z[k] > ref[k];
    if (!above) continue;
    bool dominated = false;
    for (size_t p = 0; p < got.size() && !dominated; ++p) {
      bool ge = true;
      for (int k = 0; k < m; ++k) ge = ge && F[p * m + k] >= z[k];
      dominated = ge;
    }
    int inside = 0;
    for (size_t b = 0; b < nb; ++b) {
      bool in = true;
      for (int k = 0; k < m; ++k) in = in && z[k] >= lo[b * m + k] && z[k] < hi[b * m + k];
      inside += in ? 1 : 0;
    }
    // probes exactly on a box face are skipped (the half-open convention)
    bool on_face = false;
    for (size_t b = 0; b < nb && !on_face; ++b)
      for (int k = 0; k < m; ++k)
        on_face = on_face || z[k] == lo[b * m + k] || z[k] == hi[b * m + k];
    if (on_face) continue;
    if ((dominated && inside != 0) || (!dominated && inside != 1)) {
      std::printf("FAIL boxes %s case %d (m=%d): probe dominated=%d inside=%d\n", tname, id, m,
                  dominated ? 1 : 0, inside);
      ++failures;
      return;
    }
  }
}

}  // namespace

int main() {
  std::mt19937_64 rng(12345);
  int id = 0;
  for (int m = 2; m <= 3; ++m)
    for (int n : {1, 2, 7, 40, 200})
      for (int integer = 0; integer <= 1; ++integer) {
        check_case<float>(rng, n, m, integer != 0, "float", id++);
        check_case<double>(rng, n, m, integer != 0, "double", id++);
      }
  if (failures) {
    std::printf("%d failures\n", failures);
    return 1;
  }
  std::printf("host geometry ok: %d cases\n", id);
  return 0;
}
