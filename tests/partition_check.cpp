// Host check of the adaptive partition arithmetic of the attention kernel (vmla_internal.h):
// the closed-form owner against a brute-force scan, the merge kernels' owner forms (divisions
// by floor_div) against the integer ones and floor_div against integer division, the ranges
// tiling [0, U) without empty ranges, the equal-weight case against the even split, and the
// partial-result slot bound.
#include "vmla_internal.h"
#include <cstdio>
#include <random>
using namespace vmla;

int owner_ref(const uint32_t* w, int G, int64_t U, int64_t u) {
  int best = 0;
  for (int k = 0; k < G; ++k) if (bal_start(w, G, U, k) <= u) best = k;
  return best;
}
int main() {
  std::mt19937_64 rng(1);
  long bad = 0, checks = 0;
  // floor_div against integer division: random operands over the whole range it is used in,
  // exact multiples and their neighbours, and operands at and above 2^53
  for (int it = 0; it < 2000000; ++it) {
    const int64_t d = 1 + (int64_t)(rng() % ((it % 3 == 0) ? 7u : (it % 3 == 1) ? 300000u : 2147483647u));
    int64_t n = (int64_t)(rng() >> (11 + it % 40));  // below 2^53, many magnitudes
    if (it % 4 == 1) n = (n / d) * d;
    if (it % 4 == 2) n = (n / d) * d + d - 1;
    if (it % 4 == 3) n = (int64_t(1) << 53) - 1 - (int64_t)(rng() % 1000);
    if (it % 1000 == 0) n = (int64_t(1) << 53) + (int64_t)(rng() % 1000);
    ++checks;
    if (floor_div(n, d) != n / d) { if (bad++ < 5) printf("floor_div(%ld, %ld) = %ld, not %ld\n", (long)n, (long)d, (long)floor_div(n, d), (long)(n / d)); }
  }
  // the largest quotients below 2^53 / d, at and around exact multiples
  for (int64_t d = 2; d <= 9; ++d)
    for (int64_t k = ((int64_t(1) << 53) - 1) / d - 4000; k * d + d <= (int64_t(1) << 53); ++k)
      for (int64_t n : {k * d - 1, k * d, k * d + 1, k * d + d - 1}) {
        ++checks;
        if (floor_div(n, d) != n / d) { if (bad++ < 5) printf("floor_div(%ld, %ld) = %ld, not %ld\n", (long)n, (long)d, (long)floor_div(n, d), (long)(n / d)); }
      }
  for (int it = 0; it < 3000; ++it) {
    uint32_t w[8];
    for (int x = 0; x < 8; ++x) w[x] = kBalMin + rng() % (kBalMax - kBalMin + 1);
    if (it % 5 == 0) for (int x = 0; x < 8; ++x) w[x] = kBalOne;
    const int G = 1 + rng() % (it % 3 == 0 ? 300 : 20);
    const int64_t U = G + rng() % (it % 2 ? 300000 : 2000);
    for (int s = 0; s < 200; ++s) {
      const int64_t u = s < 4 ? (s == 0 ? 0 : s == 1 ? U - 1 : bal_start(w, G, U, rng() % G)) : (int64_t)(rng() % U);
      ++checks;
      if (bal_owner(w, G, U, u) != owner_ref(w, G, U, u)) { if (bad++ < 5) printf("bad G=%d U=%ld u=%ld got %d want %d\n", G, (long)U, (long)u, bal_owner(w, G, U, u), owner_ref(w, G, U, u)); }
      if (it % 5 == 0 && bal_owner(w, G, U, u) != (int)(((u + 1) * (int64_t)G - 1) / U)) { if (bad++ < 5) printf("uniform mismatch\n"); }
      // the merge kernels' forms with the divisions done by floor_div
      if (bal_owner_fd(w, G, U, u) != bal_owner(w, G, U, u)) { if (bad++ < 5) printf("bal_owner_fd G=%d U=%ld u=%ld\n", G, (long)U, (long)u); }
      if (attend_owner_fd(u, U, G) != attend_owner(u, U, G)) { if (bad++ < 5) printf("attend_owner_fd G=%d U=%ld u=%ld\n", G, (long)U, (long)u); }
    }
    // ranges tile [0, U)
    if (bal_start(w, G, U, 0) != 0 || bal_start(w, G, U, G) != U) { bad++; printf("ends\n"); }
    // bal_max_seg bound
    const int T = 1 + rng() % 2000;
    const int ms = bal_max_seg(G, U, T);
    if (ms <= G) {
      for (int64_t rb = 0; rb * T < U; ++rb) {
        const int64_t lo = rb * T, hi = (lo + T < U ? lo + T : U) - 1;
        const int n = bal_owner(w, G, U, hi) - bal_owner(w, G, U, lo) + 1;
        if (n > ms) { bad++; printf("max_seg G=%d U=%ld T=%d n=%d ms=%d\n", G, (long)U, T, n, ms); break; }
      }
      for (int k = 0; k < G; ++k) if (bal_start(w, G, U, k + 1) <= bal_start(w, G, U, k)) { bad++; printf("empty range\n"); break; }
    }
  }
  printf("checks %ld bad %ld\n", checks, bad);
  return bad != 0;
}
