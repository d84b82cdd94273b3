// Host check of the adaptive partition arithmetic of the attention kernel (vmla_internal.h):
// the closed-form owner against a brute-force scan, the ranges tiling [0, U) without empty
// ranges, the equal-weight case against the even split, and the partial-result slot bound.
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
