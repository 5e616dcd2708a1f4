// Host check of the attention kernel's slot map (slot_map.h): for equal
// shares and for work-balanced shares, every task of [0, nt) has exactly one
// launch slot and every other slot maps to -1.  Exit status 0 and "ok N"
// when all configurations pass; the first failure is printed and exits 1.
#include <cstdint>
#include <cstdio>
#include <random>
#include <vector>

#include "slot_map.h"

namespace {

bool covers_once(int64_t nt, int64_t nslots, int64_t group, int64_t run, const int32_t* share_lo, const char* what) {
  std::vector<int> seen((size_t)nt, 0);
  for (int64_t s = 0; s < nslots; ++s) {
    const int64_t t = bsa::task_of_slot(s, nt, group, run, share_lo);
    if (t < -1 || t >= nt) {
      std::printf("FAIL %s: slot %lld maps to %lld outside [0, %lld)\n", what, (long long)s, (long long)t,
                  (long long)nt);
      return false;
    }
    if (t >= 0 && ++seen[(size_t)t] > 1) {
      std::printf("FAIL %s: task %lld twice (nt %lld group %lld run %lld)\n", what, (long long)t, (long long)nt,
                  (long long)group, (long long)run);
      return false;
    }
  }
  for (int64_t t = 0; t < nt; ++t)
    if (!seen[(size_t)t]) {
      std::printf("FAIL %s: task %lld has no slot (nt %lld group %lld run %lld, %lld slots)\n", what, (long long)t,
                  (long long)nt, (long long)group, (long long)run, (long long)nslots);
      return false;
    }
  return true;
}

}  // namespace

int main() {
  std::mt19937_64 rng(12345);
  long checks = 0;
  const int64_t groups[] = {1, 2, 4, 8};
  const int64_t runs[] = {1, 3, 8};
  // equal shares, with the default launch size
  for (int64_t nt = 0; nt <= 700; ++nt)
    for (int64_t g : groups)
      for (int64_t r : runs) {
        if (!covers_once(nt, bsa::default_slots(nt), g, r, nullptr, "equal shares")) return 1;
        ++checks;
      }
  for (int i = 0; i < 200; ++i) {
    const int64_t nt = (int64_t)(rng() % 200000);
    for (int64_t g : groups) {
      if (!covers_once(nt, bsa::default_slots(nt), g, 8, nullptr, "equal shares, large")) return 1;
      ++checks;
    }
  }
  // work-balanced shares: heads of zero, equal, skewed and random work
  for (int i = 0; i < 4000; ++i) {
    const int64_t nbh = 1 + (int64_t)(rng() % 64), npq = 1 + (int64_t)(rng() % 300);
    std::vector<int64_t> work((size_t)nbh);
    const int kind = i % 4;
    for (int64_t k = 0; k < nbh; ++k) {
      if (kind == 0) work[(size_t)k] = 0;
      else if (kind == 1) work[(size_t)k] = 1000;
      else if (kind == 2) work[(size_t)k] = (k % 7 == 0) ? 100000 : (int64_t)(rng() % 3);
      else work[(size_t)k] = (int64_t)(rng() % 5000);
    }
    for (int32_t g : {2, 4}) {
      int32_t lo[5];
      bsa::balanced_shares(work, npq, g, lo);
      const int ngroups = 8 / g;
      const int64_t nt = nbh * npq;
      if (lo[0] != 0 || lo[ngroups] != nt) {
        std::printf("FAIL shares: ends %d %d for nt %lld\n", lo[0], lo[ngroups], (long long)nt);
        return 1;
      }
      for (int k = 0; k < ngroups; ++k)
        if (lo[k] > lo[k + 1]) {
          std::printf("FAIL shares: not monotone at %d\n", k);
          return 1;
        }
      // equal work over heads that divide evenly: the shares are equal in count
      if (kind == 1 && nbh % ngroups == 0)
        for (int k = 0; k <= ngroups; ++k)
          if (lo[k] != nt / ngroups * k) {
            std::printf("FAIL shares: equal heads, share %d at %d not %lld\n", k, lo[k], (long long)(nt / ngroups * k));
            return 1;
          }
      for (int64_t r : runs) {
        if (!covers_once(nt, bsa::shares_slots(lo, g, r), g, r, lo, "balanced shares")) return 1;
        ++checks;
      }
    }
  }
  std::printf("ok %ld\n", checks);
  return 0;
}
