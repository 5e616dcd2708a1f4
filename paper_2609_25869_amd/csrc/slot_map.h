// Which task each launch slot of the attention kernel runs, and the shares of
// the task list that the XCD groups take.  Plain integer code: the kernel
// evaluates task_of_slot on the device (a constexpr function is callable from
// device code), the planner and the host tests on the host.
#pragma once

#include <cstdint>
#include <vector>

namespace bsa {

// Map launch slot `slot` to a task index in [0, nt), or -1.  Slot i runs on
// XCD i % 8.  The XCDs form 8 / group groups of `group` XCDs; group g works
// through the g-th contiguous share of the task list, and inside it its XCDs
// take turns over runs of `run` consecutive tasks (XCD member m takes runs m,
// m + group, ...), so neighbouring tasks still share an XCD while the group's
// XCDs stay on the same stretch of the list.  group = 1 gives each XCD its
// own contiguous eighth; group = 8 keeps all XCDs on one stretch.  The shares
// are equal in task count, or given (share_lo non-null: group g takes
// [share_lo[g], share_lo[g + 1]), cut by the planner so that the shares hold
// equal work; group >= 2).  The tail of a share that does not fill whole
// rounds of runs is dealt out one task per XCD.  With default_slots(nt)
// slots for equal shares, or shares_slots(...) for given ones, every task of
// [0, nt) has exactly one slot.
constexpr int64_t task_of_slot(int64_t slot, int64_t nt, int64_t group, int64_t run, const int32_t* share_lo) {
  const int64_t xcd = slot & 7, local = slot >> 3;
  if (group <= 1) {
    const int64_t per = (nt + 7) / 8;
    const int64_t t = xcd * per + local;
    return (local < per && t < nt) ? t : -1;
  }
  const int64_t ngroups = 8 / group, gi = xcd / group, mi = xcd % group;
  int64_t lo = 0, n = 0;
  if (share_lo) {
    // a select over the (at most four) groups keeps the bounds in scalar
    // registers on the device; an indexed read of the kernel argument array
    // would place it in scratch memory
    int64_t a0 = 0, a1 = 0;
    for (int i = 0; i < 4; ++i)
      if (i == gi) {
        a0 = share_lo[i];
        a1 = share_lo[i + 1];
      }
    lo = a0;
    n = a1 - a0;
  } else {
    const int64_t per = (nt + ngroups - 1) / ngroups;
    lo = gi * per;
    n = (nt < lo + per ? nt : lo + per) - lo;
    if (n < 0) n = 0;
  }
  const int64_t whole = n / (group * run);  // complete rounds of runs
  const int64_t t = local < whole * run ? (local / run) * group * run + mi * run + local % run
                                        : whole * group * run + (local - whole * run) * group + mi;
  return t < n ? lo + t : -1;
}

// Launch slots for equal shares: the task count rounded up to a multiple of 8.
constexpr int64_t default_slots(int64_t nt) { return (nt + 7) / 8 * 8; }

// Launch slots for given shares share_lo[0 .. 8 / group] (group >= 2): eight
// times the most tasks one XCD of any group takes.
constexpr int64_t shares_slots(const int32_t* share_lo, int64_t group, int64_t run) {
  int64_t most = 0;
  for (int64_t g = 0; g < 8 / group; ++g) {
    const int64_t n = (int64_t)share_lo[g + 1] - share_lo[g], whole = n / (group * run);
    const int64_t r = n - whole * group * run;
    const int64_t per_xcd = whole * run + (r + group - 1) / group;
    if (per_xcd > most) most = per_xcd;
  }
  return 8 * most;
}

// Shares of the XCD groups (group >= 2) over a split-free task list:
// contiguous stretches holding equal work.  The task list holds npq tasks
// per (b, h) in (b, head) order, whatever the dispatch order does inside a
// head, and work[k] is the work of the k-th (b, h) (its active logical
// blocks), taken as spread evenly over its tasks, so a cut may fall inside a
// head.  Requests whose heads carry equal work get equal task counts when
// the heads divide evenly among the groups.  Fills lo[0..4] (lo[g] = nt
// past the last group).
inline void balanced_shares(const std::vector<int64_t>& work, int64_t npq, int32_t group, int32_t* lo) {
  const int ngroups = 8 / group;
  const int64_t nbh = (int64_t)work.size(), nt = nbh * npq;
  std::vector<int64_t> cw(nbh + 1, 0);
  for (int64_t k = 0; k < nbh; ++k) cw[k + 1] = cw[k] + work[k];
  const int64_t total = cw[nbh];
  for (int g = 0; g <= 4; ++g) lo[g] = (int32_t)nt;
  lo[0] = 0;
  for (int g = 1; g < ngroups; ++g) {
    int64_t pos;
    if (total == 0) {
      pos = (nt * g + ngroups - 1) / ngroups;
    } else {
      const int64_t target = total * g / ngroups;
      int64_t k = 0;
      while (k + 1 < nbh && cw[k + 1] <= target) ++k;
      pos = k * npq + (work[k] > 0 ? ((target - cw[k]) * npq + work[k] / 2) / work[k] : 0);
    }
    if (pos < lo[g - 1]) pos = lo[g - 1];
    if (pos > nt) pos = nt;
    lo[g] = (int32_t)pos;
  }
}

}  // namespace bsa
