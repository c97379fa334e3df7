// Host stress of the staging planner (paper_2206_00470_amd/csrc/planner.hpp)
// under the locking protocol of the library: a worker thread signals the
// intents of batches `lookahead` clocks ahead, advances its clock (acting at
// once on intents that became due: a forced action) and checks that every
// key of its current batch holds a slot; a second thread runs rounds back to
// back (estimate, evictions, actions), as the library's round thread does.
// Both take one mutex around every planner call.  Built with thread or
// address/undefined-behaviour sanitizers; prints the totals and exits
// non-zero on a broken invariant.
#include <atomic>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <mutex>
#include <random>
#include <set>
#include <thread>
#include <vector>

#include "planner.hpp"

using adapm::Planner;

int main(int argc, char** argv) {
  const int64_t clocks = argc > 1 ? std::atol(argv[1]) : 400;
  const int64_t K = 20000;
  const int64_t begin[2] = {0, 15000};
  const int64_t cap[2] = {4000, 1500};
  const int lookahead = 2;
  Planner P;
  P.init(K, begin, cap, 2);
  std::mutex mu;
  std::atomic<bool> done{false};
  std::atomic<int> bad{0};
  const int64_t total = cap[0] + cap[1];
  std::vector<int64_t> rk(2 * total), rs(2 * total), fk(2 * total), fs(2 * total);

  auto batch = [&](int64_t c) {   // the keys of the batch used at clock c: skewed, both ranges
    std::mt19937_64 g((uint64_t)c * 7919u + 1u);
    std::vector<int64_t> v;
    for (int i = 0; i < 700; ++i) {
      const double u = std::ldexp((double)(g() >> 11), -53);
      const int64_t r0 = (int64_t)(14999.0 * u * u * u);          // range 0, hot low keys
      v.push_back(r0);
      if (i % 4 == 0) v.push_back(15000 + (int64_t)(g() % 5000));  // range 1, uniform
    }
    return v;
  };
  auto check = [&](int64_t c) {   // under the lock: the batch of clock c is resident, slots unique
    for (int64_t k : batch(c))
      if (P.slot_of(k) < 0) ++bad;
  };

  std::thread rounds([&] {
    int64_t rid = 0;
    while (!done.load()) {
      {
        std::lock_guard<std::mutex> lk(mu);
        P.clear_moves(rk.data(), rs.data());
        const int64_t h = P.timing.horizon(P.clock);
        P.evict_expired();
        P.act(h, rid++);
        if (P.nout + P.nin > 2 * total) ++bad;
      }
      std::this_thread::yield();
    }
  });

  for (int64_t c = 1; c <= lookahead; ++c) {
    std::lock_guard<std::mutex> lk(mu);
    const auto v = batch(c);
    P.signal(v.data(), (int64_t)v.size(), c, c + 1);
  }
  for (int64_t step = 0; step < clocks; ++step) {
    // some clocks leave the round thread time to act ahead, others do not
    if (step % 3 == 0) std::this_thread::sleep_for(std::chrono::microseconds(300));
    std::lock_guard<std::mutex> lk(mu);
    P.clock += 1;
    if (P.due(P.clock)) {   // a forced action, as in the library's advanceClock
      P.clear_moves(fk.data(), fs.data());
      P.evict_expired();
      P.act(P.clock + 1, -1);
      ++P.forced_total;
    }
    (void)P.take_round_for(P.clock);
    check(P.clock);
    const int64_t c = P.clock + lookahead;
    const auto v = batch(c);
    P.signal(v.data(), (int64_t)v.size(), c, c + 1);
  }
  done.store(true);
  rounds.join();

  // every slot is either free or held by exactly one key of its range
  std::set<int32_t> seen;
  int64_t held = 0;
  for (int64_t k = 0; k < K; ++k) {
    const int32_t s = P.slot_of(k);
    if (s < 0) continue;
    ++held;
    const int r = P.range_of(k);
    if (s < P.range_slot0[r] || s >= P.range_slot0[r] + cap[r] || !seen.insert(s).second) ++bad;
  }
  int64_t free_n = 0;
  for (int r = 0; r < 2; ++r)
    for (int32_t s : P.free_slots[r]) {
      ++free_n;
      if (s < P.range_slot0[r] || s >= P.range_slot0[r] + cap[r] || !seen.insert(s).second) ++bad;
    }
  if (held + free_n != total) ++bad;
  std::printf("clocks %lld staged %lld evicted %lld forced %lld stalled %lld resident %lld bad %d\n",
              (long long)P.clock, (long long)P.staged_total, (long long)P.evicted_total,
              (long long)P.forced_total, (long long)P.stalled_total, (long long)held, bad.load());
  return bad.load() ? 1 : 0;
}
