// Host side of intent-driven staging (intent signalling, Section 3;
// adaptive action timing, Section 4.2 and Algorithm 1) for one worker: the
// worker's clock, the intents signalled and not yet acted upon, the key ->
// slot assignment and a free list of slots per key range, and in each round
// the keys to stage in and the keys to write back.  Plain C++ (no device
// code), so that host builds with thread and address sanitizers can check it.
#pragma once

#include <sys/mman.h>

#include <algorithm>
#include <cmath>
#include <cstddef>
#include <cstdint>
#include <cstdlib>
#include <map>
#include <new>
#include <utility>
#include <vector>

namespace adapm {

// ------------------------------------------------------------------ action timing
// Q_Poiss(mu, p): the smallest k >= 0 with P(X <= k) >= p for X ~ Poisson(mu).
// The probability mass is carried in log space by the recurrence
// log P(k) = log P(k-1) + log mu - log k from log P(0) = -mu, so large rates
// do not underflow; the sum stops well past the mass of the distribution.
inline int64_t poisson_quantile(double mu, double p) {
  if (!(mu > 0.0)) return 0;
  const double lmu = std::log(mu);
  double lp = -mu;
  double cdf = std::exp(lp);
  int64_t k = 0;
  const int64_t kmax = (int64_t)(mu + 60.0 * std::sqrt(mu) + 200.0);
  while (cdf < p && k < kmax) {
    ++k;
    lp += lmu - std::log((double)k);
    cdf += std::exp(lp);
  }
  return k;
}

struct ActionTiming {
  double alpha = 0.1;      // smoothing factor
  double p = 0.9999;       // quantile of the soft upper bound
  double lambda = 10.0;    // clocks per round, estimated
  int64_t round_clock = 0; // worker clock at the previous round

  // Adaptive action timing (Section 4.2, Algorithm 1) for a round at worker
  // clock `clock`.  The estimate is an exponential moving average of the
  // clock advance between rounds, kept as it is by a round that saw no
  // advance.  The returned horizon is how far ahead this round acts: every
  // intent with C_start below it, the reach being a Poisson p-quantile at
  // twice the larger of the estimate and the last advance.
  int64_t horizon(int64_t clock) {
    const double advance = (double)(clock - round_clock);
    round_clock = clock;
    lambda = advance > 0.0 ? (1.0 - alpha) * lambda + alpha * advance : lambda;
    return clock + poisson_quantile(2.0 * std::max(lambda, advance), p);
  }
};

// ------------------------------------------------------------------ planner (host only)
// Allocator for the planner's per-key table (16 bytes per key, hundreds of
// MB, read at random keys): 2 MB-aligned and advised for transparent huge
// pages, so that a lookup does not also miss the TLB.  The advice is a hint
// the kernel may ignore.
template <class T>
struct HugePageAlloc {
  using value_type = T;
  HugePageAlloc() = default;
  template <class U>
  HugePageAlloc(const HugePageAlloc<U>&) {}
  T* allocate(size_t n) {
    constexpr size_t align = size_t(2) << 20;
    const size_t bytes = (n * sizeof(T) + align - 1) / align * align;
    void* p = nullptr;
    if (posix_memalign(&p, align, bytes) != 0) throw std::bad_alloc();
    (void)madvise(p, bytes, MADV_HUGEPAGE);
    return static_cast<T*>(p);
  }
  void deallocate(T* p, size_t) { std::free(p); }
  template <class U>
  bool operator==(const HugePageAlloc<U>&) const { return true; }
  template <class U>
  bool operator!=(const HugePageAlloc<U>&) const { return false; }
};

class Planner {
 public:
  struct Intent {
    int64_t end;
    std::vector<int64_t> keys;
    size_t next = 0;   // keys before it have been acted upon
  };

  int64_t num_keys = 0;
  std::vector<int64_t> range_begin;   // ascending, range_begin[0] == 0
  std::vector<int64_t> range_slot0;   // first slot of each range
  // per key, one cache line access: its slot (-1 when not resident) and,
  // while resident, the largest C_end of the intents acted upon for it
  struct KeyState {
    int64_t until;
    int32_t slot;
    int32_t pad;
  };
  std::vector<KeyState, HugePageAlloc<KeyState>> ks;
  std::vector<std::vector<int32_t>> free_slots;   // per range, a stack
  std::map<std::pair<int64_t, int64_t>, Intent> pending;   // (C_start, signal order) -> intent
  std::map<int64_t, std::vector<int64_t>> expiring;        // C_end -> keys whose `until` was set to it
  std::map<int64_t, int64_t> acted;   // C_start -> last round that finished acting on an intent starting there
  ActionTiming timing;
  int64_t clock = 0;
  int64_t seq = 0;
  // The current round's moves, written straight into the caller's buffers
  // (the pinned upload lists): nout write-backs at [0, nout), then nin
  // stage-ins at [nout, nout + nin).  A round evicts before it acts, so the
  // write-backs are complete when the first stage-in is written; the buffers
  // hold 2 x the slot count (at most every slot written back and refilled).
  int64_t* mkeys = nullptr;
  int64_t* mslots = nullptr;
  int64_t nout = 0, nin = 0;
  // totals
  int64_t staged_total = 0, evicted_total = 0, forced_total = 0, stalled_total = 0;
  // emptied key lists of finished intents and expiry buckets, kept with their
  // capacity: a round reuses them instead of faulting in new pages
  std::vector<std::vector<int64_t>> spare;

  std::vector<int64_t> take_list() {
    if (spare.empty()) return {};
    std::vector<int64_t> v = std::move(spare.back());
    spare.pop_back();
    v.clear();
    return v;
  }
  void give_list(std::vector<int64_t>&& v) {
    if (spare.size() < 16) spare.push_back(std::move(v));
  }

  void init(int64_t keys, const int64_t* begin, const int64_t* capacity, int nranges) {
    num_keys = keys;
    range_begin.assign(begin, begin + nranges);
    range_slot0.resize(nranges);
    free_slots.assign(nranges, {});
    int64_t s0 = 0;
    for (int r = 0; r < nranges; ++r) {
      range_slot0[r] = s0;
      auto& f = free_slots[r];
      f.reserve(capacity[r]);
      for (int64_t i = capacity[r] - 1; i >= 0; --i) f.push_back((int32_t)(s0 + i));   // pops ascending
      s0 += capacity[r];
    }
    ks.assign(keys, KeyState{0, -1, 0});
  }

  int32_t slot_of(int64_t key) const { return ks[key].slot; }

  int range_of(int64_t key) const {
    return (int)(std::upper_bound(range_begin.begin(), range_begin.end(), key) - range_begin.begin()) - 1;
  }

  // The range that starts exactly at `key`, or -1.
  int range_starting_at(int64_t key) const {
    auto it = std::lower_bound(range_begin.begin(), range_begin.end(), key);
    return (it != range_begin.end() && *it == key) ? (int)(it - range_begin.begin()) : -1;
  }

  void signal(const int64_t* keys, int64_t n, int64_t c_start, int64_t c_end) {
    if (c_end <= clock || c_end <= c_start) return;
    Intent it;
    it.end = c_end;
    it.keys = take_list();
    it.keys.assign(keys, keys + n);
    pending.emplace(std::make_pair(c_start, seq++), std::move(it));
  }

  bool due(int64_t c) const { return !pending.empty() && pending.begin()->first.first <= c; }

  void clear_moves(int64_t* keys, int64_t* slots) {
    mkeys = keys;
    mslots = slots;
    nout = nin = 0;
  }

  static constexpr size_t PREFETCH = 48;   // keys ahead whose state is fetched early (host DRAM latency)

  // Keys whose every acted-upon intent has expired leave the slot table.
  void evict_expired() {
    while (!expiring.empty() && expiring.begin()->first <= clock) {
      const std::vector<int64_t>& b = expiring.begin()->second;
      for (size_t i = 0; i < b.size(); ++i) {
        if (i + PREFETCH < b.size()) __builtin_prefetch(&ks[b[i + PREFETCH]]);
        const int64_t k = b[i];
        KeyState& st = ks[k];
        if (st.slot < 0 || st.until > clock) continue;   // already gone, or extended
        mkeys[nout] = k;
        mslots[nout] = st.slot;
        ++nout;
        free_slots[range_of(k)].push_back(st.slot);
        st.slot = -1;
        ++evicted_total;
      }
      give_list(std::move(expiring.begin()->second));
      expiring.erase(expiring.begin());
    }
  }

  // Act on pending intents with C_start < horizon, in (C_start, signal)
  // order; a full key range stops the acting until a later round.
  void act(int64_t horizon, int64_t round_id) {
    while (!pending.empty() && pending.begin()->first.first < horizon) {
      const int64_t c_start = pending.begin()->first.first;
      Intent& it = pending.begin()->second;
      if (it.end <= clock) {   // expired before it could be acted upon
        give_list(std::move(it.keys));
        pending.erase(pending.begin());
        continue;
      }
      auto [bpos, fresh] = expiring.try_emplace(it.end);
      if (fresh) bpos->second = take_list();
      std::vector<int64_t>& bucket = bpos->second;
      const size_t nk = it.keys.size();
      for (; it.next < nk; ++it.next) {
        if (it.next + PREFETCH < nk) {
          const int64_t kp = it.keys[it.next + PREFETCH];
          if (kp >= 0 && kp < num_keys) __builtin_prefetch(&ks[kp]);
        }
        const int64_t k = it.keys[it.next];
        if (k < 0 || k >= num_keys) continue;
        KeyState& st = ks[k];
        if (st.slot >= 0) {
          if (it.end > st.until) {
            st.until = it.end;
            bucket.push_back(k);
          }
          continue;
        }
        auto& f = free_slots[range_of(k)];
        if (f.empty()) {
          ++stalled_total;
          return;
        }
        const int32_t sl = f.back();
        f.pop_back();
        st.slot = sl;
        st.until = it.end;
        bucket.push_back(k);
        mkeys[nout + nin] = k;
        mslots[nout + nin] = sl;
        ++nin;
        ++staged_total;
      }
      auto a = acted.find(c_start);
      if (a == acted.end()) acted.emplace(c_start, round_id);
      else a->second = std::max(a->second, round_id);
      give_list(std::move(it.keys));
      pending.erase(pending.begin());
    }
  }

  // The latest round that acted on intents starting at or before `c`
  // (forgotten afterwards), or -1.
  int64_t take_round_for(int64_t c) {
    int64_t r = -1;
    while (!acted.empty() && acted.begin()->first <= c) {
      r = std::max(r, acted.begin()->second);
      acted.erase(acted.begin());
    }
    return r;
  }
};

}  // namespace adapm
