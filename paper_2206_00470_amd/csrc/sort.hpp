// Duplicate-key merge order: a stable LSD radix sort of (key, occurrence)
// pairs, then segment and chunk boundaries of the sorted keys.
//
// Radix tiles hold BLOCK * IT keys (IT = 4, 8 or 16 keys per thread, chosen
// per call from the number of keys).  Each pass is reduce-then-scan:
//   count   : per-tile digit histogram  -> counts[digit][tile]
//   scan    : one workgroup per digit turns its row of counts into global
//             offsets, seeded with the digit base from a whole-array
//             histogram that the key-intake kernel built for all passes
//   scatter : stable in-tile ranks from wavefront ballots (each lane finds
//             the lanes of its wave holding the same digit), combined
//             across the 4 waves of the tile in wave order.
// Invalid keys are mapped to the sentinel num_keys, so they sort last.
#pragma once

#include "common.hpp"

namespace adapm {

struct RadixPlan {
  int passes;
  int shift[MAX_PASSES];
  int bits[MAX_PASSES];
};

// Fill `n` 32-bit words with zero.
__global__ __launch_bounds__(BLOCK) void k_zero_words(uint32_t* p, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)BLOCK + threadIdx.x; i < n; i += (int64_t)gridDim.x * BLOCK)
    p[i] = 0u;
}

// ------------------------------------------------------------------ key intake
// Key source functors give the int64 key of occurrence i, or ABSENT.
struct KeysInt64 {
  const int64_t* keys;
  __device__ int64_t operator()(int64_t i) const { return keys[i]; }
};

// Reads every occurrence key once: range check (invalid -> sentinel and the
// sticky error flag), narrow to u32, digit-0 histogram of this tile, and the
// whole-array histograms of every pass.  Those are kept in GH_COPIES copies,
// tile t adding to copy t % GH_COPIES, so that no histogram word takes more
// than tiles / GH_COPIES atomic adds.
template <class KS, int IT>
__global__ __launch_bounds__(BLOCK) void k_keyprep(KS ks, int64_t n, uint32_t sentinel, RadixPlan plan,
                                                   uint32_t* __restrict__ kout, uint32_t* __restrict__ counts0,
                                                   int tiles, uint32_t* __restrict__ ghist,
                                                   int32_t* __restrict__ err) {
  __shared__ uint32_t h[MAX_PASSES][MAX_BINS];
  for (int i = threadIdx.x; i < MAX_PASSES * MAX_BINS; i += BLOCK) (&h[0][0])[i] = 0u;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * (BLOCK * IT);
  int bad = 0;
#pragma unroll 4
  for (int it = 0; it < IT; ++it) {
    const int64_t i = base + (int64_t)it * BLOCK + threadIdx.x;
    if (i < n) {
      const int64_t key = ks(i);
      uint32_t k;
      if (key == ABSENT) {
        k = sentinel;
      } else if (key < 0 || key >= (int64_t)sentinel) {
        k = sentinel;
        bad = 1;
      } else {
        k = (uint32_t)key;
      }
      kout[i] = k;
      for (int p = 0; p < plan.passes; ++p)
        atomicAdd(&h[p][(k >> plan.shift[p]) & ((1u << plan.bits[p]) - 1u)], 1u);
    }
  }
  bad = __syncthreads_or(bad);
  if (bad && threadIdx.x == 0 && err) atomicOr(err, 1);
  const int bins0 = 1 << plan.bits[0];
  for (int d = threadIdx.x; d < bins0; d += BLOCK) counts0[(int64_t)d * tiles + blockIdx.x] = h[0][d];
  uint32_t* gh = ghist + (int64_t)(blockIdx.x % GH_COPIES) * MAX_BINS;
  for (int p = 0; p < plan.passes; ++p) {
    const int bins = 1 << plan.bits[p];
    for (int d = threadIdx.x; d < bins; d += BLOCK)
      if (h[p][d]) atomicAdd(&gh[(int64_t)p * GH_COPIES * MAX_BINS + d], h[p][d]);
  }
}

// ------------------------------------------------------------------ count
template <int IT>
__global__ __launch_bounds__(BLOCK) void k_radix_count(const uint32_t* __restrict__ keys, int64_t n, int shift,
                                                       int bits, uint32_t* __restrict__ counts, int tiles) {
  __shared__ uint32_t h[MAX_BINS];
  const int bins = 1 << bits;
  for (int d = threadIdx.x; d < bins; d += BLOCK) h[d] = 0u;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * (BLOCK * IT);
#pragma unroll 4
  for (int it = 0; it < IT; ++it) {
    const int64_t i = base + (int64_t)it * BLOCK + threadIdx.x;
    if (i < n) atomicAdd(&h[(keys[i] >> shift) & (bins - 1)], 1u);
  }
  __syncthreads();
  for (int d = threadIdx.x; d < bins; d += BLOCK) counts[(int64_t)d * tiles + blockIdx.x] = h[d];
}

// ------------------------------------------------------------------ scan
// One workgroup per digit d: offsets[d][t] = sum_{d'<d} total[d'] + sum_{t'<t} counts[d][t'].
// ghist_pass holds the pass's GH_COPIES histogram copies ([GH_COPIES][MAX_BINS]).
__global__ __launch_bounds__(BLOCK) void k_radix_scan(uint32_t* __restrict__ counts, int tiles,
                                                      const uint32_t* __restrict__ ghist_pass) {
  __shared__ uint32_t smem[WAVES_PER_BLOCK + 1];
  __shared__ double dsm[WAVES_PER_BLOCK];
  const int d = blockIdx.x;
  // digit base: thread i sums digits i + BLOCK q over the copies (independent
  // loads), then the block adds the digits below d (exact in double: the sum
  // is below 2^31)
  static_assert(BLOCK * DIG_PER_THREAD == MAX_BINS, "every digit has a thread");
  double part = 0.0;
#pragma unroll
  for (int q = 0; q < DIG_PER_THREAD; ++q) {
    const int dd = threadIdx.x + BLOCK * q;
    uint32_t x[GH_COPIES];
#pragma unroll
    for (int c = 0; c < GH_COPIES; ++c) x[c] = ghist_pass[c * MAX_BINS + dd];
    uint32_t tot = 0;
#pragma unroll
    for (int c = 0; c < GH_COPIES; ++c) tot += x[c];
    part += dd < d ? (double)tot : 0.0;
  }
  double b = block_sum_double(part, dsm);
  __shared__ uint32_t sbase;
  if (threadIdx.x == 0) sbase = (uint32_t)b;
  __syncthreads();
  uint32_t carry = sbase;
  uint32_t* row = counts + (int64_t)d * tiles;
  for (int t0 = 0; t0 < tiles; t0 += BLOCK) {
    const int t = t0 + threadIdx.x;
    const uint32_t x = t < tiles ? row[t] : 0u;
    uint32_t tot;
    const uint32_t ex = block_exclusive_scan(x, smem, &tot);
    if (t < tiles) row[t] = carry + ex;
    carry += tot;
  }
}

// ------------------------------------------------------------------ scatter
// FIRST: the values are the occurrence indices themselves (no value input).
// RANK : also write rank[value] = destination (the inverse permutation).
template <bool FIRST, bool RANK, int IT>
__global__ __launch_bounds__(BLOCK) void k_radix_scatter(const uint32_t* __restrict__ kin,
                                                         const uint32_t* __restrict__ vin, int64_t n, int shift,
                                                         int bits, const uint32_t* __restrict__ offs, int tiles,
                                                         uint32_t* __restrict__ kout, uint32_t* __restrict__ vout,
                                                         uint32_t* __restrict__ rank) {
  static_assert(BLOCK * DIG_PER_THREAD == MAX_BINS, "every digit has a thread in the tile scan");
  __shared__ uint32_t wc[WAVES_PER_BLOCK][MAX_BINS];
  __shared__ uint32_t toff[MAX_BINS];
  __shared__ uint32_t dstart[MAX_BINS];
  __shared__ uint32_t scan_smem[WAVES_PER_BLOCK + 1];
  __shared__ uint32_t sk[(BLOCK * IT)];
  __shared__ uint32_t sv[(BLOCK * IT)];
  const int bins = 1 << bits;
  const uint32_t mask = (uint32_t)bins - 1u;
  for (int i = threadIdx.x; i < WAVES_PER_BLOCK * MAX_BINS; i += BLOCK) (&wc[0][0])[i] = 0u;
  for (int d = threadIdx.x; d < bins; d += BLOCK) toff[d] = offs[(int64_t)d * tiles + blockIdx.x];
  __syncthreads();

  const int w = threadIdx.x / WAVE;
  const int lane = lane_id();
  const uint64_t lt = lanemask_lt();
  const int64_t base = (int64_t)blockIdx.x * (BLOCK * IT) + (int64_t)w * (WAVE * IT);
  uint32_t key[IT], val[IT], rk[IT];
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int64_t i = base + it * WAVE + lane;
    const bool valid = i < n;
    key[it] = valid ? kin[i] : 0u;
    if constexpr (FIRST) val[it] = (uint32_t)i;
    else val[it] = valid ? vin[i] : 0u;
  }
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int64_t i = base + it * WAVE + lane;
    const bool valid = i < n;
    const uint32_t d = (key[it] >> shift) & mask;
    uint64_t m = __ballot(valid);
    for (int b = 0; b < bits; ++b) {
      const bool bit = (d >> b) & 1u;
      const uint64_t bb = __ballot(bit);
      m &= bit ? bb : ~bb;
    }
    const uint32_t below = __popcll(m & lt);
    const uint32_t cnt = __popcll(m);
    uint32_t r = 0;
    if (valid) {
      const uint32_t start = wc[w][d];
      r = start + below;
      if (below == cnt - 1) wc[w][d] = start + cnt;
    }
    rk[it] = r;
  }
  __syncthreads();
  // per digit: offsets of the 4 waves inside the tile's run, and the run's
  // start within the tile (exclusive scan over digits; thread i owns the
  // DIG_PER_THREAD consecutive digits from i * DIG_PER_THREAD)
  {
    uint32_t tot[DIG_PER_THREAD];
    uint32_t mine = 0;
#pragma unroll
    for (int q = 0; q < DIG_PER_THREAD; ++q) {
      const int d = threadIdx.x * DIG_PER_THREAD + q;
      tot[q] = 0;
      if (d < bins) {
        for (int ww = 0; ww < WAVES_PER_BLOCK; ++ww) {
          const uint32_t t = wc[ww][d];
          wc[ww][d] = tot[q];
          tot[q] += t;
        }
      }
      mine += tot[q];
    }
    uint32_t all;
    uint32_t run = block_exclusive_scan(mine, scan_smem, &all);
#pragma unroll
    for (int q = 0; q < DIG_PER_THREAD; ++q) {
      dstart[threadIdx.x * DIG_PER_THREAD + q] = run;
      run += tot[q];
    }
  }
  __syncthreads();
  // stage the tile in LDS in digit order ...
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int64_t i = base + it * WAVE + lane;
    if (i < n) {
      const uint32_t d = (key[it] >> shift) & mask;
      const uint32_t p = dstart[d] + wc[w][d] + rk[it];
      sk[p] = key[it];
      sv[p] = val[it];
    }
  }
  __syncthreads();
  // ... and write it out: consecutive threads write consecutive positions of a digit run
  const int64_t tile_base = (int64_t)blockIdx.x * (BLOCK * IT);
  const int cnt = (int)((n - tile_base) < (BLOCK * IT) ? (n - tile_base) : (BLOCK * IT));
  for (int p = threadIdx.x; p < cnt; p += BLOCK) {
    const uint32_t k = sk[p];
    const uint32_t v = sv[p];
    const uint32_t d = (k >> shift) & mask;
    const uint32_t pos = toff[d] + (uint32_t)p - dstart[d];
    kout[pos] = k;
    vout[pos] = v;
    if constexpr (RANK) rank[v] = pos;
  }
}

// ------------------------------------------------------------------ segments
// Sorted position j (valid key) starts a segment if its key differs from
// position j-1.  It starts a chunk if it starts a segment, or if j is a
// multiple of CHUNK and position j - CHUNK holds the same key ("cut"): a
// segment of at most CHUNK occurrences is never cut, a longer one is cut at
// the multiples of CHUNK at least CHUNK past its start, so a chunk holds at
// most 2*CHUNK-1 occurrences and a CHUNK-aligned block holds at most two
// chunk starts of cut segments (a cut at its start, a segment head inside).
__device__ __forceinline__ bool chunk_cut(const uint32_t* __restrict__ ks, int64_t j, uint32_t k) {
  return (j % CHUNK) == 0 && j >= CHUNK && ks[j - CHUNK] == k;
}

// Per tile: number of segment heads, chunk heads and valid positions.
template <int IT>
__global__ __launch_bounds__(BLOCK) void k_seg_count(const uint32_t* __restrict__ ks, int64_t n, uint32_t sentinel,
                                                     uint32_t* __restrict__ tstat /*[3][tiles]*/, int tiles) {
  __shared__ uint32_t smem[WAVES_PER_BLOCK + 1];
  const int64_t base = (int64_t)blockIdx.x * (BLOCK * IT);
  uint32_t nh = 0, nc = 0, nv = 0;
#pragma unroll 4
  for (int it = 0; it < IT; ++it) {
    const int64_t j = base + (int64_t)it * BLOCK + threadIdx.x;
    if (j < n) {
      const uint32_t k = ks[j];
      if (k < sentinel) {
        const bool head = (j == 0) || ks[j - 1] != k;
        nv += 1;
        nh += head;
        nc += head || chunk_cut(ks, j, k);
      }
    }
  }
  uint32_t th, tc, tv;
  block_exclusive_scan(nh, smem, &th);
  block_exclusive_scan(nc, smem, &tc);
  block_exclusive_scan(nv, smem, &tv);
  if (threadIdx.x == 0) {
    tstat[blockIdx.x] = th;
    tstat[tiles + blockIdx.x] = tc;
    tstat[2 * tiles + blockIdx.x] = tv;
  }
}

// Single workgroup: exclusive scans of the per-tile head and chunk counts,
// totals into the header, and the closing entries offsets[U], chunk_start[C].
__global__ __launch_bounds__(BLOCK) void k_seg_scan(uint32_t* __restrict__ tstat, int tiles, SegHeader* hdr,
                                                    int32_t* __restrict__ seg_off,
                                                    int32_t* __restrict__ chunk_start) {
  __shared__ uint32_t smem[WAVES_PER_BLOCK + 1];
  constexpr int IPT = 16;   // consecutive tiles per thread and round
  uint32_t ch = 0, cc = 0, cv = 0;
  for (int t0 = 0; t0 < tiles; t0 += BLOCK * IPT) {
    const int tb = t0 + threadIdx.x * IPT;
    uint32_t h[IPT], c[IPT];
    uint32_t sh = 0, sc = 0, sv = 0;
#pragma unroll
    for (int q = 0; q < IPT; ++q) {
      const int t = tb + q;
      h[q] = t < tiles ? tstat[t] : 0u;
      c[q] = t < tiles ? tstat[tiles + t] : 0u;
      sv += t < tiles ? tstat[2 * tiles + t] : 0u;
    }
#pragma unroll
    for (int q = 0; q < IPT; ++q) {
      sh += h[q];
      sc += c[q];
    }
    uint32_t th, tc, tv;
    uint32_t eh = block_exclusive_scan(sh, smem, &th) + ch;
    uint32_t ec = block_exclusive_scan(sc, smem, &tc) + cc;
    block_exclusive_scan(sv, smem, &tv);
#pragma unroll
    for (int q = 0; q < IPT; ++q) {
      const int t = tb + q;
      if (t < tiles) {
        tstat[t] = eh;
        tstat[tiles + t] = ec;
      }
      eh += h[q];
      ec += c[q];
    }
    ch += th;
    cc += tc;
    cv += tv;
  }
  if (threadIdx.x == 0) {
    hdr->num_unique = ch;
    hdr->num_chunks = cc;
    hdr->num_valid = cv;
    hdr->num_lo = ch;   // k_seg_write lowers these if some key reaches the split key
    hdr->chunk_lo = cc;
    seg_off[ch] = (int32_t)cv;
    chunk_start[cc] = (int32_t)cv;
  }
}

// Per tile (blocked: thread t owns positions base + t*IT ..): write
// the segment offsets (and optionally the distinct keys as int64), the chunk
// list (start position and segment of each chunk) and the number of segments
// with key < split_key.
template <int IT>
__global__ __launch_bounds__(BLOCK) void k_seg_write(const uint32_t* __restrict__ ks, int64_t n, uint32_t sentinel,
                                                     const uint32_t* __restrict__ tstat, int tiles,
                                                     int32_t* __restrict__ seg_off, int64_t* __restrict__ uniq64,
                                                     int32_t* __restrict__ chunk_start,
                                                     int32_t* __restrict__ chunk_seg,
                                                     uint32_t split_key,
                                                     SegHeader* hdr) {
  __shared__ uint32_t smem[WAVES_PER_BLOCK + 1];
  const int64_t base = (int64_t)blockIdx.x * (BLOCK * IT) + (int64_t)threadIdx.x * IT;
  uint32_t k[IT];
  uint32_t prev = (base > 0 && base - 1 < n) ? ks[base - 1] : 0xFFFFFFFFu;
#pragma unroll
  for (int q = 0; q < IT; ++q) {
    const int64_t j = base + q;
    k[q] = j < n ? ks[j] : sentinel;
  }
  uint32_t hf = 0, cf = 0;   // bit q: position base+q starts a segment / chunk
  uint32_t nh = 0, nc = 0;
#pragma unroll
  for (int q = 0; q < IT; ++q) {
    const int64_t j = base + q;
    const uint32_t p = q == 0 ? prev : k[q - 1];
    const bool valid = j < n && k[q] < sentinel;
    const bool head = valid && (j == 0 || p != k[q]);
    const bool chead = valid && (head || chunk_cut(ks, j, k[q]));
    hf |= (uint32_t)head << q;
    cf |= (uint32_t)chead << q;
    nh += head;
    nc += chead;
  }
  uint32_t th, tc;
  uint32_t hi = block_exclusive_scan(nh, smem, &th) + tstat[blockIdx.x];
  uint32_t ci = block_exclusive_scan(nc, smem, &tc) + tstat[tiles + blockIdx.x];
  // segment index of the position before this thread's first one
  int64_t cur = (int64_t)hi - 1;
#pragma unroll
  for (int q = 0; q < IT; ++q) {
    const int64_t j = base + q;
    if ((hf >> q) & 1u) {
      seg_off[hi] = (int32_t)j;
      if (uniq64) uniq64[hi] = (int64_t)k[q];
      const uint32_t pk = q == 0 ? prev : k[q - 1];
      if (k[q] >= split_key && (j == 0 || pk < split_key)) {
        hdr->num_lo = hi;
        hdr->chunk_lo = ci;   // a segment head is always a chunk head
      }
      cur = hi;
      ++hi;
    }
    if ((cf >> q) & 1u) {
      chunk_start[ci] = (int32_t)j;
      chunk_seg[ci] = (int32_t)cur;
      ++ci;
    }
  }
}

}  // namespace adapm
