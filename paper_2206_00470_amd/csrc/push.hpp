// Read access (pull) and merged write access (segmented reduce + AdaGrad).
//
// Work is mapped to "groups" of L lanes, one group per row: L is the power of
// two that covers dim/VW vectors (VW = 4 floats when dim % 4 == 0), so a
// 400-byte MF row is one 16-byte load per lane of a 32-lane half-wave and a
// wavefront serves two rows at once.
#pragma once

#include "common.hpp"

namespace adapm {

struct RowShape {
  int L;    // lanes per row group
  int NV;   // vectors per lane
  int VW;   // floats per vector
};

// ------------------------------------------------------------------ pull
// With a key -> slot map (a staged store), keys index the home table of
// map_keys keys and rows are read from their slots; a key with no slot gives
// a zero row and sets err[1].  VT: the table's value type (float or bf16_t);
// the pulled rows are fp32 either way.
// Pulled row i goes to out + i * out_ld (out_ld = dim, or the full row
// width when a wide row is pulled in column slices).
template <int L, int NV, int VW, class VT>
__global__ __launch_bounds__(BLOCK) void k_pull(const VT* __restrict__ W, int64_t ld, int64_t num_keys, int dim,
                                                const int64_t* __restrict__ keys, int64_t n,
                                                float* __restrict__ out, int64_t out_ld, int32_t* __restrict__ err,
                                                const int32_t* __restrict__ map, int64_t map_keys) {
  constexpr int GPB = BLOCK / L;
  const int gl = threadIdx.x % L;
  int bad = 0, miss = 0;
  for (int64_t i = (int64_t)blockIdx.x * GPB + threadIdx.x / L; i < n; i += (int64_t)gridDim.x * GPB) {
    int64_t key = keys[i];
    bool ok;
    if (map) {
      ok = key >= 0 && key < map_keys;
      bad |= !ok;
      const int32_t m = ok ? map[key] : -1;
      miss |= ok && m < 0;
      ok = m >= 0;
      key = m;
    } else {
      ok = key >= 0 && key < num_keys;
      bad |= !ok;
    }
    const VT* src = W + (ok ? key : 0) * ld;
    float* dst = out + i * out_ld;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int c = (gl + v * L) * VW;
      if (c < dim) {
        float x[VW];
        if (ok) load_vals<VW>(src + c, x);
        else
#pragma unroll
          for (int e = 0; e < VW; ++e) x[e] = 0.0f;
        store_frag<VW>(dst + c, x);
      }
    }
  }
  if (__syncthreads_or(bad) && threadIdx.x == 0) atomicOr(err, 1);
  if (__syncthreads_or(miss) && threadIdx.x == 0) atomicOr(err + 1, 1);
}

// ------------------------------------------------------------------ gather probe
// The row reads of a gather-bound kernel without its arithmetic (for
// measurement): row group g reads the rows keys[i] of W for i = g, g + S,
// g + 2S, ... (S row groups in the grid, UNROLL rows in flight per group)
// and adds them into fp64 lane sums; each workgroup writes the sum of its
// lanes' sums to sink[workgroup], so the loads cannot be left out.  Keys
// outside [0, rows) are skipped.
template <int L, int NV, int VW>
__global__ __launch_bounds__(BLOCK) void k_gather_probe(const float* __restrict__ W, int64_t ld, int dim,
                                                        int64_t rows, const int32_t* __restrict__ keys, int64_t n,
                                                        double* __restrict__ sink) {
  constexpr int GPB = BLOCK / L;
  constexpr int NE = NV * VW;
  constexpr int UNROLL = NE <= 4 ? 8 : 4;
  __shared__ double sm[WAVES_PER_BLOCK];
  const int gl = threadIdx.x % L;
  const int64_t S = (int64_t)gridDim.x * GPB;
  double acc[NE];
#pragma unroll
  for (int e = 0; e < NE; ++e) acc[e] = 0.0;
  auto load_row = [&](int64_t i, float* x) {
    const int32_t k = keys[i];
    const bool ok = k >= 0 && k < rows;
    const float* p = W + (ok ? (int64_t)k : 0) * ld;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int c = (gl + v * L) * VW;
      if (ok && c < dim) load_frag<VW>(p + c, x + v * VW);
      else
#pragma unroll
        for (int e = 0; e < VW; ++e) x[v * VW + e] = 0.0f;
    }
  };
  int64_t i = (int64_t)blockIdx.x * GPB + threadIdx.x / L;
  for (; i + (UNROLL - 1) * S < n; i += UNROLL * S) {
    float x[UNROLL][NE];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) load_row(i + u * S, x[u]);
#pragma unroll
    for (int u = 0; u < UNROLL; ++u)
#pragma unroll
      for (int e = 0; e < NE; ++e) acc[e] += (double)x[u][e];
  }
  for (; i < n; i += S) {
    float x[NE];
    load_row(i, x);
#pragma unroll
    for (int e = 0; e < NE; ++e) acc[e] += (double)x[e];
  }
  double t = 0.0;
#pragma unroll
  for (int e = 0; e < NE; ++e) t += acc[e];
  t = block_sum_double(t, sm);
  if (threadIdx.x == 0) sink[blockIdx.x] = t;
}

// ------------------------------------------------------------------ gradient sources
// A source describes the fp32 gradient row of the occurrence at sorted
// position j in two steps:
//   meta(j)            the per-occurrence indirections (loaded by one lane,
//                      for up to L consecutive positions at once)
//   load(m, own, ...)  the lane's fragment of the gradient row, given the
//                      broadcast metadata and, for sources that need it
//                      (kNeedsOwn), the pre-step row of the segment's key.
// Metadata travels between lanes word by word.
template <class T>
__device__ __forceinline__ T shfl_pod(const T& v, int src, int width) {
  static_assert(sizeof(T) % 4 == 0, "metadata must be whole words");
  union U {
    T t;
    uint32_t w[sizeof(T) / 4];
  } in, out;
  in.t = v;
#pragma unroll
  for (int i = 0; i < (int)(sizeof(T) / 4); ++i) out.w[i] = __shfl(in.w[i], src, width);
  return out.t;
}

// Gradient rows in occurrence order, ld floats apart, read through the sort
// permutation.
struct SrcIndirect {
  static constexpr bool kNeedsOwn = false;
  const float* grads;
  const uint32_t* perm;
  int dim;
  int64_t ld;
  struct Meta {
    const float* row;
  };
  __device__ __forceinline__ Meta meta(int64_t j) const { return {grads + (int64_t)perm[j] * ld}; }
  template <int L, int NV, int VW>
  __device__ __forceinline__ void load(const Meta& m, const float*, int gl, float* x) const {
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int c = (gl + v * L) * VW;
      if (c < dim) load_frag<VW>(m.row + c, x + v * VW);
    }
  }
};

// Gradient rows already stored at their sorted positions, ld floats apart.
struct SrcSorted {
  static constexpr bool kNeedsOwn = false;
  const float* grads;
  int dim;
  int64_t ld;
  struct Meta {
    const float* row;
  };
  __device__ __forceinline__ Meta meta(int64_t j) const { return {grads + j * ld}; }
  template <int L, int NV, int VW>
  __device__ __forceinline__ void load(const Meta& m, const float*, int gl, float* x) const {
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int c = (gl + v * L) * VW;
      if (c < dim) load_frag<VW>(m.row + c, x + v * VW);
    }
  }
};

// Sources with kLoss = true also add each occurrence's loss term to a
// per-thread sum (load takes it as a last argument); the merge writes the
// workgroup totals to src.loss_part[workgroup].
template <class Src>
constexpr bool src_has_loss() {
  if constexpr (requires { Src::kLoss; }) return Src::kLoss;
  else return false;
}

template <int L, int NV, int VW, class Src>
__device__ __forceinline__ void src_load(const Src& src, const typename Src::Meta& m, const float* own, int gl,
                                         float* x, double& lsum) {
  if constexpr (src_has_loss<Src>()) src.template load<L, NV, VW>(m, own, gl, x, lsum);
  else src.template load<L, NV, VW>(m, own, gl, x);
}

// ------------------------------------------------------------------ reduce
struct SegView {
  const uint32_t* keys;        // sorted u32 keys
  const int32_t* seg_off;      // [U+1]
  const int32_t* chunk_start;  // [nchunks+1]
  const int32_t* chunk_seg;    // [nchunks]
  const SegHeader* hdr;
};

// Map a workgroup index to a group-slot so that consecutive work items stay
// on one accelerator die (workgroups are dealt round-robin over the 8 dies,
// each with its own L2): die x gets the x-th contiguous slice of the slots.
__device__ __forceinline__ int64_t xcd_slot(int64_t block, int64_t nblocks) {
  if (nblocks % NUM_XCD != 0) return block;
  const int64_t per = nblocks / NUM_XCD;
  return (block % NUM_XCD) * per + block / NUM_XCD;
}

// Chunk c covers sorted positions [chunk_start[c], chunk_start[c+1]) of one
// segment.  The group sums its gradient rows in position order in fp64: the
// metadata of up to L positions is loaded at once (one lane each) and
// broadcast, so each row load depends on one round trip only.  If the chunk
// is the whole segment the group rounds the sum to fp32 and applies AdaGrad
// to the key's row; otherwise it stores the fp64 partial in the slot of its
// CHUNK-aligned block (2 slots per block: the chunk starting at the block
// start, and the one starting inside it) for k_seg_finalize; the first chunk
// of such a segment also appends the segment to split_list.
// RW selects row-wise AdaGrad: G then holds one accumulator per key, at
// G[key * gld]; otherwise G is a table of rows at G + key * gld.
template <int L, int NV, int VW, class Src, bool RW, class VT>
__global__ __launch_bounds__(BLOCK) void k_segreduce(SegView sv, Src src, int64_t n, VT* __restrict__ W,
                                                     float* __restrict__ G, int64_t ld, int64_t gld, int dim,
                                                     float lr, float eps,
                                                     double* __restrict__ partial,
                                                     int32_t* __restrict__ split_list, SegHeader* split_hdr,
                                                     int part) {
  constexpr int GPB = BLOCK / L;
  constexpr int NE = NV * VW;
  constexpr int UNROLL = src_has_loss<Src>() ? 1 : (NE <= 4 ? 4 : 2);
  using Meta = typename Src::Meta;
  const int gl = threadIdx.x % L;
  // part 0: every chunk; 1: chunks whose key reaches the split key; 2: the others
  int64_t cbeg = 0, cend = sv.hdr->num_chunks;
  if (part == 1) cbeg = sv.hdr->chunk_lo;
  if (part == 2) cend = sv.hdr->chunk_lo;
  // chunks are dealt round-robin over the S row groups of the grid (hot keys'
  // chunks spread out); lane i prefetches the bounds and keys of the group's
  // i-th next chunk, so one round of loads serves L chunks
  const int64_t S = (int64_t)gridDim.x * GPB;
  double lsum = 0.0;
  for (int64_t cb = cbeg + xcd_slot(blockIdx.x, gridDim.x) * GPB + threadIdx.x / L; cb < cend; cb += S * L) {
    const int64_t left = (cend - cb + S - 1) / S;
    const int ccount = (int)(left < L ? left : L);
    int32_t my_j0 = 0, my_j1 = 0;
    uint32_t my_key = 0, my_flags = 0;
    Meta my_first{};   // metadata of the chunk's first occurrence
    if (gl < ccount) {
      my_j0 = sv.chunk_start[cb + gl * S];
      my_j1 = sv.chunk_start[cb + gl * S + 1];
      my_first = src.meta(my_j0);
      my_key = sv.keys[my_j0];
      // the chunk is a whole segment if its neighbours hold other keys
      const bool hd = my_j0 == 0 || sv.keys[my_j0 - 1] != my_key;
      const bool wh = hd && (my_j1 >= n || sv.keys[my_j1] != my_key);
      my_flags = (hd ? 1u : 0u) | (wh ? 2u : 0u);
    }
  for (int ci = 0; ci < ccount; ++ci) {
    const int64_t c = cb + ci * S;
    const int64_t j0 = __shfl(my_j0, ci, L);
    const int64_t j1 = __shfl(my_j1, ci, L);
    const uint32_t key = __shfl(my_key, ci, L);
    const uint32_t flags = __shfl(my_flags, ci, L);
    const bool head = flags & 1u;
    const bool whole = flags & 2u;
    const Meta first = shfl_pod(my_first, ci, L);
    VT* wrow = W + (int64_t)key * ld;
    float* grow = G + (int64_t)key * gld;
    float wv[NE], gv[NE];
    float gacc = 0.0f;   // RW: the key's accumulator
    if (whole || Src::kNeedsOwn) {   // issue the table reads early, they do not depend on the sum
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int col = (gl + v * L) * VW;
        if (col < dim) {
          load_vals<VW>(wrow + col, wv + v * VW);
          if (!RW && whole) load_frag<VW>(grow + col, gv + v * VW);
        }
      }
      if (RW && whole) gacc = *grow;
    }
    double acc[NE];
#pragma unroll
    for (int e = 0; e < NE; ++e) acc[e] = 0.0;
    for (int64_t jb = j0; jb < j1; jb += L) {
      const int cnt = (int)((j1 - jb) < L ? (j1 - jb) : L);
      Meta mine{};
      if (jb == j0 && gl == 0) mine = first;            // prefetched with the chunk bounds
      else if (gl < cnt) mine = src.meta(jb + gl);
      int q = 0;
      for (; q + UNROLL <= cnt; q += UNROLL) {
        float x[UNROLL][NE];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) src_load<L, NV, VW>(src, shfl_pod(mine, q + u, L), wv, gl, x[u], lsum);
#pragma unroll
        for (int u = 0; u < UNROLL; ++u)
#pragma unroll
          for (int e = 0; e < NE; ++e) acc[e] += (double)x[u][e];
      }
      for (; q < cnt; ++q) {
        float x[NE];
        src_load<L, NV, VW>(src, shfl_pod(mine, q, L), wv, gl, x, lsum);
#pragma unroll
        for (int e = 0; e < NE; ++e) acc[e] += (double)x[e];
      }
    }
    if (whole && RW) {
      float g[NE];
      double sq = 0.0;
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int col = (gl + v * L) * VW;
#pragma unroll
        for (int e = 0; e < VW; ++e) {
          g[v * VW + e] = (float)acc[v * VW + e];
          if (col < dim) sq += (double)g[v * VW + e] * (double)g[v * VW + e];
        }
      }
      sq = group_sum<L>(sq);
      const float den = rowwise_den(gacc, sq, dim, eps);
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int col = (gl + v * L) * VW;
        if (col < dim) {
#pragma unroll
          for (int e = 0; e < VW; ++e) rowwise_elem(wv[v * VW + e], g[v * VW + e], den, lr);
          store_vals<VW>(wrow + col, wv + v * VW);
        }
      }
      if (gl == 0) *grow = gacc;
    } else if (whole) {
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int col = (gl + v * L) * VW;
        if (col < dim) {
#pragma unroll
          for (int e = 0; e < VW; ++e)
            adagrad_elem(wv[v * VW + e], gv[v * VW + e], (float)acc[v * VW + e], lr, eps);
          store_vals<VW>(wrow + col, wv + v * VW);
          store_frag<VW>(grow + col, gv + v * VW);
        }
      }
    } else {
      if (head && gl == 0) split_list[atomicAdd(&split_hdr->num_split, 1u)] = sv.chunk_seg[c];
      const int64_t slot = 2 * (j0 / CHUNK) + ((j0 % CHUNK) != 0);
      double* p = partial + slot * dim;
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int col = (gl + v * L) * VW;
        if (col < dim)
#pragma unroll
          for (int e = 0; e < VW; ++e) p[col + e] = acc[v * VW + e];
      }
    }
  }
  }
  if constexpr (src_has_loss<Src>()) {
    __shared__ double sm[WAVES_PER_BLOCK];
    lsum = block_sum_double(lsum, sm);
    if (threadIdx.x == 0) src.loss_part[blockIdx.x] = lsum;
  }
}

// Block-wide fixed-order sum of `count` fp64 rows of dim values: row group g
// adds rows g, g + GPB, g + 2 GPB, ... (FU rows in flight), in that order,
// and leaves its sum in lds[g][*]; the caller adds the GPB group sums in
// group order.  row(i) returns the address of row i.
template <int L, int NV, int VW, class RowAt>
__device__ __forceinline__ void group_sum_rows(RowAt row, int64_t count, int dim, double* lds) {
  constexpr int GPB = BLOCK / L;
  constexpr int NE = NV * VW;
  constexpr int FU = NE <= 4 ? 8 : 4;
  const int gl = threadIdx.x % L;
  const int g = threadIdx.x / L;
  double acc[NE];
#pragma unroll
  for (int q = 0; q < NE; ++q) acc[q] = 0.0;
  int64_t k = g;
  for (; k + (FU - 1) * GPB < count; k += FU * GPB) {
    double x[FU][NE];
#pragma unroll
    for (int f = 0; f < FU; ++f) {
      const double* p = row(k + f * GPB);
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int col = (gl + v * L) * VW;
#pragma unroll
        for (int q = 0; q < VW; ++q) x[f][v * VW + q] = col < dim ? p[col + q] : 0.0;
      }
    }
#pragma unroll
    for (int f = 0; f < FU; ++f)
#pragma unroll
      for (int q = 0; q < NE; ++q) acc[q] += x[f][q];
  }
  for (; k < count; k += GPB) {
    const double* p = row(k);
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int col = (gl + v * L) * VW;
      if (col < dim)
#pragma unroll
        for (int q = 0; q < VW; ++q) acc[v * VW + q] += p[col + q];
    }
  }
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int col = (gl + v * L) * VW;
    if (col < dim)
#pragma unroll
      for (int q = 0; q < VW; ++q) lds[g * dim + col + q] = acc[v * VW + q];
  }
}

// Chunk partials of a long segment are folded ahead of the finalize in runs
// of FOLD_SB CHUNK-aligned blocks ("super-blocks"): super-block s covers
// sorted positions [P0, P1) = [s*FOLD_SB*CHUNK, (s+1)*FOLD_SB*CHUNK).  When
// positions P0 - CHUNK .. P1 - 1 all hold one key, the start of every block
// in it is a cut of that key's segment, whose partial sits in the block's
// even slot; one workgroup adds those FOLD_SB partials in fixed order into
// fold[s].  A hot key's segment then needs a few fold rows plus the partials
// at its two ragged ends instead of one partial per chunk.
constexpr int FOLD_SB = 64;

template <int L, int NV, int VW>
__global__ __launch_bounds__(BLOCK) void k_seg_fold(SegView sv, int64_t nsb, uint32_t sentinel, int dim,
                                                    const double* __restrict__ partial,
                                                    double* __restrict__ fold) {
  constexpr int GPB = BLOCK / L;
  extern __shared__ double lds[];   // [GPB][dim]
  for (int64_t s = blockIdx.x; s < nsb; s += gridDim.x) {
    const int64_t p0 = s * FOLD_SB * CHUNK;
    if (p0 < CHUNK) continue;
    const uint32_t key = sv.keys[p0];
    // uniform over the block
    if (key >= sentinel || sv.keys[p0 - CHUNK] != key || sv.keys[p0 + FOLD_SB * CHUNK - 1] != key) continue;
    const int64_t b0 = s * FOLD_SB;
    group_sum_rows<L, NV, VW>([&](int64_t k) { return partial + 2 * (b0 + k) * dim; }, FOLD_SB, dim, lds);
    __syncthreads();
    for (int col = threadIdx.x; col < dim; col += BLOCK) {
      double t = 0.0;
      for (int gg = 0; gg < GPB; ++gg) t += lds[gg * dim + col];
      fold[s * dim + col] = t;
    }
    __syncthreads();
  }
}

// Segments cut into several chunks: one workgroup per such segment (listed by
// k_segreduce).  The segment's rows are, in position order: the partial of
// its first chunk, the partials of its cuts before its first foldable
// super-block, the fold rows of its foldable super-blocks, then the partials
// of the cuts after them.  They are added by group_sum_rows, the group
// results in group order, rounded once and applied with AdaGrad (row-wise
// when RW, with the accumulator at G[key * gld]).  The order is fixed, so
// the result is deterministic.
template <int L, int NV, int VW, bool RW, class VT>
__global__ __launch_bounds__(BLOCK) void k_seg_finalize(SegView sv, VT* __restrict__ W, float* __restrict__ G,
                                                        int64_t ld, int64_t gld, int dim, float lr, float eps,
                                                        const double* __restrict__ partial,
                                                        const double* __restrict__ fold,
                                                        const int32_t* __restrict__ split_list, LossTotal lt) {
  constexpr int GPB = BLOCK / L;
  extern __shared__ double lds[];   // [GPB][dim]
  __shared__ double sm[WAVES_PER_BLOCK];
  __shared__ float den_sh;
  // the step's loss, from the partials of its loss kernel (already complete:
  // that kernel ran earlier on this stream)
  if (lt.out && blockIdx.x == 0) sum_loss_parts(lt, sm);
  const int64_t nsplit = sv.hdr->num_split;
  for (int64_t e = blockIdx.x; e < nsplit; e += gridDim.x) {
    const int32_t u = split_list[e];
    const int64_t s0 = sv.seg_off[u];
    const int64_t s1 = sv.seg_off[u + 1];
    const uint32_t key = sv.keys[s0];
    const int64_t b0 = s0 / CHUNK;
    const int64_t f = (s0 + 2 * CHUNK - 1) / CHUNK;     // block of the first cut
    const int64_t bl = (s1 - 1) / CHUNK;                // block of the last cut
    const int64_t sa = (f + FOLD_SB - 1) / FOLD_SB;     // foldable super-blocks: [sa, sb)
    const int64_t sb = s1 / (FOLD_SB * CHUNK);
    const int64_t nf = sb > sa ? sb - sa : 0;
    const int64_t n1 = nf ? sa * FOLD_SB - f : bl - f + 1;   // cut partials before the folds
    const int64_t n3 = nf ? bl - sb * FOLD_SB + 1 : 0;       // cut partials after them
    auto row = [=](int64_t i) -> const double* {
      if (i == 0) return partial + (2 * b0 + ((s0 % CHUNK) != 0)) * dim;
      if (i <= n1) return partial + 2 * (f + (i - 1)) * dim;
      if (i <= n1 + nf) return fold + (sa + (i - 1 - n1)) * dim;
      return partial + 2 * (sb * FOLD_SB + (i - 1 - n1 - nf)) * dim;
    };
    group_sum_rows<L, NV, VW>(row, 1 + n1 + nf + n3, dim, lds);
    __syncthreads();
    VT* wrow = W + (int64_t)key * ld;
    float* grow = G + (int64_t)key * gld;
    if constexpr (RW) {
      // each thread keeps the fp32 sums of its own columns in lds[col]
      double sq = 0.0;
      for (int col = threadIdx.x; col < dim; col += BLOCK) {
        double t = 0.0;
        for (int gg = 0; gg < GPB; ++gg) t += lds[gg * dim + col];
        const float g = (float)t;
        lds[col] = g;
        sq += (double)g * (double)g;
      }
      sq = block_sum_double(sq, sm);
      if (threadIdx.x == 0) {
        float a = *grow;
        den_sh = rowwise_den(a, sq, dim, eps);
        *grow = a;
      }
      __syncthreads();
      const float den = den_sh;
      for (int col = threadIdx.x; col < dim; col += BLOCK) {
        float w = val_load(wrow + col);
        rowwise_elem(w, (float)lds[col], den, lr);
        val_store(wrow + col, w);
      }
    } else {
      for (int col = threadIdx.x; col < dim; col += BLOCK) {
        double t = 0.0;
        for (int gg = 0; gg < GPB; ++gg) t += lds[gg * dim + col];
        float w = val_load(wrow + col), a = grow[col];
        adagrad_elem(w, a, (float)t, lr, eps);
        val_store(wrow + col, w);
        grow[col] = a;
      }
    }
    __syncthreads();
  }
}

}  // namespace adapm
