// Intent-driven staging of parameter rows between a home table in pinned host
// memory and a table of slots in HBM (intent signalling, Section 3; adaptive
// action timing, Section 4.2 and Algorithm 1), for one worker: the GPU.
//
// Host side (planner.hpp): the planner keeps the worker's clock, the intents signalled and
// not yet acted upon, the key -> slot assignment and a free list of slots per
// key range, and decides in each round which keys to stage in and which to
// write back.  Device side: row moves between the two tables, updates of the
// device copy of the key -> slot map, and the translation of a batch's ids
// into slot ids so that the step kernels run unchanged on the slot table.
#pragma once

#include <cstdint>

#include "common.hpp"
#include "planner.hpp"

namespace adapm {

// ------------------------------------------------------------------ kernels
__global__ __launch_bounds__(BLOCK) void k_map_fill(int32_t* __restrict__ map, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * BLOCK + threadIdx.x; i < n; i += (int64_t)gridDim.x * BLOCK) map[i] = -1;
}

// map[keys[i]] = slots[i] (or -1 without slots).
__global__ __launch_bounds__(BLOCK) void k_map_set(int32_t* __restrict__ map, const int64_t* __restrict__ keys,
                                                   const int64_t* __restrict__ slots, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * BLOCK + threadIdx.x; i < n; i += (int64_t)gridDim.x * BLOCK)
    map[keys[i]] = slots ? (int32_t)slots[i] : -1;
}

// Row i of the move: the value and accumulator rows at index from[i] of the
// source tables are copied to index to[i] of the destination tables.  One
// group of L lanes per row; a source or destination may be host memory
// mapped into the device's address space.
template <int L, int NV, int VW>
__global__ __launch_bounds__(BLOCK) void k_move_rows(const float* __restrict__ sW, const float* __restrict__ sG,
                                                     int64_t sld, const int64_t* __restrict__ from,
                                                     float* __restrict__ dW, float* __restrict__ dG, int64_t dld,
                                                     const int64_t* __restrict__ to, int64_t n, int dim) {
  constexpr int GPB = BLOCK / L;
  const int gl = threadIdx.x % L;
  for (int64_t i = (int64_t)blockIdx.x * GPB + threadIdx.x / L; i < n; i += (int64_t)gridDim.x * GPB) {
    const int64_t a = from[i] * sld;
    const int64_t b = to[i] * dld;
    float w[NV * VW], g[NV * VW];
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int c = (gl + v * L) * VW;
      if (c < dim) {
        load_frag<VW>(sW + a + c, w + v * VW);
        load_frag<VW>(sG + a + c, g + v * VW);
      }
    }
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int c = (gl + v * L) * VW;
      if (c < dim) {
        store_frag<VW>(dW + b + c, w + v * VW);
        store_frag<VW>(dG + b + c, g + v * VW);
      }
    }
  }
}

// A batch's 32-bit ids in slot space: id (a key of key_off + id) becomes
// map[key_off + id] - slot_off.  Negative ids pass through unchanged (they
// keep the meaning the step gives them); an id beyond the key range becomes
// INT32_MAX (out of range for the step, which skips and flags it); a key
// with no slot also becomes INT32_MAX and sets status[1].
__global__ __launch_bounds__(BLOCK) void k_translate_ids(const int32_t* __restrict__ in, int64_t n,
                                                         const int32_t* __restrict__ map, int64_t key_off,
                                                         int64_t id_limit, int64_t slot_off,
                                                         int32_t* __restrict__ out, int32_t* __restrict__ status) {
  int miss = 0;
  for (int64_t i = (int64_t)blockIdx.x * BLOCK + threadIdx.x; i < n; i += (int64_t)gridDim.x * BLOCK) {
    const int32_t v = in[i];
    int32_t r = v;
    if (v >= 0) {
      r = INT32_MAX;
      if (v < id_limit) {
        const int32_t m = map[key_off + v];
        if (m >= 0) r = (int32_t)(m - slot_off);
        else miss = 1;
      }
    }
    out[i] = r;
  }
  if (__syncthreads_or(miss) && threadIdx.x == 0) atomicOr(status + 1, 1);
}

// 64-bit keys in slot space: a key in [0, num_keys) becomes its slot; a key
// outside it, or one with no slot (which also sets status[1]), becomes -1.
__global__ __launch_bounds__(BLOCK) void k_translate_keys(const int64_t* __restrict__ in, int64_t n,
                                                          const int32_t* __restrict__ map, int64_t num_keys,
                                                          int64_t* __restrict__ out, int32_t* __restrict__ status) {
  int miss = 0;
  for (int64_t i = (int64_t)blockIdx.x * BLOCK + threadIdx.x; i < n; i += (int64_t)gridDim.x * BLOCK) {
    const int64_t v = in[i];
    int64_t r = -1;
    if (v >= 0 && v < num_keys) {
      const int32_t m = map[v];
      if (m >= 0) r = m;
      else miss = 1;
    }
    out[i] = r;
  }
  if (__syncthreads_or(miss) && threadIdx.x == 0) atomicOr(status + 1, 1);
}

}  // namespace adapm
