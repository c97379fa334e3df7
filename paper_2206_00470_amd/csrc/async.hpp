// Write access without merging: the asynchronous update semantics of the
// paper's experiments (Section 5.1, asynchronous SGD), where every update
// reaches the store on its own.  Each occurrence's gradient row is applied
// as its own AdaGrad step, element by element with device-scope atomic
// adds: the accumulator add returns the value it replaced, so the
// occurrence's step uses the accumulator just after its own square was
// added, as one of the occurrences in a sequence would.  Occurrences of one
// key land in whatever order their atomics reach memory; no sort, no
// segments, no workspace.
#pragma once

#include "common.hpp"
#include "tasks.hpp"

namespace adapm {

struct KeysList {
  const int64_t* keys;
  __device__ int64_t operator()(int64_t i) const { return keys[i]; }
};

// One row group per occurrence i (grid-stride): key keys(i), gradient row
// grads[i * dim ..].  An occurrence with a key outside [0, num_keys) is
// skipped and raises the sticky error flag.  RW: row-wise AdaGrad, the
// key's single accumulator at G[key * gld] gets the mean square of the row.
template <int L, int NV, int VW, bool RW, class Keys>
__global__ __launch_bounds__(BLOCK) void k_push_async(Keys keys, const float* __restrict__ grads, int64_t n,
                                                      float* __restrict__ W, float* __restrict__ G, int64_t ld,
                                                      int64_t gld, int dim, int64_t num_keys, float lr, float eps,
                                                      int32_t* __restrict__ err) {
  constexpr int GPB = BLOCK / L;
  constexpr int NE = NV * VW;
  const int gl = threadIdx.x % L;
  int bad = 0;
  for (int64_t i = (int64_t)blockIdx.x * GPB + threadIdx.x / L; i < n; i += (int64_t)gridDim.x * GPB) {
    const int64_t key = keys(i);   // the same for every lane of the group
    if (key < 0 || key >= num_keys) {
      bad = 1;
      continue;
    }
    float g[NE];
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int c = (gl + v * L) * VW;
      if (c < dim) load_frag<VW>(grads + i * dim + c, g + v * VW);
    }
    float* wrow = W + key * ld;
    float* grow = G + key * gld;
    if constexpr (RW) {
      double sq = 0.0;
#pragma unroll
      for (int v = 0; v < NV; ++v)
        if ((gl + v * L) * VW < dim)
#pragma unroll
          for (int q = 0; q < VW; ++q) sq += (double)g[v * VW + q] * (double)g[v * VW + q];
      sq = group_sum<L>(sq);
      const float t = (float)(sq / (double)dim);
      float a = 0.0f;
      if (gl == 0) a = unsafeAtomicAdd(grow, t) + t;
      a = __shfl(a, 0, L);
      const float den = __builtin_sqrtf(a) + eps;
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int c = (gl + v * L) * VW;
        if (c < dim)
#pragma unroll
          for (int q = 0; q < VW; ++q) {
            const float step = lr * (g[v * VW + q] / den);
            unsafeAtomicAdd(wrow + c + q, -step);
          }
      }
    } else {
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int c = (gl + v * L) * VW;
        if (c < dim)
#pragma unroll
          for (int q = 0; q < VW; ++q) {
            const float gq = g[v * VW + q];
            const float t = gq * gq;
            const float a = unsafeAtomicAdd(grow + c + q, t) + t;   // the value this add left
            const float den = __builtin_sqrtf(a) + eps;
            const float step = lr * (gq / den);
            unsafeAtomicAdd(wrow + c + q, -step);
          }
      }
    }
  }
  if (__syncthreads_or(bad) && threadIdx.x == 0) atomicOr(err, 1);
}

// The MF step's gradient rows from the pre-step table, one row group per
// entry b (u = W[row], m = W[col_off + col], y): e = y - <u,m> in fp64,
// rows 2b = lam*u - e*m and 2b+1 = lam*m - e*u (fp32) in entry order, and
// loss e^2/2 + lam/2 (|u|^2 + |m|^2) summed per workgroup into
// loss_part[blockIdx.x].  Invalid entries write nothing (the apply skips
// their keys).
template <int L, int NV, int VW>
__global__ __launch_bounds__(BLOCK) void k_mf_grad_rows(const float* __restrict__ W, int64_t ld, int dim,
                                                        const int32_t* __restrict__ row,
                                                        const int32_t* __restrict__ col,
                                                        const float* __restrict__ val, int64_t B, int64_t col_off,
                                                        int64_t num_keys, double lam, float* __restrict__ grads,
                                                        double* __restrict__ loss_part) {
  constexpr int GPB = BLOCK / L;
  constexpr int NE = NV * VW;
  const int gl = threadIdx.x % L;
  double lsum = 0.0;
  for (int64_t b = (int64_t)blockIdx.x * GPB + threadIdx.x / L; b < B; b += (int64_t)gridDim.x * GPB) {
    const int32_t r = row[b], c = col[b];
    if (!mf_entry_ok(r, c, col_off, num_keys)) continue;
    const float* u = W + (int64_t)r * ld;
    const float* m = W + (col_off + (int64_t)c) * ld;
    float uv[NE], mv[NE];
    double dot = 0.0, nu = 0.0, nm = 0.0;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int e = (gl + v * L) * VW;
      if (e < dim) {
        load_frag<VW>(u + e, uv + v * VW);
        load_frag<VW>(m + e, mv + v * VW);
      }
    }
#pragma unroll
    for (int v = 0; v < NV; ++v)
      if ((gl + v * L) * VW < dim)
#pragma unroll
        for (int q = 0; q < VW; ++q) {
          // products of two floats are exact in fp64
          const double uq = (double)uv[v * VW + q], mq = (double)mv[v * VW + q];
          dot = __builtin_fma(uq, mq, dot);
          nu = __builtin_fma(uq, uq, nu);
          nm = __builtin_fma(mq, mq, nm);
        }
    dot = group_sum<L>(dot);
    nu = group_sum<L>(nu);
    nm = group_sum<L>(nm);
    const double err = (double)val[b] - dot;
    if (gl == 0) lsum += 0.5 * err * err + 0.5 * lam * (nu + nm);
    float* gu = grads + (2 * b) * dim;
    float* gm = gu + dim;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int e = (gl + v * L) * VW;
      if (e < dim) {
        float a[VW], z[VW];
#pragma unroll
        for (int q = 0; q < VW; ++q) {
          const double uq = (double)uv[v * VW + q], mq = (double)mv[v * VW + q];
          a[q] = (float)(lam * uq - err * mq);
          z[q] = (float)(lam * mq - err * uq);
        }
        store_frag<VW>(gu + e, a);
        store_frag<VW>(gm + e, z);
      }
    }
  }
  __shared__ double sm[WAVES_PER_BLOCK];
  lsum = block_sum_double(lsum, sm);
  if (threadIdx.x == 0) loss_part[blockIdx.x] = lsum;
}

}  // namespace adapm
