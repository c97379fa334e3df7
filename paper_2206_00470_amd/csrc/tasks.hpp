// Per-task gradient kernels: each reads the pre-step rows it needs, computes
// the per-occurrence gradients in fp64 and writes them (rounded once to fp32)
// where the merge kernel will read them, plus a per-workgroup loss partial.
#pragma once

#include "common.hpp"

namespace adapm {

// Sum loss partials in index order (deterministic), then write the total.
__global__ __launch_bounds__(BLOCK) void k_sum_loss(const double* __restrict__ part, int64_t n,
                                                    double* __restrict__ out) {
  __shared__ double sm[WAVES_PER_BLOCK];
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += BLOCK) s += part[i];
  s = block_sum_double(s, sm);
  if (threadIdx.x == 0) *out = s;
}

// ------------------------------------------------------------------ MF
// Key occurrences of entry b: 2b = row key, 2b+1 = column key.  An entry with
// a key outside the table yields the (invalid) key -1 for both occurrences.
struct KeysMF {
  const int32_t* row;
  const int32_t* col;
  int64_t col_off;
  int64_t num_keys;
  __device__ int64_t operator()(int64_t i) const {
    const int64_t b = i >> 1;
    const int64_t ku = row[b];
    const int64_t km = col_off + (int64_t)col[b];
    const bool ok = ku >= 0 && ku < num_keys && col[b] >= 0 && km < num_keys;
    if (!ok) return -1;
    return (i & 1) ? km : ku;
  }
};

// One row group per entry (u = W[row], m = W[col_off + col], e = v - <u,m>):
//   grad_u = lam u - e m ,  grad_m = lam m - e u     (fp64, rounded to fp32)
//   loss  += e^2/2 + lam/2 (|u|^2 + |m|^2)
// The two gradient rows go to the sorted positions rank[2b], rank[2b+1], or
// to occurrence positions 2b, 2b+1 when rank is null.
template <int L, int NV, int VW>
__global__ __launch_bounds__(BLOCK) void k_mf_grad(const float* __restrict__ W, int64_t num_keys, int dim,
                                                   const int32_t* __restrict__ row, const int32_t* __restrict__ col,
                                                   const float* __restrict__ val, int64_t B, int64_t col_off,
                                                   float lam, const uint32_t* __restrict__ rank,
                                                   float* __restrict__ grads, double* __restrict__ loss_part) {
  constexpr int GPB = BLOCK / L;
  constexpr int NE = NV * VW;
  __shared__ double sm[WAVES_PER_BLOCK];
  const int gl = threadIdx.x % L;
  const double lamd = (double)lam;
  double lsum = 0.0;
  for (int64_t b = (int64_t)blockIdx.x * GPB + threadIdx.x / L; b < B; b += (int64_t)gridDim.x * GPB) {
    const int64_t ku = row[b];
    const int64_t km = col_off + (int64_t)col[b];
    if (!(ku >= 0 && ku < num_keys && col[b] >= 0 && km < num_keys)) continue;
    const float* up = W + ku * dim;
    const float* mp = W + km * dim;
    float u[NE], m[NE];
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int c = (gl + v * L) * VW;
      if (c < dim) {
        load_frag<VW>(up + c, u + v * VW);
        load_frag<VW>(mp + c, m + v * VW);
      } else {
#pragma unroll
        for (int e = 0; e < VW; ++e) u[v * VW + e] = m[v * VW + e] = 0.0f;
      }
    }
    double dot = 0.0, nu = 0.0, nm = 0.0;
#pragma unroll
    for (int e = 0; e < NE; ++e) {
      dot += (double)u[e] * (double)m[e];
      nu += (double)u[e] * (double)u[e];
      nm += (double)m[e] * (double)m[e];
    }
    dot = group_sum<L>(dot);
    nu = group_sum<L>(nu);
    nm = group_sum<L>(nm);
    const double err = (double)val[b] - dot;
    if (gl == 0) lsum += 0.5 * err * err + 0.5 * lamd * (nu + nm);
    float gu[NE], gm[NE];
#pragma unroll
    for (int e = 0; e < NE; ++e) {
      gu[e] = (float)(lamd * (double)u[e] - err * (double)m[e]);
      gm[e] = (float)(lamd * (double)m[e] - err * (double)u[e]);
    }
    float* du = grads + (rank ? (int64_t)rank[2 * b] : 2 * b) * dim;
    float* dm = grads + (rank ? (int64_t)rank[2 * b + 1] : 2 * b + 1) * dim;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int c = (gl + v * L) * VW;
      if (c < dim) {
        store_frag<VW>(du + c, gu + v * VW);
        store_frag<VW>(dm + c, gm + v * VW);
      }
    }
  }
  lsum = block_sum_double(lsum, sm);
  if (threadIdx.x == 0) loss_part[blockIdx.x] = lsum;
}

}  // namespace adapm
