// The deep part of the Wide & Deep click-through-rate model (Appendix C,
// "Click-through-rate prediction"): an MLP over the concatenated field
// embeddings, forward and backward in fp64 on the matrix cores.
//
// The products are the only dense contractions of the store's tasks; they
// run on v_mfma_f64_16x16x4f64, whose operands and results a wavefront holds
// as: lane l passes a = A[l % 16][l / 16] (16 x 4) and b = B[l / 16][l % 16]
// (4 x 16) and holds c[v] = C[l / 16 + 4 v][l % 16] of the 16 x 16 result.
#pragma once

#include "common.hpp"

namespace adapm {

typedef double f64x4 __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------------ GEMM
// C[M][N] = op(A)[M][K] op(B)[K][N] with an epilogue, all sums in fp64.
// op(A)[m][k] = TA ? A[k * lda + m] : A[m * lda + k]; op(B) likewise with
// TB.  B's elements are fp32 (the dense parameters) or fp64.
// Epilogues: store; add bias[n] (fp32) then ReLU; keep only where
// mask[m * ldm + n] > 0 (the ReLU derivative of the layer below).
enum { EPI_STORE = 0, EPI_BIAS_RELU = 1, EPI_MASK = 2 };

constexpr int GEMM_BM = 64, GEMM_BN = 64, GEMM_BK = 16;
constexpr int GEMM_PAD = 2;   // doubles of padding per LDS row

template <bool TA, bool TB, typename BT, int EPI>
__global__ __launch_bounds__(BLOCK) void k_gemm_f64(int64_t M, int64_t N, int64_t K, const double* __restrict__ A,
                                                    int64_t lda, const BT* __restrict__ B, int64_t ldb,
                                                    double* __restrict__ C, int64_t ldc,
                                                    const float* __restrict__ bias, const double* __restrict__ mask,
                                                    int64_t ldm) {
  __shared__ double As[GEMM_BK][GEMM_BM + GEMM_PAD];   // [k][m]
  __shared__ double Bs[GEMM_BK][GEMM_BN + GEMM_PAD];   // [k][n]
  const int t = threadIdx.x;
  const int lane = t % WAVE;
  const int wave = t / WAVE;
  const int64_t m0 = (int64_t)blockIdx.y * GEMM_BM;
  const int64_t n0 = (int64_t)blockIdx.x * GEMM_BN;
  const int wm = (wave / 2) * 32;   // the wave's 32 x 32 quarter of the tile
  const int wn = (wave % 2) * 32;
  f64x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f64x4{0.0, 0.0, 0.0, 0.0};

  for (int64_t k0 = 0; k0 < K; k0 += GEMM_BK) {
    // A tile: 64 x 16 elements, 4 per thread, read along A's contiguous axis
    if constexpr (!TA) {
      const int r = t / 4, kq = (t % 4) * 4;
      const int64_t m = m0 + r;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t k = k0 + kq + e;
        As[kq + e][r] = (m < M && k < K) ? A[m * lda + k] : 0.0;
      }
    } else {
      const int kk = t / 16, mq = (t % 16) * 4;
      const int64_t k = k0 + kk;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t m = m0 + mq + e;
        As[kk][mq + e] = (m < M && k < K) ? A[k * lda + m] : 0.0;
      }
    }
    // B tile: 16 x 64
    if constexpr (!TB) {
      const int kk = t / 16, nq = (t % 16) * 4;
      const int64_t k = k0 + kk;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t n = n0 + nq + e;
        Bs[kk][nq + e] = (n < N && k < K) ? (double)B[k * ldb + n] : 0.0;
      }
    } else {
      const int c = t / 4, kq = (t % 4) * 4;
      const int64_t n = n0 + c;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t k = k0 + kq + e;
        Bs[kq + e][c] = (n < N && k < K) ? (double)B[n * ldb + k] : 0.0;
      }
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < GEMM_BK; ks += 4) {
      const int kr = ks + lane / 16;
      double a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) a[i] = As[kr][wm + i * 16 + lane % 16];
#pragma unroll
      for (int j = 0; j < 2; ++j) b[j] = Bs[kr][wn + j * 16 + lane % 16];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t m = m0 + wm + i * 16 + lane / 16 + 4 * v;
        const int64_t n = n0 + wn + j * 16 + lane % 16;
        if (m < M && n < N) {
          double x = acc[i][j][v];
          if constexpr (EPI == EPI_BIAS_RELU) {
            x += (double)bias[n];
            x = x > 0.0 ? x : 0.0;
          } else if constexpr (EPI == EPI_MASK) {
            x = mask[m * ldm + n] > 0.0 ? x : 0.0;
          }
          C[m * ldc + n] = x;
        }
      }
}

// ------------------------------------------------------------------ inputs and head
// X[b][f * E + c] = W[key(b, f)][c] in fp64 (zero rows for skipped samples):
// one group of L lanes per (sample, field) row.
template <int L, int NV, int VW>
__global__ __launch_bounds__(BLOCK) void k_wd_gather(const float* __restrict__ W, int64_t ld,
                                                     const int64_t* __restrict__ keys, int64_t B, int F, int E,
                                                     const uint8_t* __restrict__ ok, double* __restrict__ X) {
  constexpr int GPB = BLOCK / L;
  const int gl = threadIdx.x % L;
  const int64_t n = B * F;
  for (int64_t i = (int64_t)blockIdx.x * GPB + threadIdx.x / L; i < n; i += (int64_t)gridDim.x * GPB) {
    const int64_t b = i / F;
    const bool valid = ok[b];
    const float* row = W + (valid ? keys[i] : 0) * ld;
    double* out = X + i * E;   // row b, field f: X + (b * F + f) * E
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int c = (gl + v * L) * VW;
      if (c < E) {
        float x[VW];
        if (valid) load_frag<VW>(row + c, x);
#pragma unroll
        for (int e = 0; e < VW; ++e)
          if (c + e < E) out[c + e] = valid ? (double)x[e] : 0.0;
      }
    }
  }
}

// One wavefront per sample: logit = h_L . w + c + sum of the F wide weights
// (field order), the logistic loss, dlogit = sigmoid(logit) - label (0 for
// skipped samples) and dH_L = dlogit w, masked by h_L > 0 when h_L is a
// ReLU layer (relu = 0: no hidden layer, h_L is the input x itself).
__global__ __launch_bounds__(BLOCK) void k_wd_head(const double* __restrict__ H, int64_t Hn,
                                                   const float* __restrict__ w, const float* __restrict__ c,
                                                   const float* __restrict__ W, int64_t ld, int E,
                                                   const int64_t* __restrict__ keys, int F,
                                                   const float* __restrict__ label, const uint8_t* __restrict__ ok,
                                                   int64_t B, int relu, double* __restrict__ dlogit,
                                                   double* __restrict__ dH, double* __restrict__ loss_part) {
  const int lane = threadIdx.x % WAVE;
  double lsum = 0.0;
  for (int64_t b = (int64_t)blockIdx.x * WAVES_PER_BLOCK + threadIdx.x / WAVE; b < B;
       b += (int64_t)gridDim.x * WAVES_PER_BLOCK) {
    const double* h = H + b * Hn;
    double s = 0.0;
    for (int64_t n = lane; n < Hn; n += WAVE) s += h[n] * (double)w[n];
    s = group_sum<WAVE>(s);
    double wide = 0.0;
    const bool valid = ok[b];
    if (valid)
      for (int f = 0; f < F; ++f) wide += (double)W[keys[b * F + f] * ld + E];
    const double logit = s + (double)c[0] + wide;
    const double y = (double)label[b];
    double g = 0.0;
    if (valid) {
      // softplus(z) - y z, and sigmoid(z) - y, in forms that do not overflow
      const double sp = logit > 0.0 ? logit + log1p(exp(-logit)) : log1p(exp(logit));
      if (lane == 0) lsum += sp - y * logit;
      g = (logit >= 0.0 ? 1.0 / (1.0 + exp(-logit)) : exp(logit) / (1.0 + exp(logit))) - y;
    }
    if (lane == 0) dlogit[b] = g;
    for (int64_t n = lane; n < Hn; n += WAVE) dH[b * Hn + n] = (!relu || h[n] > 0.0) ? g * (double)w[n] : 0.0;
  }
  __shared__ double sm[WAVES_PER_BLOCK];
  lsum = block_sum_double(lsum, sm);
  if (threadIdx.x == 0) loss_part[blockIdx.x] = lsum;
}

// Column sums out[n] = sum_b A[b][n] s[b] (s = 1 without a scale), in two
// deterministic stages: block (x, y) sums rows [y R, (y+1) R) of columns
// x*BLOCK .. into part[y][n]; then the parts are added in y order.
constexpr int64_t COLSUM_ROWS = 256;

__global__ __launch_bounds__(BLOCK) void k_colsum_part(const double* __restrict__ A, int64_t rows, int64_t cols,
                                                       const double* __restrict__ s, double* __restrict__ part) {
  const int64_t n = (int64_t)blockIdx.x * BLOCK + threadIdx.x;
  if (n >= cols) return;
  const int64_t r0 = (int64_t)blockIdx.y * COLSUM_ROWS;
  const int64_t r1 = r0 + COLSUM_ROWS < rows ? r0 + COLSUM_ROWS : rows;
  double t = 0.0;
  for (int64_t r = r0; r < r1; ++r) t += s ? A[r * cols + n] * s[r] : A[r * cols + n];
  part[(int64_t)blockIdx.y * cols + n] = t;
}

__global__ __launch_bounds__(BLOCK) void k_colsum_final(const double* __restrict__ part, int64_t nparts, int64_t cols,
                                                        double* __restrict__ out) {
  const int64_t n = (int64_t)blockIdx.x * BLOCK + threadIdx.x;
  if (n >= cols) return;
  double t = 0.0;
  for (int64_t y = 0; y < nparts; ++y) t += part[y * cols + n];
  out[n] = t;
}

// Per-occurrence gradient rows at the occurrence's sorted position:
// [dX[b][f E .. f E + E) | dlogit[b] | 0 ...] rounded to fp32 (zeros for
// skipped samples, whose occurrences sort last and are not merged).
__global__ __launch_bounds__(BLOCK) void k_wd_rows(const double* __restrict__ dX, const double* __restrict__ dlogit,
                                                   int64_t B, int F, int E, int dim, const uint32_t* __restrict__ rank,
                                                   float* __restrict__ grads) {
  const int64_t n = B * F;
  for (int64_t i = (int64_t)blockIdx.x * WAVES_PER_BLOCK + threadIdx.x / WAVE; i < n;
       i += (int64_t)gridDim.x * WAVES_PER_BLOCK) {
    const int lane = threadIdx.x % WAVE;
    const int64_t b = i / F;
    float* out = grads + (int64_t)rank[i] * dim;
    const double* src = dX + i * E;
    for (int c = lane; c < dim; c += WAVE)
      out[c] = c < E ? (float)src[c] : (c == E ? (float)dlogit[b] : 0.0f);
  }
}

// Per-element AdaGrad of the dense buffer from its fp64 gradient, rounded
// once to fp32.
__global__ __launch_bounds__(BLOCK) void k_dense_adagrad(float* __restrict__ w, float* __restrict__ acc,
                                                         const double* __restrict__ g, int64_t n, float lr,
                                                         float eps) {
  for (int64_t i = (int64_t)blockIdx.x * BLOCK + threadIdx.x; i < n; i += (int64_t)gridDim.x * BLOCK) {
    float wi = w[i], ai = acc[i];
    adagrad_elem(wi, ai, (float)g[i], lr, eps);
    w[i] = wi;
    acc[i] = ai;
  }
}

}  // namespace adapm
