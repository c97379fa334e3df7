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
// C[M][N] = op(A)[M][K] op(B)[K][N], all sums in fp64.
// op(A)[m][k] = TA ? A[k * lda + m] : A[m * lda + k]; op(B) likewise with
// TB.  B's elements are fp32 (the dense parameters) or fp64.  The bias and
// ReLU of a forward layer and the ReLU mask of a backward one are applied
// by k_bias_relu / k_relu_mask afterwards: an epilogue with arithmetic would
// copy the 128 accumulator registers into ordinary ones and halve the
// workgroups a compute unit holds.
//
// A workgroup computes a 128 x 128 tile of C, each of its four wavefronts a
// 64 x 64 quarter as 4 x 4 products of 16 x 16.  K advances 16 at a time
// through two LDS buffers, one barrier per step; the operands of the step
// after next are loaded into registers while the matrix cores work on the
// current buffer (two register sets, so each load has two steps to land),
// and the next step's registers are stored to the other buffer.  With gridDim.z = S > 1 the K range
// is split into S slices and slice z writes its partial product to
// C + z * M * N (plain store only); k_sum_slices adds them in slice order.
constexpr int GEMM_BM = 128, GEMM_BN = 128, GEMM_BK = 16;
constexpr int GEMM_PAD = 0;   // doubles of padding per LDS row (padding measured no faster)

template <bool TA, bool TB, typename BT>
__global__ __launch_bounds__(BLOCK, 2) void k_gemm_f64(int64_t M, int64_t N, int64_t K, const double* __restrict__ A,
                                                    int64_t lda, const BT* __restrict__ B, int64_t ldb,
                                                    double* __restrict__ C, int64_t ldc, int64_t kslice) {
  __shared__ double As[2][GEMM_BK][GEMM_BM + GEMM_PAD];   // [buffer][k][m]
  __shared__ double Bs[2][GEMM_BK][GEMM_BN + GEMM_PAD];   // [buffer][k][n]
  const int t = threadIdx.x;
  const int lane = t % WAVE;
  const int wave = t / WAVE;
  const int64_t m0 = (int64_t)blockIdx.y * GEMM_BM;
  const int64_t n0 = (int64_t)blockIdx.x * GEMM_BN;
  const int64_t kbeg = (int64_t)blockIdx.z * kslice;
  const int64_t kend = kbeg + kslice < K ? kbeg + kslice : K;
  if (gridDim.z > 1) C += (int64_t)blockIdx.z * M * N;
  const int wm = (wave / 2) * 64;   // the wave's 64 x 64 quarter of the tile
  const int wn = (wave % 2) * 64;

  // the thread's 8 elements of each operand tile: A (TA = false) rows t/2,
  // k (t%2)*8..+8; A (TA) k t/16, m (t%16)*8..+8; B likewise
  const int ar = TA ? t / 16 : t / 2;            // TA: k row; else m row
  const int aq = TA ? (t % 16) * 8 : (t % 2) * 8;
  const int br = TB ? t / 2 : t / 16;            // TB: n row; else k row
  const int bq = TB ? (t % 2) * 8 : (t % 16) * 8;
  double ra_[2][8], rb_[2][8];
  auto load = [&]<int R>(int64_t k0) {
    double* ra = ra_[R];
    double* rb = rb_[R];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if constexpr (!TA) {
        const int64_t m = m0 + ar, k = k0 + aq + e;
        ra[e] = (m < M && k < kend) ? A[m * lda + k] : 0.0;
      } else {
        const int64_t k = k0 + ar, m = m0 + aq + e;
        ra[e] = (m < M && k < kend) ? A[k * lda + m] : 0.0;
      }
      if constexpr (!TB) {
        const int64_t k = k0 + br, n = n0 + bq + e;
        rb[e] = (n < N && k < kend) ? (double)B[k * ldb + n] : 0.0;
      } else {
        const int64_t n = n0 + br, k = k0 + bq + e;
        rb[e] = (n < N && k < kend) ? (double)B[n * ldb + k] : 0.0;
      }
    }
  };
  auto stash = [&]<int R>(int buf) {
    const double* ra = ra_[R];
    const double* rb = rb_[R];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if constexpr (!TA) As[buf][aq + e][ar] = ra[e];
      else As[buf][ar][aq + e] = ra[e];
      if constexpr (!TB) Bs[buf][br][bq + e] = rb[e];
      else Bs[buf][bq + e][br] = rb[e];
    }
  };

  f64x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f64x4{0.0, 0.0, 0.0, 0.0};

  auto products = [&](int buf) {
#pragma unroll
    for (int ks = 0; ks < GEMM_BK; ks += 4) {
      const int kr = ks + lane / 16;
      double a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[buf][kr][wm + i * 16 + lane % 16];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[buf][kr][wn + j * 16 + lane % 16];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  };
  // step s: LDS buffer s % 2 holds its operands, register set (s + 1) % 2
  // those of step s + 1; set s % 2 is free (stored at the end of step s - 1)
  // and receives step s + 2.  The other buffer was last read in step s - 1,
  // which every wave finished before that step's barrier.
  const int64_t nsteps = kbeg < kend ? (kend - kbeg + GEMM_BK - 1) / GEMM_BK : 0;
  auto step = [&]<int P>(int64_t s) {
    if (s + 2 < nsteps) load.template operator()<P>(kbeg + (s + 2) * GEMM_BK);
    products(P);
    if (s + 1 < nsteps) stash.template operator()<1 - P>(1 - P);
    __syncthreads();
  };
  if (nsteps > 0) {
    load.template operator()<0>(kbeg);
    stash.template operator()<0>(0);
    if (nsteps > 1) load.template operator()<1>(kbeg + GEMM_BK);
  }
  __syncthreads();
  for (int64_t s = 0; s < nsteps; s += 2) {
    step.template operator()<0>(s);
    if (s + 1 < nsteps) step.template operator()<1>(s + 1);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t m = m0 + wm + i * 16 + lane / 16 + 4 * v;
        const int64_t n = n0 + wn + j * 16 + lane % 16;
        if (m < M && n < N) C[m * ldc + n] = acc[i][j][v];
      }
}

// H[m][n] = max(H[m][n] + bias[n], 0): a forward layer's bias and ReLU.
__global__ __launch_bounds__(BLOCK) void k_bias_relu(double* __restrict__ H, int64_t M, int64_t N,
                                                     const float* __restrict__ bias) {
  const int64_t n_all = M * N;
  for (int64_t i = (int64_t)blockIdx.x * BLOCK + threadIdx.x; i < n_all; i += (int64_t)gridDim.x * BLOCK) {
    const double x = H[i] + (double)bias[i % N];
    H[i] = x > 0.0 ? x : 0.0;
  }
}

// D[m][n] = 0 where H[m][n] <= 0: the ReLU derivative of the layer below.
__global__ __launch_bounds__(BLOCK) void k_relu_mask(double* __restrict__ D, const double* __restrict__ H,
                                                     int64_t count) {
  for (int64_t i = (int64_t)blockIdx.x * BLOCK + threadIdx.x; i < count; i += (int64_t)gridDim.x * BLOCK)
    if (!(H[i] > 0.0)) D[i] = 0.0;
}

// out[i] = sum over z of part[z * count + i], z = 0 .. S-1 in order.
__global__ __launch_bounds__(BLOCK) void k_sum_slices(const double* __restrict__ part, int64_t S, int64_t count,
                                                      double* __restrict__ out) {
  for (int64_t i = (int64_t)blockIdx.x * BLOCK + threadIdx.x; i < count; i += (int64_t)gridDim.x * BLOCK) {
    double t = 0.0;
    for (int64_t z = 0; z < S; ++z) t += part[z * count + i];
    out[i] = t;
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
