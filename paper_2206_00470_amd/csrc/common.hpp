// Shared device helpers and constants of the gfx950 parameter-store kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>

#include <cstddef>
#include <cstdint>

namespace adapm {

constexpr int WAVE = 64;                 // CDNA wavefront width
constexpr int BLOCK = 256;               // threads per workgroup for every kernel here
constexpr int WAVES_PER_BLOCK = BLOCK / WAVE;
constexpr int MAX_PASSES = 4;            // 32-bit keys, at most 9 bits per pass
constexpr int MAX_BINS = 512;            // digits of up to 9 bits
constexpr int DIG_PER_THREAD = MAX_BINS / 256;   // digits per thread in the per-digit loops of a 256-thread block
constexpr int GH_COPIES = 32;             // copies of the whole-array histograms (spreads the atomics)
constexpr int CHUNK = 32;               // cut length of long segments (chunks hold < 2*CHUNK occurrences)
constexpr int NUM_XCD = 8;               // MI355X: 8 accelerator dies, each with its own L2
constexpr int64_t ABSENT = INT64_MIN;    // a key source's "no occurrence here" marker

// Device-side counters written by the segment kernels and read by the
// reduce kernels, so that no host round trip is needed to size grids.
struct SegHeader {
  uint32_t num_unique;   // U: distinct valid keys
  uint32_t num_chunks;   // reduce work items
  uint32_t num_valid;    // occurrences with a valid key (a prefix of the sorted order)
  uint32_t num_split;    // segments longer than one chunk, listed for the finalize pass
  uint32_t num_lo;       // segments whose key is below the split key given to k_seg_write
  uint32_t chunk_lo;     // chunks whose key is below that split key (they come first)
  uint32_t pad[2];
};

// ------------------------------------------------------------------ lanes
__device__ __forceinline__ int lane_id() { return __lane_id(); }

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int l = lane_id();
  return l == 0 ? 0ull : (~0ull >> (64 - l));
}

// Butterfly sum over aligned groups of L lanes (L a power of two <= 64).
// Every lane of the group ends with the same value: a+b and b+a round alike.
template <int L>
__device__ __forceinline__ double group_sum(double v) {
#pragma unroll
  for (int o = L / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, L);
  return v;
}

// Sums J values over a group of L lanes at once (J <= L, both powers of two):
// log2(J) halving stages in which each lane keeps half of its values and adds
// the partner's copy of that half, then a butterfly over the remaining L/J
// lanes.  Lane gl returns the group total of value gl / (L/J).  The addition
// tree is fixed, so the result is deterministic.
template <int L, int J>
__device__ __forceinline__ double group_multi_sum(double (&v)[J], int gl) {
  static_assert(J >= 1 && J <= L, "J must not exceed the group width");
#pragma unroll
  for (int k = 0; (J >> k) > 1; ++k) {
    const int half = (J >> k) / 2;
    const int mask = L >> (k + 1);
    const bool upper = (gl & mask) != 0;
#pragma unroll
    for (int i = 0; i < J / 2; ++i) {
      if (i < half) {
        const double keep = upper ? v[i + half] : v[i];
        const double send = upper ? v[i] : v[i + half];
        v[i] = keep + __shfl_xor(send, mask, L);
      }
    }
  }
  double s = v[0];
#pragma unroll
  for (int o = L / J / 2; o > 0; o >>= 1) s += __shfl_xor(s, o, L);
  return s;
}

// ------------------------------------------------------------------ block scan
// Exclusive scan of one uint32 per thread over a 256-thread block; returns the
// thread's exclusive prefix and writes the block total to *total.
// `smem` needs WAVES_PER_BLOCK + 1 words.
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t x, uint32_t* smem, uint32_t* total) {
  const int lane = lane_id();
  const int w = threadIdx.x / WAVE;
  uint32_t inc = x;
#pragma unroll
  for (int o = 1; o < WAVE; o <<= 1) {
    uint32_t y = __shfl_up(inc, o, WAVE);
    if (lane >= o) inc += y;
  }
  if (lane == WAVE - 1) smem[w] = inc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t run = 0;
    for (int i = 0; i < WAVES_PER_BLOCK; ++i) {
      uint32_t t = smem[i];
      smem[i] = run;
      run += t;
    }
    smem[WAVES_PER_BLOCK] = run;
  }
  __syncthreads();
  uint32_t res = smem[w] + inc - x;
  *total = smem[WAVES_PER_BLOCK];
  __syncthreads();
  return res;
}

// Sum of one double per thread over the block (fixed order: waves, then
// wave totals in wave order), result valid in thread 0.
__device__ __forceinline__ double block_sum_double(double v, double* smem) {
  v = group_sum<WAVE>(v);
  const int w = threadIdx.x / WAVE;
  if (lane_id() == 0) smem[w] = v;
  __syncthreads();
  double r = 0.0;
  if (threadIdx.x == 0) {
    for (int i = 0; i < WAVES_PER_BLOCK; ++i) r += smem[i];
  }
  __syncthreads();
  return r;
}

// ------------------------------------------------------------------ loss totals
// The loss kernels leave one fp64 value per workgroup in part[]; a kernel
// that runs after them on the same stream (the merge's finalize pass) adds
// part[0 .. n) in index order with one workgroup: eight independent loads
// per thread and round, then the fixed block tree, so the total does not
// depend on the launch or on timing.
struct LossTotal {
  const double* part;
  int64_t n;
  double* out;   // NULL: no total wanted
};

__device__ __forceinline__ void sum_loss_parts(const LossTotal& lt, double* smem) {
  double s = 0.0;
  int64_t i = threadIdx.x;
  for (; i + 7 * BLOCK < lt.n; i += 8 * BLOCK) {
    double x[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) x[k] = lt.part[i + k * BLOCK];
#pragma unroll
    for (int k = 0; k < 8; ++k) s += x[k];
  }
  for (; i < lt.n; i += BLOCK) s += lt.part[i];
  s = block_sum_double(s, smem);
  if (threadIdx.x == 0) *lt.out = s;
}

// ------------------------------------------------------------------ AdaGrad
// One element, fp32, in the fixed order G' = G + g*g; W' = W - lr*(g/(sqrt(G')+eps)).
// Built with -ffp-contract=off and correctly rounded sqrt/div, so each
// operation rounds once exactly as written.
__device__ __forceinline__ void adagrad_elem(float& w, float& acc, float g, float lr, float eps) {
  float t = g * g;
  float a = acc + t;
  float s = __builtin_sqrtf(a);
  float den = s + eps;
  float q = g / den;
  float step = lr * q;
  acc = a;
  w = w - step;
}

// Row-wise AdaGrad: one accumulator per row, advanced by the row mean of the
// squared merged gradient (fp32 values, squared and summed in fp64, the mean
// rounded once); every element of the row then steps with the row's shared
// denominator, in the element-wise order q = g/den, step = lr*q, w - step.
__device__ __forceinline__ float rowwise_den(float& acc, double sumsq, int dim, float eps) {
  const float t = (float)(sumsq / (double)dim);
  const float a = acc + t;
  acc = a;
  const float s = __builtin_sqrtf(a);
  return s + eps;
}

__device__ __forceinline__ void rowwise_elem(float& w, float g, float den, float lr) {
  float q = g / den;
  float step = lr * q;
  w = w - step;
}

// ------------------------------------------------------------------ row fragments
// A group of L lanes covers one row of `dim` floats: lane `gl` owns the
// VW-wide vectors at columns (gl + v*L)*VW for v < NV.
template <int VW> struct vec_t;
template <> struct vec_t<1> { using type = float; };
template <> struct vec_t<2> { using type = float2; };
template <> struct vec_t<4> { using type = float4; };

template <int VW>
__device__ __forceinline__ void load_frag(const float* p, float* out) {
  if constexpr (VW == 4) {
    float4 x = *reinterpret_cast<const float4*>(p);
    out[0] = x.x; out[1] = x.y; out[2] = x.z; out[3] = x.w;
  } else if constexpr (VW == 2) {
    float2 x = *reinterpret_cast<const float2*>(p);
    out[0] = x.x; out[1] = x.y;
  } else {
    out[0] = *p;
  }
}

template <int VW>
__device__ __forceinline__ void store_frag(float* p, const float* in) {
  if constexpr (VW == 4) {
    *reinterpret_cast<float4*>(p) = make_float4(in[0], in[1], in[2], in[3]);
  } else if constexpr (VW == 2) {
    *reinterpret_cast<float2*>(p) = make_float2(in[0], in[1]);
  } else {
    *p = in[0];
  }
}

// ------------------------------------------------------------------ bf16 values
// A store may keep its values as bf16 words (the upper half of an fp32
// word): widening is exact, narrowing rounds to the nearest bf16 with ties
// to the even word (a NaN stays a quiet NaN).  Arithmetic is unchanged.
struct bf16_t {
  uint16_t bits;
};

__device__ __forceinline__ float bf16_widen(uint32_t bits16) { return __uint_as_float(bits16 << 16); }

__device__ __forceinline__ uint32_t bf16_narrow(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;   // a carry moves into the exponent, as it should
}

// VW values of type VT at p <-> VW floats (VT = float or bf16_t).
template <int VW, class VT>
__device__ __forceinline__ void load_vals(const VT* p, float* out) {
  if constexpr (std::is_same_v<VT, float>) {
    load_frag<VW>(p, out);
  } else if constexpr (VW == 4) {
    const uint2 x = *reinterpret_cast<const uint2*>(p);
    out[0] = bf16_widen(x.x & 0xffffu);
    out[1] = bf16_widen(x.x >> 16);
    out[2] = bf16_widen(x.y & 0xffffu);
    out[3] = bf16_widen(x.y >> 16);
  } else if constexpr (VW == 2) {
    const uint32_t x = *reinterpret_cast<const uint32_t*>(p);
    out[0] = bf16_widen(x & 0xffffu);
    out[1] = bf16_widen(x >> 16);
  } else {
    out[0] = bf16_widen(p->bits);
  }
}

template <int VW, class VT>
__device__ __forceinline__ void store_vals(VT* p, const float* in) {
  if constexpr (std::is_same_v<VT, float>) {
    store_frag<VW>(p, in);
  } else if constexpr (VW == 4) {
    uint2 x;
    x.x = bf16_narrow(in[0]) | (bf16_narrow(in[1]) << 16);
    x.y = bf16_narrow(in[2]) | (bf16_narrow(in[3]) << 16);
    *reinterpret_cast<uint2*>(p) = x;
  } else if constexpr (VW == 2) {
    *reinterpret_cast<uint32_t*>(p) = bf16_narrow(in[0]) | (bf16_narrow(in[1]) << 16);
  } else {
    p->bits = (uint16_t)bf16_narrow(in[0]);
  }
}

__device__ __forceinline__ float val_load(const float* p) { return *p; }
__device__ __forceinline__ float val_load(const bf16_t* p) { return bf16_widen(p->bits); }
__device__ __forceinline__ void val_store(float* p, float x) { *p = x; }
__device__ __forceinline__ void val_store(bf16_t* p, float x) { p->bits = (uint16_t)bf16_narrow(x); }

// Non-temporal fragment store for streams that are read back only once.
template <int VW>
__device__ __forceinline__ void store_frag_nt(float* p, const float* in) {
#pragma unroll
  for (int e = 0; e < VW; ++e) __builtin_nontemporal_store(in[e], p + e);
}

}  // namespace adapm
