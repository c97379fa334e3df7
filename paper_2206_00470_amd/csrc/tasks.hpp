// Per-task gradient kernels: each reads the pre-step rows it needs, computes
// the per-occurrence gradients in fp64 and writes them (rounded once to fp32)
// where the merge kernel will read them, plus a per-workgroup loss partial.
#pragma once

#include "common.hpp"
#include "fp64math.hpp"

namespace adapm {

// Sum loss partials in index order (deterministic), then write the total.
__global__ __launch_bounds__(BLOCK) void k_sum_loss(LossTotal lt) {
  __shared__ double sm[WAVES_PER_BLOCK];
  sum_loss_parts(lt, sm);
}

// ------------------------------------------------------------------ MF
// Key occurrences of entry b: 2b = row key, 2b+1 = column key.  Row factors
// are keys [0, col_off), column factors [col_off, num_keys); an entry with a
// key outside its range yields the (invalid) key -1 for both occurrences.
__device__ __forceinline__ bool mf_entry_ok(int64_t ku, int32_t c, int64_t col_off, int64_t num_keys) {
  return ku >= 0 && ku < col_off && c >= 0 && col_off + (int64_t)c < num_keys;
}

struct KeysMF {
  const int32_t* row;
  const int32_t* col;
  int64_t col_off;
  int64_t num_keys;
  __device__ int64_t operator()(int64_t i) const {
    const int64_t b = i >> 1;
    if (!mf_entry_ok(row[b], col[b], col_off, num_keys)) return -1;
    return (i & 1) ? col_off + (int64_t)col[b] : (int64_t)row[b];
  }
};

// What the row-key merge needs of one MF entry, stored at the sorted
// position of its row occurrence: the column key, the observed value and the
// sorted position of the column occurrence.
struct MFEntry {
  uint32_t col_key;
  float y;
  uint32_t col_pos;
  uint32_t pad;
};

// Entry b -> its MFEntry at the row occurrence's sorted position (rank[2b]);
// reads are in entry order, the write is one 16-byte scatter.
__global__ __launch_bounds__(BLOCK) void k_mf_pack(const int32_t* __restrict__ row, const int32_t* __restrict__ col,
                                                   const float* __restrict__ val, int64_t B, int64_t col_off,
                                                   int64_t num_keys, const uint32_t* __restrict__ rank,
                                                   MFEntry* __restrict__ pe) {
  for (int64_t b = (int64_t)blockIdx.x * BLOCK + threadIdx.x; b < B; b += (int64_t)gridDim.x * BLOCK) {
    const int32_t c = col[b];
    if (!mf_entry_ok(row[b], c, col_off, num_keys)) continue;
    const uint2 rk = *reinterpret_cast<const uint2*>(rank + 2 * b);
    pe[rk.x] = MFEntry{(uint32_t)(col_off + (int64_t)c), val[b], rk.y, 0u};
  }
}

// MF row keys, merged before any column key is updated.  For the row
// occurrence of entry (u = W[row], m = W[col_off + col], y) the merge has the
// pre-step row u of the segment key; this source reads m and forms
//   e = y - <u,m>   (fp64)
//   row gradient      lam*u - e*m   (returned, fp32)
//   column gradient   lam*m - e*u   (fp32, stored at the column occurrence's
//                                    sorted position for the column-key merge)
//   loss += e^2/2 + lam/2 (|u|^2 + |m|^2)
// Row stride (floats) of the column-occurrence gradient rows: dim rounded
// up to MF_GRAD_ALIGN floats (64 bytes), and the row merge writes the
// padding too, so its scattered row writes cover whole 64-byte pieces of
// memory (400-byte rows at a 448-byte stride: 1% off the row merge).
constexpr int MF_GRAD_ALIGN = 16;
__host__ __device__ constexpr int64_t mf_grad_ld(int dim) {
  return (dim + MF_GRAD_ALIGN - 1) / MF_GRAD_ALIGN * MF_GRAD_ALIGN;
}

template <class VT>
struct SrcMFRow {
  static constexpr bool kNeedsOwn = true;
  static constexpr bool kLoss = true;
  using Value = VT;   // the table's value type
  const MFEntry* pe;
  const VT* W;
  int64_t ld;
  float* grads;
  double* loss_part;
  double lam;
  int dim;
  int64_t gld;   // row stride of grads
  struct Meta {
    const VT* partner;
    float y;
    uint32_t col_pos;
  };
  __device__ __forceinline__ Meta meta(int64_t j) const {
    const MFEntry r = pe[j];
    return {W + (int64_t)r.col_key * ld, r.y, r.col_pos};
  }
  template <int L, int NV, int VW>
  __device__ __forceinline__ void load(const Meta& m, const float* own, int gl, float* x, double& lsum) const {
    float p[NV * VW];
    double dot = 0.0, nu = 0.0, nm = 0.0;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int c = (gl + v * L) * VW;
      if (c < dim) {
        load_vals<VW>(m.partner + c, p + v * VW);
#pragma unroll
        for (int q = 0; q < VW; ++q) {
          // a product of two floats is exact in fp64, so a fused multiply-add
          // rounds exactly like the separate multiply and add
          const double uq = (double)own[v * VW + q], mq = (double)p[v * VW + q];
          dot = __builtin_fma(uq, mq, dot);
          nu = __builtin_fma(uq, uq, nu);
          nm = __builtin_fma(mq, mq, nm);
        }
      }
    }
    dot = group_sum<L>(dot);
    nu = group_sum<L>(nu);
    nm = group_sum<L>(nm);
    const double err = (double)m.y - dot;
    if (gl == 0) lsum += 0.5 * err * err + 0.5 * lam * (nu + nm);
    float* gc = grads + (int64_t)m.col_pos * gld;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int c = (gl + v * L) * VW;
      if (c < dim) {
        float g[VW];
#pragma unroll
        for (int q = 0; q < VW; ++q) {
          const double uq = (double)own[v * VW + q], mq = (double)p[v * VW + q];
          x[v * VW + q] = (float)(lam * uq - err * mq);
          g[q] = (float)(lam * mq - err * uq);
        }
        store_frag<VW>(gc + c, g);
      } else if (c < gld) {
        float z[VW] = {};
        store_frag<VW>(gc + c, z);
      }
    }
  }
};

// ------------------------------------------------------------------ shared pieces
// sigmoid and softplus of the logistic losses: fp64math.hpp.

// Per-unit validity: a unit (sample, triple, centre) with any id outside its
// table is skipped entirely and raises the sticky error flag.
template <class V>
// One wavefront per unit: its lanes check the unit's ids (V::ids, V::id_ok)
// side by side.  The grid also zeroes clear[0, clear_words): the key sort's
// header and histograms, which the sort that follows would otherwise clear
// with a launch of its own.
__global__ __launch_bounds__(BLOCK) void k_unit_valid(V v, int64_t B, uint8_t* __restrict__ ok,
                                                      int32_t* __restrict__ err, uint32_t* __restrict__ clear,
                                                      int64_t clear_words) {
  for (int64_t i = (int64_t)blockIdx.x * BLOCK + threadIdx.x; i < clear_words; i += (int64_t)gridDim.x * BLOCK)
    clear[i] = 0u;
  const int lane = lane_id();
  int bad = 0;
  for (int64_t b = (int64_t)blockIdx.x * WAVES_PER_BLOCK + threadIdx.x / WAVE; b < B;
       b += (int64_t)gridDim.x * WAVES_PER_BLOCK) {
    const int n = v.ids(b);
    bool good = true;
    for (int i = lane; i < n; i += WAVE) good = good && v.id_ok(b, i);
    const bool all = __ballot(!good) == 0;
    if (lane == 0) ok[b] = all;
    bad |= !all;
  }
  if (__syncthreads_or(bad) && threadIdx.x == 0) atomicOr(err, 1);
}

// ------------------------------------------------------------------ CTR
struct ValidCTR {
  const int64_t* keys;
  int F;
  int64_t num_keys;
  __device__ int ids(int64_t) const { return F; }
  __device__ bool id_ok(int64_t b, int f) const {
    const int64_t k = keys[b * F + f];
    return k >= 0 && k < num_keys;
  }
};

struct KeysCTR {
  const int64_t* keys;
  int F;
  const uint8_t* ok;
  __device__ int64_t operator()(int64_t i) const {
    return ok[(uint32_t)i / (uint32_t)F] ? keys[i] : ABSENT;
  }
};

// One row group per sample (e_f = W[keys[b,f]], label y):
//   S = sum_f e_f ;  z = sum_{f<g} <e_f, e_g> = (|S|^2 - sum_f |e_f|^2) / 2
//   loss += softplus(z) - y z ;  grad e_f = (sigmoid(z) - y)(S - e_f)
// Gradient rows are written in occurrence order (row b*F + f), so the
// kernel needs nothing from the key sort and runs beside it.
template <int L, int NV, int VW>
__global__ __launch_bounds__(BLOCK) void k_ctr_grad(const float* __restrict__ W, int64_t ld, int dim,
                                                    const int64_t* __restrict__ keys,
                                                    const float* __restrict__ label, int64_t B, int F,
                                                    const uint8_t* __restrict__ ok, float* __restrict__ grads,
                                                    double* __restrict__ loss_part) {
  constexpr int GPB = BLOCK / L;
  constexpr int NE = NV * VW;
  __shared__ double sm[WAVES_PER_BLOCK];
  const int gl = threadIdx.x % L;
  double lsum = 0.0;
  for (int64_t b = (int64_t)blockIdx.x * GPB + threadIdx.x / L; b < B; b += (int64_t)gridDim.x * GPB) {
    if (!ok[b]) continue;
    double S[NE];
#pragma unroll
    for (int e = 0; e < NE; ++e) S[e] = 0.0;
    double sq = 0.0;
    // the sample's keys are loaded L at a time, one per lane, and FU rows are
    // in flight at once; the sums still take the fields in order
    constexpr int FU = 4;
    for (int f0 = 0; f0 < F; f0 += L) {
      const int nf = F - f0 < L ? F - f0 : L;
      const int64_t my_key = gl < nf ? keys[b * F + f0 + gl] : 0;
      for (int f = 0; f < nf; f += FU) {
        float x[FU][NE];
#pragma unroll
        for (int u = 0; u < FU; ++u) {
          const int64_t key = __shfl(my_key, (f + u) % L, L);
          const float* row = W + key * ld;
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            const int c = (gl + v * L) * VW;
            if (f + u < nf && c < dim) load_frag<VW>(row + c, x[u] + v * VW);
            else
#pragma unroll
              for (int e = 0; e < VW; ++e) x[u][v * VW + e] = 0.0f;
          }
        }
#pragma unroll
        for (int u = 0; u < FU; ++u)
          if (f + u < nf)
#pragma unroll
            for (int e = 0; e < NE; ++e) {
              S[e] += (double)x[u][e];
              sq = __builtin_fma((double)x[u][e], (double)x[u][e], sq);   // exact product: same rounding as mul + add
            }
      }
    }
    double ss = 0.0;
#pragma unroll
    for (int e = 0; e < NE; ++e) ss += S[e] * S[e];
    ss = group_sum<L>(ss);
    sq = group_sum<L>(sq);
    const double z = 0.5 * (ss - sq);
    const double y = (double)label[b];
    double sig, sp;
    sigmoid_softplus(z, &sig, &sp);
    const double a = sig - y;
    if (gl == 0) lsum += sp - y * z;
    for (int f0 = 0; f0 < F; f0 += L) {
      const int nf = F - f0 < L ? F - f0 : L;
      const int64_t my_key = gl < nf ? keys[b * F + f0 + gl] : 0;
      for (int f = 0; f < nf; f += FU) {
        float x[FU][NE];
#pragma unroll
        for (int u = 0; u < FU; ++u) {
          const float* row = W + __shfl(my_key, (f + u) % L, L) * ld;
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            const int c = (gl + v * L) * VW;
            if (f + u < nf && c < dim) load_frag<VW>(row + c, x[u] + v * VW);
          }
        }
#pragma unroll
        for (int u = 0; u < FU; ++u) {
          float* dst = grads + (b * F + f0 + f + u) * (int64_t)dim;
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            const int c = (gl + v * L) * VW;
            if (f + u < nf && c < dim) {
              float g[VW];
#pragma unroll
              for (int e = 0; e < VW; ++e) g[e] = (float)(a * (S[v * VW + e] - (double)x[u][v * VW + e]));
              store_frag<VW>(dst + c, g);
            }
          }
        }
      }
    }
  }
  lsum = block_sum_double(lsum, sm);
  if (threadIdx.x == 0) loss_part[blockIdx.x] = lsum;
}

// ------------------------------------------------------------------ KGE (ComplEx)
struct ValidKGE {
  const int32_t *head, *rel, *tail, *neg;
  int n_neg;
  int64_t rel_off, num_keys;
  __device__ int ids(int64_t) const { return 3 + n_neg; }
  // id 0 = head, 1 = tail, 2 = relation, 3 + j = negative j
  __device__ bool id_ok(int64_t t, int i) const {
    auto okk = [&](int64_t k) { return k >= 0 && k < num_keys; };
    if (i == 0) return okk(head[t]);
    if (i == 1) return okk(tail[t]);
    if (i == 2) return rel[t] >= 0 && okk(rel_off + rel[t]);
    return okk(neg[t * n_neg + (i - 3)]);
  }
};

// Occurrences of triple t: 0 = head, 1 = relation, 2 = tail, 3 + j = negative j.
struct KeysKGE {
  const int32_t *head, *rel, *tail, *neg;
  int per, n_neg;
  int64_t rel_off;
  const uint8_t* ok;
  __device__ int64_t operator()(int64_t i) const {
    const uint32_t t = (uint32_t)i / (uint32_t)per;
    const uint32_t q = (uint32_t)i - t * (uint32_t)per;
    if (!ok[t]) return ABSENT;
    if (q == 0) return head[t];
    if (q == 1) return rel_off + rel[t];
    if (q == 2) return tail[t];
    return neg[(int64_t)t * n_neg + (q - 3)];
  }
};

// One wavefront per triple; lane l holds complex components k = l + 64 i.
// A row is [Re(0..C-1) | Im(0..C-1)].  With f = d phi/d s at (r, o) and
// h = d phi/d o at (s, r), a head-corrupted triple scores phi(x,r,o) = <x, f>
// and a tail-corrupted one phi(s,r,x) = <x, h>, so the gradient row of each
// negative occurrence is (its coefficient) x (f or h): the kernel stores the
// fp64 rows f, h per triple and one fp64 coefficient per negative, and
// writes the full fp32 gradient rows of s, r and o.  The negatives' terms in
// those three rows are linear in x, so the kernel sums c_j x_j over the
// head-corrupted and over the tail-corrupted negatives (fp64) and multiplies
// the two sums by (r, o) and (s, r) once per triple.
template <int KPL>
__global__ __launch_bounds__(BLOCK) void k_kge_grad(const float* __restrict__ W, int64_t ld, int dim,
                                                    const int32_t* __restrict__ head,
                                                    const int32_t* __restrict__ rel,
                                                    const int32_t* __restrict__ tail,
                                                    const int32_t* __restrict__ neg, int64_t B, int n_neg,
                                                    int n_head, int64_t rel_off, const uint8_t* __restrict__ ok,
                                                    float* __restrict__ mat, double* __restrict__ base,
                                                    double* __restrict__ coef, double* __restrict__ loss_part) {
  constexpr int JB = 4;   // negatives in flight, scored together (8 costs occupancy)
  __shared__ double sm[WAVES_PER_BLOCK];
  // per-thread fp64 gradient rows of s, r, o (Re, Im) of the true triple's
  // term, and the current batch of negative rows, kept in LDS: the
  // coefficient's fp64 transcendentals would otherwise run with all of them
  // in registers
  __shared__ double gacc[6 * KPL][BLOCK];
  __shared__ float xstash[2 * JB * KPL][BLOCK];
  const int cdim = dim / 2;
  const int lane = lane_id();
  const int64_t per = 3 + n_neg;
  double lsum = 0.0;
  for (int64_t t = (int64_t)blockIdx.x * WAVES_PER_BLOCK + threadIdx.x / WAVE; t < B;
       t += (int64_t)gridDim.x * WAVES_PER_BLOCK) {
    if (!ok[t]) continue;
    const float* sp = W + (int64_t)head[t] * ld;
    const float* rp = W + (rel_off + rel[t]) * ld;
    const float* op = W + (int64_t)tail[t] * ld;
    // the rows as loaded (fp32; each use converts exactly to fp64)
    float sRf[KPL], sIf[KPL], rRf[KPL], rIf[KPL], oRf[KPL], oIf[KPL];
#pragma unroll
    for (int i = 0; i < KPL; ++i) {
      const int k = lane + WAVE * i;
      const bool in = k < cdim;
      sRf[i] = in ? sp[k] : 0.0f; sIf[i] = in ? sp[cdim + k] : 0.0f;
      rRf[i] = in ? rp[k] : 0.0f; rIf[i] = in ? rp[cdim + k] : 0.0f;
      oRf[i] = in ? op[k] : 0.0f; oIf[i] = in ? op[cdim + k] : 0.0f;
    }
    double fR[KPL], fI[KPL], hR[KPL], hI[KPL];
    double* const gsR = gacc[0 * KPL] + threadIdx.x;   // element i at [i * BLOCK]
    double* const gsI = gacc[1 * KPL] + threadIdx.x;
    double* const grR = gacc[2 * KPL] + threadIdx.x;
    double* const grI = gacc[3 * KPL] + threadIdx.x;
    double* const goR = gacc[4 * KPL] + threadIdx.x;
    double* const goI = gacc[5 * KPL] + threadIdx.x;
    double part = 0.0;
#pragma unroll
    for (int i = 0; i < KPL; ++i) {
      fR[i] = (double)rRf[i] * (double)oRf[i] + (double)rIf[i] * (double)oIf[i];
      fI[i] = (double)rRf[i] * (double)oIf[i] - (double)rIf[i] * (double)oRf[i];
      hR[i] = (double)sRf[i] * (double)rRf[i] - (double)sIf[i] * (double)rIf[i];
      hI[i] = (double)sIf[i] * (double)rRf[i] + (double)sRf[i] * (double)rIf[i];
      part += (double)sRf[i] * (double)rRf[i] * (double)oRf[i];
      part += (double)sIf[i] * (double)rRf[i] * (double)oIf[i];
      part += (double)sRf[i] * (double)rIf[i] * (double)oIf[i];
      part -= (double)sIf[i] * (double)rIf[i] * (double)oRf[i];
    }
    const double phi = group_sum<WAVE>(part);
    double c, sp0;
    sigmoid_softplus(-phi, &c, &sp0);
    c = -c;
    if (lane == 0) lsum += sp0;
#pragma unroll
    for (int i = 0; i < KPL; ++i) {
      gsR[i * BLOCK] = c * fR[i];
      gsI[i * BLOCK] = c * fI[i];
      grR[i * BLOCK] = c * ((double)sRf[i] * (double)oRf[i] + (double)sIf[i] * (double)oIf[i]);
      grI[i * BLOCK] = c * ((double)sRf[i] * (double)oIf[i] - (double)sIf[i] * (double)oRf[i]);
      goR[i * BLOCK] = c * hR[i];
      goI[i * BLOCK] = c * hI[i];
      const int k = lane + WAVE * i;
      if (k < cdim) {
        double* fb = base + (2 * t) * dim;
        double* hb = base + (2 * t + 1) * dim;
        fb[k] = fR[i]; fb[cdim + k] = fI[i];
        hb[k] = hR[i]; hb[cdim + k] = hI[i];
      }
    }
    // lane l holds the id of negative 64 i + l of the current tile i; the
    // next tile's ids are loaded one tile ahead, so the row loads of a batch
    // never wait for an id load
    const int32_t* nt = neg + t * n_neg;
    int32_t id_cur = lane < n_neg ? nt[lane] : 0;
    int32_t id_nxt = WAVE + lane < n_neg ? nt[WAVE + lane] : 0;
    // the rows of the batch of negatives starting at jb (a multiple of JB,
    // inside the id tile held in id_cur)
    float xR[JB][KPL], xI[JB][KPL];
    auto load_batch = [&](int jb) {
#pragma unroll
      for (int jj = 0; jj < JB; ++jj) {
        const int j = jb + jj;
        const int32_t id = __shfl(id_cur, jb % WAVE + jj, WAVE);
        const float* xp = W + (int64_t)(j < n_neg ? id : 0) * ld;
#pragma unroll
        for (int i = 0; i < KPL; ++i) {
          const int k = lane + WAVE * i;
          const bool in = k < cdim && j < n_neg;
          xR[jj][i] = in ? xp[k] : 0.0f;
          xI[jj][i] = in ? xp[cdim + k] : 0.0f;
        }
      }
    };
    // sums over the negatives of c_j x_j (head-corrupted: Xh, tail-corrupted: Xt)
    double XhR[KPL], XhI[KPL], XtR[KPL], XtI[KPL];
#pragma unroll
    for (int i = 0; i < KPL; ++i) XhR[i] = XhI[i] = XtR[i] = XtI[i] = 0.0;
    if (n_neg > 0) load_batch(0);
    for (int j0 = 0; j0 < n_neg; j0 += JB) {
      // convert s, r, o per batch instead of holding fp64 copies across the loop
#pragma unroll
      for (int i = 0; i < KPL; ++i)
        asm volatile("" : "+v"(sRf[i]), "+v"(sIf[i]), "+v"(rRf[i]), "+v"(rIf[i]), "+v"(oRf[i]), "+v"(oIf[i]));
      double ph[JB];
#pragma unroll
      for (int jj = 0; jj < JB; ++jj) {
        const bool hd = j0 + jj < n_head;
        double p = 0.0;
#pragma unroll
        for (int i = 0; i < KPL; ++i)
          p += hd ? ((double)xR[jj][i] * fR[i] + (double)xI[jj][i] * fI[i])
                  : ((double)xR[jj][i] * hR[i] + (double)xI[jj][i] * hI[i]);
        ph[jj] = p;
      }
#pragma unroll
      for (int jj = 0; jj < JB; ++jj)
#pragma unroll
        for (int i = 0; i < KPL; ++i) {
          xstash[(jj * KPL + i) * 2][threadIdx.x] = xR[jj][i];
          xstash[(jj * KPL + i) * 2 + 1][threadIdx.x] = xI[jj][i];
        }
      asm volatile("" ::: "memory");   // read them back from LDS, not from registers
      // the next batch's rows load while this batch's coefficients are formed
      if (j0 + JB < n_neg) {
        if ((j0 + JB) % WAVE == 0) {
          id_cur = id_nxt;
          id_nxt = j0 + JB + WAVE + lane < n_neg ? nt[j0 + JB + WAVE + lane] : 0;
        }
        load_batch(j0 + JB);
      }
      // lane finishes the score of negative j0 + lane / (WAVE / JB) and its coefficient
      const double phi_my = group_multi_sum<WAVE, JB>(ph, lane);
      const int j_my = j0 + lane / (WAVE / JB);
      double c_my = 0.0;
      if (j_my < n_neg) {
        double sp;
        sigmoid_softplus(phi_my, &c_my, &sp);
        if (lane % (WAVE / JB) == 0) {
          lsum += sp;
          coef[t * per + 3 + j_my] = c_my;
        }
      }
#pragma unroll
      for (int jj = 0; jj < JB; ++jj) {
        const int j = j0 + jj;
        const double cj = __shfl(c_my, jj * (WAVE / JB), WAVE);
        if (j >= n_neg) break;
        const bool hd = j < n_head;
#pragma unroll
        for (int i = 0; i < KPL; ++i) {
          const double x_r = xstash[(jj * KPL + i) * 2][threadIdx.x];
          const double x_i = xstash[(jj * KPL + i) * 2 + 1][threadIdx.x];
          if (hd) {
            XhR[i] = __builtin_fma(cj, x_r, XhR[i]);
            XhI[i] = __builtin_fma(cj, x_i, XhI[i]);
          } else {
            XtR[i] = __builtin_fma(cj, x_r, XtR[i]);
            XtI[i] = __builtin_fma(cj, x_i, XtI[i]);
          }
        }
      }
    }
#pragma unroll
    for (int i = 0; i < KPL; ++i) {
      const double sR = sRf[i], sI = sIf[i], rR = rRf[i], rI = rIf[i], oR = oRf[i], oI = oIf[i];
      grR[i * BLOCK] += (XhR[i] * oR + XhI[i] * oI) + (sR * XtR[i] + sI * XtI[i]);
      grI[i * BLOCK] += (XhR[i] * oI - XhI[i] * oR) + (sR * XtI[i] - sI * XtR[i]);
      goR[i * BLOCK] += XhR[i] * rR - XhI[i] * rI;
      goI[i * BLOCK] += XhI[i] * rR + XhR[i] * rI;
      gsR[i * BLOCK] += rR * XtR[i] + rI * XtI[i];
      gsI[i * BLOCK] += rR * XtI[i] - rI * XtR[i];
    }
    float* ms = mat + (3 * t) * dim;
#pragma unroll
    for (int i = 0; i < KPL; ++i) {
      const int k = lane + WAVE * i;
      if (k < cdim) {
        ms[k] = (float)gsR[i * BLOCK];
        ms[cdim + k] = (float)gsI[i * BLOCK];
        ms[dim + k] = (float)grR[i * BLOCK];
        ms[dim + cdim + k] = (float)grI[i * BLOCK];
        ms[2 * dim + k] = (float)goR[i * BLOCK];
        ms[2 * dim + cdim + k] = (float)goI[i * BLOCK];
      }
    }
  }
  lsum = block_sum_double(lsum, sm);
  if (threadIdx.x == 0) loss_part[blockIdx.x] = lsum;
}

// Gradient source of the KGE push.
struct SrcKGE {
  static constexpr bool kNeedsOwn = false;
  const uint32_t* perm;
  const float* mat;
  const double* base;
  const double* coef;
  int per, n_head, dim;
  struct Meta {
    const void* row;    // fp32 stored row (s, r, o) or fp64 base row (negatives)
    double c;           // coefficient of a negative
    uint32_t scaled;    // 1: row is fp64 and scaled by c
    uint32_t pad;
  };
  __device__ __forceinline__ Meta meta(int64_t j) const {
    const uint32_t occ = perm[j];
    const uint32_t t = occ / (uint32_t)per;
    const uint32_t q = occ - t * (uint32_t)per;
    if (q < 3) return {mat + ((int64_t)t * 3 + q) * dim, 0.0, 0u, 0u};
    return {base + ((int64_t)t * 2 + ((int)q - 3 < n_head ? 0 : 1)) * dim, coef[occ], 1u, 0u};
  }
  template <int L, int NV, int VW>
  __device__ __forceinline__ void load(const Meta& m, const float*, int gl, float* x) const {
    if (!m.scaled) {
      const float* row = static_cast<const float*>(m.row);
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int c = (gl + v * L) * VW;
        if (c < dim) load_frag<VW>(row + c, x + v * VW);
      }
    } else {
      const double* row = static_cast<const double*>(m.row);
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int c = (gl + v * L) * VW;
        if (c < dim)
#pragma unroll
          for (int e = 0; e < VW; ++e) x[v * VW + e] = (float)(m.c * row[c + e]);
      }
    }
  }
};

// ------------------------------------------------------------------ SGNS
struct ValidSGNS {
  const int32_t *centre, *ctx, *neg;
  int slots, K;
  int64_t out_off, num_keys;
  __device__ int ids(int64_t) const { return 1 + slots * (K + 1); }
  // id 0 = centre; then per slot q the context word and its K negatives
  // (an absent slot, context -1, passes)
  __device__ bool id_ok(int64_t b, int i) const {
    if (i == 0) {
      const int64_t c = centre[b];
      return c >= 0 && c < out_off && c < num_keys;
    }
    const int q = (i - 1) / (K + 1);
    const int k = (i - 1) - q * (K + 1);
    const int64_t x = ctx[b * slots + q];
    if (x == -1) return true;
    const int64_t vout = num_keys - out_off;
    const int64_t y = k == 0 ? x : (int64_t)neg[(b * slots + q) * K + (k - 1)];
    return y >= 0 && y < vout;
  }
};

// Occurrences of centre b: 0 = centre (input table), then for slot q the
// context word and its K negatives (output table); absent slots are ABSENT.
struct KeysSGNS {
  const int32_t *centre, *ctx, *neg;
  int per, slots, K;
  int64_t out_off;
  const uint8_t* ok;
  __device__ int64_t operator()(int64_t i) const {
    const uint32_t b = (uint32_t)i / (uint32_t)per;
    const uint32_t q = (uint32_t)i - b * (uint32_t)per;
    if (!ok[b]) return ABSENT;
    if (q == 0) return centre[b];
    const uint32_t r = q - 1;
    const uint32_t slot = r / (uint32_t)(K + 1);
    const uint32_t k = r - slot * (uint32_t)(K + 1);
    const int64_t cx = ctx[(int64_t)b * slots + slot];
    if (cx == -1) return ABSENT;
    if (k == 0) return out_off + cx;
    return out_off + neg[((int64_t)b * slots + slot) * K + (k - 1)];
  }
};

// One row group per centre (v = input row of the centre word): for each
// present slot, the context word (x = <u, v>, a = -sigmoid(-x), loss
// softplus(-x)) and its negatives (a = sigmoid(x), loss softplus(x)).
// Stores one fp64 coefficient a per output occurrence (its gradient row is
// a*v) and the centre's fp32 gradient row sum(a*u).
template <int L, int NV, int VW>
__global__ __launch_bounds__(BLOCK) void k_sgns_grad(const float* __restrict__ W, int64_t ld, int dim,
                                                     const int32_t* __restrict__ centre,
                                                     const int32_t* __restrict__ ctx,
                                                     const int32_t* __restrict__ neg, int64_t B, int slots, int K,
                                                     int64_t out_off, const uint8_t* __restrict__ ok,
                                                     float* __restrict__ mat, double* __restrict__ coef,
                                                     double* __restrict__ loss_part) {
  constexpr int GPB = BLOCK / L;
  constexpr int NE = NV * VW;
  constexpr int JB = L >= 4 ? 4 : L;   // output rows scored together (power of two <= L)
  __shared__ double sm[WAVES_PER_BLOCK];
  __shared__ float ustash[JB * NE][BLOCK];   // one batch of rows, lane-major
  __shared__ double gacc[NE][BLOCK];
  const int gl = threadIdx.x % L;
  const int64_t per = 1 + (int64_t)slots * (K + 1);
  double lsum = 0.0;
  for (int64_t b = (int64_t)blockIdx.x * GPB + threadIdx.x / L; b < B; b += (int64_t)gridDim.x * GPB) {
    if (!ok[b]) continue;
    const float* vp = W + (int64_t)centre[b] * ld;
    float v[NE];
    double* gv = gacc[0] + threadIdx.x;   // gv[e] is gacc[e][thread]: the centre gradient in fp64
#pragma unroll
    for (int q = 0; q < NV; ++q) {
      const int c = (gl + q * L) * VW;
      if (c < dim) load_frag<VW>(vp + c, v + q * VW);
      else
#pragma unroll
        for (int e = 0; e < VW; ++e) v[q * VW + e] = 0.0f;
    }
#pragma unroll
    for (int e = 0; e < NE; ++e) gv[e * BLOCK] = 0.0;
    // the output rows of the centre's present slots in occurrence order: row
    // r is slot r / (K+1), position r % (K+1) (0 = the context word, then the
    // negatives).  The loop runs over "live" rows rp, the rows of present
    // slots only (a slot whose context is -1 has no rows), mapped to r
    // through a bit mask of the present slots (up to 64 slots; with more,
    // every slot is visited and absent ones are skipped row by row).  Lane i
    // holds the table id of live row t*L + i of the current tile t of L rows
    // (-1: absent or past the end); the next tile's ids are loaded one tile
    // ahead, so the row loads never wait for an id load.
    uint64_t present = 0;
    bool compact = false;   // some slot absent, and at most 64 slots
    if (slots <= 64) {
      for (int q = 0; q < slots; ++q) present |= (uint64_t)(ctx[b * slots + q] != -1) << q;
      compact = __popcll(present) < slots;
    }
    const int rows = (compact ? __popcll(present) : slots) * (K + 1);
    auto map_row = [&](int rp) -> int {   // live row -> row of the centre
      if (!compact) return rp;
      const int nth = rp / (K + 1);
      uint64_t m = present;
      for (int i = 0; i < nth; ++i) m &= m - 1;   // drop the nth lowest present slots
      return __builtin_ctzll(m) * (K + 1) + (rp - nth * (K + 1));
    };
    // table id of live row rp (-1: absent or past the end) and its row r
    auto row_id = [&](int rp, int& r) -> int64_t {
      r = 0;
      if (rp >= rows) return -1;
      r = map_row(rp);
      const int q = r / (K + 1);
      const int k = r - q * (K + 1);
      const int64_t cx = ctx[b * slots + q];
      const int64_t ng = k == 0 ? 0 : (int64_t)neg[(b * slots + q) * K + (k - 1)];
      return cx == -1 ? -1 : (k == 0 ? cx : ng);
    };
    int r_cur, r_nxt;
    int64_t id_cur = row_id(gl, r_cur);
    int64_t id_nxt = row_id(L + gl, r_nxt);
    // the rows of live rows rb .. rb + JB - 1 (rb a multiple of JB, inside
    // the id tile held in id_cur)
    float u[JB][NE];
    bool live[JB];
    auto load_batch = [&](int rb) {
#pragma unroll
      for (int jj = 0; jj < JB; ++jj) {
        const int64_t id = __shfl(id_cur, rb % L + jj, L);
        live[jj] = id != -1;
        const float* up = W + (out_off + (live[jj] ? id : 0)) * ld;
#pragma unroll
        for (int q2 = 0; q2 < NV; ++q2) {
          const int c = (gl + q2 * L) * VW;
          if (c < dim) load_frag<VW>(up + c, u[jj] + q2 * VW);
          else
#pragma unroll
            for (int e = 0; e < VW; ++e) u[jj][q2 * VW + e] = 0.0f;
        }
      }
    };
    if (rows > 0) load_batch(0);
    for (int r0 = 0; r0 < rows; r0 += JB) {
      double x[JB];
#pragma unroll
      for (int e = 0; e < NE; ++e) asm volatile("" : "+v"(v[e]));   // convert v per batch, not once for the loop
#pragma unroll
      for (int jj = 0; jj < JB; ++jj) {
        double p = 0.0;
#pragma unroll
        for (int e = 0; e < NE; ++e) p = __builtin_fma((double)u[jj][e], (double)v[e], p);   // exact product
        x[jj] = p;
      }
      // park the rows in LDS while the coefficients are computed (the fp64
      // transcendentals need many registers; the rows come back for the update)
#pragma unroll
      for (int jj = 0; jj < JB; ++jj)
#pragma unroll
        for (int e = 0; e < NE; ++e) ustash[jj * NE + e][threadIdx.x] = u[jj][e];
      // lane finishes the score of live row r0 + gl / (L / JB) and its coefficient
      const double x_my = group_multi_sum<L, JB>(x, gl);
      const bool live_my = __shfl(id_cur, r0 % L + gl / (L / JB), L) != -1;   // also false past the end
      const int r_my = __shfl(r_cur, r0 % L + gl / (L / JB), L);
      bool used[JB];
#pragma unroll
      for (int jj = 0; jj < JB; ++jj) used[jj] = live[jj];
      // the next batch's rows load while this batch's coefficients are formed
      if (r0 + JB < rows) {
        if ((r0 + JB) % L == 0) {
          id_cur = id_nxt;
          r_cur = r_nxt;
          id_nxt = row_id(r0 + JB + L + gl, r_nxt);
        }
        load_batch(r0 + JB);
      }
      double a_my = 0.0;
      if (live_my) {
        const int q_my = r_my / (K + 1);
        const int k_my = r_my - q_my * (K + 1);
        // context word: a = -sigmoid(-x), loss softplus(-x); negative: a = sigmoid(x), loss softplus(x)
        const double sgn = k_my == 0 ? -1.0 : 1.0;
        double sig, sp;
        sigmoid_softplus(sgn * x_my, &sig, &sp);
        a_my = sgn * sig;
        if (gl % (L / JB) == 0) {
          lsum += sp;
          coef[b * per + 1 + r_my] = a_my;
        }
      }
#pragma unroll
      for (int jj = 0; jj < JB; ++jj) {
        const double aj = __shfl(a_my, jj * (L / JB), L);
        if (used[jj])
#pragma unroll
          for (int e = 0; e < NE; ++e) gv[e * BLOCK] += aj * (double)ustash[jj * NE + e][threadIdx.x];
      }
    }
    float* dst = mat + b * dim;
#pragma unroll
    for (int q = 0; q < NV; ++q) {
      const int c = (gl + q * L) * VW;
      if (c < dim) {
        float g[VW];
#pragma unroll
        for (int e = 0; e < VW; ++e) g[e] = (float)gv[(q * VW + e) * BLOCK];
        store_frag<VW>(dst + c, g);
      }
    }
  }
  lsum = block_sum_double(lsum, sm);
  if (threadIdx.x == 0) loss_part[blockIdx.x] = lsum;
}

// Gradient source of the SGNS push: the centre occurrence reads its stored
// row; an output occurrence of centre b is a * v with v the centre's input
// row, read from the table before the input rows are updated.
struct SrcSGNS {
  static constexpr bool kNeedsOwn = false;
  const uint32_t* perm;
  const float* mat;
  const double* coef;
  const int32_t* centre;
  const float* W;
  int64_t ld;
  int per, dim;
  struct Meta {
    const float* row;   // the centre's stored gradient row, or its input row
    double a;           // coefficient of an output occurrence
    uint32_t scaled;    // 1: row is the input row, scaled by a
    uint32_t pad;
  };
  __device__ __forceinline__ Meta meta(int64_t j) const {
    const uint32_t occ = perm[j];
    const uint32_t b = occ / (uint32_t)per;
    const uint32_t q = occ - b * (uint32_t)per;
    if (q == 0) return {mat + (int64_t)b * dim, 1.0, 0u, 0u};
    return {W + (int64_t)centre[b] * ld, coef[occ], 1u, 0u};
  }
  template <int L, int NV, int VW>
  __device__ __forceinline__ void load(const Meta& m, const float*, int gl, float* x) const {
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int c = (gl + v * L) * VW;
      if (c < dim) {
        float t[VW];
        load_frag<VW>(m.row + c, t);
#pragma unroll
        for (int e = 0; e < VW; ++e) x[v * VW + e] = m.scaled ? (float)(m.a * (double)t[e]) : t[e];
      }
    }
  }
};

}  // namespace adapm
