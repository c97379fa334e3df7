// C ABI of the gfx950 parameter store: argument checks, workspace layout and
// the launch sequence of each call.  See include/adapm.h for the contract.
#include "adapm.h"

#include <atomic>
#include <chrono>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <initializer_list>
#include <mutex>
#include <string>
#include <thread>
#include <utility>
#include <vector>

#include "async.hpp"
#include "common.hpp"
#include "mlp.hpp"
#include "push.hpp"
#include "sort.hpp"
#include "staging.hpp"
#include "tasks.hpp"

using namespace adapm;

// ======================================================================== errors
namespace {

thread_local std::string g_last_error;

ps_status fail(ps_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

#define HIP_TRY(expr)                                                                        \
  do {                                                                                       \
    hipError_t e_ = (expr);                                                                  \
    if (e_ != hipSuccess) return fail(PS_ERR_DEVICE, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

#define LAUNCHED(name) HIP_TRY(hipGetLastError())

constexpr int64_t MAX_OCC = (int64_t(1) << 31) - (int64_t(1) << 20);
// Rows of up to ROW_MAX floats are one row group's; wider rows (up to
// WIDE_MAX floats, a multiple of 4) are pulled and pushed in column slices
// of ROW_MAX floats, each slice a row of the kernels that serve ROW_MAX.
constexpr int ROW_MAX = 512;
constexpr int WIDE_MAX = 16384;
constexpr int NUM_TIMED = 8;
constexpr size_t MAX_TIMED_LAUNCHES = 1 << 14;

}  // namespace

// ======================================================================== static scratch
// Workspace of the allocation-free push (ps_push_noalloc): one array per
// device, held from the first store created on that device until the
// process ends.  In host code the array's name is not a device address;
// host code reaches it only through the address hipGetSymbolAddress gives
// for the current device (scratch_address below).
static_assert(PS_NOALLOC_SCRATCH_BYTES % 256 == 0, "scratch size must keep the workspace alignment");
static __device__ __align__(256) unsigned char scratch[PS_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch[MAX_DEVICES] = {};

// The device address of `scratch` on the current device, looked up once per
// device and kept.
ps_status scratch_address(int* device, void** out) {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= MAX_DEVICES) return fail(PS_ERR_UNSUPPORTED, "device %d beyond the scratch table", dev);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    g_scratch[dev] = p;
  }
  *device = dev;
  *out = g_scratch[dev];
  return PS_OK;
}

}  // namespace

// ======================================================================== store
// Staging state of a store whose slot table caches rows of a home table in
// pinned host memory.
struct Staging {
  static constexpr int RING = 256;   // round events kept
  Planner plan;
  std::mutex mu;                     // planner and enqueue order
  int64_t num_keys = 0;              // keys of the home table
  int64_t total_slots = 0;
  const float* hW = nullptr;         // device addresses of the home tables
  const float* hG = nullptr;
  int64_t hld = 0;
  int32_t* map = nullptr;            // device: key -> slot (caller-owned)
  hipStream_t st = nullptr;          // the staging stream
  hipEvent_t clock_ev = nullptr;     // worker stream at its last clock advance
  hipEvent_t flush_ev = nullptr;
  std::vector<hipEvent_t> round_ev;
  int64_t round_id = 0;              // rounds (and forced actions) enqueued so far
  int64_t rounds = 0;                // of which regular rounds
  int64_t waited = -1;               // latest round the worker stream waits for
  int64_t* d_keys = nullptr;         // device move lists [2 * total_slots]
  int64_t* d_slots = nullptr;
  int64_t* h_list[2] = {nullptr, nullptr};   // pinned: keys then slots, [4 * total_slots]
  hipEvent_t list_ev[2] = {nullptr, nullptr};
  int list_i = 0;
  std::thread auto_thread;
  std::atomic<bool> auto_on{false};
  std::atomic<int32_t> auto_status{0};
  int64_t plan_us = 0;               // host time spent in rounds (planning and enqueueing the moves)
};

struct ps_store {
  int64_t num_keys;
  int64_t ld;        // row stride (floats) of W
  int64_t gld;       // stride (floats) between consecutive keys' accumulator rows or values
  int32_t dim;
  bool rowwise = false;   // one AdaGrad accumulator per key instead of per element
  bool bf16 = false;      // values stored as bf16 words (W then points at bf16_t)
  float* W;
  float* G;
  float lr;
  float eps;
  int32_t* status;   // device: [0] sticky key-range flag
  int device = 0;           // the device current at creation
  void* scratch = nullptr;  // that device's address of the static scratch array
  uint32_t timing = 0;   // bit k: bracket launches of kernel id k
  // a second stream for key work that runs beside a step's task kernel
  hipStream_t aux = nullptr;
  hipEvent_t fork_ev = nullptr;
  hipEvent_t join_ev = nullptr;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> events[NUM_TIMED];
  size_t used[NUM_TIMED] = {};
  Staging* stg = nullptr;   // set for stores over a slot table (ps_create_staged)
};

namespace {

// Brackets one launch with HIP events on its stream while timing is enabled.
struct Timed {
  ps_store* s;
  int id;
  hipStream_t st;
  hipEvent_t end = nullptr;
  Timed(ps_store* s_, int id_, hipStream_t st_) : s(s_), id(id_), st(st_) {
    if (!s || !((s->timing >> id) & 1u) || s->used[id] >= MAX_TIMED_LAUNCHES) return;
    auto& v = s->events[id];
    if (s->used[id] == v.size()) {
      hipEvent_t a, b;
      if (hipEventCreate(&a) != hipSuccess) return;
      if (hipEventCreate(&b) != hipSuccess) {
        (void)hipEventDestroy(a);
        return;
      }
      v.emplace_back(a, b);
    }
    auto& pr = v[s->used[id]];
    if (hipEventRecord(pr.first, st) != hipSuccess) return;
    end = pr.second;
  }
  ~Timed() {
    if (end && hipEventRecord(end, st) == hipSuccess) s->used[id] += 1;
  }
};

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// ------------------------------------------------------------------ row shapes
bool row_shape(int dim, bool vec_ok, RowShape* s) {
  if (dim <= 0) return false;
  if (vec_ok && dim % 4 == 0) {
    const int nvec = dim / 4;
    s->VW = 4;
    if (nvec <= 4) { s->L = 4; s->NV = 1; }
    else if (nvec <= 8) { s->L = 8; s->NV = 1; }
    else if (nvec <= 16) { s->L = 16; s->NV = 1; }
    else if (nvec <= 32) { s->L = 32; s->NV = 1; }
    else if (nvec <= 64) { s->L = 64; s->NV = 1; }
    else if (nvec <= 128) { s->L = 64; s->NV = 2; }
    // wider rows are not supported: their register-heavy kernel variants are disabled
    else return false;
    return true;
  }
  s->VW = 1;
  s->L = 64;
  if (dim <= 64) s->NV = 1;
  else if (dim <= 128) s->NV = 2;
  else if (dim <= 256) s->NV = 4;
  else if (dim <= 512) s->NV = 8;
  else return false;
  return true;
}

template <class F>
ps_status with_shape(const RowShape& s, F&& f) {
#define ADAPM_SHAPE(L_, NV_, VW_) \
  if (s.L == L_ && s.NV == NV_ && s.VW == VW_) return f.template operator()<L_, NV_, VW_>();
  ADAPM_SHAPE(4, 1, 4)
  ADAPM_SHAPE(8, 1, 4)
  ADAPM_SHAPE(16, 1, 4)
  ADAPM_SHAPE(32, 1, 4)
  ADAPM_SHAPE(64, 1, 4)
  ADAPM_SHAPE(64, 2, 4)
  ADAPM_SHAPE(64, 1, 1)
  ADAPM_SHAPE(64, 2, 1)
  ADAPM_SHAPE(64, 4, 1)
  ADAPM_SHAPE(64, 8, 1)
#undef ADAPM_SHAPE
  return fail(PS_ERR_UNSUPPORTED, "no kernel for row shape L=%d NV=%d VW=%d", s.L, s.NV, s.VW);
}

// ------------------------------------------------------------------ workspace
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base(static_cast<char*>(b)) {}
  template <class T>
  T* take(size_t count) {
    off = (off + 255) & ~size_t(255);
    T* p = reinterpret_cast<T*>(base ? base + off : nullptr);
    off += count * sizeof(T);
    return p;
  }
};

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

RadixPlan radix_plan(int64_t num_keys) {
  // the sentinel num_keys must be representable
  int bits = 0;
  while (bits < 32 && (uint64_t(1) << bits) <= uint64_t(num_keys)) ++bits;
  RadixPlan p{};
  p.passes = (bits + 8) / 9;   // digits of at most 9 bits
  if (p.passes < 1) p.passes = 1;
  const int per = (bits + p.passes - 1) / p.passes;
  for (int i = 0; i < p.passes; ++i) {
    p.shift[i] = i * per;
    int b = bits - i * per;
    p.bits[i] = b < per ? (b < 1 ? 1 : b) : per;
  }
  return p;
}

// Buffers of the sort + segment pipeline, carved from the workspace.
struct SortBufs {
  SegHeader* hdr;
  uint32_t* ghist;        // [MAX_PASSES][GH_COPIES][MAX_BINS]
  uint32_t* counts;       // [MAX_BINS][tiles]
  uint32_t* k[2];
  uint32_t* v[2];
  uint32_t* rank;         // [n] (steps that scatter gradients to sorted order)
  uint32_t* tstat;        // [3][tiles]
  int32_t* seg_off;       // [n+1]
  int32_t* chunk_start;   // [n+1]
  int32_t* chunk_seg;     // [n]
  int32_t* split_list;    // [n/CHUNK + 2]
  double* partial;        // [2*(n/CHUNK+1)][dim]
  double* fold;           // [n/(FOLD_SB*CHUNK)+1][dim]
  int64_t tiles;
  int items;              // keys per thread of a radix tile (tile = BLOCK * items keys)
};

// Keys per thread of the radix tiles: small sorts get more, smaller tiles
// (more workgroups), large ones bigger tiles (fewer per-tile counts).
int sort_items(int64_t n) { return n < (int64_t(1) << 19) ? 4 : (n > (int64_t(1) << 23) ? 16 : 8); }

template <class F>
ps_status with_items(int items, F&& f) {
  if (items == 4) return f.template operator()<4>();
  if (items == 16) return f.template operator()<16>();
  return f.template operator()<8>();
}

void carve_sort(Carver& c, int64_t n, int dim, bool want_rank, bool want_segments, SortBufs* b) {
  b->items = sort_items(n);
  b->tiles = ceil_div(n, int64_t(BLOCK) * b->items);
  b->hdr = c.take<SegHeader>(16);   // header and histogram are cleared together
  b->ghist = c.take<uint32_t>(MAX_PASSES * GH_COPIES * MAX_BINS);
  b->counts = c.take<uint32_t>(size_t(MAX_BINS) * b->tiles);
  b->k[0] = c.take<uint32_t>(n);
  b->k[1] = c.take<uint32_t>(n);
  b->v[0] = c.take<uint32_t>(n);
  b->v[1] = c.take<uint32_t>(n);
  b->rank = want_rank ? c.take<uint32_t>(n) : nullptr;
  b->tstat = c.take<uint32_t>(3 * b->tiles);
  b->seg_off = want_segments ? c.take<int32_t>(n + 1) : nullptr;
  b->chunk_start = c.take<int32_t>(n + 1);
  b->chunk_seg = c.take<int32_t>(n);
  b->split_list = c.take<int32_t>(n / CHUNK + 2);
  const int rdim = dim < ROW_MAX ? dim : ROW_MAX;   // wide rows are merged one column slice at a time
  b->partial = c.take<double>(size_t(2) * (n / CHUNK + 1) * rdim);
  b->fold = c.take<double>(size_t(n / (FOLD_SB * CHUNK) + 1) * rdim);
}

struct Plan {
  SortBufs sb;
  float* grads = nullptr;      // per-occurrence gradient rows (MF, CTR)
  float* mat = nullptr;        // gradient rows stored per unit (KGE: s, r, o; SGNS: centre)
  double* base = nullptr;      // KGE: fp64 rows d phi/d s (r,o) and d phi/d o (s,r) per triple
  double* coef = nullptr;      // KGE, SGNS: fp64 coefficient per occurrence
  uint8_t* ok = nullptr;       // per-unit validity
  MFEntry* pe = nullptr;       // MF: entry data at the sorted position of its row occurrence
  double* loss_part = nullptr;
  char* trans = nullptr;        // a staged store's ids in slot space (8 bytes per occurrence)
  size_t bytes = 0;
};

constexpr int64_t LOSS_GRID = 2048;
constexpr int64_t MERGE_GRID_MAX = 8192;   // largest merge grid (see reduce_grid)

bool plan_op(void* ws, int64_t num_keys, int dim, int op, int64_t units, int64_t per_unit, Plan* p) {
  (void)num_keys;
  const int64_t n = units * per_unit;
  Carver c(ws);
  switch (op) {
    case PS_OP_PUSH:
      carve_sort(c, n, dim, false, true, &p->sb);
      break;
    case PS_OP_DEDUP:
      carve_sort(c, n, dim, false, false, &p->sb);
      break;
    case PS_OP_STEP_MF:
      carve_sort(c, n, dim, true, true, &p->sb);
      // row keys sort below column keys, so row occurrences hold positions [0, units)
      p->pe = c.take<MFEntry>(units);
      p->grads = c.take<float>(size_t(n) * mf_grad_ld(dim));   // column-occurrence gradient rows, sorted positions
      p->loss_part = c.take<double>(MERGE_GRID_MAX);   // written by the row-key merge
      break;
    case PS_OP_STEP_CTR:
      carve_sort(c, n, dim, false, true, &p->sb);
      p->grads = c.take<float>(size_t(n) * dim);   // occurrence order
      p->loss_part = c.take<double>(LOSS_GRID);
      p->ok = c.take<uint8_t>(units);
      break;
    case PS_OP_STEP_KGE:
      carve_sort(c, n, dim, false, true, &p->sb);
      p->mat = c.take<float>(size_t(3) * units * dim);
      p->base = c.take<double>(size_t(2) * units * dim);
      p->coef = c.take<double>(n);
      p->loss_part = c.take<double>(LOSS_GRID);
      p->ok = c.take<uint8_t>(units);
      break;
    case PS_OP_STEP_MF_ASYNC:
      p->grads = c.take<float>(size_t(n) * dim);   // both gradient rows of each entry, entry order
      p->loss_part = c.take<double>(LOSS_GRID);
      break;
    case PS_OP_STEP_SGNS:
      carve_sort(c, n, dim, false, true, &p->sb);
      p->mat = c.take<float>(size_t(units) * dim);
      p->coef = c.take<double>(n);
      p->loss_part = c.take<double>(LOSS_GRID);
      p->ok = c.take<uint8_t>(units);
      break;
    default:
      return false;
  }
  if (op != PS_OP_DEDUP && op != PS_OP_STEP_MF_ASYNC) p->trans = c.take<char>(size_t(n) * 8);
  p->bytes = c.off + 256;
  return true;
}

// ------------------------------------------------------------------ pipeline pieces
// The sort's header and whole-array histograms, cleared together before
// each sort (by the sort itself, or by the unit-validity kernel before it).
int64_t header_words(const SortBufs& b) {
  return (reinterpret_cast<char*>(b.ghist + MAX_PASSES * GH_COPIES * MAX_BINS) - reinterpret_cast<char*>(b.hdr)) / 4;
}

void clear_header(const SortBufs& b, hipStream_t st) {
  const int64_t words = header_words(b);
  hipLaunchKernelGGL(k_zero_words, dim3(ceil_div(words, 4 * BLOCK)), dim3(BLOCK), 0, st,
                     reinterpret_cast<uint32_t*>(b.hdr), words);
}

// Stable radix sort of the keys produced by `ks`.  Returns the sorted keys;
// the permutation ends in `perm_out` if given, else in a workspace buffer
// (*perm).  With want_rank, b.rank receives the inverse permutation.
template <class KS>
ps_status run_sort(ps_store* s, KS ks, int64_t n, int64_t num_keys, SortBufs& b, int32_t* err,
                   uint32_t* perm_out, bool want_rank, hipStream_t st, uint32_t** keys_sorted,
                   uint32_t** perm, bool header_cleared = false) {
  const RadixPlan plan = radix_plan(num_keys);
  const int tiles = (int)b.tiles;
  if (!header_cleared) {
    clear_header(b, st);
    LAUNCHED(k_zero_words);
  }
  return with_items(b.items, [&]<int IT>() -> ps_status {
    hipLaunchKernelGGL((k_keyprep<KS, IT>), dim3(tiles), dim3(BLOCK), 0, st, ks, n, (uint32_t)num_keys, plan, b.k[0],
                       b.counts, tiles, b.ghist, err);
    LAUNCHED(k_keyprep);
    int src = 0;
    for (int p = 0; p < plan.passes; ++p) {
      const int bins = 1 << plan.bits[p];
      const bool last = p == plan.passes - 1;
      if (p > 0) {
        hipLaunchKernelGGL(k_radix_count<IT>, dim3(tiles), dim3(BLOCK), 0, st, b.k[src], n, plan.shift[p],
                           plan.bits[p], b.counts, tiles);
        LAUNCHED(k_radix_count);
      }
      hipLaunchKernelGGL(k_radix_scan, dim3(bins), dim3(BLOCK), 0, st, b.counts, tiles,
                         b.ghist + p * GH_COPIES * MAX_BINS);
      LAUNCHED(k_radix_scan);
      uint32_t* vout = (last && perm_out) ? perm_out : b.v[1 - src];
      uint32_t* rank = (last && want_rank) ? b.rank : nullptr;
      Timed t(s, PS_KERNEL_SCATTER, st);
      if (p == 0 && rank)
        hipLaunchKernelGGL((k_radix_scatter<true, true, IT>), dim3(tiles), dim3(BLOCK), 0, st, b.k[src], nullptr, n,
                           plan.shift[p], plan.bits[p], b.counts, tiles, b.k[1 - src], vout, rank);
      else if (p == 0)
        hipLaunchKernelGGL((k_radix_scatter<true, false, IT>), dim3(tiles), dim3(BLOCK), 0, st, b.k[src], nullptr, n,
                           plan.shift[p], plan.bits[p], b.counts, tiles, b.k[1 - src], vout, nullptr);
      else if (rank)
        hipLaunchKernelGGL((k_radix_scatter<false, true, IT>), dim3(tiles), dim3(BLOCK), 0, st, b.k[src], b.v[src], n,
                           plan.shift[p], plan.bits[p], b.counts, tiles, b.k[1 - src], vout, rank);
      else
        hipLaunchKernelGGL((k_radix_scatter<false, false, IT>), dim3(tiles), dim3(BLOCK), 0, st, b.k[src], b.v[src],
                           n, plan.shift[p], plan.bits[p], b.counts, tiles, b.k[1 - src], vout, nullptr);
      LAUNCHED(k_radix_scatter);
      src = 1 - src;
      if (last) *perm = vout;
    }
    *keys_sorted = b.k[src];
    return PS_OK;
  });
}

ps_status run_segments(const SortBufs& b, const uint32_t* ks, int64_t n, int64_t num_keys, int32_t* seg_off,
                       int64_t* uniq64, hipStream_t st, uint32_t split_key = 0) {
  const int tiles = (int)b.tiles;
  return with_items(b.items, [&]<int IT>() -> ps_status {
    hipLaunchKernelGGL(k_seg_count<IT>, dim3(tiles), dim3(BLOCK), 0, st, ks, n, (uint32_t)num_keys, b.tstat, tiles);
    LAUNCHED(k_seg_count);
    hipLaunchKernelGGL(k_seg_scan, dim3(1), dim3(BLOCK), 0, st, b.tstat, tiles, b.hdr, seg_off, b.chunk_start);
    LAUNCHED(k_seg_scan);
    hipLaunchKernelGGL(k_seg_write<IT>, dim3(tiles), dim3(BLOCK), 0, st, ks, n, (uint32_t)num_keys, b.tstat, tiles,
                       seg_off, uniq64, b.chunk_start, b.chunk_seg, split_key, b.hdr);
    LAUNCHED(k_seg_write);
    return PS_OK;
  });
}

// The skip-gram gradient kernel's lane layout.  For rows of 257..384 floats
// (300 in the paper's word vectors) float4 fragments would fill 64 lanes
// twice with most of the second pass idle (75 vectors for dim 300); float2
// fragments three times fill 78% of the lanes and need a quarter fewer
// registers and LDS per lane (measured 9-11% faster).  Other widths use the
// common layout.
template <class F>
ps_status with_sgns_shape(int dim, int64_t ld, F&& f) {
  if (dim % 2 == 0 && ld % 2 == 0 && dim > 256 && dim <= 384) return f.template operator()<64, 3, 2>();
  RowShape shape;
  if (!row_shape(dim, true, &shape)) return fail(PS_ERR_UNSUPPORTED, "dim %d not supported", dim);
  return with_shape(shape, f);
}

// Columns [col0, col0 + dim) of every row: a column slice of a wide row
// (dim 0: the whole row of the store).
struct ColSlice {
  int64_t col0 = 0;
  int dim = 0;
};

int64_t reduce_grid(int64_t n, int L, int64_t cap = MERGE_GRID_MAX) {
  const int64_t gpb = BLOCK / L;
  // one row group per chunk up to a cap (there are at most n + n/CHUNK + 1 chunks)
  int64_t g = ceil_div(n + n / CHUNK + 1, gpb);
  if (g > cap) g = cap;
  g = ceil_div(g, NUM_XCD) * NUM_XCD;
  return g;
}

// Segmented fp64 reduce of the occurrences' gradients + AdaGrad, one launch
// per part of the chunk list in the given order (a later part may update
// rows that an earlier part's source reads), then one finalize pass for all
// segments longer than a chunk.  Parts split the sorted keys at the split key
// given to run_segments: PART_UPPER = keys >= split, PART_LOWER = keys below.
enum { PART_ALL = 0, PART_UPPER = 1, PART_LOWER = 2 };

// Value types a gradient source can run on: the MF row source reads rows of
// its own value type; the sources of stored gradient rows read no table row.
template <class Src> struct SrcValue { using type = void; };
template <class VT> struct SrcValue<SrcMFRow<VT>> { using type = VT; };
template <class Src, class VT>
constexpr bool src_runs_on() {
  using T = typename SrcValue<Src>::type;
  if constexpr (std::is_same_v<VT, bf16_t>)   // bf16 stores: pull, push and the MF step
    return std::is_same_v<Src, SrcIndirect> || std::is_same_v<Src, SrcSorted> || std::is_same_v<T, bf16_t>;
  else
    return std::is_same_v<T, void> || std::is_same_v<T, VT>;
}

// grid_cap 0: the default cap, 1,024 workgroups for rows of at most 32
// lanes (each row group then walks more chunks, whose metadata it fetches
// 32 at a time; measured on pushes of 400-byte rows: 0.937 -> 0.917 ms, of
// 256-byte rows 0.123 -> 0.112 ms), MERGE_GRID_MAX for wider rows (no gain
// there, 1% lost on 1,200-byte rows).
template <class Src>
ps_status launch_segreduce(ps_store* s, const SortBufs& b, const uint32_t* ks, Src src, int64_t n, int part,
                           hipStream_t st, int timing_id = PS_KERNEL_SEGREDUCE, int64_t grid_cap = 0,
                           ColSlice cs = ColSlice{}) {
  const int dim = cs.dim ? cs.dim : s->dim;
  RowShape shape;
  if (!row_shape(dim, true, &shape)) return fail(PS_ERR_UNSUPPORTED, "dim %d not supported", dim);
  SegView sv{ks, b.seg_off, b.chunk_start, b.chunk_seg, b.hdr};
  float* W = s->W + (s->bf16 ? 0 : cs.col0);
  bf16_t* Wb = reinterpret_cast<bf16_t*>(s->W) + (s->bf16 ? cs.col0 : 0);
  float* G = s->G + (s->rowwise ? 0 : cs.col0);
  return with_shape(shape, [&]<int L, int NV, int VW>() -> ps_status {
    const int64_t grid = reduce_grid(n, L, grid_cap ? grid_cap : (L <= 32 ? 1024 : MERGE_GRID_MAX));
    Timed t(s, timing_id, st);
    if (s->bf16) {
      if constexpr (src_runs_on<Src, bf16_t>())
        hipLaunchKernelGGL((k_segreduce<L, NV, VW, Src, false, bf16_t>), dim3(grid), dim3(BLOCK), 0, st, sv, src, n,
                           Wb, G, s->ld, s->gld, dim, s->lr, s->eps, b.partial, b.split_list, b.hdr, part);
      else
        return fail(PS_ERR_UNSUPPORTED, "this step does not run on bf16 values");
    } else if constexpr (src_runs_on<Src, float>()) {
      if (s->rowwise)
        hipLaunchKernelGGL((k_segreduce<L, NV, VW, Src, true, float>), dim3(grid), dim3(BLOCK), 0, st, sv, src, n,
                           W, G, s->ld, s->gld, dim, s->lr, s->eps, b.partial, b.split_list, b.hdr, part);
      else
        hipLaunchKernelGGL((k_segreduce<L, NV, VW, Src, false, float>), dim3(grid), dim3(BLOCK), 0, st, sv, src, n,
                           W, G, s->ld, s->gld, dim, s->lr, s->eps, b.partial, b.split_list, b.hdr, part);
    } else {
      return fail(PS_ERR_UNSUPPORTED, "this step does not run on fp32 values");
    }
    LAUNCHED(k_segreduce);
    return PS_OK;
  });
}

ps_status launch_finalize(ps_store* s, const SortBufs& b, const uint32_t* ks, int64_t n, hipStream_t st,
                          LossTotal lt = LossTotal{nullptr, 0, nullptr}, ColSlice cs = ColSlice{}) {
  const int dim = cs.dim ? cs.dim : s->dim;
  RowShape shape;
  if (!row_shape(dim, true, &shape)) return fail(PS_ERR_UNSUPPORTED, "dim %d not supported", dim);
  SegView sv{ks, b.seg_off, b.chunk_start, b.chunk_seg, b.hdr};
  float* W = s->W + (s->bf16 ? 0 : cs.col0);
  bf16_t* Wb = reinterpret_cast<bf16_t*>(s->W) + (s->bf16 ? cs.col0 : 0);
  float* G = s->G + (s->rowwise ? 0 : cs.col0);
  return with_shape(shape, [&]<int L, int NV, int VW>() -> ps_status {
    const size_t lds = size_t(BLOCK / L) * dim * sizeof(double);
    const int64_t nsb = n / (FOLD_SB * CHUNK);   // super-blocks wholly inside [0, n)
    if (nsb > 0) {
      hipLaunchKernelGGL((k_seg_fold<L, NV, VW>), dim3(nsb < 1024 ? nsb : 1024), dim3(BLOCK), lds, st, sv, nsb,
                         (uint32_t)s->num_keys, dim, b.partial, b.fold);
      LAUNCHED(k_seg_fold);
    }
    // at most n / CHUNK + 1 split segments; blocks beyond their count exit at once
    int64_t fgrid = n / CHUNK + 1;
    if (fgrid > 16384) fgrid = 16384;
    if (s->bf16)
      hipLaunchKernelGGL((k_seg_finalize<L, NV, VW, false, bf16_t>), dim3(fgrid), dim3(BLOCK), lds, st, sv, Wb, G,
                         s->ld, s->gld, dim, s->lr, s->eps, b.partial, b.fold, b.split_list, lt);
    else if (s->rowwise)
      hipLaunchKernelGGL((k_seg_finalize<L, NV, VW, true, float>), dim3(fgrid), dim3(BLOCK), lds, st, sv, W, G,
                         s->ld, s->gld, dim, s->lr, s->eps, b.partial, b.fold, b.split_list, lt);
    else
      hipLaunchKernelGGL((k_seg_finalize<L, NV, VW, false, float>), dim3(fgrid), dim3(BLOCK), lds, st, sv, W, G,
                         s->ld, s->gld, dim, s->lr, s->eps, b.partial, b.fold, b.split_list, lt);
    LAUNCHED(k_seg_finalize);
    return PS_OK;
  });
}

template <class Src>
ps_status run_reduce(ps_store* s, const SortBufs& b, const uint32_t* ks, Src src, int64_t n,
                     std::initializer_list<int> parts, hipStream_t st,
                     LossTotal lt = LossTotal{nullptr, 0, nullptr}) {
  for (int part : parts)
    if (ps_status r = launch_segreduce(s, b, ks, src, n, part, st)) return r;
  return launch_finalize(s, b, ks, n, st, lt);
}


int64_t small_grid(int64_t units, int64_t per_block, int64_t cap) {
  int64_t g = ceil_div(units, per_block);
  if (g > cap) g = cap;
  return g < 1 ? 1 : g;
}

ps_status check_ws(const Plan& p, void* ws, size_t ws_bytes) {
  if (!ws) return fail(PS_ERR_INVALID, "workspace pointer is NULL");
  if (ws_bytes < p.bytes) return fail(PS_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, p.bytes);
  return PS_OK;
}

ps_status check_store(const ps_store* s) {
  if (!s) return fail(PS_ERR_INVALID, "store is NULL");
  return PS_OK;
}

// The task steps and unmerged updates work on whole rows of at most ROW_MAX
// floats; wider rows have pull and push only.
ps_status check_row_width(const ps_store* s) {
  if (s->dim > ROW_MAX)
    return fail(PS_ERR_UNSUPPORTED, "rows of %d floats: this call handles rows of at most %d (wider rows: pull and push)",
                s->dim, ROW_MAX);
  return PS_OK;
}

ps_status check_n(int64_t n, int64_t per_unit) {
  if (n < 0) return fail(PS_ERR_INVALID, "negative size %lld", (long long)n);
  if (per_unit > 0 && n > MAX_OCC / per_unit)
    return fail(PS_ERR_UNSUPPORTED, "%lld units x %lld occurrences exceed the 32-bit occurrence index",
                (long long)n, (long long)per_unit);
  return PS_OK;
}

hipStream_t as_stream(void* p) { return static_cast<hipStream_t>(p); }

// Fork/join with the store's second stream: work enqueued on s->aux after
// fork() runs beside what the caller then enqueues on st; join() makes st
// wait for it.  Both are event record/wait pairs, so a step stays capturable
// in a HIP graph.
ps_status fork_aux(ps_store* s, hipStream_t st) {
  HIP_TRY(hipEventRecord(s->fork_ev, st));
  HIP_TRY(hipStreamWaitEvent(s->aux, s->fork_ev, 0));
  return PS_OK;
}

ps_status join_aux(ps_store* s, hipStream_t st) {
  HIP_TRY(hipEventRecord(s->join_ev, s->aux));
  HIP_TRY(hipStreamWaitEvent(st, s->join_ev, 0));
  return PS_OK;
}

// The MF step in two phases.  Prepare reads only the batch: the key sort,
// segments and the per-entry records, all in the workspace.  Apply reads the
// workspace and W: the row-key merge (with the loss), the column-key merge
// and the long-segment finalize.
ps_status mf_prepare(ps_store* s, const int32_t* row, const int32_t* col, const float* val, int64_t B,
                     int64_t col_key_offset, Plan& p, hipStream_t st) {
  const int64_t n = 2 * B;
  uint32_t *ks, *perm;
  KeysMF kmf{row, col, col_key_offset, s->num_keys};
  if (ps_status r = run_sort(s, kmf, n, s->num_keys, p.sb, s->status, nullptr, true, st, &ks, &perm)) return r;
  const uint32_t split = (uint32_t)(col_key_offset < s->num_keys ? col_key_offset : s->num_keys);
  if (ps_status r = run_segments(p.sb, ks, n, s->num_keys, p.sb.seg_off, nullptr, st, split)) return r;
  Timed t(s, PS_KERNEL_TASKGRAD, st);
  hipLaunchKernelGGL(k_mf_pack, dim3(small_grid(B, BLOCK, MERGE_GRID_MAX)), dim3(BLOCK), 0, st, row, col, val, B,
                     col_key_offset, s->num_keys, p.sb.rank, p.pe);
  LAUNCHED(k_mf_pack);
  return PS_OK;
}

ps_status mf_apply(ps_store* s, int64_t B, float lambda, double* loss, Plan& p, hipStream_t st,
                   hipEvent_t rows_done = nullptr) {
  const int64_t n = 2 * B;
  const uint32_t* ks = p.sb.k[radix_plan(s->num_keys).passes % 2];   // where the sort left the keys
  // Row keys first: their source reads the column rows before any column
  // update, forms e, the loss and the column-occurrence gradients; then the
  // column keys merge those stored rows.
  // (about one key per chunk here: a smaller grid gives each group a longer
  // run of chunks whose metadata it prefetches together)
  constexpr int64_t kRowMergeGrid = 2048;
  ps_status r = s->bf16
      ? launch_segreduce(s, p.sb, ks,
                         SrcMFRow<bf16_t>{p.pe, reinterpret_cast<const bf16_t*>(s->W), s->ld, p.grads, p.loss_part,
                                          (double)lambda, s->dim, mf_grad_ld(s->dim)},
                         n, PART_LOWER, st, PS_KERNEL_MF_ROWMERGE, kRowMergeGrid)
      : launch_segreduce(s, p.sb, ks,
                         SrcMFRow<float>{p.pe, s->W, s->ld, p.grads, p.loss_part, (double)lambda, s->dim, mf_grad_ld(s->dim)}, n,
                         PART_LOWER, st, PS_KERNEL_MF_ROWMERGE, kRowMergeGrid);
  if (r) return r;
  if (rows_done) HIP_TRY(hipEventRecord(rows_done, st));
  // A caller that takes the event runs the next batch's key work beside the
  // column-key merge: a grid of 3 workgroups per CU leaves that work room
  // (measured: MF step 1.035 -> 1.011 ms overlapped; alone, the full grid is
  // faster).
  const int64_t col_grid = rows_done ? 768 : MERGE_GRID_MAX;
  if (ps_status r = launch_segreduce(s, p.sb, ks, SrcSorted{p.grads, s->dim, mf_grad_ld(s->dim)}, n, PART_UPPER, st,
                                     PS_KERNEL_SEGREDUCE, col_grid))
    return r;
  // the finalize pass also totals the row-key merge's loss partials
  RowShape shape;
  row_shape(s->dim, true, &shape);
  return launch_finalize(s, p.sb, ks, n, st, LossTotal{p.loss_part, reduce_grid(n, shape.L, kRowMergeGrid), loss});
}

ps_status zero_loss(double* loss, hipStream_t st) {
  if (loss) {
    hipLaunchKernelGGL(k_zero_words, dim3(1), dim3(BLOCK), 0, st, reinterpret_cast<uint32_t*>(loss), int64_t(2));
    LAUNCHED(k_zero_words);
  }
  return PS_OK;
}

// Checks shared by the store constructors: key count, row shape, value
// table, learning rate.
ps_status check_values(int64_t num_keys, int32_t dim, int64_t row_stride, const float* values, float lr, float eps,
                       bool wide_ok = false) {
  if (num_keys < 1 || num_keys > INT32_MAX) return fail(PS_ERR_INVALID, "num_keys %lld outside [1, 2^31-1]", (long long)num_keys);
  RowShape shape;
  const bool wide = wide_ok && dim > ROW_MAX && dim <= WIDE_MAX && dim % 4 == 0;
  if (dim < 1 || (!wide && !row_shape(dim, true, &shape)))
    return fail(PS_ERR_UNSUPPORTED, "dim %d unsupported (at most 512; per-element stores up to %d, a multiple of 4)",
                dim, WIDE_MAX);
  if (row_stride < dim) return fail(PS_ERR_INVALID, "row_stride %lld < dim %d", (long long)row_stride, dim);
  if (!values) return fail(PS_ERR_INVALID, "table pointer is NULL");
  if (dim % 4 == 0 && (!aligned16(values) || row_stride % 4 != 0))
    return fail(PS_ERR_INVALID, "tables must be 16-byte aligned with a row stride that is a multiple of 4");
  if (!(lr > 0.0f) || !(eps >= 0.0f)) return fail(PS_ERR_INVALID, "need lr > 0 and eps >= 0");
  return PS_OK;
}

// Allocates the store, its status block (cleared on `stream`), second stream
// and events.
ps_status make_store(ps_store** out, int64_t num_keys, int32_t dim, int64_t row_stride, float* values, float* accum,
                     int64_t accum_stride, bool rowwise, float lr, float eps, void* stream) {
  ps_store* s = new ps_store();
  s->num_keys = num_keys;
  s->ld = row_stride;
  s->gld = accum_stride;
  s->dim = dim;
  s->rowwise = rowwise;
  s->W = values;
  s->G = accum;
  s->lr = lr;
  s->eps = eps;
  hipError_t e = hipMalloc(&s->status, 256);
  if (e != hipSuccess) {
    delete s;
    return fail(PS_ERR_DEVICE, "hipMalloc(status): %s", hipGetErrorString(e));
  }
  if (ps_status r = scratch_address(&s->device, &s->scratch)) {
    (void)hipFree(s->status);
    delete s;
    return r;
  }
  hipStream_t st = as_stream(stream);
  hipLaunchKernelGGL(k_zero_words, dim3(1), dim3(BLOCK), 0, st, reinterpret_cast<uint32_t*>(s->status), int64_t(64));
  e = hipGetLastError();
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e == hipSuccess) e = hipStreamCreateWithFlags(&s->aux, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&s->fork_ev, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&s->join_ev, hipEventDisableTiming);
  if (e != hipSuccess) {
    if (s->join_ev) (void)hipEventDestroy(s->join_ev);
    if (s->fork_ev) (void)hipEventDestroy(s->fork_ev);
    if (s->aux) (void)hipStreamDestroy(s->aux);
    (void)hipFree(s->status);
    delete s;
    return fail(PS_ERR_DEVICE, "store set-up: %s", hipGetErrorString(e));
  }
  *out = s;
  return PS_OK;
}

// ------------------------------------------------------------------ Wide & Deep
constexpr int WD_MAX_HIDDEN = 8;

// Offsets of the dense buffer: per hidden layer W (fan_in x fan_out) then b,
// then the output vector w and bias c.
struct DenseLayout {
  int64_t offW[WD_MAX_HIDDEN], offb[WD_MAX_HIDDEN], offw, offc, total, widest;
};

DenseLayout dense_layout(int64_t K0, int L, const int32_t* hidden) {
  DenseLayout d{};
  int64_t off = 0, fan = K0;
  d.widest = K0;
  for (int l = 0; l < L; ++l) {
    d.offW[l] = off;
    off += fan * hidden[l];
    d.offb[l] = off;
    off += hidden[l];
    fan = hidden[l];
    d.widest = std::max<int64_t>(d.widest, fan);
  }
  d.offw = off;
  off += fan;
  d.offc = off;
  d.total = off + 1;
  return d;
}

struct PlanWD {
  Plan base;                 // the CTR step's sort, segments, gradient rows, loss, validity, translation
  double* X = nullptr;       // [B][F*E] inputs of the first layer
  double* H[WD_MAX_HIDDEN] = {};   // [B][h_l] activations
  double* dA = nullptr;      // [B][widest] gradients, ping-pong
  double* dB = nullptr;
  double* dlogit = nullptr;  // [B]
  double* dg = nullptr;      // dense gradient, fp64, in the dense layout
  double* part = nullptr;    // column-sum partials
  double* slices = nullptr;  // split-K partial products of the weight gradients
};

// K slices of a weight-gradient product (K = the batch): enough workgroups
// to fill the chip (about 1024), slices of at least 256 rows.
int64_t wgrad_slices(int64_t M, int64_t N, int64_t K) {
  const int64_t blocks = ceil_div(M, GEMM_BM) * ceil_div(N, GEMM_BN);
  int64_t S = ceil_div(1024, blocks);
  S = std::min<int64_t>(S, std::max<int64_t>(1, K / 256));
  return std::max<int64_t>(1, std::min<int64_t>(S, 32));
}

void plan_wd(void* ws, int dim, int64_t B, int F, int E, int L, const int32_t* hidden, PlanWD* p) {
  const int64_t n = B * F;
  const DenseLayout d = dense_layout((int64_t)F * E, L, hidden);
  Carver c(ws);
  carve_sort(c, n, dim, true, true, &p->base.sb);
  p->base.grads = c.take<float>(size_t(n) * dim);
  p->base.loss_part = c.take<double>(LOSS_GRID);
  p->base.ok = c.take<uint8_t>(B);
  p->base.trans = c.take<char>(size_t(n) * 8);
  p->X = c.take<double>(size_t(B) * F * E);
  for (int l = 0; l < L; ++l) p->H[l] = c.take<double>(size_t(B) * hidden[l]);
  p->dA = c.take<double>(size_t(B) * d.widest);
  p->dB = c.take<double>(size_t(B) * d.widest);
  p->dlogit = c.take<double>(B);
  p->dg = c.take<double>(d.total);
  p->part = c.take<double>(size_t(ceil_div(B, COLSUM_ROWS)) * d.widest);
  int64_t sl = 0, fan = (int64_t)F * E;
  for (int l = 0; l < L; ++l) {
    const int64_t S = wgrad_slices(fan, hidden[l], B);
    if (S > 1) sl = std::max<int64_t>(sl, S * fan * hidden[l]);
    fan = hidden[l];
  }
  p->slices = c.take<double>(size_t(sl));
  p->base.bytes = c.off + 256;
}

// One product; with S > 1 K is split into S slices whose partial products go
// to `slices` (S * M * N doubles) and are then added in order into C (which
// must then be dense: ldc = N, plain store).
template <bool TA, bool TB, typename BT>
ps_status gemm(ps_store* s, int64_t M, int64_t N, int64_t K, const double* A, int64_t lda, const BT* B, int64_t ldb,
               double* C, int64_t ldc, hipStream_t st, int64_t S = 1, double* slices = nullptr) {
  const int64_t gy = ceil_div(M, GEMM_BM), gx = ceil_div(N, GEMM_BN);
  if (gy > 65535) return fail(PS_ERR_UNSUPPORTED, "%lld rows exceed the product kernel's grid", (long long)M);
  const int64_t kslice = S > 1 ? ceil_div(ceil_div(K, S), GEMM_BK) * GEMM_BK : K;
  S = S > 1 ? ceil_div(K, kslice) : 1;
  {
    Timed t(s, PS_KERNEL_MLP, st);
    hipLaunchKernelGGL((k_gemm_f64<TA, TB, BT>), dim3(gx, gy, S), dim3(BLOCK), 0, st, M, N, K, A, lda, B, ldb,
                       S > 1 ? slices : C, S > 1 ? N : ldc, kslice);
    LAUNCHED(k_gemm_f64);
    if (S > 1) {
      hipLaunchKernelGGL(k_sum_slices, dim3(small_grid(M * N, BLOCK, 4096)), dim3(BLOCK), 0, st, slices, S, M * N, C);
      LAUNCHED(k_sum_slices);
    }
  }
  return PS_OK;
}

ps_status colsum(const double* A, int64_t rows, int64_t cols, const double* scale, double* part, double* out,
                 hipStream_t st) {
  const int64_t ny = ceil_div(rows, COLSUM_ROWS);
  hipLaunchKernelGGL(k_colsum_part, dim3(ceil_div(cols, BLOCK), ny), dim3(BLOCK), 0, st, A, rows, cols, scale, part);
  LAUNCHED(k_colsum_part);
  hipLaunchKernelGGL(k_colsum_final, dim3(ceil_div(cols, BLOCK)), dim3(BLOCK), 0, st, part, ny, cols, out);
  LAUNCHED(k_colsum_final);
  return PS_OK;
}

// ------------------------------------------------------------------ staged stores
// A staged store's step translates the batch's ids into slot ids first, into
// the workspace region Plan::trans.

// The first slot of the key range that starts at key_off (a key offset of a
// step must start a range, so that slot ids keep the step's id split).
ps_status slot_offset(const ps_store* s, int64_t key_off, const char* what, int64_t* out) {
  const int r = s->stg->plan.range_starting_at(key_off);
  if (r < 0)
    return fail(PS_ERR_INVALID, "%s %lld does not start a key range of the staged store", what, (long long)key_off);
  *out = s->stg->plan.range_slot0[r];
  return PS_OK;
}

ps_status translate_ids(ps_store* s, const int32_t* in, int64_t n, int64_t key_off, int64_t slot_off, int32_t* out,
                        hipStream_t st) {
  if (n <= 0 || !in) return PS_OK;
  hipLaunchKernelGGL(k_translate_ids, dim3(small_grid(n, BLOCK, 4096)), dim3(BLOCK), 0, st, in, n, s->stg->map,
                     key_off, s->stg->num_keys - key_off, slot_off, out, s->status);
  LAUNCHED(k_translate_ids);
  return PS_OK;
}

ps_status translate_keys(ps_store* s, const int64_t* in, int64_t n, int64_t* out, hipStream_t st) {
  if (n <= 0 || !in) return PS_OK;
  hipLaunchKernelGGL(k_translate_keys, dim3(small_grid(n, BLOCK, 4096)), dim3(BLOCK), 0, st, in, n, s->stg->map,
                     s->stg->num_keys, out, s->status);
  LAUNCHED(k_translate_keys);
  return PS_OK;
}

// Rows between the home tables and the slot table: `from` indexes the
// source, `to` the destination (both device lists of n entries).
ps_status move_rows(ps_store* s, bool to_home, const int64_t* from, const int64_t* to, int64_t n, hipStream_t st) {
  Staging& g = *s->stg;
  RowShape shape;
  row_shape(s->dim, true, &shape);
  return with_shape(shape, [&]<int L, int NV, int VW>() -> ps_status {
    const int64_t grid = small_grid(n, BLOCK / L, 16384);
    Timed t(s, PS_KERNEL_STAGE, st);
    if (to_home)
      hipLaunchKernelGGL((k_move_rows<L, NV, VW>), dim3(grid), dim3(BLOCK), 0, st, s->W, s->G, s->ld, from,
                         const_cast<float*>(g.hW), const_cast<float*>(g.hG), g.hld, to, n, s->dim);
    else
      hipLaunchKernelGGL((k_move_rows<L, NV, VW>), dim3(grid), dim3(BLOCK), 0, st, g.hW, g.hG, g.hld, from, s->W, s->G,
                         s->ld, to, n, s->dim);
    LAUNCHED(k_move_rows);
    return PS_OK;
  });
}

// Uploads a round's moves (written by the planner into pinned list b: keys
// at h_list[b], slots 2 * total_slots further) and enqueues them on the
// staging stream: write-backs (slot -> home, map entry cleared) before
// stage-ins (home -> slot, map entry set), so a slot freed in this round
// can be reused by it.
ps_status enqueue_moves(ps_store* s, int b, int64_t nout, int64_t nin) {
  Staging& g = *s->stg;
  if (nout + nin == 0) return PS_OK;
  g.list_i = b ^ 1;
  int64_t* hk = g.h_list[b];
  int64_t* hs = hk + 2 * g.total_slots;
  HIP_TRY(hipMemcpyAsync(g.d_keys, hk, size_t(nout + nin) * 8, hipMemcpyHostToDevice, g.st));
  HIP_TRY(hipMemcpyAsync(g.d_slots, hs, size_t(nout + nin) * 8, hipMemcpyHostToDevice, g.st));
  HIP_TRY(hipEventRecord(g.list_ev[b], g.st));
  if (nout) {
    if (ps_status r = move_rows(s, true, g.d_slots, g.d_keys, nout, g.st)) return r;
    hipLaunchKernelGGL(k_map_set, dim3(small_grid(nout, BLOCK, 4096)), dim3(BLOCK), 0, g.st, g.map, g.d_keys,
                       (const int64_t*)nullptr, nout);
    LAUNCHED(k_map_set);
  }
  if (nin) {
    if (ps_status r = move_rows(s, false, g.d_keys + nout, g.d_slots + nout, nin, g.st)) return r;
    hipLaunchKernelGGL(k_map_set, dim3(small_grid(nin, BLOCK, 4096)), dim3(BLOCK), 0, g.st, g.map, g.d_keys + nout,
                       g.d_slots + nout, nin);
    LAUNCHED(k_map_set);
  }
  return PS_OK;
}

// One round (forced: act only on intents already active, no rate update),
// with the planner lock held.  The staging stream first waits for the
// worker's steps before its last clock advance, so a write-back never races
// a step that still uses the row.
ps_status stage_round_locked(ps_store* s, bool forced, int64_t* rid_out, int64_t* moved) {
  Staging& g = *s->stg;
  Planner& P = g.plan;
  const auto t0 = std::chrono::steady_clock::now();
  const int b = g.list_i;   // the pinned list this round's moves are written into
  HIP_TRY(hipEventSynchronize(g.list_ev[b]));   // its previous upload has been read
  P.clear_moves(g.h_list[b], g.h_list[b] + 2 * g.total_slots);
  const int64_t rid = g.round_id;
  const int64_t horizon = forced ? P.clock + 1 : P.timing.horizon(P.clock);
  P.evict_expired();
  P.act(horizon, rid);
  if (forced) ++P.forced_total;
  else ++g.rounds;
  HIP_TRY(hipStreamWaitEvent(g.st, g.clock_ev, 0));
  if (ps_status r = enqueue_moves(s, b, P.nout, P.nin)) return r;
  HIP_TRY(hipEventRecord(g.round_ev[rid % Staging::RING], g.st));
  g.plan_us += std::chrono::duration_cast<std::chrono::microseconds>(std::chrono::steady_clock::now() - t0).count();
  g.round_id = rid + 1;
  if (rid_out) *rid_out = rid;
  if (moved) *moved = P.nout + P.nin;
  return PS_OK;
}

// Rounds back to back on a thread of the library: each lasts until its
// moves are done, an idle one 100 us.
void auto_rounds(ps_store* s) {
  Staging& g = *s->stg;
  while (g.auto_on.load()) {
    hipEvent_t ev = nullptr;
    int64_t moved = 0;
    {
      std::lock_guard<std::mutex> lk(g.mu);
      int64_t rid = 0;
      ps_status r = stage_round_locked(s, false, &rid, &moved);
      if (r != PS_OK) {
        g.auto_status.store(r);
        g.auto_on.store(false);
        return;
      }
      ev = g.round_ev[rid % Staging::RING];
    }
    if (hipEventSynchronize(ev) != hipSuccess) {
      g.auto_status.store(PS_ERR_DEVICE);
      g.auto_on.store(false);
      return;
    }
    if (moved == 0) std::this_thread::sleep_for(std::chrono::microseconds(100));
  }
}

void stop_auto(Staging& g) {
  g.auto_on.store(false);
  if (g.auto_thread.joinable()) g.auto_thread.join();
}

void free_staging(Staging* g) {
  if (!g) return;
  stop_auto(*g);
  if (g->st) (void)hipStreamSynchronize(g->st);
  for (hipEvent_t e : g->round_ev)
    if (e) (void)hipEventDestroy(e);
  for (int i = 0; i < 2; ++i) {
    if (g->list_ev[i]) (void)hipEventDestroy(g->list_ev[i]);
    if (g->h_list[i]) (void)hipHostFree(g->h_list[i]);
  }
  if (g->clock_ev) (void)hipEventDestroy(g->clock_ev);
  if (g->flush_ev) (void)hipEventDestroy(g->flush_ev);
  if (g->d_keys) (void)hipFree(g->d_keys);
  if (g->d_slots) (void)hipFree(g->d_slots);
  if (g->st) (void)hipStreamDestroy(g->st);
  delete g;
}

ps_status check_staged(ps_store* s) {
  if (ps_status st = check_store(s)) return st;
  if (!s->stg) return fail(PS_ERR_INVALID, "not a staged store (ps_create_staged)");
  return PS_OK;
}

// ------------------------------------------------------------------ unmerged (asynchronous) updates
ps_status check_async(const ps_store* s) {
  if (s->stg) return fail(PS_ERR_UNSUPPORTED, "unmerged updates are not available on a staged store");
  if (s->bf16) return fail(PS_ERR_UNSUPPORTED, "unmerged updates run on fp32 values only");
  return PS_OK;
}

template <class Keys>
ps_status launch_push_async(ps_store* s, Keys keys, const float* grads, int64_t n, hipStream_t st) {
  // one float per lane and atomic instruction, consecutive lanes on
  // consecutive floats: a wave's atomic touches whole cache lines (four
  // times faster than four consecutive floats per lane)
  RowShape shape;
  if (!row_shape(s->dim, false, &shape)) return fail(PS_ERR_UNSUPPORTED, "dim %d not supported", s->dim);
  return with_shape(shape, [&]<int L, int NV, int VW>() -> ps_status {
    const int64_t grid = small_grid(n, BLOCK / L, int64_t(1) << 16);
    Timed t(s, PS_KERNEL_ASYNC, st);
    if (s->rowwise)
      hipLaunchKernelGGL((k_push_async<L, NV, VW, true, Keys>), dim3(grid), dim3(BLOCK), 0, st, keys, grads, n, s->W,
                         s->G, s->ld, s->gld, s->dim, s->num_keys, s->lr, s->eps, s->status);
    else
      hipLaunchKernelGGL((k_push_async<L, NV, VW, false, Keys>), dim3(grid), dim3(BLOCK), 0, st, keys, grads, n, s->W,
                         s->G, s->ld, s->gld, s->dim, s->num_keys, s->lr, s->eps, s->status);
    LAUNCHED(k_push_async);
    return PS_OK;
  });
}

}  // namespace

// ======================================================================== C ABI
extern "C" {

const char* ps_status_string(ps_status st) {
  switch (st) {
    case PS_OK: return "ok";
    case PS_ERR_INVALID: return "invalid argument";
    case PS_ERR_KEY_RANGE: return "key outside [0, num_keys)";
    case PS_ERR_WORKSPACE: return "workspace too small";
    case PS_ERR_DEVICE: return "HIP runtime error";
    case PS_ERR_UNSUPPORTED: return "unsupported size";
    case PS_ERR_NOT_RESIDENT: return "key not resident in the staged store";
    default: return "unknown status";
  }
}

const char* ps_last_error_message(void) { return g_last_error.c_str(); }

ps_status ps_create(ps_store** out, int64_t num_keys, int32_t dim, float* values, float* accum, float lr,
                    float eps, void* stream) {
  return ps_create_strided(out, num_keys, dim, dim, values, accum, lr, eps, stream);
}

ps_status ps_create_strided(ps_store** out, int64_t num_keys, int32_t dim, int64_t row_stride, float* values,
                            float* accum, float lr, float eps, void* stream) {
  if (!out) return fail(PS_ERR_INVALID, "out is NULL");
  *out = nullptr;
  if (ps_status r = check_values(num_keys, dim, row_stride, values, lr, eps, true)) return r;
  if (!accum) return fail(PS_ERR_INVALID, "table pointer is NULL");
  {
    // rows of W and G must not overlap: either two separate tables, or rows
    // interleaved in one allocation with a gap of at least dim on each side
    const int64_t d = (int64_t)(accum - values);
    const int64_t ad = d < 0 ? -d : d;
    const bool separate = ad >= num_keys * row_stride;
    const int64_t r = ((d % row_stride) + row_stride) % row_stride;
    const bool interleaved = row_stride >= 2 * (int64_t)dim && r >= dim && r <= row_stride - dim;
    if (!separate && !interleaved) return fail(PS_ERR_INVALID, "values and accumulator rows overlap");
  }
  if (dim % 4 == 0 && !aligned16(accum)) return fail(PS_ERR_INVALID, "accumulator table must be 16-byte aligned");
  return make_store(out, num_keys, dim, row_stride, values, accum, row_stride, false, lr, eps, stream);
}

ps_status ps_create_bf16(ps_store** out, int64_t num_keys, int32_t dim, uint16_t* values, int64_t value_stride,
                         float* accum, int64_t accum_stride, float lr, float eps, void* stream) {
  if (!out) return fail(PS_ERR_INVALID, "out is NULL");
  *out = nullptr;
  if (num_keys < 1 || num_keys > INT32_MAX) return fail(PS_ERR_INVALID, "num_keys %lld outside [1, 2^31-1]", (long long)num_keys);
  RowShape shape;
  if (dim < 1 || !row_shape(dim, true, &shape)) return fail(PS_ERR_UNSUPPORTED, "dim %d unsupported (at most 512)", dim);
  if (!values || !accum) return fail(PS_ERR_INVALID, "table pointer is NULL");
  if (value_stride < dim || accum_stride < dim) return fail(PS_ERR_INVALID, "a row stride is smaller than dim");
  if (dim % 4 == 0 && ((reinterpret_cast<uintptr_t>(values) & 7u) != 0 || value_stride % 4 != 0 || !aligned16(accum) ||
                       accum_stride % 4 != 0))
    return fail(PS_ERR_INVALID, "values must be 8-byte and accumulators 16-byte aligned, strides multiples of 4");
  if (!(lr > 0.0f) || !(eps >= 0.0f)) return fail(PS_ERR_INVALID, "need lr > 0 and eps >= 0");
  {
    // two separate allocations, or rows interleaved in one: the same byte
    // stride, each key's accumulator row between its value row and the next
    const int64_t vs = value_stride * 2, as = accum_stride * 4;
    const int64_t d = (int64_t)(reinterpret_cast<uintptr_t>(accum) - reinterpret_cast<uintptr_t>(values));
    const bool separate = d >= num_keys * vs || -d >= num_keys * as;
    const int64_t r = vs > 0 ? ((d % vs) + vs) % vs : 0;
    const bool interleaved = vs == as && r >= 2 * (int64_t)dim && r <= vs - 4 * (int64_t)dim;
    if (!separate && !interleaved) return fail(PS_ERR_INVALID, "values and accumulators overlap");
  }
  if (ps_status r = make_store(out, num_keys, dim, value_stride, reinterpret_cast<float*>(values), accum, accum_stride,
                               false, lr, eps, stream))
    return r;
  (*out)->bf16 = true;
  return PS_OK;
}

ps_status ps_create_rowwise(ps_store** out, int64_t num_keys, int32_t dim, int64_t row_stride, float* values,
                            float* accum, int64_t accum_stride, float lr, float eps, void* stream) {
  if (!out) return fail(PS_ERR_INVALID, "out is NULL");
  *out = nullptr;
  if (ps_status r = check_values(num_keys, dim, row_stride, values, lr, eps)) return r;
  if (!accum) return fail(PS_ERR_INVALID, "accumulator pointer is NULL");
  if (accum_stride < 1) return fail(PS_ERR_INVALID, "accum_stride %lld < 1", (long long)accum_stride);
  {
    // no accumulator may lie inside a value row: either the accumulators
    // are wholly outside W's extent, or they sit in the rows' padding
    // (accum_stride == row_stride, offset within the row in [dim, row_stride))
    const int64_t d = (int64_t)(accum - values);
    const int64_t w_end = (num_keys - 1) * row_stride + dim;        // W spans [0, w_end)
    const int64_t a_last = d + (num_keys - 1) * accum_stride;       // last accumulator
    const bool separate = a_last < 0 || d >= w_end;
    const int64_t r = ((d % row_stride) + row_stride) % row_stride;
    const bool padded = accum_stride == row_stride && r >= dim;
    if (!separate && !padded) return fail(PS_ERR_INVALID, "accumulators overlap the value rows");
  }
  return make_store(out, num_keys, dim, row_stride, values, accum, accum_stride, true, lr, eps, stream);
}

ps_status ps_destroy(ps_store* s) {
  if (!s) return PS_OK;
  free_staging(s->stg);
  s->stg = nullptr;
  hipError_t e = hipDeviceSynchronize();
  for (auto& v : s->events)
    for (auto& pr : v) {
      (void)hipEventDestroy(pr.first);
      (void)hipEventDestroy(pr.second);
    }
  (void)hipEventDestroy(s->join_ev);
  (void)hipEventDestroy(s->fork_ev);
  (void)hipStreamDestroy(s->aux);
  hipError_t f = hipFree(s->status);
  delete s;
  if (e != hipSuccess) return fail(PS_ERR_DEVICE, "hipDeviceSynchronize: %s", hipGetErrorString(e));
  if (f != hipSuccess) return fail(PS_ERR_DEVICE, "hipFree: %s", hipGetErrorString(f));
  return PS_OK;
}

size_t ps_workspace_bytes(int64_t num_keys, int32_t dim, int32_t op, int64_t units, int64_t per_unit) {
  if (num_keys < 1 || dim < 1 || units < 0 || per_unit < 1) return 0;
  if (op == PS_OP_PULL) return 0;
  if (units > MAX_OCC / per_unit) return 0;
  Plan p;
  if (!plan_op(nullptr, num_keys, dim, op, units, per_unit, &p)) return 0;
  return p.bytes;
}

ps_status ps_pull(ps_store* s, const int64_t* keys, int64_t n, float* out, void* stream) {
  if (ps_status st = check_store(s)) return st;
  if (ps_status st = check_n(n, 1)) return st;
  if (n == 0) return PS_OK;
  if (!keys || !out) return fail(PS_ERR_INVALID, "keys or out is NULL");
  hipStream_t st = as_stream(stream);
  // rows of up to ROW_MAX floats in one pass; wider rows one column slice at a time
  for (int64_t col0 = 0; col0 < s->dim; col0 += ROW_MAX) {
    const int dim = (int)std::min<int64_t>(ROW_MAX, s->dim - col0);
    RowShape shape;
    row_shape(dim, aligned16(out) && s->dim % 4 == 0, &shape);
    ps_status r = with_shape(shape, [&]<int L, int NV, int VW>() -> ps_status {
      int64_t grid = ceil_div(n, BLOCK / L);
      if (grid > 65536) grid = 65536;
      Timed t(s, PS_KERNEL_PULL, st);
      if (s->bf16)
        hipLaunchKernelGGL((k_pull<L, NV, VW, bf16_t>), dim3(grid), dim3(BLOCK), 0, st,
                           reinterpret_cast<const bf16_t*>(s->W) + col0, s->ld, s->num_keys, dim, keys, n,
                           out + col0, (int64_t)s->dim, s->status, (const int32_t*)nullptr, int64_t(0));
      else
        hipLaunchKernelGGL((k_pull<L, NV, VW, float>), dim3(grid), dim3(BLOCK), 0, st, s->W + col0, s->ld,
                           s->num_keys, dim, keys, n, out + col0, (int64_t)s->dim, s->status,
                           s->stg ? s->stg->map : nullptr, s->stg ? s->stg->num_keys : int64_t(0));
      LAUNCHED(k_pull);
      return PS_OK;
    });
    if (r) return r;
  }
  return PS_OK;
}

// The push in two phases: the key work (intake, sort, segments; workspace
// only) and the merge of the gradient rows into the table.
static ps_status push_prepare(ps_store* s, const int64_t* keys, int64_t n, Plan& p, hipStream_t st) {
  uint32_t *ks, *perm;
  if (ps_status r = run_sort(s, KeysInt64{keys}, n, s->num_keys, p.sb, s->status, nullptr, false, st, &ks, &perm))
    return r;
  return run_segments(p.sb, ks, n, s->num_keys, p.sb.seg_off, nullptr, st);
}

static ps_status push_apply(ps_store* s, int64_t n, const float* grads, Plan& p, hipStream_t st) {
  const int passes = radix_plan(s->num_keys).passes;   // where the sort left keys and permutation
  const uint32_t* ks = p.sb.k[passes % 2];
  const uint32_t* perm = p.sb.v[passes % 2];
  if (s->dim <= ROW_MAX) return run_reduce(s, p.sb, ks, SrcIndirect{grads, perm, s->dim, s->dim}, n, {PART_ALL}, st);
  // a wide row: each column slice merged and updated on its own (per-element
  // AdaGrad and per-element sums do not mix columns, so this is the same
  // update); the segments are the sort's, the partials reused slice after
  // slice, the list of cut segments rebuilt by each slice's merge
  for (int64_t col0 = 0; col0 < s->dim; col0 += ROW_MAX) {
    const ColSlice cs{col0, (int)std::min<int64_t>(ROW_MAX, s->dim - col0)};
    if (col0 > 0) {
      hipLaunchKernelGGL(k_zero_words, dim3(1), dim3(BLOCK), 0, st, &p.sb.hdr->num_split, int64_t(1));
      LAUNCHED(k_zero_words);
    }
    if (ps_status r = launch_segreduce(s, p.sb, ks, SrcIndirect{grads + col0, perm, cs.dim, s->dim}, n, PART_ALL, st,
                                       PS_KERNEL_SEGREDUCE, 0, cs))
      return r;
    if (ps_status r = launch_finalize(s, p.sb, ks, n, st, LossTotal{nullptr, 0, nullptr}, cs)) return r;
  }
  return PS_OK;
}

static ps_status check_grads(const ps_store* s, const float* grads) {
  if (!grads) return fail(PS_ERR_INVALID, "grads is NULL");
  if (s->dim % 4 == 0 && !aligned16(grads)) return fail(PS_ERR_INVALID, "grads must be 16-byte aligned");
  return PS_OK;
}

static ps_status push_impl(ps_store* s, const int64_t* keys, int64_t n, const float* grads, void* ws, size_t ws_bytes,
                           void* stream) {
  if (ps_status st = check_store(s)) return st;
  if (ps_status st = check_n(n, 1)) return st;
  if (n == 0) return PS_OK;
  if (!keys) return fail(PS_ERR_INVALID, "keys is NULL");
  if (ps_status st = check_grads(s, grads)) return st;
  Plan p;
  plan_op(ws, s->num_keys, s->dim, PS_OP_PUSH, n, 1, &p);
  if (ps_status st = check_ws(p, ws, ws_bytes)) return st;
  hipStream_t st = as_stream(stream);
  if (ps_status r = push_prepare(s, keys, n, p, st)) return r;
  return push_apply(s, n, grads, p, st);
}

ps_status ps_push_prepare(ps_store* s, const int64_t* keys, int64_t n, void* ws, size_t ws_bytes, void* stream) {
  if (ps_status st = check_store(s)) return st;
  if (s->stg) return fail(PS_ERR_UNSUPPORTED, "the two-phase push is not available on a staged store");
  if (ps_status st = check_n(n, 1)) return st;
  if (n == 0) return PS_OK;
  if (!keys) return fail(PS_ERR_INVALID, "keys is NULL");
  Plan p;
  plan_op(ws, s->num_keys, s->dim, PS_OP_PUSH, n, 1, &p);
  if (ps_status st = check_ws(p, ws, ws_bytes)) return st;
  return push_prepare(s, keys, n, p, as_stream(stream));
}

ps_status ps_push_apply(ps_store* s, int64_t n, const float* grads, void* ws, size_t ws_bytes, void* stream) {
  if (ps_status st = check_store(s)) return st;
  if (s->stg) return fail(PS_ERR_UNSUPPORTED, "the two-phase push is not available on a staged store");
  if (ps_status st = check_n(n, 1)) return st;
  if (n == 0) return PS_OK;
  if (ps_status st = check_grads(s, grads)) return st;
  Plan p;
  plan_op(ws, s->num_keys, s->dim, PS_OP_PUSH, n, 1, &p);
  if (ps_status st = check_ws(p, ws, ws_bytes)) return st;
  return push_apply(s, n, grads, p, as_stream(stream));
}

ps_status ps_dedup(int64_t num_keys, const int64_t* keys, int64_t n, int64_t* uniq, int32_t* perm,
                   int32_t* offsets, int32_t* num_unique, int32_t* err, void* ws, size_t ws_bytes, void* stream) {
  if (num_keys < 1 || num_keys > INT32_MAX) return fail(PS_ERR_INVALID, "num_keys %lld outside [1, 2^31-1]", (long long)num_keys);
  if (ps_status st = check_n(n, 1)) return st;
  if (!offsets || !num_unique) return fail(PS_ERR_INVALID, "offsets or num_unique is NULL");
  hipStream_t st = as_stream(stream);
  if (n == 0) {
    hipLaunchKernelGGL(k_zero_words, dim3(1), dim3(BLOCK), 0, st, reinterpret_cast<uint32_t*>(offsets), int64_t(1));
    LAUNCHED(k_zero_words);
    hipLaunchKernelGGL(k_zero_words, dim3(1), dim3(BLOCK), 0, st, reinterpret_cast<uint32_t*>(num_unique), int64_t(1));
    LAUNCHED(k_zero_words);
    return PS_OK;
  }
  if (!keys || !uniq || !perm) return fail(PS_ERR_INVALID, "keys, uniq or perm is NULL");
  Plan p;
  plan_op(ws, num_keys, 1, PS_OP_DEDUP, n, 1, &p);
  if (ps_status r = check_ws(p, ws, ws_bytes)) return r;
  uint32_t *ks, *pm;
  if (ps_status r = run_sort(nullptr, KeysInt64{keys}, n, num_keys, p.sb, err, reinterpret_cast<uint32_t*>(perm),
                             false, st, &ks, &pm))
    return r;
  if (ps_status r = run_segments(p.sb, ks, n, num_keys, offsets, uniq, st)) return r;
  HIP_TRY(hipMemcpyAsync(num_unique, &p.sb.hdr->num_unique, sizeof(int32_t), hipMemcpyDeviceToDevice, st));
  return PS_OK;
}

static ps_status step_mf_impl(ps_store* s, const int32_t* row, const int32_t* col, const float* val, int64_t B,
                              int64_t col_key_offset, float lambda, double* loss, void* ws, size_t ws_bytes, void* stream) {
  if (ps_status st = check_store(s)) return st;
  if (ps_status st = check_row_width(s)) return st;
  if (ps_status st = check_n(B, 2)) return st;
  hipStream_t st = as_stream(stream);
  if (B == 0) return zero_loss(loss, st);
  if (!row || !col || !val) return fail(PS_ERR_INVALID, "row, col or val is NULL");
  if (col_key_offset < 0) return fail(PS_ERR_INVALID, "negative col_key_offset");
  Plan p;
  plan_op(ws, s->num_keys, s->dim, PS_OP_STEP_MF, B, 2, &p);
  if (ps_status r = check_ws(p, ws, ws_bytes)) return r;
  if (ps_status r = mf_prepare(s, row, col, val, B, col_key_offset, p, st)) return r;
  return mf_apply(s, B, lambda, loss, p, st);
}

ps_status ps_step_mf_prepare(ps_store* s, const int32_t* row, const int32_t* col, const float* val, int64_t B,
                             int64_t col_key_offset, void* ws, size_t ws_bytes, void* stream) {
  if (ps_status st = check_store(s)) return st;
  if (ps_status st = check_row_width(s)) return st;
  if (s->stg) return fail(PS_ERR_UNSUPPORTED, "the two-phase MF step is not available on a staged store");
  if (ps_status st = check_n(B, 2)) return st;
  if (B == 0) return PS_OK;
  if (!row || !col || !val) return fail(PS_ERR_INVALID, "row, col or val is NULL");
  if (col_key_offset < 0) return fail(PS_ERR_INVALID, "negative col_key_offset");
  Plan p;
  plan_op(ws, s->num_keys, s->dim, PS_OP_STEP_MF, B, 2, &p);
  if (ps_status r = check_ws(p, ws, ws_bytes)) return r;
  return mf_prepare(s, row, col, val, B, col_key_offset, p, as_stream(stream));
}

ps_status ps_step_mf_apply(ps_store* s, int64_t B, float lambda, double* loss, void* ws, size_t ws_bytes,
                           void* stream, void* rows_done) {
  if (ps_status st = check_store(s)) return st;
  if (ps_status st = check_row_width(s)) return st;
  if (s->stg) return fail(PS_ERR_UNSUPPORTED, "the two-phase MF step is not available on a staged store");
  if (ps_status st = check_n(B, 2)) return st;
  hipStream_t st = as_stream(stream);
  if (B == 0) return zero_loss(loss, st);
  Plan p;
  plan_op(ws, s->num_keys, s->dim, PS_OP_STEP_MF, B, 2, &p);
  if (ps_status r = check_ws(p, ws, ws_bytes)) return r;
  return mf_apply(s, B, lambda, loss, p, st, static_cast<hipEvent_t>(rows_done));
}

// Where the key sort of a workspace left the sorted keys and the
// permutation (no caller-owned permutation, so the sort's own buffers).
static void sorted_view(const ps_store* s, const Plan& p, const uint32_t** ks, const uint32_t** perm) {
  const int passes = radix_plan(s->num_keys).passes;
  *ks = p.sb.k[passes % 2];
  *perm = p.sb.v[passes % 2];
}

// The pieces of the ComplEx step: validity of the triples, the key work
// (sort and segments; workspace only), the gradient kernel (table reads,
// per-triple rows and per-negative coefficients) and the merge.
static ps_status check_kge(ps_store* s, int64_t B, int32_t n_neg, int32_t n_head_neg) {
  if (ps_status st = check_store(s)) return st;
  if (ps_status st = check_row_width(s)) return st;
  if (s->bf16) return fail(PS_ERR_UNSUPPORTED, "this step runs on fp32 values only (bf16 stores: pull, push, MF)");
  if (n_neg < 0 || n_head_neg < 0 || n_head_neg > n_neg)
    return fail(PS_ERR_INVALID, "need 0 <= n_head_neg <= n_neg");
  if (ps_status st = check_n(B, 3 + (int64_t)n_neg)) return st;
  if (s->dim % 2 != 0) return fail(PS_ERR_UNSUPPORTED, "ComplEx rows need an even dim");
  return PS_OK;
}

static ps_status check_kge_ids(const int32_t* head, const int32_t* rel, const int32_t* tail, const int32_t* neg,
                               int32_t n_neg, int64_t rel_key_offset) {
  if (!head || !rel || !tail || (n_neg > 0 && !neg)) return fail(PS_ERR_INVALID, "head, rel, tail or neg is NULL");
  if (rel_key_offset < 0) return fail(PS_ERR_INVALID, "negative rel_key_offset");
  return PS_OK;
}

static ps_status kge_keywork(ps_store* s, const int32_t* head, const int32_t* rel, const int32_t* tail,
                             const int32_t* neg, int64_t B, int32_t n_neg, int64_t rel_key_offset, Plan& p,
                             hipStream_t st) {
  const int per = 3 + n_neg;
  uint32_t *ks, *perm;
  KeysKGE kk{head, rel, tail, neg, per, n_neg, rel_key_offset, p.ok};
  if (ps_status r = run_sort(s, kk, B * per, s->num_keys, p.sb, s->status, nullptr, false, st, &ks, &perm, true))
    return r;
  return run_segments(p.sb, ks, B * per, s->num_keys, p.sb.seg_off, nullptr, st);
}

static ps_status kge_valid(ps_store* s, const int32_t* head, const int32_t* rel, const int32_t* tail,
                           const int32_t* neg, int64_t B, int32_t n_neg, int64_t rel_key_offset, Plan& p,
                           hipStream_t st) {
  hipLaunchKernelGGL(k_unit_valid<ValidKGE>, dim3(small_grid(B, WAVES_PER_BLOCK, 4096)), dim3(BLOCK), 0, st,
                     ValidKGE{head, rel, tail, neg, n_neg, rel_key_offset, s->num_keys}, B, p.ok, s->status,
                     reinterpret_cast<uint32_t*>(p.sb.hdr), header_words(p.sb));
  LAUNCHED(k_unit_valid);
  return PS_OK;
}

// Launches the gradient kernel; *grid receives its number of loss partials.
static ps_status kge_grad(ps_store* s, const int32_t* head, const int32_t* rel, const int32_t* tail,
                          const int32_t* neg, int64_t B, int32_t n_neg, int32_t n_head_neg, int64_t rel_key_offset,
                          Plan& p, hipStream_t st, int64_t* grid) {
  const int cdim = s->dim / 2;
  *grid = small_grid(B, WAVES_PER_BLOCK, LOSS_GRID);
  auto launch = [&](auto kernel) -> ps_status {
    Timed t(s, PS_KERNEL_TASKGRAD, st);
    hipLaunchKernelGGL(kernel, dim3(*grid), dim3(BLOCK), 0, st, s->W, s->ld, s->dim, head, rel, tail, neg, B, n_neg,
                       n_head_neg, rel_key_offset, p.ok, p.mat, p.base, p.coef, p.loss_part);
    LAUNCHED(k_kge_grad);
    return PS_OK;
  };
  if (cdim <= 64) return launch(k_kge_grad<1>);
  if (cdim <= 128) return launch(k_kge_grad<2>);
  return launch(k_kge_grad<4>);   // cdim <= 256: the store holds rows of at most 512 floats
}

static ps_status kge_merge(ps_store* s, int64_t B, int32_t n_neg, int32_t n_head_neg, double* loss, Plan& p,
                           hipStream_t st, int64_t grid) {
  const uint32_t *ks, *perm;
  sorted_view(s, p, &ks, &perm);
  const int per = 3 + n_neg;
  return run_reduce(s, p.sb, ks, SrcKGE{perm, p.mat, p.base, p.coef, per, n_head_neg, s->dim}, B * per, {PART_ALL},
                    st, LossTotal{p.loss_part, grid, loss});
}

static ps_status step_kge_impl(ps_store* s, const int32_t* head, const int32_t* rel, const int32_t* tail, const int32_t* neg,
                               int64_t B, int32_t n_neg, int32_t n_head_neg, int64_t rel_key_offset, double* loss, void* ws,
                               size_t ws_bytes, void* stream) {
  if (ps_status st = check_kge(s, B, n_neg, n_head_neg)) return st;
  hipStream_t st = as_stream(stream);
  if (B == 0) return zero_loss(loss, st);
  if (ps_status r = check_kge_ids(head, rel, tail, neg, n_neg, rel_key_offset)) return r;
  Plan p;
  plan_op(ws, s->num_keys, s->dim, PS_OP_STEP_KGE, B, 3 + n_neg, &p);
  if (ps_status r = check_ws(p, ws, ws_bytes)) return r;
  if (ps_status r = kge_valid(s, head, rel, tail, neg, B, n_neg, rel_key_offset, p, st)) return r;
  // the key sort and segments (workspace only) run on the second stream
  // beside the gradient kernel (table reads, per-unit rows)
  if (ps_status r = fork_aux(s, st)) return r;
  if (ps_status r = kge_keywork(s, head, rel, tail, neg, B, n_neg, rel_key_offset, p, s->aux)) return r;
  int64_t grid = 0;
  if (ps_status r = kge_grad(s, head, rel, tail, neg, B, n_neg, n_head_neg, rel_key_offset, p, st, &grid)) return r;
  if (ps_status r = join_aux(s, st)) return r;
  return kge_merge(s, B, n_neg, n_head_neg, loss, p, st, grid);
}

ps_status ps_step_kge_prepare(ps_store* s, const int32_t* head, const int32_t* rel, const int32_t* tail,
                              const int32_t* neg, int64_t B, int32_t n_neg, int64_t rel_key_offset, void* ws,
                              size_t ws_bytes, void* stream) {
  if (ps_status st = check_store(s)) return st;
  if (s->stg) return fail(PS_ERR_UNSUPPORTED, "the two-phase ComplEx step is not available on a staged store");
  if (ps_status st = check_kge(s, B, n_neg, 0)) return st;
  if (B == 0) return PS_OK;
  if (ps_status r = check_kge_ids(head, rel, tail, neg, n_neg, rel_key_offset)) return r;
  Plan p;
  plan_op(ws, s->num_keys, s->dim, PS_OP_STEP_KGE, B, 3 + n_neg, &p);
  if (ps_status r = check_ws(p, ws, ws_bytes)) return r;
  hipStream_t st = as_stream(stream);
  if (ps_status r = kge_valid(s, head, rel, tail, neg, B, n_neg, rel_key_offset, p, st)) return r;
  return kge_keywork(s, head, rel, tail, neg, B, n_neg, rel_key_offset, p, st);
}

ps_status ps_step_kge_apply(ps_store* s, const int32_t* head, const int32_t* rel, const int32_t* tail,
                            const int32_t* neg, int64_t B, int32_t n_neg, int32_t n_head_neg, int64_t rel_key_offset,
                            double* loss, void* ws, size_t ws_bytes, void* stream) {
  if (ps_status st = check_store(s)) return st;
  if (s->stg) return fail(PS_ERR_UNSUPPORTED, "the two-phase ComplEx step is not available on a staged store");
  if (ps_status st = check_kge(s, B, n_neg, n_head_neg)) return st;
  hipStream_t st = as_stream(stream);
  if (B == 0) return zero_loss(loss, st);
  if (ps_status r = check_kge_ids(head, rel, tail, neg, n_neg, rel_key_offset)) return r;
  Plan p;
  plan_op(ws, s->num_keys, s->dim, PS_OP_STEP_KGE, B, 3 + n_neg, &p);
  if (ps_status r = check_ws(p, ws, ws_bytes)) return r;
  int64_t grid = 0;
  if (ps_status r = kge_grad(s, head, rel, tail, neg, B, n_neg, n_head_neg, rel_key_offset, p, st, &grid)) return r;
  return kge_merge(s, B, n_neg, n_head_neg, loss, p, st, grid);
}

// The pieces of the skip-gram step, as for ComplEx.
static ps_status check_sgns(ps_store* s, int64_t B, int32_t window, int32_t n_neg, int64_t out_key_offset) {
  if (ps_status st = check_store(s)) return st;
  if (ps_status st = check_row_width(s)) return st;
  if (s->bf16) return fail(PS_ERR_UNSUPPORTED, "this step runs on fp32 values only (bf16 stores: pull, push, MF)");
  if (window < 0 || n_neg < 0) return fail(PS_ERR_INVALID, "negative window or n_neg");
  if (ps_status st = check_n(B, 1 + 2 * (int64_t)window * (1 + (int64_t)n_neg))) return st;
  if (out_key_offset < 1 || out_key_offset >= s->num_keys)
    return fail(PS_ERR_INVALID, "out_key_offset must split the table into input and output rows");
  return PS_OK;
}

static ps_status check_sgns_ids(const int32_t* centre, const int32_t* ctx, const int32_t* neg, int32_t window,
                                int32_t n_neg) {
  if (!centre || (window > 0 && !ctx) || (window > 0 && n_neg > 0 && !neg))
    return fail(PS_ERR_INVALID, "centre, ctx or neg is NULL");
  return PS_OK;
}

static ps_status sgns_valid(ps_store* s, const int32_t* centre, const int32_t* ctx, const int32_t* neg, int64_t B,
                            int32_t window, int32_t n_neg, int64_t out_key_offset, Plan& p, hipStream_t st) {
  hipLaunchKernelGGL(k_unit_valid<ValidSGNS>, dim3(small_grid(B, WAVES_PER_BLOCK, 4096)), dim3(BLOCK), 0, st,
                     ValidSGNS{centre, ctx, neg, 2 * window, n_neg, out_key_offset, s->num_keys}, B, p.ok, s->status,
                     reinterpret_cast<uint32_t*>(p.sb.hdr), header_words(p.sb));
  LAUNCHED(k_unit_valid);
  return PS_OK;
}

static ps_status sgns_keywork(ps_store* s, const int32_t* centre, const int32_t* ctx, const int32_t* neg, int64_t B,
                              int32_t window, int32_t n_neg, int64_t out_key_offset, Plan& p, hipStream_t st) {
  const int slots = 2 * window;
  const int64_t per = 1 + (int64_t)slots * (1 + n_neg);
  uint32_t *ks, *perm;
  KeysSGNS kk{centre, ctx, neg, (int)per, slots, n_neg, out_key_offset, p.ok};
  if (ps_status r = run_sort(s, kk, B * per, s->num_keys, p.sb, s->status, nullptr, false, st, &ks, &perm, true))
    return r;
  return run_segments(p.sb, ks, B * per, s->num_keys, p.sb.seg_off, nullptr, st, (uint32_t)out_key_offset);
}

// Launches the gradient kernel; *grid receives its number of loss partials.
static ps_status sgns_grad(ps_store* s, const int32_t* centre, const int32_t* ctx, const int32_t* neg, int64_t B,
                           int32_t window, int32_t n_neg, int64_t out_key_offset, Plan& p, hipStream_t st,
                           int64_t* grid) {
  const int slots = 2 * window;
  return with_sgns_shape(s->dim, s->ld, [&]<int L, int NV, int VW>() -> ps_status {
    *grid = small_grid(B, BLOCK / L, LOSS_GRID);
    {
      Timed t(s, PS_KERNEL_TASKGRAD, st);
      hipLaunchKernelGGL((k_sgns_grad<L, NV, VW>), dim3(*grid), dim3(BLOCK), 0, st, s->W, s->ld, s->dim, centre, ctx,
                         neg, B, slots, n_neg, out_key_offset, p.ok, p.mat, p.coef, p.loss_part);
    }
    LAUNCHED(k_sgns_grad);
    return PS_OK;
  });
}

static ps_status sgns_merge(ps_store* s, const int32_t* centre, int64_t B, int32_t window, int32_t n_neg,
                            double* loss, Plan& p, hipStream_t st, int64_t grid) {
  const uint32_t *ks, *perm;
  sorted_view(s, p, &ks, &perm);
  const int64_t per = 1 + 2 * (int64_t)window * (1 + n_neg);
  // output rows first: their gradients read the input rows, which are updated second
  SrcSGNS src{perm, p.mat, p.coef, centre, s->W, s->ld, (int)per, s->dim};
  return run_reduce(s, p.sb, ks, src, B * per, {PART_UPPER, PART_LOWER}, st, LossTotal{p.loss_part, grid, loss});
}

static ps_status step_sgns_impl(ps_store* s, const int32_t* centre, const int32_t* ctx, const int32_t* neg, int64_t B,
                                int32_t window, int32_t n_neg, int64_t out_key_offset, double* loss, void* ws,
                                size_t ws_bytes, void* stream) {
  if (ps_status st = check_sgns(s, B, window, n_neg, out_key_offset)) return st;
  hipStream_t st = as_stream(stream);
  if (B == 0) return zero_loss(loss, st);
  if (ps_status r = check_sgns_ids(centre, ctx, neg, window, n_neg)) return r;
  const int64_t per = 1 + 2 * (int64_t)window * (1 + n_neg);
  Plan p;
  plan_op(ws, s->num_keys, s->dim, PS_OP_STEP_SGNS, B, per, &p);
  if (ps_status r = check_ws(p, ws, ws_bytes)) return r;
  if (ps_status r = sgns_valid(s, centre, ctx, neg, B, window, n_neg, out_key_offset, p, st)) return r;
  // the key sort and segments (workspace only) run on the second stream
  // beside the gradient kernel (table reads, per-unit rows)
  if (ps_status r = fork_aux(s, st)) return r;
  if (ps_status r = sgns_keywork(s, centre, ctx, neg, B, window, n_neg, out_key_offset, p, s->aux)) return r;
  int64_t grid = 0;
  if (ps_status r = sgns_grad(s, centre, ctx, neg, B, window, n_neg, out_key_offset, p, st, &grid)) return r;
  if (ps_status r = join_aux(s, st)) return r;
  return sgns_merge(s, centre, B, window, n_neg, loss, p, st, grid);
}

ps_status ps_step_sgns_prepare(ps_store* s, const int32_t* centre, const int32_t* ctx, const int32_t* neg, int64_t B,
                               int32_t window, int32_t n_neg, int64_t out_key_offset, void* ws, size_t ws_bytes,
                               void* stream) {
  if (ps_status st = check_store(s)) return st;
  if (s->stg) return fail(PS_ERR_UNSUPPORTED, "the two-phase skip-gram step is not available on a staged store");
  if (ps_status st = check_sgns(s, B, window, n_neg, out_key_offset)) return st;
  if (B == 0) return PS_OK;
  if (ps_status r = check_sgns_ids(centre, ctx, neg, window, n_neg)) return r;
  Plan p;
  plan_op(ws, s->num_keys, s->dim, PS_OP_STEP_SGNS, B, 1 + 2 * (int64_t)window * (1 + n_neg), &p);
  if (ps_status r = check_ws(p, ws, ws_bytes)) return r;
  hipStream_t st = as_stream(stream);
  if (ps_status r = sgns_valid(s, centre, ctx, neg, B, window, n_neg, out_key_offset, p, st)) return r;
  return sgns_keywork(s, centre, ctx, neg, B, window, n_neg, out_key_offset, p, st);
}

ps_status ps_step_sgns_apply(ps_store* s, const int32_t* centre, const int32_t* ctx, const int32_t* neg, int64_t B,
                             int32_t window, int32_t n_neg, int64_t out_key_offset, double* loss, void* ws,
                             size_t ws_bytes, void* stream) {
  if (ps_status st = check_store(s)) return st;
  if (s->stg) return fail(PS_ERR_UNSUPPORTED, "the two-phase skip-gram step is not available on a staged store");
  if (ps_status st = check_sgns(s, B, window, n_neg, out_key_offset)) return st;
  hipStream_t st = as_stream(stream);
  if (B == 0) return zero_loss(loss, st);
  if (ps_status r = check_sgns_ids(centre, ctx, neg, window, n_neg)) return r;
  Plan p;
  plan_op(ws, s->num_keys, s->dim, PS_OP_STEP_SGNS, B, 1 + 2 * (int64_t)window * (1 + n_neg), &p);
  if (ps_status r = check_ws(p, ws, ws_bytes)) return r;
  int64_t grid = 0;
  if (ps_status r = sgns_grad(s, centre, ctx, neg, B, window, n_neg, out_key_offset, p, st, &grid)) return r;
  return sgns_merge(s, centre, B, window, n_neg, loss, p, st, grid);
}

// The pieces of the CTR step: the key work (sort and segments; workspace
// only), the gradient kernel (table reads, gradient rows in occurrence order)
// and the merge of those rows.
static ps_status ctr_keywork(ps_store* s, const int64_t* keys, int64_t B, int32_t F, Plan& p, hipStream_t st) {
  uint32_t *ks, *perm;
  if (ps_status r = run_sort(s, KeysCTR{keys, F, p.ok}, B * F, s->num_keys, p.sb, s->status, nullptr, false, st, &ks,
                             &perm, true))
    return r;
  return run_segments(p.sb, ks, B * F, s->num_keys, p.sb.seg_off, nullptr, st);
}

static ps_status ctr_valid(ps_store* s, const int64_t* keys, int64_t B, int32_t F, Plan& p, hipStream_t st) {
  hipLaunchKernelGGL(k_unit_valid<ValidCTR>, dim3(small_grid(B, WAVES_PER_BLOCK, 4096)), dim3(BLOCK), 0, st,
                     ValidCTR{keys, F, s->num_keys}, B, p.ok, s->status, reinterpret_cast<uint32_t*>(p.sb.hdr),
                     header_words(p.sb));
  LAUNCHED(k_unit_valid);
  return PS_OK;
}

// Launches the gradient kernel; *grid receives its number of loss partials.
static ps_status ctr_grad(ps_store* s, const int64_t* keys, const float* label, int64_t B, int32_t F, Plan& p,
                          hipStream_t st, int64_t* grid) {
  RowShape shape;
  row_shape(s->dim, true, &shape);
  return with_shape(shape, [&]<int L, int NV, int VW>() -> ps_status {
    *grid = small_grid(B, BLOCK / L, LOSS_GRID);
    {
      Timed t(s, PS_KERNEL_TASKGRAD, st);
      hipLaunchKernelGGL((k_ctr_grad<L, NV, VW>), dim3(*grid), dim3(BLOCK), 0, st, s->W, s->ld, s->dim, keys, label, B,
                         F, p.ok, p.grads, p.loss_part);
    }
    LAUNCHED(k_ctr_grad);
    return PS_OK;
  });
}

static ps_status ctr_merge(ps_store* s, int64_t B, int32_t F, double* loss, Plan& p, hipStream_t st, int64_t grid) {
  const uint32_t *ks, *perm;
  sorted_view(s, p, &ks, &perm);
  return run_reduce(s, p.sb, ks, SrcIndirect{p.grads, perm, s->dim, s->dim}, B * F, {PART_ALL}, st,
                    LossTotal{p.loss_part, grid, loss});
}

static ps_status check_ctr(ps_store* s, int64_t B, int32_t F) {
  if (ps_status st = check_store(s)) return st;
  if (ps_status st = check_row_width(s)) return st;
  if (s->bf16) return fail(PS_ERR_UNSUPPORTED, "this step runs on fp32 values only (bf16 stores: pull, push, MF)");
  if (F < 1) return fail(PS_ERR_INVALID, "need F >= 1");
  return check_n(B, F);
}

static ps_status step_ctr_impl(ps_store* s, const int64_t* keys, const float* label, int64_t B, int32_t F, double* loss,
                               void* ws, size_t ws_bytes, void* stream) {
  if (ps_status st = check_ctr(s, B, F)) return st;
  hipStream_t st = as_stream(stream);
  if (B == 0) return zero_loss(loss, st);
  if (!keys || !label) return fail(PS_ERR_INVALID, "keys or label is NULL");
  Plan p;
  plan_op(ws, s->num_keys, s->dim, PS_OP_STEP_CTR, B, F, &p);
  if (ps_status r = check_ws(p, ws, ws_bytes)) return r;
  if (ps_status r = ctr_valid(s, keys, B, F, p, st)) return r;
  // the key sort and segments (workspace only) run on the second stream
  // beside the gradient kernel
  if (ps_status r = fork_aux(s, st)) return r;
  if (ps_status r = ctr_keywork(s, keys, B, F, p, s->aux)) return r;
  int64_t grid = 0;
  if (ps_status r = ctr_grad(s, keys, label, B, F, p, st, &grid)) return r;
  if (ps_status r = join_aux(s, st)) return r;
  return ctr_merge(s, B, F, loss, p, st, grid);
}

ps_status ps_step_ctr_prepare(ps_store* s, const int64_t* keys, int64_t B, int32_t F, void* ws, size_t ws_bytes,
                              void* stream) {
  if (ps_status st = check_store(s)) return st;
  if (s->stg) return fail(PS_ERR_UNSUPPORTED, "the two-phase CTR step is not available on a staged store");
  if (ps_status st = check_ctr(s, B, F)) return st;
  if (B == 0) return PS_OK;
  if (!keys) return fail(PS_ERR_INVALID, "keys is NULL");
  Plan p;
  plan_op(ws, s->num_keys, s->dim, PS_OP_STEP_CTR, B, F, &p);
  if (ps_status r = check_ws(p, ws, ws_bytes)) return r;
  hipStream_t st = as_stream(stream);
  if (ps_status r = ctr_valid(s, keys, B, F, p, st)) return r;
  return ctr_keywork(s, keys, B, F, p, st);
}

ps_status ps_step_ctr_apply(ps_store* s, const int64_t* keys, const float* label, int64_t B, int32_t F, double* loss,
                            void* ws, size_t ws_bytes, void* stream) {
  if (ps_status st = check_store(s)) return st;
  if (s->stg) return fail(PS_ERR_UNSUPPORTED, "the two-phase CTR step is not available on a staged store");
  if (ps_status st = check_ctr(s, B, F)) return st;
  hipStream_t st = as_stream(stream);
  if (B == 0) return zero_loss(loss, st);
  if (!keys || !label) return fail(PS_ERR_INVALID, "keys or label is NULL");
  Plan p;
  plan_op(ws, s->num_keys, s->dim, PS_OP_STEP_CTR, B, F, &p);
  if (ps_status r = check_ws(p, ws, ws_bytes)) return r;
  int64_t grid = 0;
  if (ps_status r = ctr_grad(s, keys, label, B, F, p, st, &grid)) return r;
  return ctr_merge(s, B, F, loss, p, st, grid);
}

// ---------------------------------------------------------------- public steps
// A staged store translates the call's ids into slot ids (the plan's
// translation region of the workspace) and runs the same step on its slot
// table.
ps_status ps_push(ps_store* s, const int64_t* keys, int64_t n, const float* grads, void* ws, size_t ws_bytes,
                  void* stream) {
  if (ps_status st = check_store(s)) return st;
  if (!s->stg || n <= 0 || !keys) return push_impl(s, keys, n, grads, ws, ws_bytes, stream);
  if (ps_status st = check_n(n, 1)) return st;
  Plan p;
  plan_op(ws, s->num_keys, s->dim, PS_OP_PUSH, n, 1, &p);
  if (ps_status r = check_ws(p, ws, ws_bytes)) return r;
  char* t = p.trans;
  int64_t* tk = reinterpret_cast<int64_t*>(t);
  if (ps_status r = translate_keys(s, keys, n, tk, as_stream(stream))) return r;
  return push_impl(s, tk, n, grads, ws, ws_bytes, stream);
}

ps_status ps_push_noalloc(ps_store* s, const int64_t* keys, int64_t n, const float* grads, void* stream) {
  if (ps_status st = check_store(s)) return st;
  if (ps_status st = check_n(n, 1)) return st;
  if (n == 0) return PS_OK;
  const size_t need = ps_workspace_bytes(s->num_keys, s->dim, PS_OP_PUSH, n, 1);
  if (need == 0 || need > PS_NOALLOC_SCRATCH_BYTES)
    return fail(PS_ERR_UNSUPPORTED, "a push of %lld keys of dim %d needs %zu bytes of scratch, the static scratch holds %zu",
                (long long)n, s->dim, need, (size_t)PS_NOALLOC_SCRATCH_BYTES);
  if (!s->scratch) return fail(PS_ERR_DEVICE, "no scratch address for the store's device");
  return ps_push(s, keys, n, grads, s->scratch, PS_NOALLOC_SCRATCH_BYTES, stream);
}

// ------------------------------------------------------------------ unmerged (asynchronous) updates
ps_status ps_push_async(ps_store* s, const int64_t* keys, int64_t n, const float* grads, void* stream) {
  if (ps_status st = check_store(s)) return st;
  if (ps_status st = check_row_width(s)) return st;
  if (ps_status st = check_async(s)) return st;
  if (ps_status st = check_n(n, 1)) return st;
  if (n == 0) return PS_OK;
  if (!keys || !grads) return fail(PS_ERR_INVALID, "keys or grads is NULL");
  return launch_push_async(s, KeysList{keys}, grads, n, as_stream(stream));
}

ps_status ps_step_mf_async(ps_store* s, const int32_t* row, const int32_t* col, const float* val, int64_t B,
                           int64_t col_key_offset, float lambda, double* loss, void* ws, size_t ws_bytes,
                           void* stream) {
  if (ps_status st = check_store(s)) return st;
  if (ps_status st = check_row_width(s)) return st;
  if (ps_status st = check_async(s)) return st;
  if (ps_status st = check_n(B, 2)) return st;
  hipStream_t st = as_stream(stream);
  if (B == 0) return zero_loss(loss, st);
  if (!row || !col || !val) return fail(PS_ERR_INVALID, "row, col or val is NULL");
  if (col_key_offset < 0) return fail(PS_ERR_INVALID, "negative col_key_offset");
  Plan p;
  plan_op(ws, s->num_keys, s->dim, PS_OP_STEP_MF_ASYNC, B, 2, &p);
  if (ps_status r = check_ws(p, ws, ws_bytes)) return r;
  RowShape shape;
  if (!row_shape(s->dim, true, &shape)) return fail(PS_ERR_UNSUPPORTED, "dim %d not supported", s->dim);
  const int64_t grid = small_grid(B, BLOCK / shape.L, LOSS_GRID);
  ps_status r = with_shape(shape, [&]<int L, int NV, int VW>() -> ps_status {
    Timed t(s, PS_KERNEL_TASKGRAD, st);
    hipLaunchKernelGGL((k_mf_grad_rows<L, NV, VW>), dim3(grid), dim3(BLOCK), 0, st, s->W, s->ld, s->dim, row, col,
                       val, B, col_key_offset, s->num_keys, (double)lambda, p.grads, p.loss_part);
    LAUNCHED(k_mf_grad_rows);
    return PS_OK;
  });
  if (r) return r;
  if (loss) {
    hipLaunchKernelGGL(k_sum_loss, dim3(1), dim3(BLOCK), 0, st, LossTotal{p.loss_part, grid, loss});
    LAUNCHED(k_sum_loss);
  }
  return launch_push_async(s, KeysMF{row, col, col_key_offset, s->num_keys}, p.grads, 2 * B, st);
}

ps_status ps_step_mf(ps_store* s, const int32_t* row, const int32_t* col, const float* val, int64_t B,
                     int64_t col_key_offset, float lambda, double* loss, void* ws, size_t ws_bytes, void* stream) {
  if (ps_status st = check_store(s)) return st;
  if (!s->stg || B <= 0 || !row || !col || col_key_offset < 0)
    return step_mf_impl(s, row, col, val, B, col_key_offset, lambda, loss, ws, ws_bytes, stream);
  if (ps_status st = check_n(B, 2)) return st;
  int64_t off;
  if (ps_status r = slot_offset(s, col_key_offset, "col_key_offset", &off)) return r;
  Plan p;
  plan_op(ws, s->num_keys, s->dim, PS_OP_STEP_MF, B, 2, &p);
  if (ps_status r = check_ws(p, ws, ws_bytes)) return r;
  char* t = p.trans;
  int32_t* tr = reinterpret_cast<int32_t*>(t);
  int32_t* tc = tr + B;
  hipStream_t st = as_stream(stream);
  if (ps_status r = translate_ids(s, row, B, 0, 0, tr, st)) return r;
  if (ps_status r = translate_ids(s, col, B, col_key_offset, off, tc, st)) return r;
  return step_mf_impl(s, tr, tc, val, B, off, lambda, loss, ws, ws_bytes, stream);
}

ps_status ps_step_kge(ps_store* s, const int32_t* head, const int32_t* rel, const int32_t* tail, const int32_t* neg,
                      int64_t B, int32_t n_neg, int32_t n_head_neg, int64_t rel_key_offset, double* loss, void* ws,
                      size_t ws_bytes, void* stream) {
  if (ps_status st = check_store(s)) return st;
  if (!s->stg || B <= 0 || !head || !rel || !tail || (n_neg > 0 && !neg) || n_neg < 0 || rel_key_offset < 0)
    return step_kge_impl(s, head, rel, tail, neg, B, n_neg, n_head_neg, rel_key_offset, loss, ws, ws_bytes, stream);
  if (ps_status st = check_n(B, 3 + (int64_t)n_neg)) return st;
  int64_t off;
  if (ps_status r = slot_offset(s, rel_key_offset, "rel_key_offset", &off)) return r;
  const int64_t per = 3 + (int64_t)n_neg;
  Plan p;
  plan_op(ws, s->num_keys, s->dim, PS_OP_STEP_KGE, B, per, &p);
  if (ps_status r = check_ws(p, ws, ws_bytes)) return r;
  char* t = p.trans;
  int32_t* th = reinterpret_cast<int32_t*>(t);
  int32_t* tt = th + B;
  int32_t* trl = tt + B;
  int32_t* tn = trl + B;
  hipStream_t st = as_stream(stream);
  if (ps_status r = translate_ids(s, head, B, 0, 0, th, st)) return r;
  if (ps_status r = translate_ids(s, tail, B, 0, 0, tt, st)) return r;
  if (ps_status r = translate_ids(s, rel, B, rel_key_offset, off, trl, st)) return r;
  if (ps_status r = translate_ids(s, neg, B * n_neg, 0, 0, tn, st)) return r;
  return step_kge_impl(s, th, trl, tt, n_neg > 0 ? tn : neg, B, n_neg, n_head_neg, off, loss, ws, ws_bytes, stream);
}

ps_status ps_step_sgns(ps_store* s, const int32_t* centre, const int32_t* ctx, const int32_t* neg, int64_t B,
                       int32_t window, int32_t n_neg, int64_t out_key_offset, double* loss, void* ws,
                       size_t ws_bytes, void* stream) {
  if (ps_status st = check_store(s)) return st;
  const int64_t slots = 2 * (int64_t)window;
  if (!s->stg || B <= 0 || !centre || window < 0 || n_neg < 0 || (slots > 0 && !ctx) ||
      (slots > 0 && n_neg > 0 && !neg))
    return step_sgns_impl(s, centre, ctx, neg, B, window, n_neg, out_key_offset, loss, ws, ws_bytes, stream);
  const int64_t per = 1 + slots * (1 + (int64_t)n_neg);
  if (ps_status st = check_n(B, per)) return st;
  int64_t off;
  if (ps_status r = slot_offset(s, out_key_offset, "out_key_offset", &off)) return r;
  Plan p;
  plan_op(ws, s->num_keys, s->dim, PS_OP_STEP_SGNS, B, per, &p);
  if (ps_status r = check_ws(p, ws, ws_bytes)) return r;
  char* t = p.trans;
  int32_t* tce = reinterpret_cast<int32_t*>(t);
  int32_t* tcx = tce + B;
  int32_t* tn = tcx + B * slots;
  hipStream_t st = as_stream(stream);
  if (ps_status r = translate_ids(s, centre, B, 0, 0, tce, st)) return r;
  if (ps_status r = translate_ids(s, ctx, B * slots, out_key_offset, off, tcx, st)) return r;
  if (ps_status r = translate_ids(s, neg, B * slots * n_neg, out_key_offset, off, tn, st)) return r;
  return step_sgns_impl(s, tce, slots > 0 ? tcx : ctx, (slots > 0 && n_neg > 0) ? tn : neg, B, window, n_neg, off,
                        loss, ws, ws_bytes, stream);
}

ps_status ps_step_ctr(ps_store* s, const int64_t* keys, const float* label, int64_t B, int32_t F, double* loss,
                      void* ws, size_t ws_bytes, void* stream) {
  if (ps_status st = check_store(s)) return st;
  if (!s->stg || B <= 0 || F < 1 || !keys) return step_ctr_impl(s, keys, label, B, F, loss, ws, ws_bytes, stream);
  if (ps_status st = check_n(B, F)) return st;
  Plan p;
  plan_op(ws, s->num_keys, s->dim, PS_OP_STEP_CTR, B, F, &p);
  if (ps_status r = check_ws(p, ws, ws_bytes)) return r;
  char* t = p.trans;
  int64_t* tk = reinterpret_cast<int64_t*>(t);
  if (ps_status r = translate_keys(s, keys, B * F, tk, as_stream(stream))) return r;
  return step_ctr_impl(s, tk, label, B, F, loss, ws, ws_bytes, stream);
}

// ---------------------------------------------------------------- Wide & Deep CTR
size_t ps_ctr_wd_workspace_bytes(int64_t num_keys, int32_t dim, int64_t B, int32_t F, int32_t emb_dim,
                                 int32_t n_hidden, const int32_t* hidden) {
  if (num_keys < 1 || dim < 1 || B < 0 || F < 1 || emb_dim < 1 || emb_dim >= dim || n_hidden < 0 ||
      n_hidden > WD_MAX_HIDDEN || (n_hidden > 0 && !hidden))
    return 0;
  for (int l = 0; l < n_hidden; ++l)
    if (hidden[l] < 1) return 0;
  if (B > MAX_OCC / F) return 0;
  PlanWD p;
  plan_wd(nullptr, dim, B, F, emb_dim, n_hidden, hidden, &p);
  return p.base.bytes;
}

ps_status ps_step_ctr_wd(ps_store* s, const int64_t* keys, const float* label, int64_t B, int32_t F, int32_t emb_dim,
                         int32_t n_hidden, const int32_t* hidden, float* dense, float* dense_accum, double* loss,
                         void* ws, size_t ws_bytes, void* stream) {
  if (ps_status st = check_store(s)) return st;
  if (ps_status st = check_row_width(s)) return st;
  if (s->bf16) return fail(PS_ERR_UNSUPPORTED, "this step runs on fp32 values only (bf16 stores: pull, push, MF)");
  if (F < 1) return fail(PS_ERR_INVALID, "need F >= 1");
  if (emb_dim < 1 || emb_dim >= s->dim) return fail(PS_ERR_INVALID, "need 1 <= emb_dim < dim (the row holds the wide weight)");
  if (n_hidden < 0 || n_hidden > WD_MAX_HIDDEN || (n_hidden > 0 && !hidden))
    return fail(PS_ERR_INVALID, "need 0 <= n_hidden <= %d hidden widths", WD_MAX_HIDDEN);
  for (int l = 0; l < n_hidden; ++l)
    if (hidden[l] < 1) return fail(PS_ERR_INVALID, "hidden width %d < 1", hidden[l]);
  if (ps_status st = check_n(B, F)) return st;
  hipStream_t st = as_stream(stream);
  if (B == 0) return zero_loss(loss, st);
  if (!keys || !label || !dense || !dense_accum) return fail(PS_ERR_INVALID, "keys, label or a dense buffer is NULL");
  const int L = n_hidden;
  const int E = emb_dim;
  const int64_t K0 = (int64_t)F * E;
  const int64_t n = B * F;
  PlanWD p;
  plan_wd(ws, s->dim, B, F, E, L, hidden, &p);
  if (ps_status r = check_ws(p.base, ws, ws_bytes)) return r;
  const DenseLayout d = dense_layout(K0, L, hidden);
  if (s->stg) {
    int64_t* tk = reinterpret_cast<int64_t*>(p.base.trans);
    if (ps_status r = translate_keys(s, keys, n, tk, st)) return r;
    keys = tk;
  }
  hipLaunchKernelGGL(k_unit_valid<ValidCTR>, dim3(small_grid(B, WAVES_PER_BLOCK, 4096)), dim3(BLOCK), 0, st,
                     ValidCTR{keys, F, s->num_keys}, B, p.base.ok, s->status,
                     reinterpret_cast<uint32_t*>(p.base.sb.hdr), header_words(p.base.sb));
  LAUNCHED(k_unit_valid);
  // the key sort and segments run beside the MLP on the store's second stream
  if (ps_status r = fork_aux(s, st)) return r;
  uint32_t *ks, *perm;
  if (ps_status r = run_sort(s, KeysCTR{keys, F, p.base.ok}, n, s->num_keys, p.base.sb, s->status, nullptr, true,
                             s->aux, &ks, &perm, true))
    return r;
  if (ps_status r = run_segments(p.base.sb, ks, n, s->num_keys, p.base.sb.seg_off, nullptr, s->aux)) return r;
  // inputs
  RowShape shape;
  row_shape(E, E % 4 == 0 && s->ld % 4 == 0, &shape);
  if (ps_status r = with_shape(shape, [&]<int Lw, int NV, int VW>() -> ps_status {
        hipLaunchKernelGGL((k_wd_gather<Lw, NV, VW>), dim3(small_grid(n, BLOCK / Lw, 16384)), dim3(BLOCK), 0, st, s->W,
                           s->ld, keys, B, F, E, p.base.ok, p.X);
        LAUNCHED(k_wd_gather);
        return PS_OK;
      }))
    return r;
  // forward
  const double* h = p.X;
  int64_t fan = K0;
  for (int l = 0; l < L; ++l) {
    if (ps_status r = gemm<false, false, float>(s, B, hidden[l], fan, h, fan, dense + d.offW[l], hidden[l], p.H[l],
                                                hidden[l], st))
      return r;
    hipLaunchKernelGGL(k_bias_relu, dim3(small_grid(B * hidden[l], BLOCK, 8192)), dim3(BLOCK), 0, st, p.H[l], B,
                       (int64_t)hidden[l], dense + d.offb[l]);
    LAUNCHED(k_bias_relu);
    h = p.H[l];
    fan = hidden[l];
  }
  const int64_t head_grid = small_grid(B, WAVES_PER_BLOCK, LOSS_GRID);
  hipLaunchKernelGGL(k_wd_head, dim3(head_grid), dim3(BLOCK), 0, st, h, fan, dense + d.offw, dense + d.offc, s->W,
                     s->ld, E, keys, F, label, p.base.ok, B, L > 0 ? 1 : 0, p.dlogit, p.dA, p.base.loss_part);
  LAUNCHED(k_wd_head);
  if (loss) {
    hipLaunchKernelGGL(k_sum_loss, dim3(1), dim3(BLOCK), 0, st, LossTotal{p.base.loss_part, head_grid, loss});
    LAUNCHED(k_sum_loss);
  }
  // output layer gradients
  if (ps_status r = colsum(h, B, fan, p.dlogit, p.part, p.dg + d.offw, st)) return r;
  if (ps_status r = colsum(p.dlogit, B, 1, nullptr, p.part, p.dg + d.offc, st)) return r;
  // backward through the hidden layers
  double* cur = p.dA;
  for (int l = L - 1; l >= 0; --l) {
    const double* hp = l > 0 ? p.H[l - 1] : p.X;
    const int64_t fin = l > 0 ? hidden[l - 1] : K0;
    const int64_t fout = hidden[l];
    if (ps_status r = gemm<true, false, double>(s, fin, fout, B, hp, fin, cur, fout, p.dg + d.offW[l], fout, st,
                                                wgrad_slices(fin, fout, B), p.slices))
      return r;
    if (ps_status r = colsum(cur, B, fout, nullptr, p.part, p.dg + d.offb[l], st)) return r;
    double* next = cur == p.dA ? p.dB : p.dA;
    if (ps_status r = gemm<false, true, float>(s, B, fin, fout, cur, fout, dense + d.offW[l], fout, next, fin, st))
      return r;
    if (l > 0) {
      hipLaunchKernelGGL(k_relu_mask, dim3(small_grid(B * fin, BLOCK, 8192)), dim3(BLOCK), 0, st, next, hp, B * fin);
      LAUNCHED(k_relu_mask);
    }
    cur = next;
  }
  // per-occurrence embedding gradient rows, at their sorted positions
  if (ps_status r = join_aux(s, st)) return r;
  hipLaunchKernelGGL(k_wd_rows, dim3(small_grid(n, WAVES_PER_BLOCK, 16384)), dim3(BLOCK), 0, st, cur, p.dlogit, B, F,
                     E, s->dim, p.base.sb.rank, p.base.grads);
  LAUNCHED(k_wd_rows);
  if (ps_status r = run_reduce(s, p.base.sb, ks, SrcSorted{p.base.grads, s->dim, s->dim}, n, {PART_ALL}, st)) return r;
  hipLaunchKernelGGL(k_dense_adagrad, dim3(small_grid(d.total, BLOCK, 4096)), dim3(BLOCK), 0, st, dense, dense_accum,
                     p.dg, d.total, s->lr, s->eps);
  LAUNCHED(k_dense_adagrad);
  return PS_OK;
}

// ---------------------------------------------------------------- staged stores
ps_status ps_create_staged(ps_store** out, int64_t num_keys, int32_t dim, float* home_values, float* home_accum,
                           int64_t home_stride, float* values, float* accum, int64_t row_stride, int32_t* key_slot,
                           int32_t num_ranges, const int64_t* range_begin, const int64_t* range_slots, float lr,
                           float eps, void* stream) {
  if (!out) return fail(PS_ERR_INVALID, "out is NULL");
  *out = nullptr;
  if (num_keys < 1 || num_keys > INT32_MAX) return fail(PS_ERR_INVALID, "num_keys %lld outside [1, 2^31-1]", (long long)num_keys);
  if (!home_values || !home_accum || !key_slot) return fail(PS_ERR_INVALID, "home table or key_slot is NULL");
  if (num_ranges < 1 || !range_begin || !range_slots) return fail(PS_ERR_INVALID, "need at least one key range");
  if (range_begin[0] != 0) return fail(PS_ERR_INVALID, "the first key range must begin at key 0");
  int64_t total = 0;
  for (int r = 0; r < num_ranges; ++r) {
    if (r > 0 && range_begin[r] <= range_begin[r - 1]) return fail(PS_ERR_INVALID, "key ranges must ascend");
    if (range_begin[r] >= num_keys) return fail(PS_ERR_INVALID, "key range %d begins past num_keys", r);
    const int64_t len = (r + 1 < num_ranges ? range_begin[r + 1] : num_keys) - range_begin[r];
    if (range_slots[r] < 1 || range_slots[r] > len)
      return fail(PS_ERR_INVALID, "key range %d needs between 1 and %lld slots", r, (long long)len);
    total += range_slots[r];
  }
  if (total > INT32_MAX) return fail(PS_ERR_INVALID, "more than 2^31-1 slots");
  if (dim > ROW_MAX) return fail(PS_ERR_UNSUPPORTED, "a staged store holds rows of at most %d floats", ROW_MAX);
  if (home_stride < dim) return fail(PS_ERR_INVALID, "home_stride %lld < dim %d", (long long)home_stride, dim);
  {
    const int64_t d = (int64_t)(home_accum - home_values);
    const int64_t ad = d < 0 ? -d : d;
    const bool separate = ad >= num_keys * home_stride;
    const int64_t r = ((d % home_stride) + home_stride) % home_stride;
    const bool interleaved = home_stride >= 2 * (int64_t)dim && r >= dim && r <= home_stride - dim;
    if (!separate && !interleaved) return fail(PS_ERR_INVALID, "home value and accumulator rows overlap");
  }
  if (dim % 4 == 0 && (!aligned16(home_values) || !aligned16(home_accum) || home_stride % 4 != 0))
    return fail(PS_ERR_INVALID, "home tables must be 16-byte aligned with a stride that is a multiple of 4");
  void* hw = nullptr;
  void* hg = nullptr;
  if (hipHostGetDevicePointer(&hw, home_values, 0) != hipSuccess ||
      hipHostGetDevicePointer(&hg, home_accum, 0) != hipSuccess) {
    (void)hipGetLastError();
    return fail(PS_ERR_INVALID, "home tables must be pinned host memory (hipHostMalloc)");
  }
  ps_store* s = nullptr;
  if (ps_status r = ps_create_strided(&s, total, dim, row_stride, values, accum, lr, eps, stream)) return r;
  Staging* g = new Staging();
  s->stg = g;
  g->num_keys = num_keys;
  g->total_slots = total;
  g->hW = static_cast<const float*>(hw);
  g->hG = static_cast<const float*>(hg);
  g->hld = home_stride;
  g->map = key_slot;
  g->plan.init(num_keys, range_begin, range_slots, num_ranges);
  hipError_t e = hipStreamCreateWithFlags(&g->st, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&g->clock_ev, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&g->flush_ev, hipEventDisableTiming);
  g->round_ev.assign(Staging::RING, nullptr);
  for (int i = 0; i < Staging::RING && e == hipSuccess; ++i)
    e = hipEventCreateWithFlags(&g->round_ev[i], hipEventDisableTiming);
  for (int i = 0; i < 2 && e == hipSuccess; ++i) {
    e = hipEventCreateWithFlags(&g->list_ev[i], hipEventDisableTiming);
    if (e == hipSuccess) e = hipHostMalloc(reinterpret_cast<void**>(&g->h_list[i]), size_t(4) * total * 8);
  }
  if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&g->d_keys), size_t(2) * total * 8);
  if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&g->d_slots), size_t(2) * total * 8);
  if (e == hipSuccess) {
    hipStream_t st = as_stream(stream);
    hipLaunchKernelGGL(k_map_fill, dim3(small_grid(num_keys, BLOCK, 4096)), dim3(BLOCK), 0, st, key_slot, num_keys);
    e = hipGetLastError();
    if (e == hipSuccess) e = hipStreamSynchronize(st);
  }
  if (e != hipSuccess) {
    (void)ps_destroy(s);
    return fail(PS_ERR_DEVICE, "staged store set-up: %s", hipGetErrorString(e));
  }
  *out = s;
  return PS_OK;
}

ps_status ps_set_action_timing(ps_store* s, double alpha, double p, double lambda0) {
  if (ps_status st = check_staged(s)) return st;
  if (!(alpha > 0.0 && alpha <= 1.0) || !(p > 0.0 && p < 1.0) || !(lambda0 >= 0.0))
    return fail(PS_ERR_INVALID, "need 0 < alpha <= 1, 0 < p < 1 and lambda0 >= 0");
  std::lock_guard<std::mutex> lk(s->stg->mu);
  ActionTiming& t = s->stg->plan.timing;
  t.alpha = alpha;
  t.p = p;
  t.lambda = lambda0;
  return PS_OK;
}

ps_status ps_intent(ps_store* s, const int64_t* keys, int64_t n, int64_t c_start, int64_t c_end) {
  if (ps_status st = check_staged(s)) return st;
  if (n < 0 || (n > 0 && !keys)) return fail(PS_ERR_INVALID, "keys is NULL or n < 0");
  if (c_end <= c_start) return fail(PS_ERR_INVALID, "need c_start < c_end");
  std::lock_guard<std::mutex> lk(s->stg->mu);
  s->stg->plan.signal(keys, n, c_start, c_end);
  return PS_OK;
}

ps_status ps_advance_clock(ps_store* s, void* stream) {
  if (ps_status st = check_staged(s)) return st;
  Staging& g = *s->stg;
  std::lock_guard<std::mutex> lk(g.mu);
  hipStream_t st = as_stream(stream);
  g.plan.clock += 1;
  HIP_TRY(hipEventRecord(g.clock_ev, st));
  if (g.plan.due(g.plan.clock))
    if (ps_status r = stage_round_locked(s, true, nullptr, nullptr)) return r;
  const int64_t r = g.plan.take_round_for(g.plan.clock);
  if (r > g.waited) {
    HIP_TRY(hipStreamWaitEvent(st, g.round_ev[r % Staging::RING], 0));
    g.waited = r;
  }
  return PS_OK;
}

ps_status ps_stage_round(ps_store* s, int32_t wait) {
  if (ps_status st = check_staged(s)) return st;
  Staging& g = *s->stg;
  if (g.auto_on.load()) return fail(PS_ERR_INVALID, "rounds are running on the library's thread");
  int64_t rid = 0;
  {
    std::lock_guard<std::mutex> lk(g.mu);
    if (ps_status r = stage_round_locked(s, false, &rid, nullptr)) return r;
  }
  if (wait) HIP_TRY(hipEventSynchronize(g.round_ev[rid % Staging::RING]));
  return PS_OK;
}

ps_status ps_stage_auto(ps_store* s, int32_t on) {
  if (ps_status st = check_staged(s)) return st;
  Staging& g = *s->stg;
  if (!on) {
    stop_auto(g);
    const int32_t r = g.auto_status.exchange(0);
    return r ? fail(r, "a round on the library's thread failed") : PS_OK;
  }
  if (g.auto_on.load()) return PS_OK;
  if (g.auto_thread.joinable()) g.auto_thread.join();
  g.auto_on.store(true);
  g.auto_thread = std::thread(auto_rounds, s);
  return PS_OK;
}

ps_status ps_stage_flush(ps_store* s, void* stream) {
  if (ps_status st = check_staged(s)) return st;
  Staging& g = *s->stg;
  std::lock_guard<std::mutex> lk(g.mu);
  HIP_TRY(hipEventRecord(g.flush_ev, as_stream(stream)));
  HIP_TRY(hipStreamWaitEvent(g.st, g.flush_ev, 0));
  std::vector<int64_t> keys, slots, none;
  const Planner& P = g.plan;
  for (int64_t k = 0; k < g.num_keys; ++k)
    if (P.slot_of(k) >= 0) {
      keys.push_back(k);
      slots.push_back(P.slot_of(k));
    }
  // every resident row is written back; it stays resident
  if (!keys.empty()) {
    const int b = g.list_i;
    g.list_i ^= 1;
    HIP_TRY(hipEventSynchronize(g.list_ev[b]));
    int64_t* hk = g.h_list[b];
    int64_t* hs = hk + 2 * g.total_slots;
    std::copy(keys.begin(), keys.end(), hk);
    std::copy(slots.begin(), slots.end(), hs);
    const int64_t n = (int64_t)keys.size();
    HIP_TRY(hipMemcpyAsync(g.d_keys, hk, size_t(n) * 8, hipMemcpyHostToDevice, g.st));
    HIP_TRY(hipMemcpyAsync(g.d_slots, hs, size_t(n) * 8, hipMemcpyHostToDevice, g.st));
    HIP_TRY(hipEventRecord(g.list_ev[b], g.st));
    if (ps_status r = move_rows(s, true, g.d_slots, g.d_keys, n, g.st)) return r;
  }
  HIP_TRY(hipStreamSynchronize(g.st));
  return PS_OK;
}

ps_status ps_stage_stats(ps_store* s, int64_t* counts, int32_t n, double* lambda) {
  if (ps_status st = check_staged(s)) return st;
  if (n < 0 || (n > 0 && !counts)) return fail(PS_ERR_INVALID, "counts is NULL");
  Staging& g = *s->stg;
  std::lock_guard<std::mutex> lk(g.mu);
  const Planner& P = g.plan;
  int64_t resident = g.total_slots;
  for (const auto& f : P.free_slots) resident -= (int64_t)f.size();
  int64_t pending = 0;
  for (const auto& kv : P.pending) pending += (int64_t)(kv.second.keys.size() - kv.second.next);
  const int64_t v[PS_STAGE_NUM_STATS] = {P.clock, g.rounds, P.forced_total, P.staged_total, P.evicted_total,
                                         resident, pending, P.stalled_total, g.plan_us};
  for (int i = 0; i < n && i < PS_STAGE_NUM_STATS; ++i) counts[i] = v[i];
  if (lambda) *lambda = P.timing.lambda;
  return PS_OK;
}

ps_status ps_stage_resident(ps_store* s, int64_t* keys, int64_t capacity, int64_t* count) {
  if (ps_status st = check_staged(s)) return st;
  if (!count || capacity < 0 || (capacity > 0 && !keys)) return fail(PS_ERR_INVALID, "bad output arguments");
  Staging& g = *s->stg;
  std::lock_guard<std::mutex> lk(g.mu);
  int64_t c = 0;
  for (int64_t k = 0; k < g.num_keys; ++k)
    if (g.plan.slot_of(k) >= 0) {
      if (c < capacity) keys[c] = k;
      ++c;
    }
  *count = c;
  return PS_OK;
}

ps_status ps_action_timing(double lambda_prev, int64_t c_prev, int64_t c_now, double alpha, double p,
                           double* lambda_new, int64_t* horizon) {
  if (!lambda_new || !horizon) return fail(PS_ERR_INVALID, "output pointer is NULL");
  if (!(alpha > 0.0 && alpha <= 1.0) || !(p > 0.0 && p < 1.0)) return fail(PS_ERR_INVALID, "bad alpha or p");
  ActionTiming t;
  t.alpha = alpha;
  t.p = p;
  t.lambda = lambda_prev;
  t.round_clock = c_prev;
  *horizon = t.horizon(c_now);
  *lambda_new = t.lambda;
  return PS_OK;
}

ps_status ps_get_error(ps_store* s, void* stream) {
  if (ps_status st = check_store(s)) return st;
  HIP_TRY(hipStreamSynchronize(as_stream(stream)));
  int32_t flag[2] = {0, 0};
  HIP_TRY(hipMemcpy(flag, s->status, sizeof flag, hipMemcpyDeviceToHost));
  if (flag[0] || flag[1]) {
    HIP_TRY(hipMemset(s->status, 0, sizeof flag));
    HIP_TRY(hipDeviceSynchronize());
    if (flag[1]) return fail(PS_ERR_NOT_RESIDENT, "a key with no slot (no intent acted upon) was accessed");
    return fail(PS_ERR_KEY_RANGE, "a key outside [0, %lld) was seen",
                (long long)(s->stg ? s->stg->num_keys : s->num_keys));
  }
  return PS_OK;
}

ps_status ps_probe_gather(ps_store* s, const int32_t* keys, int64_t n, double* sink, void* stream) {
  if (ps_status st = check_store(s)) return st;
  if (s->bf16) return fail(PS_ERR_UNSUPPORTED, "the gather probe reads fp32 values only");
  if (n < 0) return fail(PS_ERR_INVALID, "negative size %lld", (long long)n);
  if (!sink || (n > 0 && !keys)) return fail(PS_ERR_INVALID, "keys or sink is NULL");
  RowShape shape;
  if (!row_shape(s->dim, true, &shape)) return fail(PS_ERR_UNSUPPORTED, "dim %d not supported", s->dim);
  hipStream_t st = as_stream(stream);
  return with_shape(shape, [&]<int L, int NV, int VW>() -> ps_status {
    hipLaunchKernelGGL((k_gather_probe<L, NV, VW>), dim3(PS_PROBE_GRID), dim3(BLOCK), 0, st, s->W, s->ld, s->dim,
                       s->num_keys, keys, n, sink);
    LAUNCHED(k_gather_probe);
    return PS_OK;
  });
}

ps_status ps_set_timing(ps_store* s, int32_t mask) {
  if (ps_status st = check_store(s)) return st;
  s->timing = (uint32_t)mask;
  return PS_OK;
}

ps_status ps_read_timing(ps_store* s, int32_t kernel_id, double* total_ms, int64_t* launches) {
  if (ps_status st = check_store(s)) return st;
  if (kernel_id < 0 || kernel_id >= NUM_TIMED || !total_ms || !launches)
    return fail(PS_ERR_INVALID, "bad kernel id or output pointer");
  double tot = 0.0;
  auto& v = s->events[kernel_id];
  for (size_t i = 0; i < s->used[kernel_id]; ++i) {
    HIP_TRY(hipEventSynchronize(v[i].second));
    float ms = 0.0f;
    HIP_TRY(hipEventElapsedTime(&ms, v[i].first, v[i].second));
    tot += ms;
  }
  *total_ms = tot;
  *launches = (int64_t)s->used[kernel_id];
  s->used[kernel_id] = 0;
  return PS_OK;
}

}  // extern "C"
