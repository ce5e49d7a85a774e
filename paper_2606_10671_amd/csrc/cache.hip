// FadeMem bounded memory on the device: pool layout, the C ABI, and the
// bookkeeping kernels (insert copy, schedule, merge).
//
// Paper: FadeMem, arXiv 2606.10671 -- Sec. 3.1 (bounded ordered memory),
// Sec. 3.3 (insertion, distance-aware scheduling, consolidation operator,
// boundary handling) and Algorithm S1 (the complete update).
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <new>
#include <vector>

#include "fademem_internal.h"

using namespace fademem;

namespace {

// Host replay of the memory's metadata and slot table.  The device decides
// every consolidation itself; the host replays the same steps on the same
// integers (Alg. S1 with the schedule of select_pair, the slot bookkeeping
// of the kernels) so that it knows, without reading anything back, which
// slots are free (the addresses of staged frames) and which entries changed
// (the re-indexed K views).  fademem_verify and serialize mode compare it
// with the device state.
struct Mirror {
  std::vector<int64_t> first, pos_sum, span;  // held entries, oldest first
  std::vector<int32_t> order;                 // logical -> slot, all slots
};

}  // namespace

struct fademem_cache {
  fademem_config cfg;
  Layout lay;
  char* pool;
  int64_t count;        // entries held (mirrors the device state exactly)
  int64_t newest;       // newest inserted position
  int64_t inserted;     // blocks inserted so far
  int cur;              // metadata copy holding the current state (0 or 1)
  bool any_inserted;
  bool serialize;       // FADEMEM_SERIALIZE set at creation: every call waits for its work and checks it
  int last_hip_error;
  Mirror mirror;
  // Re-indexed K views (rope_pairs > 0): view block s of layer l holds the
  // K of slot s with its temporal pairs rotated to index view_index, built
  // when the slot held the entry covering [view_first, view_first +
  // view_span) (span 0: nothing valid).  An entry's covered range fixes its
  // contents for the life of a cache: positions strictly increase and ranges
  // only grow by merging.  An entry that only moved to another index (a
  // merge before it) needs its temporal pairs rotated again, nothing else.
  std::vector<int64_t> view_first, view_span;
  std::vector<int32_t> view_index;
};

namespace {

inline size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// End of an asynchronous call: in serialize mode (a debugging aid), wait for
// the call's work and report a failure at the call that caused it.
int verify_mirror(fademem_cache* c, void* stream);

int finish(fademem_cache* c, void* stream) {
  if (!c->serialize) return FADEMEM_OK;
  hipError_t e = hipStreamSynchronize(reinterpret_cast<hipStream_t>(stream));
  if (e == hipSuccess) e = hipGetLastError();
  if (e != hipSuccess) {
    c->last_hip_error = int(e);
    return FADEMEM_EHIP;
  }
  return verify_mirror(c, stream);
}

int hip_fail(fademem_cache* c, hipError_t e) {
  if (c) c->last_hip_error = int(e);
  return FADEMEM_EHIP;
}

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Typed views of one metadata copy.
struct Meta {
  int64_t* first;
  int64_t* pos_sum;
  int64_t* span;
  int32_t* order;
};
__host__ __device__ inline Meta meta_of(char* pool, const Layout& lay, int copy) {
  Meta m;
  m.first = reinterpret_cast<int64_t*>(pool + lay.off_first[copy]);
  m.pos_sum = reinterpret_cast<int64_t*>(pool + lay.off_pos_sum[copy]);
  m.span = reinterpret_cast<int64_t*>(pool + lay.off_span[copy]);
  m.order = reinterpret_cast<int32_t*>(pool + lay.off_order[copy]);
  return m;
}

// ---------------------------------------------------------------------------
// Kernels
// ---------------------------------------------------------------------------

// Empty memory: both order copies = identity permutation, counters cleared.
__global__ void init_kernel(char* pool, Layout lay) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i == 0) {
    DevHeader* hdr = reinterpret_cast<DevHeader*>(pool);
    hdr->merges_total = 0;
    hdr->anchor_merges = 0;
  }
  if (i < lay.slots) {
    meta_of(pool, lay, 0).order[i] = int32_t(i);
    meta_of(pool, lay, 1).order[i] = int32_t(i);
  }
}

struct InsertArgs {
  const void* k[kMaxLayersPerLaunch];
  const void* v[kMaxLayersPerLaunch];
  char* pool;
  Layout lay;
  int64_t layer0;      // first layer of this launch
  int64_t units;       // 16-byte units per block
  int64_t index;       // logical index of the new entry (= count before insert)
  int64_t position;    // t
  int cur;             // current metadata copy
  int write_meta;      // 1 in exactly one launch of an insert
};

// Append (K_t, V_t, t, 1): copy each layer's block into the free slot
// order[index] and record first = t, pos_sum = t, span = 1 (Sec. 3.3,
// Alg. S1 Append).  grid.y = layer_in_launch * 2 + kv.
__global__ __launch_bounds__(256) void insert_kernel(InsertArgs a) {
  const int li = blockIdx.y >> 1;
  const int kv = blockIdx.y & 1;
  const Meta m = meta_of(a.pool, a.lay, a.cur);
  const int32_t slot = m.order[a.index];
  const u32x4* src = reinterpret_cast<const u32x4*>(kv ? a.v[li] : a.k[li]);
  u32x4* dst = reinterpret_cast<u32x4*>(a.pool + kv_offset(a.lay, a.layer0 + li, slot, kv));
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t u = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; u < a.units; u += stride) {
    __builtin_nontemporal_store(__builtin_nontemporal_load(src + u), dst + u);
  }
  if (a.write_meta && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) {
    m.first[a.index] = a.position;
    m.pos_sum[a.index] = a.position;
    m.span[a.index] = 1;
  }
}

// Block-wide reductions for 256-thread blocks (4 waves).
__device__ double block_min_f64(double v, double* red) {
  for (int o = 32; o > 0; o >>= 1) v = fmin(v, __shfl_xor(v, o));
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (lane == 0) red[w] = v;
  __syncthreads();
  double r = fmin(fmin(red[0], red[1]), fmin(red[2], red[3]));
  __syncthreads();
  return r;
}

__device__ int block_min_i32(int v, int* red) {
  for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o));
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (lane == 0) red[w] = v;
  __syncthreads();
  int r = min(min(red[0], red[1]), min(red[2], red[3]));
  __syncthreads();
  return r;
}

// fp64 -> fp32 with round-to-odd: the hardware conversion rounds to
// nearest; if that moved away from zero, step back one ulp (truncation),
// then set the last bit when the conversion was inexact.  Rounding the
// result to bf16 to nearest even then equals a single correct rounding of
// x to bf16, because fp32 carries 16 more significand bits than bf16.
__device__ __forceinline__ float f64_to_f32_odd(double x) {
  const float f = float(x);
  const double xd = double(f);
  uint32_t b = __float_as_uint(f);
  b -= (fabs(xd) > fabs(x)) ? 1u : 0u;
  b |= (xd != x) ? 1u : 0u;
  return __uint_as_float(b);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Two fp64 values -> packed bf16x2 (low half = lo), each rounded to nearest even.
__device__ __forceinline__ uint32_t pack_bf16_rne(double lo, double hi) {
  bf16x2_t v;
  v[0] = (__bf16)f64_to_f32_odd(lo);
  v[1] = (__bf16)f64_to_f32_odd(hi);
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ double bf16_lo(uint32_t w) { return double(__uint_as_float(w << 16)); }
__device__ __forceinline__ double bf16_hi(uint32_t w) { return double(__uint_as_float(w & 0xffff0000u)); }

// The schedule of one consolidation (Sec. 3.3 "Distance-aware scheduling",
// Alg. S1) over entries 0..n-1 (the newest is n-1), for a 256-thread block:
//   d_i = t - mu_i = (t*s_i - pos_sum_i) / s_i   (exact numerator, one fp64 division)
//   u_i = d_i^beta
//   g_i = |u_{i+1} - u_i| for the pairs i = 0..n-3 (the pair holding the
//         newest entry, n-2..n-1, is not eligible)
//   j   = lowest i with g_i - min(g) <= 1e-9 * min(g)
// Every thread returns j.  span/pos_sum may live in global or LDS memory.
__device__ int select_pair(const int64_t* span, const int64_t* pos_sum, int n, int64_t t, double beta,
                           double* u_s, double* g_s, double* red_d, int* red_i) {
#pragma clang fp contract(off)
  const int tid = threadIdx.x;
  for (int i = tid; i < n - 1; i += 256) {
    const int64_t s = span[i];
    const double d = double(t * s - pos_sum[i]) / double(s);
    u_s[i] = (beta == 1.0) ? d : pow(d, beta);
  }
  __syncthreads();
  double gmin = INFINITY;
  for (int i = tid; i < n - 2; i += 256) {
    const double g = fabs(u_s[i + 1] - u_s[i]);
    g_s[i] = g;
    gmin = fmin(gmin, g);
  }
  const double gm = block_min_f64(gmin, red_d);
  const double tol = 1e-9 * gm;
  int cand = 0x7fffffff;
  for (int i = tid; i < n - 2; i += 256) {
    if (g_s[i] - gm <= tol) cand = min(cand, i);
  }
  return block_min_i32(cand, red_i);
}

// One 16-byte unit of a merge: x is the older entry's, y the newer entry's.
// Weighted (and average): each element w_a*x + w_b*y in fp64 (two products,
// one sum) rounded once to the storage type; max pooling: the newer value
// only when strictly greater.
template <bool BF16, bool MAXOP>
__device__ __forceinline__ u32x4 merge_unit(u32x4 x, u32x4 y, double wa, double wb) {
#pragma clang fp contract(off)
  u32x4 o;
  if constexpr (MAXOP) {
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      if constexpr (BF16) {
        const uint32_t xl = x[w] << 16, yl = y[w] << 16;
        const uint32_t xh = x[w] & 0xFFFF0000u, yh = y[w] & 0xFFFF0000u;
        const uint32_t lo = (__uint_as_float(yl) > __uint_as_float(xl)) ? yl : xl;
        const uint32_t hi = (__uint_as_float(yh) > __uint_as_float(xh)) ? yh : xh;
        o[w] = (lo >> 16) | hi;
      } else {
        o[w] = (__uint_as_float(y[w]) > __uint_as_float(x[w])) ? y[w] : x[w];
      }
    }
  } else if constexpr (BF16) {
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const double lo = wa * bf16_lo(x[w]) + wb * bf16_lo(y[w]);
      const double hi = wa * bf16_hi(x[w]) + wb * bf16_hi(y[w]);
      o[w] = pack_bf16_rne(lo, hi);
    }
  } else {
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const double v = wa * double(__uint_as_float(x[w])) + wb * double(__uint_as_float(y[w]));
      o[w] = __float_as_uint(float(v));
    }
  }
  return o;
}

// Weights (w_j, w_j+1) of a merge of spans s_j, s_j+1 under `op`.
__device__ __forceinline__ void merge_weights(int op, int64_t s_j, int64_t s_j1, double* wa, double* wb) {
#pragma clang fp contract(off)
  const double rj = sqrt(double(s_j));
  const double rj1 = sqrt(double(s_j1));
  *wa = op == FADEMEM_MERGE_AVERAGE ? 0.5 : rj / (rj + rj1);
  *wb = 1.0 - *wa;
}

struct ConsolidateArgs {
  char* pool;
  Layout lay;
  int n;            // entries held (M + 1)
  int layers;
  int64_t t;        // newest position
  double beta;
  int anchor;
  int cur;          // metadata copy read; the other copy is written
  int op;           // FADEMEM_MERGE_*
  int64_t units;    // 16-byte units per K (or V) block
};

// One consolidation (Sec. 3.3 "Distance-aware scheduling" and
// "Consolidation operator", Alg. S1) in one launch.  Every block derives
// the decision (select_pair) from the current metadata copy, which no block
// writes.  Block 0 writes the spliced metadata into the other copy (spans add,
// pos_sum adds so mu is span-weighted; the anchor keeps its position, the
// slot of entry j+1 is freed) and appends j to the merge log.  Unless the
// pair holds the anchor, all blocks then merge entry j+1 into entry j's
// slot: X_new = w_j X_j + w_{j+1} X_{j+1}, each element in fp64 as two
// products and one sum, rounded once to the storage type.  The blocks of
// each (layer, K|V) plane cover it with 16-byte nontemporal loads/stores,
// UNROLL units in flight per thread (striding on if the plane needs more
// blocks than a grid row holds); grid.y = layer * 2 + kv.
template <bool BF16, int UNROLL, bool MAXOP>
__global__ __launch_bounds__(256) void consolidate_kernel(ConsolidateArgs a) {
#pragma clang fp contract(off)
  __shared__ double u_s[kMaxBudget + 1];
  __shared__ double g_s[kMaxBudget + 1];
  __shared__ double red_d[4];
  __shared__ int red_i[4];

  const Meta m = meta_of(a.pool, a.lay, a.cur);
  const int n = a.n;
  const int tid = threadIdx.x;
  const int j = select_pair(m.span, m.pos_sum, n, a.t, a.beta, u_s, g_s, red_d, red_i);

  const int64_t s_j = m.span[j], s_j1 = m.span[j + 1];
  const bool anchor_pair = a.anchor && j == 0;
  const int32_t dst_slot = m.order[j];
  const int32_t src_slot = m.order[j + 1];
  // Select Nearest keeps the newer entry's K, V: the merged entry takes its
  // slot and the older entry's slot is freed (no K/V bytes move).
  const bool select = a.op == FADEMEM_MERGE_SELECT_NEAREST && !anchor_pair;
  const int32_t keep_slot = select ? src_slot : dst_slot;
  const int32_t free_slot = select ? dst_slot : src_slot;

  if (blockIdx.x == 0 && blockIdx.y == 0) {
    const Meta w = meta_of(a.pool, a.lay, a.cur ^ 1);
    for (int i = tid; i < n; i += 256) {
      if (i < j) {
        w.first[i] = m.first[i];
        w.pos_sum[i] = m.pos_sum[i];
        w.span[i] = m.span[i];
        w.order[i] = m.order[i];
      } else if (i == j) {
        const int64_t s_new = s_j + s_j1;
        w.first[i] = m.first[j];
        w.pos_sum[i] = anchor_pair ? m.first[j] * s_new : m.pos_sum[j] + m.pos_sum[j + 1];
        w.span[i] = s_new;
        w.order[i] = keep_slot;
      } else if (i < n - 1) {
        w.first[i] = m.first[i + 1];
        w.pos_sum[i] = m.pos_sum[i + 1];
        w.span[i] = m.span[i + 1];
        w.order[i] = m.order[i + 1];
      } else {
        w.order[i] = free_slot;
      }
    }
    // order[] keeps all M+1 slots: copy the free tail beyond the held entries.
    for (int i = n + tid; i < a.lay.slots; i += 256) w.order[i] = m.order[i];
    if (tid == 0) {
      DevHeader* hdr = reinterpret_cast<DevHeader*>(a.pool);
      int32_t* log = reinterpret_cast<int32_t*>(a.pool + a.lay.off_log);
      const int64_t k = hdr->merges_total;
      log[k % kLogCap] = j;
      hdr->merges_total = k + 1;
      if (anchor_pair) hdr->anchor_merges += 1;
    }
  }
  if (anchor_pair || select) return;  // the anchor keeps its K and V; selection moves nothing

  double wa, wb;
  merge_weights(a.op, s_j, s_j1, &wa, &wb);
  const int64_t step = int64_t(gridDim.x) * 256 * UNROLL;
  {
    const int plane = blockIdx.y;  // layer * 2 + kv
    const int layer = plane >> 1, kv = plane & 1;
    u32x4* dst = reinterpret_cast<u32x4*>(a.pool + kv_offset(a.lay, layer, dst_slot, kv));
    const u32x4* src = reinterpret_cast<const u32x4*>(a.pool + kv_offset(a.lay, layer, src_slot, kv));
    for (int64_t base = int64_t(blockIdx.x) * 256 * UNROLL + tid; base < a.units; base += step) {
      u32x4 x[UNROLL], y[UNROLL];
#pragma unroll
      for (int r = 0; r < UNROLL; ++r) {
        const int64_t u = base + int64_t(r) * 256;
        if (u < a.units) {
          x[r] = __builtin_nontemporal_load(dst + u);
          y[r] = __builtin_nontemporal_load(src + u);
        }
      }
#pragma unroll
      for (int r = 0; r < UNROLL; ++r) {
        const int64_t u = base + int64_t(r) * 256;
        if (u < a.units) {
          const u32x4 o = merge_unit<BF16, MAXOP>(x[r], y[r], wa, wb);
          __builtin_nontemporal_store(o, dst + u);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Fused update: F sequential Algorithm S1 updates (append frame f, then
// consolidate if over budget) in two launches.  The plan kernel replays the
// F steps on the metadata with the same schedule arithmetic as
// consolidate_kernel and records, for every merge that computes K and V,
// its operands (an old entry's slot, a frame of the caller's chunk, or an
// earlier merge of this update) and weights, and for every entry that ends
// up new or changed, where it comes from and the slot it goes to.  The data
// kernel then streams each (layer, K|V) plane once: per 16-byte unit it
// loads each operand once, evaluates the merges in order in registers
// (each rounded to the storage type exactly as a lone merge is), and stores
// each changed entry once.  Frames consumed by a merge of the same update
// are read from the caller's buffers and never copied into the pool.
// Staged frames (the zero-copy update) already sit in free pool slots: they
// enter the plan as slot references, so a frame that survives the update
// stays where the caller wrote it and one that a merge consumes frees its
// slot.
// ---------------------------------------------------------------------------

struct PlanArgs {
  char* pool;
  Layout lay;
  int n0;                  // entries held before the update (<= M)
  int frames;              // 1..kMaxPlanFrames
  int64_t first_position;  // position of frame 0; frame f is first_position + f
  int64_t budget;          // M
  double beta;
  int anchor;
  int op;
  int cur;                 // metadata copy read; the other copy is written
  int staged;              // 1: frame f is already in slot order[n0 + f]
};

__global__ __launch_bounds__(256) void update_plan_kernel(PlanArgs a) {
#pragma clang fp contract(off)
  constexpr int kCap = kMaxBudget + 1;  // entries held at most (M + 1)
  __shared__ int64_t first_s[kCap], pos_s[kCap], span_s[kCap];
  __shared__ int32_t kind_s[kCap], idx_s[kCap];
  __shared__ int32_t free_s[kMaxBudget + kMaxPlanFrames];  // free slots: at most all M + stage_frames
  __shared__ double u_s[kCap], g_s[kCap];
  __shared__ double red_d[4];
  __shared__ int red_i[4];
  __shared__ int n_free_s;
  __shared__ UpdatePlan plan;

  const int tid = threadIdx.x;
  const Meta m = meta_of(a.pool, a.lay, a.cur);
  const int slots = int(a.lay.slots);
  for (int i = tid; i < a.n0; i += 256) {
    first_s[i] = m.first[i];
    pos_s[i] = m.pos_sum[i];
    span_s[i] = m.span[i];
    kind_s[i] = kRefSlot;
    idx_s[i] = m.order[i];
  }
  const int skip = a.staged ? a.frames : 0;  // staged frames' slots are not free
  for (int i = a.n0 + skip + tid; i < slots; i += 256) free_s[i - a.n0 - skip] = m.order[i];
  if (tid == 0) {
    n_free_s = slots - a.n0 - skip;
    plan.n_ar = 0;
    plan.n_out = 0;
  }
  __syncthreads();

  DevHeader* hdr = reinterpret_cast<DevHeader*>(a.pool);
  int32_t* log = reinterpret_cast<int32_t*>(a.pool + a.lay.off_log);
  int64_t merges = 0, anchors = 0;  // the header's counters, read once and written back at the end (thread 0)
  if (tid == 0) {
    merges = hdr->merges_total;
    anchors = hdr->anchor_merges;
  }
  int n = a.n0;
  for (int f = 0; f < a.frames; ++f) {
    const int64_t t = a.first_position + f;
    if (tid == 0) {  // Append (K_t, V_t, t, 1), its K, V still the caller's frame f (or its staging slot)
      first_s[n] = t;
      pos_s[n] = t;
      span_s[n] = 1;
      kind_s[n] = a.staged ? kRefSlot : kRefFrame;
      idx_s[n] = a.staged ? m.order[a.n0 + f] : f;
    }
    n += 1;
    __syncthreads();
    if (n <= a.budget) continue;  // within budget: nothing to consolidate (uniform)
    const int j = select_pair(span_s, pos_s, n, t, a.beta, u_s, g_s, red_d, red_i);
    if (tid == 0) {
      const bool anchor_pair = a.anchor && j == 0;
      const bool select = a.op == FADEMEM_MERGE_SELECT_NEAREST && !anchor_pair;
      const int64_t s_new = span_s[j] + span_s[j + 1];
      int32_t nk, ni;  // reference of the merged entry
      if (anchor_pair || select) {
        // The kept entry's K, V move unchanged; the other one's are dropped.
        const int keep = anchor_pair ? j : j + 1, drop = anchor_pair ? j + 1 : j;
        nk = kind_s[keep];
        ni = idx_s[keep];
        if (kind_s[drop] == kRefSlot) free_s[n_free_s++] = idx_s[drop];
      } else {
        const int k = plan.n_ar++;
        plan.a_kind[k] = kind_s[j];
        plan.a_idx[k] = idx_s[j];
        plan.b_kind[k] = kind_s[j + 1];
        plan.b_idx[k] = idx_s[j + 1];
        merge_weights(a.op, span_s[j], span_s[j + 1], &plan.wa[k], &plan.wb[k]);
        if (kind_s[j] == kRefSlot) free_s[n_free_s++] = idx_s[j];
        if (kind_s[j + 1] == kRefSlot) free_s[n_free_s++] = idx_s[j + 1];
        nk = kRefResult;
        ni = k;
      }
      pos_s[j] = anchor_pair ? first_s[j] * s_new : pos_s[j] + pos_s[j + 1];
      span_s[j] = s_new;
      kind_s[j] = nk;
      idx_s[j] = ni;
      log[merges % kLogCap] = j;
      merges += 1;
      if (anchor_pair) anchors += 1;
    }
    __syncthreads();
    // Replace: entries j+2..n-1 move down by one.
    constexpr int kPer = (kCap + 255) / 256;
    int64_t tf[kPer], tp[kPer], ts[kPer];
    int32_t tk[kPer], ti[kPer];
#pragma unroll
    for (int r = 0; r < kPer; ++r) {
      const int i = j + 1 + tid + 256 * r;
      if (i < n - 1) {
        tf[r] = first_s[i + 1];
        tp[r] = pos_s[i + 1];
        ts[r] = span_s[i + 1];
        tk[r] = kind_s[i + 1];
        ti[r] = idx_s[i + 1];
      }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kPer; ++r) {
      const int i = j + 1 + tid + 256 * r;
      if (i < n - 1) {
        first_s[i] = tf[r];
        pos_s[i] = tp[r];
        span_s[i] = ts[r];
        kind_s[i] = tk[r];
        idx_s[i] = ti[r];
      }
    }
    n -= 1;
    __syncthreads();
  }

  // Slots: kept old entries stay; every new or changed entry takes a free
  // slot (those free before, or freed by this update).
  const Meta w = meta_of(a.pool, a.lay, a.cur ^ 1);
  if (tid == 0) {
    int next = 0;
    for (int i = 0; i < n; ++i) {
      if (kind_s[i] == kRefSlot) {
        w.order[i] = idx_s[i];
      } else {
        const int o = plan.n_out++;
        const int32_t slot = free_s[next++];
        plan.o_kind[o] = kind_s[i];
        plan.o_idx[o] = idx_s[i];
        plan.o_slot[o] = slot;
        w.order[i] = slot;
      }
    }
    for (int i = n; i < slots; ++i) w.order[i] = free_s[next++];
    *reinterpret_cast<UpdatePlan*>(a.pool + a.lay.off_prog) = plan;
    hdr->merges_total = merges;
    hdr->anchor_merges = anchors;
  }
  for (int i = tid; i < n; i += 256) {
    w.first[i] = first_s[i];
    w.pos_sum[i] = pos_s[i];
    w.span[i] = span_s[i];
  }
}

struct UpdateDataArgs {
  const void* k[kMaxLayersPerLaunch];  // layer's chunk K, [frames][N][H][D]
  const void* v[kMaxLayersPerLaunch];
  char* pool;
  Layout lay;
  int64_t layer0;  // first layer of this launch
  int64_t units;   // 16-byte units per K (or V) block
};

// grid.y = layer * 2 + kv: the blocks of a (layer, K|V) plane cover it,
// one 16-byte unit per thread (striding on if the plane needs more blocks
// than a grid row holds).
template <bool BF16, bool MAXOP, int MF>
__global__ __launch_bounds__(256) void update_data_kernel(UpdateDataArgs a) {
  // Operand arrays for plans of up to MF frames: at most MF merges and 2 * MF
  // entries written.
  constexpr int kM = MF, kO = 2 * MF;
  const UpdatePlan* P = reinterpret_cast<const UpdatePlan*>(a.pool + a.lay.off_prog);
  const int n_ar = P->n_ar, n_out = P->n_out;
  // Result r of the merges computed so far (r is wave-uniform).
  auto pick = [](const u32x4 (&R)[kM], int r) {
    u32x4 x = R[0];
#pragma unroll
    for (int k = 1; k < kM; ++k)
      if (r == k) x = R[k];
    return x;
  };
  auto run_plane = [&](int li, int kv, int64_t u_begin, int64_t u_end, int64_t u_step) {
    const int64_t layer = a.layer0 + li;
    const char* chunk = static_cast<const char*>(kv ? a.v[li] : a.k[li]);
    auto ref = [&](int kind, int idx) -> const u32x4* {
      return reinterpret_cast<const u32x4*>(kind == kRefSlot ? a.pool + kv_offset(a.lay, layer, idx, kv)
                                                             : chunk + size_t(idx) * a.lay.blk_bytes);
    };
    const u32x4* pa[kM];
    const u32x4* pb[kM];
    int ra[kM], rb[kM];
    double wa[kM], wb[kM];
#pragma unroll
    for (int k = 0; k < kM; ++k) {
      const bool on = k < n_ar;
      ra[k] = on && P->a_kind[k] == kRefResult ? P->a_idx[k] : -1;
      rb[k] = on && P->b_kind[k] == kRefResult ? P->b_idx[k] : -1;
      pa[k] = on && ra[k] < 0 ? ref(P->a_kind[k], P->a_idx[k]) : nullptr;
      pb[k] = on && rb[k] < 0 ? ref(P->b_kind[k], P->b_idx[k]) : nullptr;
      wa[k] = on ? P->wa[k] : 0.0;
      wb[k] = on ? P->wb[k] : 0.0;
    }
    u32x4* po[kO];
    const u32x4* ps[kO];
    int ro[kO];
#pragma unroll
    for (int o = 0; o < kO; ++o) {
      const bool on = o < n_out;
      ro[o] = on && P->o_kind[o] == kRefResult ? P->o_idx[o] : -1;
      ps[o] = on && ro[o] < 0 ? ref(P->o_kind[o], P->o_idx[o]) : nullptr;
      po[o] = on ? reinterpret_cast<u32x4*>(a.pool + kv_offset(a.lay, layer, P->o_slot[o], kv)) : nullptr;
    }
    for (int64_t u = u_begin; u < u_end; u += u_step) {
      // Every operand of this unit is loaded before any store (stores may go
      // to a slot an operand was read from).
      u32x4 A[kM], B[kM], S[kO], R[kM];
#pragma unroll
      for (int k = 0; k < kM; ++k) {
        if (pa[k]) A[k] = __builtin_nontemporal_load(pa[k] + u);
        if (pb[k]) B[k] = __builtin_nontemporal_load(pb[k] + u);
      }
#pragma unroll
      for (int o = 0; o < kO; ++o)
        if (ps[o]) S[o] = __builtin_nontemporal_load(ps[o] + u);
#pragma unroll
      for (int k = 0; k < kM; ++k) {
        if (k < n_ar) {
          const u32x4 x = pa[k] ? A[k] : pick(R, ra[k]);
          const u32x4 y = pb[k] ? B[k] : pick(R, rb[k]);
          R[k] = merge_unit<BF16, MAXOP>(x, y, wa[k], wb[k]);
        }
      }
#pragma unroll
      for (int o = 0; o < kO; ++o)
        if (po[o]) __builtin_nontemporal_store(ps[o] ? S[o] : pick(R, ro[o]), po[o] + u);
    }
  };
  run_plane(blockIdx.y >> 1, blockIdx.y & 1, int64_t(blockIdx.x) * 256 + threadIdx.x, a.units,
            int64_t(gridDim.x) * 256);
}

// ---------------------------------------------------------------------------
// Temporal RoPE view (Sec. 3.3 "Boundary and positional handling"): memory
// keys are stored without their temporal phase; for attention, entry e is
// exposed at temporal index e.  The layer's view keeps one K block per slot:
// this kernel writes slot s's K with pairs k < P rotated by the angle e * w_k,
// w_k = theta^(-k/P) (fp64, rounded once to the storage type), e being the
// index of the entry the slot holds, into view block s.  Attention reads K
// through the slot table from the view and V from the slots.  Only listed
// slots are written: in full when the slot's entry changed, or only the
// 16-byte units holding temporal pairs when the entry just moved to another
// index.  grid = (blocks per listed slot, listed slots).
// ---------------------------------------------------------------------------

constexpr int kMaxViewPos = 64;  // listed slots per launch

struct RopeViewArgs {
  const char* kv_layer_base;  // pool + kv_offset(layer, 0, 0)
  char* view;                 // the layer's view: K block s at view + s * blk_stride
  size_t slot_stride;         // 2 * blk_stride
  size_t blk_stride;
  int64_t rows;               // N
  int heads;
  int head_dim;
  int pairs;                  // P
  double theta;
  int n_pos;
  int32_t index[kMaxViewPos];  // temporal index of the entry
  int32_t slot[kMaxViewPos];   // its slot
  int32_t full[kMaxViewPos];   // 1: every unit; 0: the units holding temporal pairs
};

template <bool BF16>
__global__ __launch_bounds__(256) void rope_view_kernel(RopeViewArgs a) {
#pragma clang fp contract(off)
  __shared__ double cs[64], sn[64];
  const int e = a.index[blockIdx.y];
  const int tid = threadIdx.x;
  const u32x4* src = reinterpret_cast<const u32x4*>(a.kv_layer_base + size_t(a.slot[blockIdx.y]) * a.slot_stride);
  u32x4* dst = reinterpret_cast<u32x4*>(a.view + size_t(a.slot[blockIdx.y]) * a.blk_stride);
  const int64_t stride = int64_t(gridDim.x) * 256;
  if (tid < a.pairs) {
    const double w = pow(a.theta, -double(tid) / double(a.pairs));
    const double ang = double(e) * w;
    cs[tid] = cos(ang);
    sn[tid] = sin(ang);
  }
  __syncthreads();
  constexpr int kElts = BF16 ? 8 : 4;  // elements per 16-byte unit (whole pairs)
  const int units_per_head = a.head_dim / kElts;
  const int t_units = (2 * a.pairs + kElts - 1) / kElts;  // units of a head holding temporal pairs
  const bool full = a.full[blockIdx.y] != 0;
  const int per_row = a.heads * (full ? units_per_head : t_units);
  const int64_t count = a.rows * per_row;
  for (int64_t i = int64_t(blockIdx.x) * 256 + tid; i < count; i += stride) {
    int64_t u = i;
    if (!full) {  // i-th temporal unit -> its unit in the block
      const int64_t row = i / per_row;
      const int r = int(i - row * per_row);
      u = (row * a.heads + r / t_units) * units_per_head + r % t_units;
    }
    u32x4 x = __builtin_nontemporal_load(src + u);
    const int d0 = int(u % units_per_head) * kElts;  // first element of the unit within its head
    if (d0 < 2 * a.pairs) {
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        if constexpr (BF16) {
          const int k = (d0 >> 1) + w;  // the word holds pair k: (element 2k, element 2k+1)
          if (k < a.pairs) {
            const double x0 = bf16_lo(x[w]), x1 = bf16_hi(x[w]);
            x[w] = pack_bf16_rne(x0 * cs[k] - x1 * sn[k], x0 * sn[k] + x1 * cs[k]);
          }
        } else {
          if (w % 2 == 0) {
            const int k = (d0 >> 1) + w / 2;
            if (k < a.pairs) {
              const double x0 = double(__uint_as_float(x[w])), x1 = double(__uint_as_float(x[w + 1]));
              x[w] = __float_as_uint(float(x0 * cs[k] - x1 * sn[k]));
              x[w + 1] = __float_as_uint(float(x0 * sn[k] + x1 * cs[k]));
            }
          }
        }
      }
    }
    __builtin_nontemporal_store(x, dst + u);
  }
}

constexpr int kMergeUnroll = 4;

// Blocks per (layer, kv) plane for a streaming pass over `units` 16-byte
// units, each thread taking `per_thread` of them.  The streaming passes of
// the insert, the merge and the fused update launch this full cover with the
// plane as grid.y: blocks are dispatched in index order, so the blocks in
// flight at any time work on a few consecutive planes, a few DRAM streams,
// rather than on every (layer, K|V) plane at once (a grid of one resident round,
// striding over all planes together, reached 0.60-0.64 of HBM peak on the
// 30-layer update and merge against 0.70-0.74 for the full cover).
unsigned plane_blocks(int64_t units, int per_thread) {
  int64_t threads = (units + per_thread - 1) / per_thread;
  int64_t b = (threads + 255) / 256;
  if (b < 1) b = 1;
  if (b > 65535) b = 65535;
  return unsigned(b);
}

// Blocks of `threads` threads that are resident on the whole device at once
// for `kernel` (0 on error).  The RoPE view pass launches one such round, so
// no block waits for a second round while most CUs idle.
int resident_blocks(const void* kernel, int threads) {
  // Cached per (device, kernel, threads): the answer never changes.
  struct Entry { int dev; const void* kernel; int threads; int blocks; };
  static Entry seen[32];
  static int n_seen = 0;
  static std::mutex mu;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  std::lock_guard<std::mutex> lock(mu);
  for (int i = 0; i < n_seen; ++i)
    if (seen[i].dev == dev && seen[i].kernel == kernel && seen[i].threads == threads) return seen[i].blocks;
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess) return 0;
  if (n_seen < 32) seen[n_seen++] = Entry{dev, kernel, threads, cus * per_cu};
  return cus * per_cu;
}

// Blocks per plane for a streaming pass over `planes` planes of `units`
// 16-byte units: one resident round spread over the planes (at least one
// block per plane), but no more than covering each plane with `per_thread`
// units per thread.
unsigned stream_blocks_per_plane(const void* kernel, unsigned planes, int64_t units, int per_thread) {
  int resident = resident_blocks(kernel, 256);
  if (resident <= 0) resident = 2048;
  unsigned per_plane = unsigned(resident) / planes;
  if (per_plane < 1) per_plane = 1;
  const unsigned cover = plane_blocks(units, per_thread);
  return per_plane < cover ? per_plane : cover;
}

bool valid_config(const fademem_config* c) {
  if (!c) return false;
  if (c->budget < 2 || c->budget > kMaxBudget) return false;
  if (c->heads < 1 || c->heads > 4096) return false;
  if (c->head_dim != 64 && c->head_dim != 128) return false;
  if (c->tokens_per_block < 1 || c->tokens_per_block > kMaxTokens) return false;
  if (!(c->beta > 0.0 && c->beta <= 1.0)) return false;
  if (c->anchor != 0 && c->anchor != 1) return false;
  if (c->dtype != FADEMEM_F32 && c->dtype != FADEMEM_BF16) return false;
  if (c->merge_op < FADEMEM_MERGE_SQRT_SPAN || c->merge_op > FADEMEM_MERGE_MAX) return false;
  if (c->layers < 1 || c->layers > 4096) return false;
  if (c->rope_pairs < 0 || c->rope_pairs > c->head_dim / 2) return false;
  if (c->rope_pairs > 0 && !(c->rope_theta > 1.0 && c->rope_theta < 1e300)) return false;
  if (c->stage_frames < 0 || c->stage_frames > kMaxPlanFrames) return false;
  return true;
}


// ---------------------------------------------------------------------------
// Host replay (Mirror).  Each function repeats, on the host's copy, what the
// corresponding kernels do to the metadata and the slot table.
// ---------------------------------------------------------------------------

// select_pair on the host: the same integers, the same fp64 operations.
int host_select_pair(const std::vector<int64_t>& span, const std::vector<int64_t>& pos_sum, int n, int64_t t,
                     double beta) {
#pragma clang fp contract(off)
  std::vector<double> u(size_t(n > 1 ? n - 1 : 1));
  for (int i = 0; i < n - 1; ++i) {
    const double d = double(t * span[i] - pos_sum[i]) / double(span[i]);
    u[i] = (beta == 1.0) ? d : pow(d, beta);
  }
  double gm = INFINITY;
  for (int i = 0; i < n - 2; ++i) gm = fmin(gm, fabs(u[i + 1] - u[i]));
  const double tol = 1e-9 * gm;
  for (int i = 0; i < n - 2; ++i)
    if (fabs(u[i + 1] - u[i]) - gm <= tol) return i;
  return 0;
}

void mirror_reset(fademem_cache* c) {
  Mirror& m = c->mirror;
  m.first.clear();
  m.pos_sum.clear();
  m.span.clear();
  m.order.resize(size_t(c->lay.slots));
  for (int64_t i = 0; i < c->lay.slots; ++i) m.order[size_t(i)] = int32_t(i);
  const size_t views = c->cfg.rope_pairs > 0 ? size_t(c->cfg.layers) * size_t(c->lay.slots) : 0;
  c->view_first.assign(views, 0);
  c->view_span.assign(views, 0);
  c->view_index.assign(views, -1);
}

// insert_kernel: the new entry goes to slot order[count].
void mirror_insert(Mirror& m, int64_t t) {
  m.first.push_back(t);
  m.pos_sum.push_back(t);
  m.span.push_back(1);
}

// consolidate_kernel's block 0.
void mirror_consolidate(fademem_cache* c) {
  Mirror& m = c->mirror;
  const int n = int(m.span.size());
  const int j = host_select_pair(m.span, m.pos_sum, n, c->newest, c->cfg.beta);
  const bool anchor_pair = c->cfg.anchor && j == 0;
  const bool select = c->cfg.merge_op == FADEMEM_MERGE_SELECT_NEAREST && !anchor_pair;
  const int32_t dst = m.order[size_t(j)], src = m.order[size_t(j) + 1];
  const int64_t s_new = m.span[size_t(j)] + m.span[size_t(j) + 1];
  m.pos_sum[size_t(j)] = anchor_pair ? m.first[size_t(j)] * s_new : m.pos_sum[size_t(j)] + m.pos_sum[size_t(j) + 1];
  m.span[size_t(j)] = s_new;
  m.first.erase(m.first.begin() + j + 1);
  m.pos_sum.erase(m.pos_sum.begin() + j + 1);
  m.span.erase(m.span.begin() + j + 1);
  m.order[size_t(j)] = select ? src : dst;
  for (int i = j + 1; i < n - 1; ++i) m.order[size_t(i)] = m.order[size_t(i) + 1];
  m.order[size_t(n) - 1] = select ? dst : src;
}

// update_plan_kernel (metadata and slots; the data program is not needed).
void mirror_update(Mirror& m, const fademem_config& cfg, int64_t n_slots, int frames, int64_t first_position,
                   bool staged) {
  const int n0 = int(m.span.size());
  const int slots = int(n_slots);
  std::vector<int32_t> kind(size_t(n0), kRefSlot), idx(m.order.begin(), m.order.begin() + n0);
  std::vector<int32_t> free_list;
  const int skip = staged ? frames : 0;
  for (int i = n0 + skip; i < slots; ++i) free_list.push_back(m.order[size_t(i)]);
  int n_ar = 0;
  for (int f = 0; f < frames; ++f) {
    const int64_t t = first_position + f;
    m.first.push_back(t);
    m.pos_sum.push_back(t);
    m.span.push_back(1);
    kind.push_back(staged ? kRefSlot : kRefFrame);
    idx.push_back(staged ? m.order[size_t(n0 + f)] : f);
    const int n = int(m.span.size());
    if (n <= cfg.budget) continue;
    const int j = host_select_pair(m.span, m.pos_sum, n, t, cfg.beta);
    const bool anchor_pair = cfg.anchor && j == 0;
    const bool select = cfg.merge_op == FADEMEM_MERGE_SELECT_NEAREST && !anchor_pair;
    const int64_t s_new = m.span[size_t(j)] + m.span[size_t(j) + 1];
    int32_t nk, ni;
    if (anchor_pair || select) {
      const int keep = anchor_pair ? j : j + 1, drop = anchor_pair ? j + 1 : j;
      nk = kind[size_t(keep)];
      ni = idx[size_t(keep)];
      if (kind[size_t(drop)] == kRefSlot) free_list.push_back(idx[size_t(drop)]);
    } else {
      if (kind[size_t(j)] == kRefSlot) free_list.push_back(idx[size_t(j)]);
      if (kind[size_t(j) + 1] == kRefSlot) free_list.push_back(idx[size_t(j) + 1]);
      nk = kRefResult;
      ni = n_ar++;
    }
    m.pos_sum[size_t(j)] = anchor_pair ? m.first[size_t(j)] * s_new : m.pos_sum[size_t(j)] + m.pos_sum[size_t(j) + 1];
    m.span[size_t(j)] = s_new;
    kind[size_t(j)] = nk;
    idx[size_t(j)] = ni;
    m.first.erase(m.first.begin() + j + 1);
    m.pos_sum.erase(m.pos_sum.begin() + j + 1);
    m.span.erase(m.span.begin() + j + 1);
    kind.erase(kind.begin() + j + 1);
    idx.erase(idx.begin() + j + 1);
  }
  const int n = int(m.span.size());
  size_t next = 0;
  for (int i = 0; i < n; ++i) m.order[size_t(i)] = kind[size_t(i)] == kRefSlot ? idx[size_t(i)] : free_list[next++];
  for (int i = n; i < slots; ++i) m.order[size_t(i)] = free_list[next++];
}

}  // namespace

namespace fademem {

int compute_layout(const fademem_config* cfg, Layout* lay) {
  if (!valid_config(cfg)) return FADEMEM_EINVAL;
  Layout L{};
  L.slots = cfg->budget + (cfg->stage_frames > 1 ? cfg->stage_frames : 1);
  size_t off = round_up(sizeof(DevHeader), 256);
  for (int c = 0; c < 2; ++c) {
    L.off_first[c] = off;   off = round_up(off + 8 * size_t(L.slots), 256);
    L.off_pos_sum[c] = off; off = round_up(off + 8 * size_t(L.slots), 256);
    L.off_span[c] = off;    off = round_up(off + 8 * size_t(L.slots), 256);
    L.off_order[c] = off;   off = round_up(off + 4 * size_t(L.slots), 256);
  }
  L.off_log = off;     off = round_up(off + 4 * size_t(kLogCap), 256);
  L.off_prog = off;    off = round_up(off + sizeof(UpdatePlan), 256);
  L.meta_bytes = off;
  L.elt = cfg->dtype == FADEMEM_BF16 ? 2 : 4;
  L.row_elems = size_t(cfg->heads) * size_t(cfg->head_dim);
  const double blk = double(cfg->tokens_per_block) * double(L.row_elems) * double(L.elt);
  if (blk > 1e15) return FADEMEM_EINVAL;
  L.blk_bytes = size_t(cfg->tokens_per_block) * L.row_elems * L.elt;
  L.blk_stride = round_up(L.blk_bytes, 256);
  L.off_ws = L.meta_bytes + size_t(cfg->layers) * size_t(L.slots) * 2 * L.blk_stride;
  L.ws_bytes = cfg->dtype == FADEMEM_BF16 ? attend_ws_bytes(cfg->head_dim) : f32_ws_bytes(cfg->head_dim);
  L.off_view = round_up(L.off_ws + L.ws_bytes, 256);
  // One K block per slot and layer: every entry the memory can expose
  // (M + 1 after an insert, or M plus the staged frames).
  L.view_bytes = cfg->rope_pairs > 0 ? size_t(cfg->layers) * size_t(L.slots) * L.blk_stride : 0;
  L.total = L.off_view + L.view_bytes;
  *lay = L;
  return FADEMEM_OK;
}

}  // namespace fademem

namespace {

// Compare the host replay with the device's current metadata copy
// (synchronises the stream).
int verify_mirror(fademem_cache* c, void* stream) {
  hipError_t e = hipStreamSynchronize(as_stream(stream));
  if (e != hipSuccess) return hip_fail(c, e);
  const Mirror& m = c->mirror;
  const size_t n = size_t(c->count);
  if (m.span.size() != n) return FADEMEM_EINTERNAL;
  std::vector<int64_t> buf(n);
  const std::vector<int64_t>* want[3] = {&m.first, &m.pos_sum, &m.span};
  const size_t offs[3] = {c->lay.off_first[c->cur], c->lay.off_pos_sum[c->cur], c->lay.off_span[c->cur]};
  for (int a = 0; a < 3; ++a) {
    if (n == 0) break;
    if ((e = hipMemcpy(buf.data(), c->pool + offs[a], n * sizeof(int64_t), hipMemcpyDeviceToHost)) != hipSuccess)
      return hip_fail(c, e);
    if (buf != *want[a]) return FADEMEM_EINTERNAL;
  }
  std::vector<int32_t> ord(size_t(c->lay.slots));
  if ((e = hipMemcpy(ord.data(), c->pool + c->lay.off_order[c->cur], ord.size() * sizeof(int32_t),
                     hipMemcpyDeviceToHost)) != hipSuccess)
    return hip_fail(c, e);
  if (ord != m.order) return FADEMEM_EINTERNAL;
  return FADEMEM_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------

extern "C" {

const char* fademem_strerror(int code) {
  switch (code) {
    case FADEMEM_OK: return "ok";
    case FADEMEM_EINVAL: return "invalid argument or configuration";
    case FADEMEM_ESTATE: return "call not allowed in the current memory state";
    case FADEMEM_ENOMEM: return "device pool too small";
    case FADEMEM_EHIP: return "HIP runtime or launch error";
    case FADEMEM_EUNSUPPORTED: return "not supported by this build";
    case FADEMEM_EINTERNAL: return "host replay of the memory state disagrees with the device";
    case FADEMEM_ESCRATCH: return "request exceeds the static scratch of the allocation-free entry point";
    default: return "unknown error";
  }
}

int fademem_pool_bytes(const fademem_config* cfg, size_t* bytes) {
  if (!bytes) return FADEMEM_EINVAL;
  Layout L;
  int rc = compute_layout(cfg, &L);
  if (rc) return rc;
  *bytes = L.total;
  return FADEMEM_OK;
}

int fademem_cache_create(const fademem_config* cfg, void* dev_pool, size_t pool_bytes, void* stream,
                         fademem_cache** out) {
  if (!out) return FADEMEM_EINVAL;
  *out = nullptr;
  Layout L;
  int rc = compute_layout(cfg, &L);
  if (rc) return rc;
  if (!dev_pool || !aligned(dev_pool, 256)) return FADEMEM_EINVAL;
  if (pool_bytes < L.total) return FADEMEM_ENOMEM;
  fademem_cache* c = new (std::nothrow) fademem_cache();
  if (!c) return FADEMEM_ENOMEM;
  c->cfg = *cfg;
  c->lay = L;
  c->pool = static_cast<char*>(dev_pool);
  c->count = 0;
  c->newest = 0;
  c->inserted = 0;
  c->cur = 0;
  c->any_inserted = false;
  const char* ser = getenv("FADEMEM_SERIALIZE");
  c->serialize = ser && ser[0] && strcmp(ser, "0") != 0;
  c->last_hip_error = 0;
  try {
    mirror_reset(c);
    c->mirror.first.reserve(size_t(L.slots));
    c->mirror.pos_sum.reserve(size_t(L.slots));
    c->mirror.span.reserve(size_t(L.slots));
  } catch (...) {
    delete c;
    return FADEMEM_ENOMEM;
  }
  (void)hipGetLastError();
  const unsigned blocks = unsigned((L.slots + 255) / 256);
  hipLaunchKernelGGL(init_kernel, dim3(blocks), dim3(256), 0, as_stream(stream), c->pool, L);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    delete c;
    return FADEMEM_EHIP;
  }
  *out = c;
  return FADEMEM_OK;
}

int fademem_cache_destroy(fademem_cache* cache) {
  delete cache;
  return FADEMEM_OK;
}

int fademem_count(const fademem_cache* cache, int64_t* count) {
  if (!cache || !count) return FADEMEM_EINVAL;
  *count = cache->count;
  return FADEMEM_OK;
}

int fademem_last_hip_error(const fademem_cache* cache) { return cache ? cache->last_hip_error : 0; }

int fademem_insert(fademem_cache* c, const void* const* k, const void* const* v, int64_t position, void* stream) {
  if (!c || !k || !v) return FADEMEM_EINVAL;
  if (position <= -kMaxPosition || position >= kMaxPosition) return FADEMEM_EINVAL;
  const int layers = c->cfg.layers;
  for (int l = 0; l < layers; ++l) {
    if (!k[l] || !v[l] || !aligned(k[l], 16) || !aligned(v[l], 16)) return FADEMEM_EINVAL;
  }
  if (c->count > c->cfg.budget) return FADEMEM_ESTATE;
  if (c->any_inserted && position <= c->newest) return FADEMEM_ESTATE;
  // t*s_i and first*s_i must stay exact in int64: |t| * (blocks ever held) < 2^62.
  {
    const unsigned __int128 mag = (unsigned __int128)(position < 0 ? -position : position) + 1;
    if (mag * (unsigned __int128)(c->inserted + 1) >= ((unsigned __int128)1 << 62)) return FADEMEM_ESTATE;
  }
  (void)hipGetLastError();
  const int64_t units = int64_t(c->lay.blk_bytes / 16);
  for (int l0 = 0; l0 < layers; l0 += kMaxLayersPerLaunch) {
    const int nl = (layers - l0) < kMaxLayersPerLaunch ? (layers - l0) : kMaxLayersPerLaunch;
    InsertArgs a;
    memset(&a, 0, sizeof(a));
    for (int l = 0; l < nl; ++l) {
      a.k[l] = k[l0 + l];
      a.v[l] = v[l0 + l];
    }
    a.pool = c->pool;
    a.lay = c->lay;
    a.layer0 = l0;
    a.units = units;
    a.index = c->count;
    a.position = position;
    a.cur = c->cur;
    a.write_meta = (l0 == 0);
    hipLaunchKernelGGL(insert_kernel, dim3(plane_blocks(units, 4), unsigned(2 * nl)), dim3(256), 0,
                       as_stream(stream), a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(c, e);
  }
  mirror_insert(c->mirror, position);  // capacity reserved at creation: no allocation
  c->count += 1;
  c->inserted += 1;
  c->newest = position;
  c->any_inserted = true;
  return finish(c, stream);
}

int fademem_consolidate(fademem_cache* c, void* stream) {
  if (!c) return FADEMEM_EINVAL;
  if (c->count <= c->cfg.budget) return FADEMEM_OK;  // Alg. S1: within budget, nothing to do
  (void)hipGetLastError();
  ConsolidateArgs a;
  a.pool = c->pool;
  a.lay = c->lay;
  a.n = int(c->count);
  a.layers = c->cfg.layers;
  a.t = c->newest;
  a.beta = c->cfg.beta;
  a.anchor = c->cfg.anchor;
  a.op = c->cfg.merge_op;
  a.cur = c->cur;
  a.units = int64_t(c->lay.blk_bytes / 16);
  const bool bf16 = c->cfg.dtype == FADEMEM_BF16, maxop = c->cfg.merge_op == FADEMEM_MERGE_MAX;
  auto kernel = bf16 ? (maxop ? consolidate_kernel<true, kMergeUnroll, true> : consolidate_kernel<true, kMergeUnroll, false>)
                     : (maxop ? consolidate_kernel<false, kMergeUnroll, true> : consolidate_kernel<false, kMergeUnroll, false>);

  // Full cover, plane-major (every block also derives the schedule: O(M)
  // work beside the 256 * kMergeUnroll units it streams).  Select Nearest
  // never moves K/V bytes: one block splices the metadata.
  const unsigned planes = unsigned(2 * c->cfg.layers);
  const bool moves_bytes = c->cfg.merge_op != FADEMEM_MERGE_SELECT_NEAREST;
  const dim3 blocks(moves_bytes ? plane_blocks(a.units, kMergeUnroll) : 1u, moves_bytes ? planes : 1u);
  hipLaunchKernelGGL(kernel, dim3(blocks), dim3(256), 0, as_stream(stream), a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(c, e);
  mirror_consolidate(c);  // erases in place: no allocation
  c->cur ^= 1;
  c->count -= 1;
  return finish(c, stream);
}

}  // extern "C"

namespace {

// The F updates of a chunk (fademem_update, fademem_update_staged).  k, v:
// the caller's chunk per layer, or NULL when the frames are staged in the
// slots order[count + f].
int update_impl(fademem_cache* c, const void* const* k, const void* const* v, int64_t frames, int64_t first_position,
                bool staged, void* stream) {
  // Every position f, first_position <= f <= first_position + frames - 1, must satisfy |f| < 2^40.
  if (first_position <= -kMaxPosition || first_position > kMaxPosition - frames) return FADEMEM_EINVAL;
  const int layers = c->cfg.layers;
  if (c->count > c->cfg.budget) return FADEMEM_ESTATE;
  if (c->any_inserted && first_position <= c->newest) return FADEMEM_ESTATE;
  // t*s_i and first*s_i must stay exact in int64 (as for fademem_insert).
  {
    const int64_t last = first_position + frames - 1;
    const int64_t a0 = first_position < 0 ? -first_position : first_position;
    const int64_t a1 = last < 0 ? -last : last;
    const unsigned __int128 mag = (unsigned __int128)(a0 > a1 ? a0 : a1) + 1;
    if (mag * (unsigned __int128)(c->inserted + frames) >= ((unsigned __int128)1 << 62)) return FADEMEM_ESTATE;
  }
  // The host replay of the whole call, committed once everything is enqueued.
  Mirror next;
  try {
    next = c->mirror;
    for (int64_t f0 = 0; f0 < frames; f0 += kMaxPlanFrames) {
      const int nf = int((frames - f0) < kMaxPlanFrames ? (frames - f0) : kMaxPlanFrames);
      mirror_update(next, c->cfg, c->lay.slots, nf, first_position + f0, staged);
    }
    // Inserts push onto these without allocating.
    next.first.reserve(size_t(c->lay.slots));
    next.pos_sum.reserve(size_t(c->lay.slots));
    next.span.reserve(size_t(c->lay.slots));
  } catch (...) {
    return FADEMEM_ENOMEM;
  }
  (void)hipGetLastError();
  const int64_t units = int64_t(c->lay.blk_bytes / 16);
  const bool bf16 = c->cfg.dtype == FADEMEM_BF16, maxop = c->cfg.merge_op == FADEMEM_MERGE_MAX;
  // Staged updates, and fused ones whose grid fits two resident rounds of
  // the four-frame instance, launch the instance sized for the plan's frames
  // (fewer registers, more resident waves: 6% faster staged at 30 layers, 6%
  // faster fused at one layer); larger fused grids keep the four-frame one,
  // which the smaller instance slowed by 2% at 30 layers.
  typedef void (*DataKernel)(UpdateDataArgs);
  static_assert(kMaxPlanFrames == 4, "one data kernel per plan size");
  static const DataKernel data_kernels[2][2][kMaxPlanFrames] = {
      {{update_data_kernel<false, false, 1>, update_data_kernel<false, false, 2>, update_data_kernel<false, false, 3>,
        update_data_kernel<false, false, 4>},
       {update_data_kernel<false, true, 1>, update_data_kernel<false, true, 2>, update_data_kernel<false, true, 3>,
        update_data_kernel<false, true, 4>}},
      {{update_data_kernel<true, false, 1>, update_data_kernel<true, false, 2>, update_data_kernel<true, false, 3>,
        update_data_kernel<true, false, 4>},
       {update_data_kernel<true, true, 1>, update_data_kernel<true, true, 2>, update_data_kernel<true, true, 3>,
        update_data_kernel<true, true, 4>}}};
  const unsigned per_plane = plane_blocks(units, 1);
  for (int64_t f0 = 0; f0 < frames; f0 += kMaxPlanFrames) {
    const int nf = int((frames - f0) < kMaxPlanFrames ? (frames - f0) : kMaxPlanFrames);
    PlanArgs pa;
    pa.pool = c->pool;
    pa.lay = c->lay;
    pa.n0 = int(c->count);
    pa.frames = nf;
    pa.first_position = first_position + f0;
    pa.budget = c->cfg.budget;
    pa.beta = c->cfg.beta;
    pa.anchor = c->cfg.anchor;
    pa.op = c->cfg.merge_op;
    pa.cur = c->cur;
    pa.staged = staged ? 1 : 0;
    hipLaunchKernelGGL(update_plan_kernel, dim3(1), dim3(256), 0, as_stream(stream), pa);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(c, e);
    for (int l0 = 0; l0 < layers; l0 += kMaxLayersPerLaunch) {
      const int nl = (layers - l0) < kMaxLayersPerLaunch ? (layers - l0) : kMaxLayersPerLaunch;
      UpdateDataArgs da;
      memset(&da, 0, sizeof(da));
      if (!staged) {
        for (int l = 0; l < nl; ++l) {
          da.k[l] = static_cast<const char*>(k[l0 + l]) + size_t(f0) * c->lay.blk_bytes;
          da.v[l] = static_cast<const char*>(v[l0 + l]) + size_t(f0) * c->lay.blk_bytes;
        }
      }
      da.pool = c->pool;
      da.lay = c->lay;
      da.layer0 = l0;
      da.units = units;
      const DataKernel wide = data_kernels[bf16][maxop][kMaxPlanFrames - 1];
      const int resident = resident_blocks(reinterpret_cast<const void*>(wide), 256);
      const bool small_grid = resident > 0 && int64_t(per_plane) * 2 * nl <= 2 * int64_t(resident);
      const DataKernel data_kernel = (staged || small_grid) ? data_kernels[bf16][maxop][nf - 1] : wide;
      hipLaunchKernelGGL(data_kernel, dim3(per_plane, unsigned(2 * nl)), dim3(256), 0, as_stream(stream), da);
      e = hipGetLastError();
      if (e != hipSuccess) return hip_fail(c, e);
    }
    // Host mirror of the count: each frame appends, then consolidates back
    // to M when over budget.
    for (int f = 0; f < nf; ++f) {
      c->count += 1;
      if (c->count > c->cfg.budget) c->count -= 1;
    }
    c->cur ^= 1;
    c->inserted += nf;
    c->newest = first_position + f0 + nf - 1;
    c->any_inserted = true;
  }
  c->mirror = std::move(next);
  return finish(c, stream);
}

// Bring layer `layer`'s re-indexed K view up to date for the first `held`
// entries (memory) and the `staged` after them (staged frames): a slot whose
// entry changed is rewritten in full, a slot whose entry only moved to
// another index has its temporal units rotated again; staged frames are
// always rewritten in full (their contents are the caller's).
int refresh_view(fademem_cache* c, int32_t layer, int held, int staged, void* stream) {
  const size_t base = size_t(layer) * size_t(c->lay.slots);
  RopeViewArgs r;
  r.kv_layer_base = c->pool + kv_offset(c->lay, layer, 0, 0);
  r.view = c->pool + c->lay.off_view + base * c->lay.blk_stride;
  r.slot_stride = 2 * c->lay.blk_stride;
  r.blk_stride = c->lay.blk_stride;
  r.rows = c->cfg.tokens_per_block;
  r.heads = c->cfg.heads;
  r.head_dim = c->cfg.head_dim;
  r.pairs = c->cfg.rope_pairs;
  r.theta = c->cfg.rope_theta;
  r.n_pos = 0;
  auto vk = c->cfg.dtype == FADEMEM_BF16 ? rope_view_kernel<true> : rope_view_kernel<false>;
  const int64_t units = int64_t(c->lay.blk_bytes / 16);
  auto flush = [&]() -> int {
    if (r.n_pos == 0) return FADEMEM_OK;
    const dim3 grid(stream_blocks_per_plane(reinterpret_cast<const void*>(vk), unsigned(r.n_pos), units, 4),
                    unsigned(r.n_pos));
    hipLaunchKernelGGL(vk, grid, dim3(256), 0, as_stream(stream), r);
    r.n_pos = 0;
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? FADEMEM_OK : hip_fail(c, e);
  };
  auto add = [&](int i, int32_t slot, bool full) -> int {
    r.index[r.n_pos] = i;
    r.slot[r.n_pos] = slot;
    r.full[r.n_pos] = full ? 1 : 0;
    return ++r.n_pos == kMaxViewPos ? flush() : FADEMEM_OK;
  };
  for (int i = 0; i < held + staged; ++i) {
    const int32_t slot = c->mirror.order[size_t(i)];
    const size_t v = base + size_t(slot);
    int rc = FADEMEM_OK;
    if (i >= held) {
      rc = add(i, slot, true);
      c->view_span[v] = 0;  // rebuilt on every use
    } else if (c->view_first[v] != c->mirror.first[size_t(i)] || c->view_span[v] != c->mirror.span[size_t(i)]) {
      rc = add(i, slot, true);
      c->view_first[v] = c->mirror.first[size_t(i)];
      c->view_span[v] = c->mirror.span[size_t(i)];
    } else if (c->view_index[v] != i) {
      rc = add(i, slot, false);
    }
    c->view_index[v] = i;
    if (rc) return rc;
  }
  return flush();
}

// Attention over [memory || staged frames || current chunk] (the staged
// frames are exposed as entries after the memory's).
int attend_impl(fademem_cache* c, int32_t layer, const void* q, int64_t q_tokens, const void* k_cur,
                const void* v_cur, int64_t cur_tokens, int64_t staged, float scale, void* out, float* lse,
                void* stream) {
  if (layer < 0 || layer >= c->cfg.layers) return FADEMEM_EINVAL;
  if (q_tokens < 0 || q_tokens > kMaxTokens || cur_tokens < 0 || cur_tokens > kMaxTokens) return FADEMEM_EINVAL;
  if (q_tokens == 0) return FADEMEM_OK;
  if (!q || !out || !aligned(q, 16) || !aligned(out, 16)) return FADEMEM_EINVAL;
  if (lse && !aligned(lse, 4)) return FADEMEM_EINVAL;
  if (cur_tokens > 0 && (!k_cur || !v_cur || !aligned(k_cur, 16) || !aligned(v_cur, 16))) return FADEMEM_EINVAL;
  const int64_t entries = c->count + staged;
  if (entries == 0 && cur_tokens == 0) return FADEMEM_EINVAL;  // no keys at all
  const double total_keys = double(entries) * double(c->cfg.tokens_per_block) + double(cur_tokens);
  if (total_keys > double(kMaxTokens)) return FADEMEM_EINVAL;
  if (!(scale >= 0.0f) || isinf(scale)) return FADEMEM_EINVAL;
  AttendArgs a;
  a.q = q;
  a.out = out;
  a.lse = lse;
  a.k_base = c->pool + kv_offset(c->lay, layer, 0, 0);
  a.k_order = reinterpret_cast<const int32_t*>(c->pool + c->lay.off_order[c->cur]);
  a.k_stride = 2 * c->lay.blk_stride;
  a.v_base = a.k_base + c->lay.blk_stride;
  a.v_order = a.k_order;
  a.v_stride = a.k_stride;
  a.k_cur = k_cur;
  a.v_cur = v_cur;
  a.n_entries = entries;
  a.tokens_per_block = c->cfg.tokens_per_block;
  a.cur_tokens = cur_tokens;
  a.q_tokens = q_tokens;
  a.ws = reinterpret_cast<float*>(c->pool + c->lay.off_ws);
  a.heads = c->cfg.heads;
  a.head_dim = c->cfg.head_dim;
  a.scale = scale > 0.0f ? scale : 1.0f / sqrtf(float(c->cfg.head_dim));
  (void)hipGetLastError();
  if (c->cfg.rope_pairs > 0 && entries > 0) {
    // Expose the memory re-indexed: keys from the layer's rotated K view
    // (one block per slot, read through the slot table), values from the
    // slots as stored.
    const int rc = refresh_view(c, layer, int(c->count), int(staged), stream);
    if (rc) return rc;
    a.k_base = c->pool + c->lay.off_view + size_t(layer) * size_t(c->lay.slots) * c->lay.blk_stride;
    a.k_stride = c->lay.blk_stride;
  }
  hipError_t e = (c->cfg.dtype == FADEMEM_BF16) ? launch_attend_bf16(a, as_stream(stream))
                                                : launch_attend_f32(a, as_stream(stream));
  if (e != hipSuccess) return hip_fail(c, e);
  return finish(c, stream);
}

bool chunk_ptrs_ok(const fademem_cache* c, const void* const* k, const void* const* v) {
  if (!k || !v) return false;
  for (int l = 0; l < c->cfg.layers; ++l)
    if (!k[l] || !v[l] || !aligned(k[l], 16) || !aligned(v[l], 16)) return false;
  return true;
}

}  // namespace

extern "C" {

int fademem_update(fademem_cache* c, const void* const* k, const void* const* v, int64_t frames,
                   int64_t first_position, void* stream) {
  if (!c) return FADEMEM_EINVAL;
  if (frames < 1 || frames > kMaxTokens) return FADEMEM_EINVAL;
  if (!chunk_ptrs_ok(c, k, v)) return FADEMEM_EINVAL;
  return update_impl(c, k, v, frames, first_position, false, stream);
}

int fademem_stage(fademem_cache* c, int64_t frames, void** k, void** v) {
  if (!c || !k || !v) return FADEMEM_EINVAL;
  if (frames < 1 || frames > c->cfg.stage_frames) return FADEMEM_EINVAL;
  if (c->count > c->cfg.budget) return FADEMEM_ESTATE;
  for (int l = 0; l < c->cfg.layers; ++l)
    for (int64_t f = 0; f < frames; ++f) {
      const int32_t slot = c->mirror.order[size_t(c->count + f)];
      k[size_t(l) * size_t(frames) + size_t(f)] = c->pool + kv_offset(c->lay, l, slot, 0);
      v[size_t(l) * size_t(frames) + size_t(f)] = c->pool + kv_offset(c->lay, l, slot, 1);
    }
  return FADEMEM_OK;
}

int fademem_update_staged(fademem_cache* c, int64_t frames, int64_t first_position, void* stream) {
  if (!c) return FADEMEM_EINVAL;
  if (frames < 1 || frames > c->cfg.stage_frames) return FADEMEM_EINVAL;
  return update_impl(c, nullptr, nullptr, frames, first_position, true, stream);
}

int fademem_attend(fademem_cache* c, int32_t layer, const void* q, int64_t q_tokens, const void* k_cur,
                   const void* v_cur, int64_t cur_tokens, float scale, void* out, float* lse, void* stream) {
  if (!c) return FADEMEM_EINVAL;
  return attend_impl(c, layer, q, q_tokens, k_cur, v_cur, cur_tokens, 0, scale, out, lse, stream);
}

int fademem_attend_staged(fademem_cache* c, int32_t layer, const void* q, int64_t q_tokens, int64_t frames,
                          float scale, void* out, float* lse, void* stream) {
  if (!c) return FADEMEM_EINVAL;
  if (frames < 1 || frames > c->cfg.stage_frames) return FADEMEM_EINVAL;
  if (c->count > c->cfg.budget) return FADEMEM_ESTATE;
  return attend_impl(c, layer, q, q_tokens, nullptr, nullptr, 0, frames, scale, out, lse, stream);
}

int fademem_verify(fademem_cache* c, void* stream) {
  if (!c) return FADEMEM_EINVAL;
  return verify_mirror(c, stream);
}

int fademem_get_state(fademem_cache* c, int64_t* count, int64_t* first, int64_t* span, int64_t* pos_sum,
                      int64_t* newest, void* stream) {
  if (!c) return FADEMEM_EINVAL;
  hipError_t e = hipStreamSynchronize(as_stream(stream));
  if (e != hipSuccess) return hip_fail(c, e);
  const size_t n = size_t(c->count);
  if (count) *count = c->count;
  if (newest) *newest = c->any_inserted ? c->newest : 0;
  struct Item { int64_t* dst; size_t off; } items[3] = {{first, c->lay.off_first[c->cur]},
                                                        {span, c->lay.off_span[c->cur]},
                                                        {pos_sum, c->lay.off_pos_sum[c->cur]}};
  for (const Item& it : items) {
    if (it.dst && n > 0) {
      e = hipMemcpy(it.dst, c->pool + it.off, n * sizeof(int64_t), hipMemcpyDeviceToHost);
      if (e != hipSuccess) return hip_fail(c, e);
    }
  }
  return FADEMEM_OK;
}

int fademem_entry_kv(fademem_cache* c, int32_t layer, int64_t i, const void** k, const void** v, void* stream) {
  if (!c || !k || !v) return FADEMEM_EINVAL;
  if (layer < 0 || layer >= c->cfg.layers || i < 0 || i >= c->count) return FADEMEM_EINVAL;
  hipError_t e = hipStreamSynchronize(as_stream(stream));
  if (e != hipSuccess) return hip_fail(c, e);
  int32_t slot = 0;
  e = hipMemcpy(&slot, c->pool + c->lay.off_order[c->cur] + 4 * size_t(i), sizeof(int32_t), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(c, e);
  *k = c->pool + kv_offset(c->lay, layer, slot, 0);
  *v = c->pool + kv_offset(c->lay, layer, slot, 1);
  return FADEMEM_OK;
}

int fademem_set_state(fademem_cache* c, int64_t count, const int64_t* first, const int64_t* span,
                      const int64_t* pos_sum, int64_t newest, const void* const* k, const void* const* v,
                      void* stream) {
  if (!c) return FADEMEM_EINVAL;
  if (c->count != 0 || c->any_inserted) return FADEMEM_ESTATE;
  if (count < 0 || count > c->cfg.budget) return FADEMEM_EINVAL;
  if (count == 0) return FADEMEM_OK;
  if (!first || !span || !pos_sum || !k || !v) return FADEMEM_EINVAL;
  if (newest <= -kMaxPosition || newest >= kMaxPosition) return FADEMEM_EINVAL;
  int64_t blocks = 0;
  for (int64_t i = 0; i < count; ++i) {
    if (first[i] <= -kMaxPosition || first[i] >= kMaxPosition || span[i] < 1 || span[i] > kMaxPosition)
      return FADEMEM_EINVAL;
    // the positions an entry covers are distinct integers after the previous entry's and up to newest
    if (i > 0 && first[i] - first[i - 1] < span[i - 1]) return FADEMEM_EINVAL;
    const __int128 lo = (__int128)first[i] * span[i], hi = (__int128)newest * span[i];
    if ((__int128)pos_sum[i] < lo || (__int128)pos_sum[i] > hi) return FADEMEM_EINVAL;
    blocks += span[i];
  }
  if (newest < first[count - 1] + span[count - 1] - 1) return FADEMEM_EINVAL;
  {
    const unsigned __int128 mag = (unsigned __int128)(newest < 0 ? -newest : newest) + 1;
    if (mag * (unsigned __int128)(blocks + 1) >= ((unsigned __int128)1 << 62)) return FADEMEM_EINVAL;
  }
  const int layers = c->cfg.layers;
  for (int64_t q = 0; q < int64_t(layers) * count; ++q)
    if (!k[q] || !v[q] || !aligned(k[q], 16) || !aligned(v[q], 16)) return FADEMEM_EINVAL;
  // Entry i goes to slot i (the slot table of a new cache is the identity),
  // metadata into copy 0.
  hipStream_t s = as_stream(stream);
  (void)hipGetLastError();
  hipError_t e = hipStreamSynchronize(s);  // the cache's initialisation has run
  if (e != hipSuccess) return hip_fail(c, e);
  const size_t n = size_t(count) * sizeof(int64_t);
  if ((e = hipMemcpy(c->pool + c->lay.off_first[0], first, n, hipMemcpyHostToDevice)) != hipSuccess ||
      (e = hipMemcpy(c->pool + c->lay.off_span[0], span, n, hipMemcpyHostToDevice)) != hipSuccess ||
      (e = hipMemcpy(c->pool + c->lay.off_pos_sum[0], pos_sum, n, hipMemcpyHostToDevice)) != hipSuccess)
    return hip_fail(c, e);
  for (int l = 0; l < layers; ++l)
    for (int64_t i = 0; i < count; ++i) {
      const size_t q = size_t(l) * size_t(count) + size_t(i);
      if ((e = hipMemcpyAsync(c->pool + kv_offset(c->lay, l, i, 0), k[q], c->lay.blk_bytes, hipMemcpyDeviceToDevice,
                              s)) != hipSuccess ||
          (e = hipMemcpyAsync(c->pool + kv_offset(c->lay, l, i, 1), v[q], c->lay.blk_bytes, hipMemcpyDeviceToDevice,
                              s)) != hipSuccess)
        return hip_fail(c, e);
    }
  if ((e = hipStreamSynchronize(s)) != hipSuccess) return hip_fail(c, e);
  try {
    mirror_reset(c);
    c->mirror.first.assign(first, first + count);
    c->mirror.span.assign(span, span + count);
    c->mirror.pos_sum.assign(pos_sum, pos_sum + count);
    c->mirror.first.reserve(size_t(c->lay.slots));
    c->mirror.pos_sum.reserve(size_t(c->lay.slots));
    c->mirror.span.reserve(size_t(c->lay.slots));
  } catch (...) {
    return FADEMEM_ENOMEM;
  }
  c->cur = 0;
  c->count = count;
  c->newest = newest;
  c->inserted = blocks;
  c->any_inserted = true;
  return FADEMEM_OK;
}

int fademem_merge_log(fademem_cache* c, int32_t* j, int64_t cap, int64_t* total, void* stream) {
  if (!c || !total || cap < 0 || (cap > 0 && !j)) return FADEMEM_EINVAL;
  hipError_t e = hipStreamSynchronize(as_stream(stream));
  if (e != hipSuccess) return hip_fail(c, e);
  DevHeader h;
  e = hipMemcpy(&h, c->pool, sizeof(h), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(c, e);
  *total = h.merges_total;
  int64_t keep = h.merges_total;
  if (keep > kLogCap) keep = kLogCap;
  if (keep > cap) keep = cap;
  if (keep == 0) return FADEMEM_OK;
  int32_t ring[kLogCap];
  e = hipMemcpy(ring, c->pool + c->lay.off_log, sizeof(ring), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(c, e);
  for (int64_t r = 0; r < keep; ++r) {
    const int64_t idx = h.merges_total - keep + r;
    j[r] = ring[idx % kLogCap];
  }
  return FADEMEM_OK;
}

int fademem_merge_counts(fademem_cache* c, int64_t* total, int64_t* anchor, void* stream) {
  if (!c) return FADEMEM_EINVAL;
  hipError_t e = hipStreamSynchronize(as_stream(stream));
  if (e != hipSuccess) return hip_fail(c, e);
  DevHeader h;
  e = hipMemcpy(&h, c->pool, sizeof(h), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(c, e);
  if (total) *total = h.merges_total;
  if (anchor) *anchor = h.anchor_merges;
  return FADEMEM_OK;
}

}  // extern "C"
