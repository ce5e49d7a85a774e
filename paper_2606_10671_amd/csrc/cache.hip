// FadeMem bounded memory on the device: pool layout, the C ABI, and the
// bookkeeping kernels (insert copy, schedule, merge).
//
// Paper: FadeMem, arXiv 2606.10671 -- Sec. 3.1 (bounded ordered memory),
// Sec. 3.3 (insertion, distance-aware scheduling, consolidation operator,
// boundary handling) and Algorithm S1 (the complete update).
#include <math.h>
#include <string.h>

#include <new>

#include "fademem_internal.h"

using namespace fademem;

struct fademem_cache {
  fademem_config cfg;
  Layout lay;
  char* pool;
  int64_t count;        // entries held (mirrors the device state exactly)
  int64_t newest;       // newest inserted position
  int64_t inserted;     // blocks inserted so far
  int cur;              // metadata copy holding the current state (0 or 1)
  bool any_inserted;
  int last_hip_error;
};

namespace {

inline size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

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
// the decision from the current metadata copy, which no block writes:
//   d_i = t - mu_i = (t*s_i - pos_sum_i) / s_i   (exact numerator, one fp64 division)
//   u_i = d_i^beta
//   g_i = |u_{i+1} - u_i| for the pairs i = 0..n-3 (the pair holding the
//         newest entry, n-2..n-1, is not eligible)
//   j   = lowest i with g_i - min(g) <= 1e-9 * min(g)
// Block 0 writes the spliced metadata into the other copy (spans add,
// pos_sum adds so mu is span-weighted; the anchor keeps its position, the
// slot of entry j+1 is freed) and appends j to the merge log.  Unless the
// pair holds the anchor, all blocks then merge entry j+1 into entry j's
// slot: X_new = w_j X_j + w_{j+1} X_{j+1}, each element in fp64 as two
// products and one sum, rounded once to the storage type.  The blocks of
// each (layer, K|V) plane stride over it with 16-byte nontemporal
// loads/stores, UNROLL units in flight per thread; grid.y = layer * 2 + kv.
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
  for (int i = tid; i < n - 1; i += 256) {
    const int64_t s = m.span[i];
    const double d = double(a.t * s - m.pos_sum[i]) / double(s);
    u_s[i] = (a.beta == 1.0) ? d : pow(d, a.beta);
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
  const int j = block_min_i32(cand, red_i);

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

  const double rj = sqrt(double(s_j));
  const double rj1 = sqrt(double(s_j1));
  const double wa = a.op == FADEMEM_MERGE_AVERAGE ? 0.5 : rj / (rj + rj1);
  const double wb = 1.0 - wa;
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
          u32x4 o;
          if constexpr (MAXOP) {
            // Max pooling: the newer value (y) only when strictly greater,
            // so equal values keep the older bits.
#pragma unroll
            for (int w = 0; w < 4; ++w) {
              if constexpr (BF16) {
                const uint32_t xl = x[r][w] << 16, yl = y[r][w] << 16;
                const uint32_t xh = x[r][w] & 0xFFFF0000u, yh = y[r][w] & 0xFFFF0000u;
                const uint32_t lo = (__uint_as_float(yl) > __uint_as_float(xl)) ? yl : xl;
                const uint32_t hi = (__uint_as_float(yh) > __uint_as_float(xh)) ? yh : xh;
                o[w] = (lo >> 16) | hi;
              } else {
                o[w] = (__uint_as_float(y[r][w]) > __uint_as_float(x[r][w])) ? y[r][w] : x[r][w];
              }
            }
          } else if constexpr (BF16) {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
              const double lo = wa * bf16_lo(x[r][w]) + wb * bf16_lo(y[r][w]);
              const double hi = wa * bf16_hi(x[r][w]) + wb * bf16_hi(y[r][w]);
              o[w] = pack_bf16_rne(lo, hi);
            }
          } else {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
              const double v = wa * double(__uint_as_float(x[r][w])) + wb * double(__uint_as_float(y[r][w]));
              o[w] = __float_as_uint(float(v));
            }
          }
          __builtin_nontemporal_store(o, dst + u);
        }
      }
    }
  }
}

constexpr int kMergeUnroll = 4;

// Blocks per (layer, kv) plane for a streaming pass over `units` 16-byte
// units, each thread taking `per_thread` of them.
unsigned plane_blocks(int64_t units, int per_thread) {
  int64_t threads = (units + per_thread - 1) / per_thread;
  int64_t b = (threads + 255) / 256;
  if (b < 1) b = 1;
  if (b > 65535) b = 65535;
  return unsigned(b);
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
  return true;
}

}  // namespace

namespace fademem {

int compute_layout(const fademem_config* cfg, Layout* lay) {
  if (!valid_config(cfg)) return FADEMEM_EINVAL;
  Layout L{};
  L.slots = cfg->budget + 1;
  size_t off = round_up(sizeof(DevHeader), 256);
  for (int c = 0; c < 2; ++c) {
    L.off_first[c] = off;   off = round_up(off + 8 * size_t(L.slots), 256);
    L.off_pos_sum[c] = off; off = round_up(off + 8 * size_t(L.slots), 256);
    L.off_span[c] = off;    off = round_up(off + 8 * size_t(L.slots), 256);
    L.off_order[c] = off;   off = round_up(off + 4 * size_t(L.slots), 256);
  }
  L.off_log = off;     off = round_up(off + 4 * size_t(kLogCap), 256);
  L.meta_bytes = off;
  L.elt = cfg->dtype == FADEMEM_BF16 ? 2 : 4;
  L.row_elems = size_t(cfg->heads) * size_t(cfg->head_dim);
  const double blk = double(cfg->tokens_per_block) * double(L.row_elems) * double(L.elt);
  if (blk > 1e15) return FADEMEM_EINVAL;
  L.blk_bytes = size_t(cfg->tokens_per_block) * L.row_elems * L.elt;
  L.blk_stride = round_up(L.blk_bytes, 256);
  L.off_ws = L.meta_bytes + size_t(cfg->layers) * size_t(L.slots) * 2 * L.blk_stride;
  L.ws_bytes = cfg->dtype == FADEMEM_BF16 ? attend_ws_bytes(cfg->head_dim) : 0;
  L.total = L.off_ws + L.ws_bytes;
  *lay = L;
  return FADEMEM_OK;
}

}  // namespace fademem

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
  c->last_hip_error = 0;
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
  c->count += 1;
  c->inserted += 1;
  c->newest = position;
  c->any_inserted = true;
  return FADEMEM_OK;
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
  // Blocks per plane: enough to cover it with UNROLL units per thread, but
  // about 2048 blocks in total (8 per CU) so that every block has work and
  // the per-block schedule evaluation stays a small fraction of the pass.
  const unsigned planes = unsigned(2 * c->cfg.layers);
  unsigned per_plane = 2048u / planes;
  if (per_plane < 1) per_plane = 1;
  const unsigned cover = plane_blocks(a.units, kMergeUnroll);
  if (per_plane > cover) per_plane = cover;
  const dim3 blocks(per_plane, planes);
  const bool bf16 = c->cfg.dtype == FADEMEM_BF16, maxop = c->cfg.merge_op == FADEMEM_MERGE_MAX;
  auto kernel = bf16 ? (maxop ? consolidate_kernel<true, kMergeUnroll, true> : consolidate_kernel<true, kMergeUnroll, false>)
                     : (maxop ? consolidate_kernel<false, kMergeUnroll, true> : consolidate_kernel<false, kMergeUnroll, false>);
  hipLaunchKernelGGL(kernel, dim3(blocks), dim3(256), 0, as_stream(stream), a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(c, e);
  c->cur ^= 1;
  c->count -= 1;
  return FADEMEM_OK;
}

int fademem_attend(fademem_cache* c, int32_t layer, const void* q, int64_t q_tokens, const void* k_cur,
                   const void* v_cur, int64_t cur_tokens, float scale, void* out, float* lse, void* stream) {
  if (!c) return FADEMEM_EINVAL;
  if (layer < 0 || layer >= c->cfg.layers) return FADEMEM_EINVAL;
  if (q_tokens < 0 || q_tokens > kMaxTokens || cur_tokens < 0 || cur_tokens > kMaxTokens) return FADEMEM_EINVAL;
  if (q_tokens == 0) return FADEMEM_OK;
  if (!q || !out || !aligned(q, 16) || !aligned(out, 16)) return FADEMEM_EINVAL;
  if (lse && !aligned(lse, 4)) return FADEMEM_EINVAL;
  if (cur_tokens > 0 && (!k_cur || !v_cur || !aligned(k_cur, 16) || !aligned(v_cur, 16))) return FADEMEM_EINVAL;
  if (c->count == 0 && cur_tokens == 0) return FADEMEM_EINVAL;  // no keys at all
  const double total_keys = double(c->count) * double(c->cfg.tokens_per_block) + double(cur_tokens);
  if (total_keys > double(kMaxTokens)) return FADEMEM_EINVAL;
  if (!(scale >= 0.0f) || isinf(scale)) return FADEMEM_EINVAL;
  AttendArgs a;
  a.q = q;
  a.out = out;
  a.lse = lse;
  a.kv_layer_base = c->pool + kv_offset(c->lay, layer, 0, 0);
  a.order = reinterpret_cast<const int32_t*>(c->pool + c->lay.off_order[c->cur]);
  a.k_cur = k_cur;
  a.v_cur = v_cur;
  a.n_entries = c->count;
  a.tokens_per_block = c->cfg.tokens_per_block;
  a.cur_tokens = cur_tokens;
  a.q_tokens = q_tokens;
  a.slot_stride = 2 * c->lay.blk_stride;
  a.v_offset = c->lay.blk_stride;
  a.ws = reinterpret_cast<float*>(c->pool + c->lay.off_ws);
  a.heads = c->cfg.heads;
  a.head_dim = c->cfg.head_dim;
  a.scale = scale > 0.0f ? scale : 1.0f / sqrtf(float(c->cfg.head_dim));
  (void)hipGetLastError();
  hipError_t e = (c->cfg.dtype == FADEMEM_BF16) ? launch_attend_bf16(a, as_stream(stream))
                                                : launch_attend_f32(a, as_stream(stream));
  if (e != hipSuccess) return hip_fail(c, e);
  return FADEMEM_OK;
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
