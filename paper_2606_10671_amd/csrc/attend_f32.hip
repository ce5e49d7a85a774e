// Attention of a chunk's queries over FadeMem's exposed cache, fp32 in and
// out (FadeMem Sec. 3.1, Sec. 4.1): O_h = softmax(scale * Q_h K_h^T) V_h,
// keys/values = [memory entries in memory order || current chunk].
//
// Vector-ALU kernel for fp32 caches (small shapes, where latency rules).
// A workgroup of 8 waves takes one (head, 64-query tile) over a range of
// the key tiles (all of them, or one of `parts` equal ranges, so that the
// call spreads over many CUs):
// * wave w runs query half w & 1 (32 queries) over key split w >> 1: key
//   tiles of 16 are dealt round-robin to the 4 splits, so 4x more waves
//   walk the key axis at once;
// * within a wave, query m = lane & 31 is held by the lane pair (m, m+32),
//   each lane owning half of the head dimension; a score is the lane's
//   half dot product plus its partner's (one permlane32 swap);
// * the two waves of a split stage its K/V tile in LDS and read it as
//   broadcasts; online softmax per tile in base 2;
// * at the end the four splits' partial (O, max, sum) are combined through
//   LDS by the split-0 waves, which write O and the LSE, or, when the key
//   axis is cut into ranges, the range's partial result to its slot;
//   attend_f32_combine_kernel then combines a query tile's ranges in order.
#include <mutex>

#include "fademem_internal.h"

namespace fademem {
namespace {

constexpr int kQ = kF32Queries;  // queries per workgroup
constexpr int kSplits = 4;    // key splits per workgroup
constexpr int kWaves = 2 * kSplits;
constexpr int kThreads = 64 * kWaves;
constexpr int kTile = 16;     // keys per tile
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float pair_add(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <int D>
struct F32Smem {
  static constexpr int HD = D / 2;  // dims per lane
  // Per split: K and V tiles [kTile][D].
  static constexpr size_t tile_floats = size_t(kSplits) * 2 * kTile * D;
  // Combine round: the two waves of one split, O halves and (m, l) per lane.
  static constexpr size_t comb_floats = size_t(2) * 64 * (HD + 2);
  static constexpr size_t floats = tile_floats > comb_floats ? tile_floats : comb_floats;
};

template <int D>
__global__ __launch_bounds__(kThreads) void attend_f32_kernel(AttendArgs args, int q_tiles, int parts,
                                                             int tiles_per_part) {
  using SM = F32Smem<D>;
  constexpr int HD = SM::HD;
  __shared__ __attribute__((aligned(16))) float smem[SM::floats];
  extern __shared__ int32_t order_s[];  // K block index of entry e at 2e, V block index at 2e + 1

  const int part = blockIdx.x % parts;
  const int h = (blockIdx.x / parts) / q_tiles;
  const int qt = (blockIdx.x / parts) % q_tiles;
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int half = wave & 1;       // query half
  const int split = wave >> 1;     // key split
  const int hf = lane >> 5;        // which half of the head dimension
  const int H = args.heads;
  const int n_entries = int(args.n_entries);
  const int N = int(args.tokens_per_block);
  const int cur = int(args.cur_tokens);
  const int mem_rows = n_entries * N;
  const int Lk = mem_rows + cur;
  const int Lq = int(args.q_tokens);
  const int q_row = qt * kQ + half * 32 + (lane & 31);
  const size_t row_bytes = size_t(H) * D * 4;
  const size_t head_off = size_t(h) * D * 4;

  for (int e = tid; e < n_entries; e += kThreads) {
    order_s[2 * e] = args.k_order ? args.k_order[e] : e;
    order_s[2 * e + 1] = args.v_order[e];
  }

  const float c2 = args.scale * kLog2e;  // scores in the log2 domain
  float q[HD], o[HD];
  {
    const float* qp = reinterpret_cast<const float*>(static_cast<const char*>(args.q) +
                                                     size_t(q_row < Lq ? q_row : Lq - 1) * row_bytes + head_off) +
                      hf * HD;
#pragma unroll
    for (int d = 0; d < HD; ++d) {
      q[d] = qp[d] * c2;
      o[d] = 0.0f;
    }
  }
  float m_run = -INFINITY, l_run = 0.0f;
  __syncthreads();

  float* k_s = smem + size_t(split) * 2 * kTile * D;
  float* v_s = k_s + kTile * D;
  const int n_tiles = (Lk + kTile - 1) / kTile;
  const int t_begin = part * tiles_per_part;
  const int t_end = min(n_tiles, t_begin + tiles_per_part);  // this workgroup's key tiles [t_begin, t_end)
  const int rounds = (t_end - t_begin + kSplits - 1) / kSplits;
  const int stage_tid = half * 64 + lane;  // 0..127 within the split
  for (int rnd = 0; rnd < rounds; ++rnd) {
    const int tile = t_begin + rnd * kSplits + split;
    const int k0 = tile * kTile;
    __syncthreads();  // the previous round's reads of this split's buffers are done
    if (tile < t_end) {
      // Stage kTile rows of K and V: 128 threads x float4 chunks.
      for (int idx = stage_tid; idx < kTile * (D / 4); idx += 128) {
        const int r = idx / (D / 4), c4 = idx % (D / 4);
        const int k = k0 + r;
        float4 kv4 = make_float4(0.f, 0.f, 0.f, 0.f), vv4 = kv4;
        if (k < Lk) {
          const char *kb, *vb;
          size_t off;
          if (k < mem_rows) {
            const int e = k / N;
            kb = args.k_base + size_t(order_s[2 * e]) * args.k_stride;
            vb = args.v_base + size_t(order_s[2 * e + 1]) * args.v_stride;
            off = size_t(k - e * N);
          } else {
            kb = static_cast<const char*>(args.k_cur);
            vb = static_cast<const char*>(args.v_cur);
            off = size_t(k - mem_rows);
          }
          kv4 = *reinterpret_cast<const float4*>(kb + off * row_bytes + head_off + c4 * 16);
          vv4 = *reinterpret_cast<const float4*>(vb + off * row_bytes + head_off + c4 * 16);
        }
        *reinterpret_cast<float4*>(k_s + r * D + 4 * c4) = kv4;
        *reinterpret_cast<float4*>(v_s + r * D + 4 * c4) = vv4;
      }
    }
    __syncthreads();
    if (tile >= t_end) continue;
    const int nk = (Lk - k0) < kTile ? (Lk - k0) : kTile;
    float s[kTile];
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < kTile; ++j) {
      float acc = 0.0f;
      const float* kr = k_s + j * D + hf * HD;
#pragma unroll
      for (int d = 0; d < HD; ++d) acc = __builtin_fmaf(q[d], kr[d], acc);
      acc = pair_add(acc);
      s[j] = (j < nk) ? acc : -INFINITY;
      mx = fmaxf(mx, s[j]);
    }
    const float m_new = fmaxf(m_run, mx);
    const float alpha = exp2f(m_run - m_new);
    m_run = m_new;
    l_run *= alpha;
#pragma unroll
    for (int d = 0; d < HD; ++d) o[d] *= alpha;
#pragma unroll
    for (int j = 0; j < kTile; ++j) {
      const float p = exp2f(s[j] - m_new);
      l_run += p;
      const float* vr = v_s + j * D + hf * HD;
#pragma unroll
      for (int d = 0; d < HD; ++d) o[d] = __builtin_fmaf(p, vr[d], o[d]);
    }
  }

  // Combine the splits into split 0: one round per other split.
  float* comb = smem;
  for (int r = 1; r < kSplits; ++r) {
    __syncthreads();
    if (split == r) {
      float* dst = comb + size_t(half * 64 + lane) * (HD + 2);
#pragma unroll
      for (int d = 0; d < HD; ++d) dst[d] = o[d];
      dst[HD] = m_run;
      dst[HD + 1] = l_run;
    }
    __syncthreads();
    if (split == 0) {
      const float* src = comb + size_t(half * 64 + lane) * (HD + 2);
      const float m_o = src[HD];
      const float m_new = fmaxf(m_run, m_o);
      if (m_new != -INFINITY) {  // both empty: nothing to add
        const float a = exp2f(m_run - m_new), b = exp2f(m_o - m_new);
        l_run = l_run * a + src[HD + 1] * b;
#pragma unroll
        for (int d = 0; d < HD; ++d) o[d] = o[d] * a + src[d] * b;
        m_run = m_new;
      }
    }
  }

  if (parts > 1) {  // this range's partial result: unnormalised O, row max and row sum per query
    if (split == 0) {
      float* slot = args.ws + size_t(blockIdx.x) * f32_part_floats(D);
      const int qi = half * 32 + (lane & 31);
      float* op = slot + size_t(qi) * D + hf * HD;
#pragma unroll
      for (int d = 0; d < HD; d += 4) *reinterpret_cast<float4*>(op + d) = make_float4(o[d], o[d + 1], o[d + 2], o[d + 3]);
      if (hf == 0) {
        slot[kQ * D + qi] = m_run;
        slot[kQ * D + kQ + qi] = l_run;
      }
    }
    return;
  }
  if (split == 0 && q_row < Lq) {
    const float inv = 1.0f / l_run;
    float* op = reinterpret_cast<float*>(static_cast<char*>(args.out) + size_t(q_row) * row_bytes + head_off) +
                hf * HD;
#pragma unroll
    for (int d = 0; d < HD; d += 4)
      *reinterpret_cast<float4*>(op + d) = make_float4(o[d] * inv, o[d + 1] * inv, o[d + 2] * inv, o[d + 3] * inv);
    if (args.lse && hf == 0) args.lse[size_t(h) * Lq + q_row] = (m_run + log2f(l_run)) * kLn2;
  }
}

// Combine the `parts` key ranges of one (head, 64-query tile): thread t
// takes query t / 4 and a quarter of the head dimension, and adds the
// ranges in order with weights 2^(m_p - max_p m_p).
constexpr int kCombThreads = 256;
template <int D>
__global__ __launch_bounds__(kCombThreads) void attend_f32_combine_kernel(AttendArgs args, int q_tiles, int parts) {
  constexpr int DQ = D / 4;
  const int h = blockIdx.x / q_tiles, qt = blockIdx.x % q_tiles;
  const int qi = threadIdx.x / 4, dq = threadIdx.x % 4;
  const int q_row = qt * kQ + qi;
  const int Lq = int(args.q_tokens);
  if (q_row >= Lq) return;
  const float* base = args.ws + size_t(blockIdx.x) * size_t(parts) * f32_part_floats(D);
  float m_max = -INFINITY;
#pragma unroll 8
  for (int p = 0; p < parts; ++p) m_max = fmaxf(m_max, base[size_t(p) * f32_part_floats(D) + kQ * D + qi]);
  float o[DQ];
#pragma unroll
  for (int d = 0; d < DQ; ++d) o[d] = 0.0f;
  float l = 0.0f;
#pragma unroll 4
  for (int p = 0; p < parts; ++p) {
    const float* slot = base + size_t(p) * f32_part_floats(D);
    const float w = exp2f(slot[kQ * D + qi] - m_max);
    l += slot[kQ * D + kQ + qi] * w;
    const float* op = slot + size_t(qi) * D + dq * DQ;
#pragma unroll
    for (int d = 0; d < DQ; ++d) o[d] += op[d] * w;
  }
  const float inv = 1.0f / l;
  const size_t row_bytes = size_t(args.heads) * D * 4;
  float* out = reinterpret_cast<float*>(static_cast<char*>(args.out) + size_t(q_row) * row_bytes + size_t(h) * D * 4) +
               dq * DQ;
#pragma unroll
  for (int d = 0; d < DQ; d += 4)
    *reinterpret_cast<float4*>(out + d) = make_float4(o[d] * inv, o[d + 1] * inv, o[d + 2] * inv, o[d + 3] * inv);
  if (args.lse && dq == 0) args.lse[size_t(h) * Lq + q_row] = (m_max + log2f(l)) * kLn2;
}

}  // namespace

namespace {

typedef void (*F32Kernel)(AttendArgs, int, int, int);
typedef void (*F32Combine)(AttendArgs, int, int);

// Key ranges per (head, query tile): enough that each workgroup's four key
// splits have about one tile each, within the kF32MaxParts slots.
hipError_t launch_f32(F32Kernel kernel, F32Combine combine, std::once_flag& attr_once, const AttendArgs& a,
                      hipStream_t stream) {
  const int64_t q_tiles64 = (a.q_tokens + kQ - 1) / kQ;
  if (q_tiles64 * a.heads > int64_t(0x7fffffff)) return hipErrorInvalidValue;
  const int q_tiles = int(q_tiles64);
  const int total = q_tiles * a.heads;
  const size_t shmem = size_t(a.n_entries) * 2 * sizeof(int32_t);  // entry tables; tile buffers are static
  if (shmem > 32 * 1024) return hipErrorInvalidValue;
  const int64_t lk = a.n_entries * a.tokens_per_block + a.cur_tokens;
  const int n_tiles = int((lk + kTile - 1) / kTile);
  int parts = 1;
  if (total * 2 <= kF32MaxParts) {
    const int want = (n_tiles + kSplits - 1) / kSplits;
    parts = want < kF32MaxParts / total ? want : kF32MaxParts / total;
    if (parts < 1) parts = 1;
  }
  const int tiles_per_part = (n_tiles + parts - 1) / parts;
  parts = (n_tiles + tiles_per_part - 1) / tiles_per_part;  // every range non-empty
  hipError_t e = hipSuccess;
  std::call_once(attr_once, [&] {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                            32 * 1024);
  });
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kernel, dim3(unsigned(total) * unsigned(parts)), dim3(kThreads), shmem, stream, a, q_tiles,
                     parts, tiles_per_part);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (parts > 1) {
    hipLaunchKernelGGL(combine, dim3(unsigned(total)), dim3(kCombThreads), 0, stream, a, q_tiles, parts);
    e = hipGetLastError();
  }
  return e;
}

std::once_flag attr_f32_d128, attr_f32_d64;

}  // namespace

hipError_t launch_attend_f32(const AttendArgs& a, hipStream_t stream) {
  if (a.head_dim == 128)
    return launch_f32(attend_f32_kernel<128>, attend_f32_combine_kernel<128>, attr_f32_d128, a, stream);
  if (a.head_dim == 64)
    return launch_f32(attend_f32_kernel<64>, attend_f32_combine_kernel<64>, attr_f32_d64, a, stream);
  return hipErrorInvalidValue;
}

}  // namespace fademem
