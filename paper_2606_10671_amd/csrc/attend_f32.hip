// Attention of a chunk's queries over FadeMem's exposed cache, fp32 in and
// out (FadeMem Sec. 3.1, Sec. 4.1): O_h = softmax(scale * Q_h K_h^T) V_h,
// keys/values = [memory entries in memory order || current chunk].
//
// Plain vector-ALU kernel for fp32 caches (small shapes): one wave per
// (head, 64 queries), one query per lane held in registers, K/V tiles of
// 32 keys staged in LDS and read as broadcasts, online softmax per tile.
#include "fademem_internal.h"

namespace fademem {
namespace {

constexpr int kQ = 64;       // queries per block (one wave)
constexpr int kTile = 32;    // keys per tile
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

template <int D>
__global__ __launch_bounds__(64) void attend_f32_kernel(AttendArgs args, int q_tiles) {
  __shared__ float k_s[kTile][D];
  __shared__ float v_s[kTile][D];
  extern __shared__ int32_t order_s[];

  const int h = blockIdx.x / q_tiles;
  const int qt = blockIdx.x % q_tiles;
  const int lane = threadIdx.x;
  const int H = args.heads;
  const int n_entries = int(args.n_entries);
  const int N = int(args.tokens_per_block);
  const int cur = int(args.cur_tokens);
  const int Lk = n_entries * N + cur;
  const int Lq = int(args.q_tokens);
  const int q_row = qt * kQ + lane;
  const size_t row_bytes = size_t(H) * D * 4;
  const size_t head_off = size_t(h) * D * 4;

  for (int e = lane; e < n_entries; e += 64) order_s[e] = args.order[e];

  const float c2 = args.scale * kLog2e;  // scores in the log2 domain
  float q[D], o[D];
  {
    const float* qp = reinterpret_cast<const float*>(static_cast<const char*>(args.q) +
                                                     size_t(q_row < Lq ? q_row : Lq - 1) * row_bytes + head_off);
#pragma unroll
    for (int d = 0; d < D; ++d) {
      q[d] = qp[d] * c2;
      o[d] = 0.0f;
    }
  }
  float m_run = -INFINITY, l_run = 0.0f;
  __syncthreads();

  for (int k0 = 0; k0 < Lk; k0 += kTile) {
    __syncthreads();
    // Stage 32 rows of K and V: 64 lanes x 4-float chunks.
    for (int idx = lane; idx < kTile * (D / 4); idx += 64) {
      const int r = idx / (D / 4), c4 = idx % (D / 4);
      const int k = k0 + r;
      float4 kv4 = make_float4(0.f, 0.f, 0.f, 0.f), vv4 = kv4;
      if (k < Lk) {
        const char *kb, *vb;
        size_t off;
        if (k < n_entries * N) {
          const int e = k / N;
          const char* slot = args.kv_layer_base + size_t(order_s[e]) * args.slot_stride;
          kb = slot;
          vb = slot + args.v_offset;
          off = size_t(k - e * N);
        } else {
          kb = static_cast<const char*>(args.k_cur);
          vb = static_cast<const char*>(args.v_cur);
          off = size_t(k - n_entries * N);
        }
        kv4 = *reinterpret_cast<const float4*>(kb + off * row_bytes + head_off + c4 * 16);
        vv4 = *reinterpret_cast<const float4*>(vb + off * row_bytes + head_off + c4 * 16);
      }
      *reinterpret_cast<float4*>(&k_s[r][4 * c4]) = kv4;
      *reinterpret_cast<float4*>(&v_s[r][4 * c4]) = vv4;
    }
    __syncthreads();
    const int nk = (Lk - k0) < kTile ? (Lk - k0) : kTile;
    float s[kTile];
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < kTile; ++j) {
      float acc = 0.0f;
#pragma unroll
      for (int d = 0; d < D; ++d) acc = __builtin_fmaf(q[d], k_s[j][d], acc);
      s[j] = (j < nk) ? acc : -INFINITY;
      mx = fmaxf(mx, s[j]);
    }
    const float m_new = fmaxf(m_run, mx);
    const float alpha = exp2f(m_run - m_new);
    m_run = m_new;
    l_run *= alpha;
#pragma unroll
    for (int d = 0; d < D; ++d) o[d] *= alpha;
#pragma unroll
    for (int j = 0; j < kTile; ++j) {
      const float p = exp2f(s[j] - m_new);
      l_run += p;
#pragma unroll
      for (int d = 0; d < D; ++d) o[d] = __builtin_fmaf(p, v_s[j][d], o[d]);
    }
  }

  if (q_row < Lq) {
    const float inv = 1.0f / l_run;
    float* op = reinterpret_cast<float*>(static_cast<char*>(args.out) + size_t(q_row) * row_bytes + head_off);
#pragma unroll
    for (int d = 0; d < D; d += 4) {
      *reinterpret_cast<float4*>(op + d) = make_float4(o[d] * inv, o[d + 1] * inv, o[d + 2] * inv, o[d + 3] * inv);
    }
    if (args.lse) args.lse[size_t(h) * Lq + q_row] = (m_run + log2f(l_run)) * kLn2;
  }
}

}  // namespace

hipError_t launch_attend_f32(const AttendArgs& a, hipStream_t stream) {
  const int64_t q_tiles64 = (a.q_tokens + kQ - 1) / kQ;
  if (q_tiles64 * a.heads > int64_t(0x7fffffff)) return hipErrorInvalidValue;
  const int q_tiles = int(q_tiles64);
  const int total = q_tiles * a.heads;
  const size_t shmem = size_t(a.n_entries) * sizeof(int32_t);
  if (a.head_dim == 128) {
    hipLaunchKernelGGL(attend_f32_kernel<128>, dim3(total), dim3(64), shmem, stream, a, q_tiles);
  } else if (a.head_dim == 64) {
    hipLaunchKernelGGL(attend_f32_kernel<64>, dim3(total), dim3(64), shmem, stream, a, q_tiles);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace fademem
