// Flash attention of a chunk's queries over FadeMem's exposed cache,
// bf16 in, fp32 accumulation, on gfx950 MFMA (v_mfma_f32_32x32x16_bf16).
//
// O_h = softmax(scale * Q_h K_h^T) V_h with the keys/values
// [memory entries in memory order || current chunk] (FadeMem Sec. 3.1 and
// Sec. 4.1: the chunk attends over the M memory entries plus its own frames).
//
// Design (one workgroup = 4 waves = 128 queries of one head):
// * Transposed scores: each wave computes S^T = K Q^T for its 32 queries,
//   so an MFMA accumulator lane holds 16 keys of ONE query.  The row max and
//   sum need one exchange between lanes l and l^32 per tile, and P leaves
//   the accumulator already in the B-operand layout of O^T = V^T P^T.
// * K tile [64 keys][D] row-major in LDS, 16-byte chunks XOR-swizzled by
//   row; V tile stored transposed [D][64 keys] (4-key groups reordered so a
//   lane's 8 keys are one 16-byte chunk), chunks XOR-swizzled by row.
// * K/V rows are gathered through the memory's logical->slot table, so a
//   tile may straddle entries and the current chunk; rows past the last key
//   read as zero and score -inf.
// * Next tile's global loads are issued before the current tile's MFMAs.
// * Block index -> (head, query tile) is remapped so that consecutive
//   tiles of one head run on the same XCD and share its L2.
#include "fademem_internal.h"

namespace fademem {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int kBM = 128;  // queries per workgroup (4 waves x 32)
constexpr int kBN = 64;   // keys per tile
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Running position of one gathered key row: entry index and row offset in
// it.  Entries [0, n_entries) are memory entries of N rows; the current
// chunk follows and is never wrapped.
struct RowPos {
  int e;
  int off;
};

__device__ __forceinline__ void advance(RowPos& p, int by, int n_entries, int N) {
  p.off += by;
  while (p.e < n_entries && p.off >= N) {
    p.off -= N;
    ++p.e;
  }
}

__device__ __forceinline__ RowPos locate(int k, int n_entries, int N) {
  RowPos p;
  const int mem_rows = n_entries * N;
  if (k < mem_rows) {
    p.e = k / N;
    p.off = k - p.e * N;
  } else {
    p.e = n_entries;
    p.off = k - mem_rows;
  }
  return p;
}

struct Gather {
  const char* kv_layer_base;
  const int32_t* order_s;  // LDS copy of logical->slot
  const char* k_cur;
  const char* v_cur;
  size_t slot_stride;
  size_t v_offset;
  size_t row_bytes;  // H*D*2
  size_t head_off;   // h*D*2
  int n_entries;
  int N;
  int cur_tokens;
};

// 16 bytes of key/value row `p` at byte column `col` (kv = 0: K, 1: V).
__device__ __forceinline__ uint4 load_row16(const Gather& g, const RowPos& p, int col, int kv) {
  const char* base;
  if (p.e < g.n_entries) {
    base = g.kv_layer_base + size_t(g.order_s[p.e]) * g.slot_stride + (kv ? g.v_offset : 0);
  } else {
    if (p.off >= g.cur_tokens) return make_uint4(0, 0, 0, 0);
    base = kv ? g.v_cur : g.k_cur;
  }
  return *reinterpret_cast<const uint4*>(base + size_t(p.off) * g.row_bytes + g.head_off + col);
}

// Select 16-bit half `hi` of x and half `hj` of y into one 32-bit word.
__device__ __forceinline__ uint32_t pack_halves(uint32_t x, int hx, uint32_t y, int hy) {
  const uint32_t a = hx ? (x >> 16) : (x & 0xffffu);
  const uint32_t b = hy ? (y & 0xffff0000u) : (y << 16);
  return a | b;
}

template <int D>
__global__ __launch_bounds__(kThreads, 2) void attend_bf16_kernel(AttendArgs args, int q_tiles, int total_blocks) {
  constexpr int CH = D / 8;          // 16-byte chunks per K row
  constexpr int KB = D / 16;         // k-steps of QK^T
  constexpr int DB = D / 32;         // 32-row blocks of O^T
  constexpr int K_ROWS_PER_PASS = kThreads / CH;
  constexpr int K_PASSES = kBN / K_ROWS_PER_PASS;      // rows of K loaded per thread
  constexpr int V_PAIRS = (kBN / 4) * CH;              // (4-key group, d-chunk) pairs
  constexpr int V_PASSES = (V_PAIRS + kThreads - 1) / kThreads;
  static_assert(kBN % K_ROWS_PER_PASS == 0, "tile rows");

  __shared__ __attribute__((aligned(16))) char k_lds[kBN * D * 2];
  __shared__ __attribute__((aligned(16))) char v_lds[D * kBN * 2];
  extern __shared__ int32_t order_s[];

  // XCD-aware block -> (head, query tile): blocks are dealt round-robin to 8
  // XCDs; give each XCD a contiguous range of (head, tile).
  const int bid = blockIdx.x;
  const int per = total_blocks / 8, rem = total_blocks % 8;
  const int xcd = bid % 8, local = bid / 8;
  const int logical = (xcd < rem) ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
  const int h = logical / q_tiles;
  const int qt = logical % q_tiles;

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int l32 = lane & 31;
  const int hh = lane >> 5;

  const int H = args.heads;
  const int n_entries = int(args.n_entries);
  const int N = int(args.tokens_per_block);
  const int Lk = n_entries * N + int(args.cur_tokens);
  const int Lq = int(args.q_tokens);

  for (int e = tid; e < n_entries; e += kThreads) order_s[e] = args.order[e];

  Gather g;
  g.kv_layer_base = args.kv_layer_base;
  g.order_s = order_s;
  g.k_cur = static_cast<const char*>(args.k_cur);
  g.v_cur = static_cast<const char*>(args.v_cur);
  g.slot_stride = args.slot_stride;
  g.v_offset = args.v_offset;
  g.row_bytes = size_t(H) * D * 2;
  g.head_off = size_t(h) * D * 2;
  g.n_entries = n_entries;
  g.N = N;
  g.cur_tokens = int(args.cur_tokens);

  // Q fragment (B operand of S^T = K Q^T): query m = l32, d = 16*kb + 8*hh + 0..7.
  const int q_row = qt * kBM + wave * 32 + l32;
  bf16x8 qf[KB];
  {
    const char* qbase = static_cast<const char*>(args.q) + (size_t(q_row < Lq ? q_row : Lq - 1) * H + h) * D * 2;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      uint4 w = *reinterpret_cast<const uint4*>(qbase + (16 * kb + 8 * hh) * 2);
      qf[kb] = __builtin_bit_cast(bf16x8, w);
    }
  }

  __syncthreads();  // order_s visible

  // Row positions of the rows this thread loads.
  RowPos kpos[K_PASSES];
  const int k_col = (tid % CH) * 16;
#pragma unroll
  for (int i = 0; i < K_PASSES; ++i) kpos[i] = locate(tid / CH + i * K_ROWS_PER_PASS, n_entries, N);
  RowPos vpos[V_PASSES][4];
  int v_kg[V_PASSES], v_c[V_PASSES];
#pragma unroll
  for (int i = 0; i < V_PASSES; ++i) {
    const int pair = tid + i * kThreads;
    v_kg[i] = pair % (kBN / 4);
    v_c[i] = pair / (kBN / 4);
#pragma unroll
    for (int r = 0; r < 4; ++r) vpos[i][r] = locate(4 * v_kg[i] + r, n_entries, N);
  }

  uint4 kreg[K_PASSES];
  uint4 vreg[V_PASSES][4];
  auto load_tile = [&](int tile) {
    const int k0 = tile * kBN;
#pragma unroll
    for (int i = 0; i < K_PASSES; ++i) {
      const int row = k0 + tid / CH + i * K_ROWS_PER_PASS;
      kreg[i] = (row < Lk) ? load_row16(g, kpos[i], k_col, 0) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < V_PASSES; ++i) {
      const bool active = (tid + i * kThreads) < V_PAIRS;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = k0 + 4 * v_kg[i] + r;
        vreg[i][r] = (active && row < Lk) ? load_row16(g, vpos[i][r], v_c[i] * 16, 1) : make_uint4(0, 0, 0, 0);
      }
    }
  };
  auto advance_rows = [&]() {
#pragma unroll
    for (int i = 0; i < K_PASSES; ++i) advance(kpos[i], kBN, n_entries, N);
#pragma unroll
    for (int i = 0; i < V_PASSES; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) advance(vpos[i][r], kBN, n_entries, N);
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int i = 0; i < K_PASSES; ++i) {
      const int n = tid / CH + i * K_ROWS_PER_PASS;
      const int c = tid % CH;
      const int pc = c ^ (n % CH);
      *reinterpret_cast<uint4*>(k_lds + n * D * 2 + pc * 16) = kreg[i];
    }
#pragma unroll
    for (int i = 0; i < V_PASSES; ++i) {
      if ((tid + i * kThreads) >= V_PAIRS) continue;
      const int kg = v_kg[i], c = v_c[i];
      // key group kg -> position among the 16-key group's 4-key slots
      const int grp = kg >> 2, sub = kg & 3;
      const int p4 = (sub == 1) ? 2 : (sub == 2) ? 1 : sub;
      const int np = 16 * grp + 4 * p4;  // n' of the group's first key
      const uint32_t* w0 = reinterpret_cast<const uint32_t*>(&vreg[i][0]);
      const uint32_t* w1 = reinterpret_cast<const uint32_t*>(&vreg[i][1]);
      const uint32_t* w2 = reinterpret_cast<const uint32_t*>(&vreg[i][2]);
      const uint32_t* w3 = reinterpret_cast<const uint32_t*>(&vreg[i][3]);
#pragma unroll
      for (int di = 0; di < 8; ++di) {
        const int d = 8 * c + di;
        const int word = di >> 1, half = di & 1;
        uint2 out;
        out.x = pack_halves(w0[word], half, w1[word], half);
        out.y = pack_halves(w2[word], half, w3[word], half);
        const int chunk = np >> 3;
        const int pc = chunk ^ (d & 7);
        *reinterpret_cast<uint2*>(v_lds + d * kBN * 2 + pc * 16 + (np & 7) * 2) = out;
      }
    }
  };

  const float c2 = args.scale * kLog2e;
  f32x16 o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.0f;
  float m_run = -INFINITY;  // running max of raw scores for query l32
  float l_run = 0.0f;       // this lane's partial sum of 2^(s*c2 - m*c2)

  const int tiles = (Lk + kBN - 1) / kBN;
  load_tile(0);
  for (int tile = 0; tile < tiles; ++tile) {
    __syncthreads();
    store_tile();
    __syncthreads();
    if (tile + 1 < tiles) {
      advance_rows();
      load_tile(tile + 1);
    }

    // S^T = K Q^T for 2 blocks of 32 keys.
    f32x16 s[2];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[nb][r] = 0.0f;
      const int n = 32 * nb + l32;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        const int pc = (2 * kb + hh) ^ (n % CH);
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(k_lds + n * D * 2 + pc * 16);
        s[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kb], s[nb], 0, 0, 0);
      }
    }
    // Mask keys past the end (only the last tile can have them).
    const int k0 = tile * kBN;
    if (k0 + kBN > Lk) {
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = k0 + 32 * nb + 8 * (r >> 2) + 4 * hh + (r & 3);
          if (key >= Lk) s[nb][r] = -INFINITY;
        }
    }
    // Online softmax for query l32 (lanes l32 and l32+32 share it).
    float mx = s[0][0];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[nb][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * c2);
    const float mc = m_new * c2;
    m_run = m_new;
    float psum = 0.0f;
    bf16x8 pf[4];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[nb][r], c2, -mc));
        psum += p;
        pf[2 * nb + (r >> 3)][r & 7] = (__bf16)p;
      }
    }
    l_run = l_run * alpha + psum;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
    // O^T += V^T P^T.
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int d = 32 * db + l32;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const int pc = (2 * ks + hh) ^ (d & 7);
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(v_lds + d * kBN * 2 + pc * 16);
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf[ks], o[db], 0, 0, 0);
      }
    }
  }

  // Epilogue: O / l, LSE = scale*m + ln(l).
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = 1.0f / l_tot;
  if (q_row < Lq) {
    char* obase = static_cast<char*>(args.out) + (size_t(q_row) * H + h) * D * 2;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        bf16x4 v;
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = (__bf16)(o[db][4 * g4 + r] * inv);
        const int d = 32 * db + 8 * g4 + 4 * hh;
        *reinterpret_cast<bf16x4*>(obase + d * 2) = v;
      }
    if (args.lse && hh == 0) args.lse[size_t(h) * Lq + q_row] = (m_run * c2 + __log2f(l_tot)) * kLn2;
  }
}

}  // namespace

hipError_t launch_attend_bf16(const AttendArgs& a, hipStream_t stream) {
  const int64_t q_tiles64 = (a.q_tokens + kBM - 1) / kBM;
  if (q_tiles64 * a.heads > int64_t(0x7fffffff)) return hipErrorInvalidValue;
  const int q_tiles = int(q_tiles64);
  const int total = q_tiles * a.heads;
  const size_t shmem = size_t(a.n_entries) * sizeof(int32_t);
  if (a.head_dim == 128) {
    hipLaunchKernelGGL(attend_bf16_kernel<128>, dim3(total), dim3(kThreads), shmem, stream, a, q_tiles, total);
  } else if (a.head_dim == 64) {
    hipLaunchKernelGGL(attend_bf16_kernel<64>, dim3(total), dim3(kThreads), shmem, stream, a, q_tiles, total);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace fademem
