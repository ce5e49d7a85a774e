// Flash attention of a chunk's queries over FadeMem's exposed cache,
// bf16 in, fp32 accumulation, on gfx950 MFMA (v_mfma_f32_32x32x16_bf16).
//
// O_h = softmax(scale * Q_h K_h^T) V_h with the keys/values
// [memory entries in memory order || current chunk] (FadeMem Sec. 3.1 and
// Sec. 4.1: the chunk attends over the memory entries plus its own frames).
//
// Design (workgroup = 4 waves = 128 queries of one head; two workgroups per
// CU, i.e. two waves per SIMD, so one wave's softmax overlaps the other's
// MFMAs):
// * Transposed scores: a wave computes S^T = K Q^T for its 32 queries, so an
//   accumulator lane holds 16 keys of ONE query.  Row max and sum need one
//   lane-pair exchange (permlane32 swap) per tile, and P leaves the
//   accumulator already in the B-operand layout of O^T = V^T P^T.
// * K/V tiles (64 keys) go from global memory straight into LDS
//   (global_load_lds, 16 bytes per lane), double-buffered: the next tile's
//   loads fly during the current tile's math; one barrier per tile.
// * K is read with 16-byte LDS loads; V stays row-major in LDS and its V^T
//   operand is built with the transposing LDS read (ds_read_b64_tr_b16).
//   Both buffers are XOR-swizzled by row so the read patterns spread over all
//   LDS banks.
// * Rows are gathered through the memory's logical->slot table; a tile may
//   straddle entries and the current chunk.  The entry of the tile's first
//   row is tracked per wave; each lane resolves its own row from it.  Rows
//   past the last key load the last key again and score -inf.
// * Online softmax in base 2 with the scale folded into one FMA; O is
//   rescaled only when a row max grows by more than 2^8 (the stale max
//   cancels in the final normalisation).
// * Block index -> (head, query tile) is remapped so that consecutive tiles
//   of one head run on the same XCD and share its L2.
#include "fademem_internal.h"

namespace fademem {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
#define LDS_AS __attribute__((address_space(3)))

constexpr int kThreads = 256;
constexpr int kBM = 128;  // queries per workgroup (4 waves x 32)
constexpr int kBN = 64;   // keys per tile
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kRescaleLog2 = 8.0f;  // rescale O when the max grows by > 2^8

template <int D>
struct Shape {
  static constexpr int CH = D / 8;                 // 16-byte chunks per row
  static constexpr int KB = D / 16;                // k-steps of S^T = K Q^T
  static constexpr int DB = D / 32;                // 32-row blocks of O^T
  static constexpr int RPB = 256 / (2 * D);        // rows per 256 bytes of LDS
  static constexpr int TILE_BYTES = kBN * D * 2;
  static constexpr int LOADS = kBN * CH / kThreads;  // 16-byte loads per lane per tile (per K and V)
  static_assert(LOADS * kThreads == kBN * CH, "tile split");
};

// Swizzles: LDS 16-byte position of chunk c of row n is c ^ swz(n).
template <int D>
__device__ __forceinline__ int kswz(int n) {
  return (n / Shape<D>::RPB) % Shape<D>::CH;
}
template <int D>
__device__ __forceinline__ int vswz(int n) {
  return 4 * ((n / Shape<D>::RPB) % (4 / Shape<D>::RPB));
}

__device__ __forceinline__ float pair_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <int D>
__device__ __forceinline__ void attend_bf16_body(const AttendArgs& args, int q_tiles, int total_blocks) {
  using S = Shape<D>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  char* tile_buf = smem;                                          // [2 bufs][K, V][TILE_BYTES]
  // Entry table: K address of row 0 (this head) of each memory entry, and
  // the current chunk as entry n_entries; V is at K + vdelta.
  const char** ent_k = reinterpret_cast<const char**>(smem + 4 * S::TILE_BYTES);
  long long* ent_vd = reinterpret_cast<long long*>(smem + 4 * S::TILE_BYTES + 8 * (args.n_entries + 2));

  // XCD-aware block -> (head, query tile).
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
  const size_t row_bytes = size_t(H) * D * 2;
  const size_t head_off = size_t(h) * D * 2;
  const char* layer_base = args.kv_layer_base;
  const char* k_cur = static_cast<const char*>(args.k_cur);
  const long long cur_vdelta = static_cast<const char*>(args.v_cur) - k_cur;

  for (int e = tid; e < n_entries + 2; e += kThreads) {
    if (e < n_entries) {
      ent_k[e] = layer_base + size_t(args.order[e]) * args.slot_stride + head_off;
      ent_vd[e] = (long long)args.v_offset;
    } else {
      ent_k[e] = k_cur + head_off;
      ent_vd[e] = cur_vdelta;
    }
  }

  // Q fragment (B operand of S^T = K Q^T): query m = l32, d = 16*kb + 8*hh + 0..7.
  const int q_row = qt * kBM + wave * 32 + l32;
  bf16x8 qf[S::KB];
  {
    const char* qbase = static_cast<const char*>(args.q) + (size_t(q_row < Lq ? q_row : Lq - 1) * H + h) * D * 2;
#pragma unroll
    for (int kb = 0; kb < S::KB; ++kb) qf[kb] = *reinterpret_cast<const bf16x8*>(qbase + (16 * kb + 8 * hh) * 2);
  }
  __syncthreads();  // entry table visible

  // Tile t's first row lies in entry e0 at row off0 (e0 == n_entries: the
  // current chunk, which is never wrapped).
  int e0 = 0, off0 = 0;
  const bool wide = N >= kBN;  // then a tile spans at most two entries
  const double inv_n = 1.0 / double(N);
  const int mem_rows = n_entries * N;

  auto entry_base = [&](int e, const char*& kb, long long& vd) {
    kb = ent_k[e];
    vd = ent_vd[e];
  };

  // Per-lane constants of the tile loads: load i writes destination chunk
  // q = (4i + wave)*64 + lane = row n0, LDS position p; it fetches global
  // chunk p ^ swz(n0) of that row.
  int ld_row[S::LOADS];
  uint32_t ld_koff[S::LOADS], ld_voff[S::LOADS];
#pragma unroll
  for (int i = 0; i < S::LOADS; ++i) {
    const int q = (i * 4 + wave) * 64 + lane;
    const int n0 = q / S::CH, p = q % S::CH;
    ld_row[i] = n0;
    ld_koff[i] = uint32_t(size_t(n0) * row_bytes) + uint32_t((p ^ kswz<D>(n0)) * 16);
    ld_voff[i] = uint32_t(size_t(n0) * row_bytes) + uint32_t((p ^ vswz<D>(n0)) * 16);
  }

  // Issue the global->LDS loads of tile `tile` into buffer BUF.
  auto issue_tile = [&](int tile, char* kb_lds) {
    char* vb_lds = kb_lds + S::TILE_BYTES;
    const int k0 = tile * kBN;
    if (wide && k0 + kBN <= Lk) {
      // Rows n < ncross are entry e0's rows off0 + n; the rest are entry
      // e0+1's rows n - ncross.  Row n's address = base + n*row_bytes.
      const char* kb0;
      const char* kb1;
      long long vd0, vd1;
      entry_base(e0, kb0, vd0);
      entry_base(e0 + 1, kb1, vd1);
      const int ncross = (e0 < n_entries) ? N - off0 : kBN;
      const char* base0 = kb0 + (long long)off0 * (long long)row_bytes;
      const char* base1 = kb1 - (long long)ncross * (long long)row_bytes;
#pragma unroll
      for (int i = 0; i < S::LOADS; ++i) {
        const bool cross = ld_row[i] >= ncross;
        const char* kb = cross ? base1 : base0;
        const char* vb = cross ? base1 + vd1 : base0 + vd0;
        const int j = i * 4 + wave;
        __builtin_amdgcn_global_load_lds(kb + ld_koff[i], (LDS_AS void*)(kb_lds + j * 1024), 16, 0, 0);
        __builtin_amdgcn_global_load_lds(vb + ld_voff[i], (LDS_AS void*)(vb_lds + j * 1024), 16, 0, 0);
      }
    } else {
      // General rows (last tile, or entries shorter than a tile): resolve
      // each row by division; rows past the last key reload the last key.
#pragma unroll
      for (int i = 0; i < S::LOADS; ++i) {
        const int q = (i * 4 + wave) * 64 + lane;
        const int n0 = q / S::CH, p = q % S::CH;
        const int k = (k0 + n0 < Lk) ? k0 + n0 : Lk - 1;
        int e = int((double(k) + 0.5) * inv_n);
        if (e > n_entries) e = n_entries;
        const bool in_mem = k < mem_rows;
        const int off = in_mem ? k - e * N : k - mem_rows;
        const char* kb;
        long long vd;
        entry_base(in_mem ? e : n_entries, kb, vd);
        const char* krow = kb + size_t(off) * row_bytes;
        const int j = i * 4 + wave;
        __builtin_amdgcn_global_load_lds(krow + (p ^ kswz<D>(n0)) * 16, (LDS_AS void*)(kb_lds + j * 1024), 16, 0, 0);
        __builtin_amdgcn_global_load_lds(krow + vd + (p ^ vswz<D>(n0)) * 16, (LDS_AS void*)(vb_lds + j * 1024), 16, 0,
                                         0);
      }
    }
  };
  auto advance_tile_start = [&](int next_k0) {
    if (wide) {
      off0 += kBN;
      if (e0 < n_entries && off0 >= N) {
        off0 -= N;
        ++e0;
      }
    } else if (next_k0 < mem_rows) {
      e0 = int((double(next_k0) + 0.5) * inv_n);
      off0 = next_k0 - e0 * N;
    } else {
      e0 = n_entries;
      off0 = next_k0 - mem_rows;
    }
  };

  // Per-lane LDS read offsets (loop-invariant; the buffer and the (nb, ks)
  // parts are compile-time immediates).
  //   K fragment (row 32nb + l32, chunk 2kb + hh): kswz(32nb + l32) = kswz(l32).
  //   V^T transposing read (row 16ks + 8*second + 4hh + sl/4, d = 32db +
  //   16(g&1) + 4(sl&3)): vswz of that row depends on the lane only.
  const int g = lane >> 4, sl = lane & 15;
  int k_rd[S::KB];
#pragma unroll
  for (int kb = 0; kb < S::KB; ++kb) k_rd[kb] = l32 * D * 2 + (((2 * kb + hh) ^ kswz<D>(l32)) * 16);
  int v_rd[S::DB];
  {
    const int n_lane = 4 * hh + (sl >> 2);
    const int vs = vswz<D>(n_lane);
#pragma unroll
    for (int db = 0; db < S::DB; ++db) {
      const int d = 32 * db + 16 * (g & 1) + 4 * (sl & 3);
      v_rd[db] = n_lane * D * 2 + (((d >> 3) ^ vs) * 16) + ((d >> 2) & 1) * 8;
    }
  }

  const float c2 = args.scale * kLog2e;
  f32x16 o[S::DB];
#pragma unroll
  for (int db = 0; db < S::DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.0f;
  float m_run = -INFINITY;  // running (possibly stale) max of raw scores for query l32
  float l_run = 0.0f;       // this lane's partial sum of 2^(s*c2 - m_run*c2)

  const int tiles = (Lk + kBN - 1) / kBN;

  // One tile: wait for its loads, start the next tile's loads into the other
  // buffer, then S^T = K Q^T, online softmax, O^T += V^T P^T.
  auto step = [&](int tile, char* cur_k, char* next_k) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();  // tile landed for every wave; the other buffer is free
    if (tile + 1 < tiles) {
      advance_tile_start((tile + 1) * kBN);
      issue_tile(tile + 1, next_k);
    }
    const char* kb_lds = cur_k;
    const char* vb_lds = cur_k + S::TILE_BYTES;

    f32x16 s[2];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[nb][r] = 0.0f;
    {
      bf16x8 ka[2][2];  // [nb][k-step parity]: fragments read one k-step ahead
      ka[0][0] = *reinterpret_cast<const bf16x8*>(kb_lds + k_rd[0]);
      ka[1][0] = *reinterpret_cast<const bf16x8*>(kb_lds + k_rd[0] + 32 * D * 2);
#pragma unroll
      for (int kb = 0; kb < S::KB; ++kb) {
        if (kb + 1 < S::KB) {
          ka[0][(kb + 1) & 1] = *reinterpret_cast<const bf16x8*>(kb_lds + k_rd[kb + 1]);
          ka[1][(kb + 1) & 1] = *reinterpret_cast<const bf16x8*>(kb_lds + k_rd[kb + 1] + 32 * D * 2);
        }
        s[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[0][kb & 1], qf[kb], s[0], 0, 0, 0);
        s[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[1][kb & 1], qf[kb], s[1], 0, 0, 0);
      }
    }
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
    float mx = s[0][0];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[nb][r]);
    mx = pair_max(mx);
    if (__any((mx - m_run) * c2 > kRescaleLog2)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * c2);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < S::DB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
    }
    const float mc = m_run * c2;
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
    l_run += psum;

#pragma unroll
    for (int db = 0; db < S::DB; ++db) {
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        bf16x8 a;
#pragma unroll
        for (int second = 0; second < 2; ++second) {
          const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (LDS_AS s16x4*)((LDS_AS const char*)(vb_lds) + v_rd[db] + (16 * ks + 8 * second) * D * 2));
          const bf16x4 vb = __builtin_bit_cast(bf16x4, v);
#pragma unroll
          for (int e = 0; e < 4; ++e) a[4 * second + e] = vb[e];
        }
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf[ks], o[db], 0, 0, 0);
      }
    }
  };

  char* buf0 = tile_buf;
  char* buf1 = tile_buf + 2 * S::TILE_BYTES;
  issue_tile(0, buf0);
  for (int tile = 0; tile < tiles; tile += 2) {
    step(tile, buf0, buf1);
    if (tile + 1 < tiles) step(tile + 1, buf1, buf0);
  }

  // Epilogue: O / l, LSE = scale*m + ln(l).
  const float l_tot = pair_sum(l_run);
  const float inv = 1.0f / l_tot;
  if (q_row < Lq) {
    char* obase = static_cast<char*>(args.out) + (size_t(q_row) * H + h) * D * 2;
#pragma unroll
    for (int db = 0; db < S::DB; ++db)
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

__global__ __launch_bounds__(kThreads, 2) void attend_bf16_d128(AttendArgs args, int q_tiles, int total_blocks) {
  attend_bf16_body<128>(args, q_tiles, total_blocks);
}
__global__ __launch_bounds__(kThreads, 2) void attend_bf16_d64(AttendArgs args, int q_tiles, int total_blocks) {
  attend_bf16_body<64>(args, q_tiles, total_blocks);
}

namespace {

template <int D, typename Kernel>
hipError_t launch_d(Kernel kernel, const AttendArgs& a, hipStream_t stream) {
  const int64_t q_tiles64 = (a.q_tokens + kBM - 1) / kBM;
  if (q_tiles64 * a.heads > int64_t(0x7fffffff)) return hipErrorInvalidValue;
  const int q_tiles = int(q_tiles64);
  const int total = q_tiles * a.heads;
  const size_t shmem = 4 * size_t(Shape<D>::TILE_BYTES) + size_t(a.n_entries + 2) * 16;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 96 * 1024);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  if (shmem > 96 * 1024) return hipErrorInvalidValue;
  hipLaunchKernelGGL(kernel, dim3(total), dim3(kThreads), shmem, stream, a, q_tiles, total);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attend_bf16(const AttendArgs& a, hipStream_t stream) {
  if (a.head_dim == 128) return launch_d<128>(attend_bf16_d128, a, stream);
  if (a.head_dim == 64) return launch_d<64>(attend_bf16_d64, a, stream);
  return hipErrorInvalidValue;
}

}  // namespace fademem
