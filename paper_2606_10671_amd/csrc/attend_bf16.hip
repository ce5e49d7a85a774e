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
// * Work split: the (query tile, key tile) iterations of all heads are cut
//   into equal contiguous shares, one per resident workgroup (stream-K).
//   A share may end or start inside a query tile; that part's unnormalised
//   O, running max and partial sums go to a scratch slot, and a second
//   kernel merges the parts of each split tile.  Every SIMD then carries
//   the same work, where whole 128-query tiles would leave part of the chip
//   idle in the last round (e.g. 444 tiles on 512 workgroup slots).
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
//   cancels in the final normalisation).  The denominator sums the
//   bf16-rounded weights that enter the P.V product.
// * Workgroup index -> share is remapped so that consecutive shares (the
//   query tiles of one head) run on the same XCD and share its L2.
#include <mutex>

#include "fademem_internal.h"

namespace fademem {

// Work split over G resident workgroups.  Query tiles are numbered
// qg = head * q_tiles + tile within the head, Q of them.  The first
// rounds*G tiles run whole, round k giving tile k*G + g to group g.  Of the
// rem = Q - rounds*G remaining tiles, tile i's keys [0, head_len) go to
// group i (i < rem) and its tail [head_len, tiles) to group
// rem + i / tails_per: the G - rem tail groups each take tails_per
// consecutive tails.  head_len = tiles - tail_len, tail_len =
// tiles / (tails_per + 1), so a tail group's tails_per tails are no more
// work than one head part.  Every group starts its parts at the same key
// tile at the same time, so the groups of one XCD read the same K/V tiles
// together and those come from its L2.  A split tile leaves its head part
// in scratch slot i and its tail in slot rem + i; a second kernel merges
// the two.
struct SkPlan {
  int tiles;      // key tiles per query tile
  int q_tiles;    // query tiles per head
  int groups;     // G
  int rounds;     // whole rounds
  int rem;        // query tiles left after the whole rounds, < G
  int head_len;   // key tiles of a remaining tile's head part
  int tail_len;   // key tiles of its tail part (0: remaining tiles run whole)
  int tails_per;  // tails per tail group
};

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
#define LDS_AS __attribute__((address_space(3)))

constexpr int kThreads = kAttnThreads;
constexpr int kBM = kAttnQueries;  // queries per workgroup (4 waves x 32)
constexpr int kBN = 64;            // keys per tile
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
  static_assert(kBM * D == 4 * DB * 16 * 64, "scratch slot holds the four waves' O registers");
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

// Round two weights to bf16 and add the ROUNDED values to an fp32 sum in one
// v_dot2 against (1, 1): the denominator then sums exactly the weights the
// P.V product uses, so O is a convex combination of V rows.
__device__ __forceinline__ bf16x2 round_and_sum(float p0, float p1, float& sum) {
  bf16x2 pk;
  pk[0] = (__bf16)p0;
  pk[1] = (__bf16)p1;
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  sum = __builtin_amdgcn_fdot2_f32_bf16(pk, ones, sum, false);
  return pk;
}

__device__ __forceinline__ float pair_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// XCD-aware group index: blocks are dealt to the 8 XCDs round-robin, so
// block b runs on XCD b % 8; give each XCD a contiguous run of groups.
__device__ __forceinline__ int xcd_group(int bid, int groups) {
  const int per = groups / 8, rem = groups % 8;
  const int xcd = bid % 8, local = bid / 8;
  return (xcd < rem) ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
}

// Final output of one lane: O row (query q_row, head h) from the O^T
// accumulators divided by the row sum, and the row's LSE.
template <int D>
__device__ __forceinline__ void store_out(const AttendArgs& args, const f32x16 (&o)[Shape<D>::DB], float m_scaled,
                                          float l_tot, int q_row, int h, int hh) {
  const int H = args.heads;
  const int Lq = int(args.q_tokens);
  if (q_row >= Lq) return;
  const float inv = 1.0f / l_tot;
  char* obase = static_cast<char*>(args.out) + (size_t(q_row) * H + h) * D * 2;
#pragma unroll
  for (int db = 0; db < Shape<D>::DB; ++db)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      bf16x4 v;
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = (__bf16)(o[db][4 * g4 + r] * inv);
      const int d = 32 * db + 8 * g4 + 4 * hh;
      *reinterpret_cast<bf16x4*>(obase + d * 2) = v;
    }
  if (args.lse && hh == 0) args.lse[size_t(h) * Lq + q_row] = (m_scaled + __log2f(l_tot)) * kLn2;
}

template <int D>
__device__ __forceinline__ void attend_bf16_body(const AttendArgs& args, const SkPlan& plan) {
  using S = Shape<D>;
  // Tile buffers: separate LDS objects, so the compiler can tell the reads
  // of one buffer from the in-flight direct-to-LDS loads into the other and
  // does not wait for those loads before reading.
  __shared__ __attribute__((aligned(16))) char k_lds0[S::TILE_BYTES];
  __shared__ __attribute__((aligned(16))) char v_lds0[S::TILE_BYTES];
  __shared__ __attribute__((aligned(16))) char k_lds1[S::TILE_BYTES];
  __shared__ __attribute__((aligned(16))) char v_lds1[S::TILE_BYTES];
  // Entry table: K address of row 0 (head 0) of each memory entry, and the
  // current chunk as entry n_entries; V is v_offset (memory) or v_cur-k_cur
  // (current chunk) bytes further.
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const char** ent_k = reinterpret_cast<const char**>(smem);

  const int g = xcd_group(blockIdx.x, gridDim.x);
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
  const char* k_cur = static_cast<const char*>(args.k_cur);
  const long long mem_vdelta = (long long)args.v_offset;
  const long long cur_vdelta = static_cast<const char*>(args.v_cur) - k_cur;

  for (int e = tid; e < n_entries + 1; e += kThreads)
    ent_k[e] = (e < n_entries) ? args.kv_layer_base + size_t(args.order[e]) * args.slot_stride : k_cur;

  const bool wide = N >= kBN;  // then a tile spans at most two entries
  const double inv_n = 1.0 / double(N);
  const int mem_rows = n_entries * N;

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

  // Per-lane LDS read offsets (loop-invariant; the buffer and the (nb, ks)
  // parts are compile-time immediates).
  //   K fragment (row 32nb + l32, chunk 2kb + hh): kswz(32nb + l32) = kswz(l32).
  //   V^T transposing read (row 16ks + 8*second + 4hh + sl/4, d = 32db +
  //   16(g&1) + 4(sl&3)): vswz of that row depends on the lane only.
  const int g16 = lane >> 4, sl = lane & 15;
  int k_rd[S::KB];
#pragma unroll
  for (int kb = 0; kb < S::KB; ++kb) k_rd[kb] = l32 * D * 2 + (((2 * kb + hh) ^ kswz<D>(l32)) * 16);
  int v_rd[S::DB];
  {
    const int n_lane = 4 * hh + (sl >> 2);
    const int vs = vswz<D>(n_lane);
#pragma unroll
    for (int db = 0; db < S::DB; ++db) {
      const int d = 32 * db + 16 * (g16 & 1) + 4 * (sl & 3);
      v_rd[db] = n_lane * D * 2 + (((d >> 3) ^ vs) * 16) + ((d >> 2) & 1) * 8;
    }
  }
  const float c2 = args.scale * kLog2e;

  // One query tile's key tiles [kt0, kt1); the result goes to the output
  // (slot < 0, the range is the whole key axis) or, partial, to scratch slot
  // `slot`.
  auto segment = [&](int h, int qt, int kt0, int kt1, int slot) {
    const size_t head_off = size_t(h) * D * 2;
    auto entry_base = [&](int e, const char*& kb, long long& vd) {
      kb = ent_k[e] + head_off;
      vd = (e < n_entries) ? mem_vdelta : cur_vdelta;
    };

    // Q fragment (B operand of S^T = K Q^T): query m = l32, d = 16*kb + 8*hh + 0..7.
    const int q_row = qt * kBM + wave * 32 + l32;
    bf16x8 qf[S::KB];
    {
      const char* qbase = static_cast<const char*>(args.q) + (size_t(q_row < Lq ? q_row : Lq - 1) * H + h) * D * 2;
#pragma unroll
      for (int kb = 0; kb < S::KB; ++kb) qf[kb] = *reinterpret_cast<const bf16x8*>(qbase + (16 * kb + 8 * hh) * 2);
    }

    // Tile t's first row lies in entry e0 at row off0 (e0 == n_entries: the
    // current chunk, which is never wrapped).
    int e0, off0;
    auto locate = [&](int k0) {
      if (k0 < mem_rows) {
        e0 = k0 / N;
        off0 = k0 - e0 * N;
      } else {
        e0 = n_entries;
        off0 = k0 - mem_rows;
      }
    };
    locate(kt0 * kBN);

    // Issue the global->LDS loads of tile `tile` into the given buffers.
    auto issue_tile = [&](int tile, char* kb_lds, char* vb_lds) {
      const int k0 = tile * kBN;
      if (wide && k0 + kBN <= Lk) {
        // Rows n < ncross are entry e0's rows off0 + n; the rest are entry
        // e0+1's rows n - ncross.  Row n's address = base + n*row_bytes.
        const char* kb0;
        const char* kb1;
        long long vd0, vd1;
        entry_base(e0, kb0, vd0);
        entry_base(e0 + 1 <= n_entries ? e0 + 1 : n_entries, kb1, vd1);
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
          __builtin_amdgcn_global_load_lds(krow + (p ^ kswz<D>(n0)) * 16, (LDS_AS void*)(kb_lds + j * 1024), 16, 0,
                                           0);
          __builtin_amdgcn_global_load_lds(krow + vd + (p ^ vswz<D>(n0)) * 16, (LDS_AS void*)(vb_lds + j * 1024), 16,
                                           0, 0);
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
      } else {
        locate(next_k0);
      }
    };

    f32x16 o[S::DB];
#pragma unroll
    for (int db = 0; db < S::DB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[db][r] = 0.0f;
    float m_run = -INFINITY;  // running (possibly stale) max of raw scores for query l32
    float l_run = 0.0f;       // this lane's partial sum of 2^(s*c2 - m_run*c2)

    // One tile: wait for its loads, start the next tile's loads into the
    // other buffers, then S^T = K Q^T, online softmax, O^T += V^T P^T.
    auto step = [&](int tile, const char* kb_lds, const char* vb_lds, char* next_k, char* next_v) {
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();  // tile landed for every wave; the other buffers are free
      if (tile + 1 < kt1) {
        advance_tile_start((tile + 1) * kBN);
        issue_tile(tile + 1, next_k, next_v);
      }

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
      float mx;
      {
        float m8[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) m8[i] = fmaxf(fmaxf(s[0][i], s[0][i + 8]), fmaxf(s[1][i], s[1][i + 8]));
#pragma unroll
        for (int w = 4; w >= 1; w >>= 1)
#pragma unroll
          for (int i = 0; i < w; ++i) m8[i] = fmaxf(m8[i], m8[i + w]);
        mx = pair_max(m8[0]);
      }
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
      float ps[4] = {0.f, 0.f, 0.f, 0.f};
      u32x4 pw[4];  // P as packed bf16 pairs: k-step 2*nb + r/8, word (r%8)/2
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
#pragma unroll
        for (int r = 0; r < 16; r += 2) {
          const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[nb][r], c2, -mc));
          const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[nb][r + 1], c2, -mc));
          pw[2 * nb + (r >> 3)][(r & 7) >> 1] = __builtin_bit_cast(uint32_t, round_and_sum(p0, p1, ps[(r >> 1) & 3]));
        }
      }
      l_run += (ps[0] + ps[1]) + (ps[2] + ps[3]);

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
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, __builtin_bit_cast(bf16x8, pw[ks]), o[db], 0, 0, 0);
        }
      }
    };

    __syncthreads();  // entry table visible; the previous segment's reads of the buffers are done
    issue_tile(kt0, k_lds0, v_lds0);
    for (int tile = kt0; tile < kt1; tile += 2) {
      step(tile, k_lds0, v_lds0, k_lds1, v_lds1);
      if (tile + 1 < kt1) step(tile + 1, k_lds1, v_lds1, k_lds0, v_lds0);
    }

    if (slot < 0) {
      store_out<D>(args, o, m_run * c2, pair_sum(l_run), q_row, h, hh);
    } else {
      // Partial: the O^T registers lane-major, then per-thread m and l.
      float* ws = args.ws + size_t(slot) * attend_slot_floats(D);
#pragma unroll
      for (int db = 0; db < S::DB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) ws[((wave * S::DB + db) * 16 + r) * 64 + lane] = o[db][r];
      ws[kBM * D + tid] = m_run;
      ws[kBM * D + kThreads + tid] = l_run;
    }
  };

  // The group's parts: its whole tiles, then its head part or its tails.
  const int base = plan.rounds * plan.groups;
  const int i0 = (g - plan.rem) * plan.tails_per;  // first tail (tail groups)
  int parts = plan.rounds;
  if (g < plan.rem) {
    parts += 1;
  } else if (plan.tail_len > 0 && i0 < plan.rem) {
    parts += (i0 + plan.tails_per < plan.rem ? plan.tails_per : plan.rem - i0);
  }
  for (int part = 0; part < parts; ++part) {
    int qg, kt0 = 0, kt1 = plan.tiles, slot = -1;
    if (part < plan.rounds) {
      qg = part * plan.groups + g;
    } else if (g < plan.rem) {
      qg = base + g;
      kt1 = plan.head_len;
      slot = plan.tail_len > 0 ? g : -1;
    } else {
      const int i = i0 + part - plan.rounds;
      qg = base + i;
      kt0 = plan.head_len;
      slot = plan.rem + i;
    }
    segment(qg / plan.q_tiles, qg % plan.q_tiles, kt0, kt1, slot);
  }
}

// Merge of split query tiles: block i combines remaining tile i's head part
// (slot i) and tail part (slot rem + i) and writes the output.
template <int D>
__device__ __forceinline__ void attend_bf16_merge_body(const AttendArgs& args, const SkPlan& plan) {
  using S = Shape<D>;
  const int i = blockIdx.x;
  const int qg = plan.rounds * plan.groups + i;
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int l32 = lane & 31;
  const int hh = lane >> 5;
  const float c2 = args.scale * kLog2e;
  const float* part[2] = {args.ws + size_t(i) * attend_slot_floats(D),
                          args.ws + size_t(plan.rem + i) * attend_slot_floats(D)};
  const float m_max = fmaxf(part[0][kBM * D + tid], part[1][kBM * D + tid]);
  f32x16 o[S::DB];
#pragma unroll
  for (int db = 0; db < S::DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.0f;
  float l_tot = 0.0f;
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const float* ws = part[p];
    const float f = __builtin_amdgcn_exp2f((ws[kBM * D + tid] - m_max) * c2);
    l_tot += f * pair_sum(ws[kBM * D + kThreads + tid]);
#pragma unroll
    for (int db = 0; db < S::DB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[db][r] += f * ws[((wave * S::DB + db) * 16 + r) * 64 + lane];
  }
  store_out<D>(args, o, m_max * c2, l_tot, (qg % plan.q_tiles) * kBM + wave * 32 + l32, qg / plan.q_tiles, hh);
}

}  // namespace

__global__ __launch_bounds__(kThreads, 2) void attend_bf16_d128(AttendArgs args, SkPlan plan) {
  attend_bf16_body<128>(args, plan);
}
__global__ __launch_bounds__(kThreads, 2) void attend_bf16_d64(AttendArgs args, SkPlan plan) {
  attend_bf16_body<64>(args, plan);
}
__global__ __launch_bounds__(kThreads) void attend_bf16_merge_d128(AttendArgs args, SkPlan plan) {
  attend_bf16_merge_body<128>(args, plan);
}
__global__ __launch_bounds__(kThreads) void attend_bf16_merge_d64(AttendArgs args, SkPlan plan) {
  attend_bf16_merge_body<64>(args, plan);
}

namespace {

template <typename Kernel>
hipError_t launch_d(Kernel kernel, Kernel merge, std::once_flag& attr_once, const AttendArgs& a,
                    hipStream_t stream) {
  const int64_t q_tiles64 = (a.q_tokens + kBM - 1) / kBM;
  if (q_tiles64 * a.heads > int64_t(0x7fffffff)) return hipErrorInvalidValue;
  const int64_t lk = a.n_entries * a.tokens_per_block + a.cur_tokens;
  SkPlan plan;
  plan.q_tiles = int(q_tiles64);
  plan.tiles = int((lk + kBN - 1) / kBN);
  const int total = plan.q_tiles * a.heads;
  const size_t shmem = size_t(a.n_entries + 1) * 8;  // entry table; tile buffers are static
  if (shmem > 32 * 1024) return hipErrorInvalidValue;
  hipError_t e = hipSuccess;
  std::call_once(attr_once, [&] {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                            32 * 1024);
  });
  if (e != hipSuccess) return e;
  int dev = 0, cus = 0, per_cu = 0;
  if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
  if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
  if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(kernel), kThreads,
                                                        shmem)) != hipSuccess)
    return e;
  long long groups = (long long)(cus > 0 ? cus : 1) * (per_cu > 0 ? per_cu : 1);
  if (groups > kSkMaxGroups) groups = kSkMaxGroups;
  plan.groups = int(groups);
  plan.rounds = total / plan.groups;
  plan.rem = total - plan.rounds * plan.groups;
  plan.tails_per = plan.rem > 0 ? (plan.rem + (plan.groups - plan.rem) - 1) / (plan.groups - plan.rem) : 1;
  plan.tail_len = plan.tiles / (plan.tails_per + 1);
  plan.head_len = plan.tiles - plan.tail_len;
  const int launched = plan.rounds > 0 ? plan.groups : plan.rem + (plan.tail_len > 0 ? (plan.rem + plan.tails_per - 1) / plan.tails_per : 0);
  hipLaunchKernelGGL(kernel, dim3(launched), dim3(kThreads), shmem, stream, a, plan);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (plan.rem > 0 && plan.tail_len > 0) {
    hipLaunchKernelGGL(merge, dim3(plan.rem), dim3(kThreads), 0, stream, a, plan);
    e = hipGetLastError();
  }
  return e;
}

std::once_flag attr_d128, attr_d64;

}  // namespace

hipError_t launch_attend_bf16(const AttendArgs& a, hipStream_t stream) {
  if (a.head_dim == 128) return launch_d(attend_bf16_d128, attend_bf16_merge_d128, attr_d128, a, stream);
  if (a.head_dim == 64) return launch_d(attend_bf16_d64, attend_bf16_merge_d64, attr_d64, a, stream);
  return hipErrorInvalidValue;
}

}  // namespace fademem
