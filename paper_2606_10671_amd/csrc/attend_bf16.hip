// Flash attention of a chunk's queries over FadeMem's exposed cache,
// bf16 in, fp32 accumulation, on gfx950 MFMA (v_mfma_f32_32x32x16_bf16).
//
// O_h = softmax(scale * Q_h K_h^T) V_h with the keys/values
// [memory entries in memory order || current chunk] (FadeMem Sec. 3.1 and
// Sec. 4.1: the chunk attends over the memory entries plus its own frames).
//
// Design (workgroup = 8 waves x 32 queries of one head, one workgroup per
// CU, two waves per SIMD; the steady-state loop keeps every value in the 256
// architectural VGPRs of a wave, while the last tiles and the epilogue
// spill):
// * The 256 queries of a workgroup share each K/V tile, which is streamed
//   from L2 into LDS once for all of them.
// * Transposed scores: S^T = K Q^T puts 16 keys of ONE query in each
//   accumulator lane.  Row max and sum need one lane-pair exchange
//   (permlane32 swap) per tile, and P leaves the accumulator already in the
//   B-operand layout of O^T = V^T P^T.
// * Software pipeline over key tiles of 64: iteration t runs block A =
//   [S(t+1) = K(t+1) Q^T] beside the exponentials of S(t)'s second 32 keys,
//   then block B = [O += V(t) P(t)] beside the exponentials of S(t+1)'s
//   first 32 keys.  Each block is cut into fenced steps of two MFMAs that
//   carry their share of the softmax VALU work and the LDS reads of the next
//   step, so one wave always has MFMAs and independent VALU work in flight.
//   Block A's first step also issues all global->LDS loads of tile t+2: the
//   earliest point at which their ring buffer is free, which gives them the
//   most time to land before the next barrier.
// * K/V tiles go from global memory straight into LDS (global_load_lds,
//   16 bytes per lane), issued two tiles ahead into three-deep rings (each
//   buffer its own LDS object, so the compiler can tell the reads of one
//   buffer from the loads in flight into another); one barrier per tile.
// * K is read with 16-byte LDS loads; V stays row-major in LDS and its V^T
//   operand is built with the transposing LDS read (ds_read_b64_tr_b16).
//   Both buffers are XOR-swizzled by row so the read patterns spread over all
//   LDS banks.
// * Rows are gathered through the memory's logical->slot table; a tile may
//   straddle two entries and the current chunk.  Row addresses come from
//   two wave-uniform entry bases per tile (entries of at least 64 rows), or
//   from a per-row lookup (shorter entries).  Rows past the last key load the
//   last key again and score -inf.
// * Online softmax in base 2 with the scale folded into one FMA; O is
//   rescaled only when a row max grows by more than 2^8 (the stale max
//   cancels in the final normalisation).  The row sum adds the fp32
//   weights before their bf16 rounding for the P.V product: it normalises O
//   (within 2^-9 of the rounded weights' sum) and gives the log-sum-exp
//   exact to fp32 rounding.  Two plain adds per pair of weights cost less
//   beside the MFMAs than summing the rounded pair with a v_dot2.
// * Workgroup index -> work is remapped so that one XCD runs a contiguous
//   range of (head, query tile) and shares K/V in its L2.
// * In a head's last query tile, usually partial, the waves whose 32
//   queries all lie past the last one only issue their share of the tile
//   loads and meet the barriers: no MFMAs, no softmax, no result.
#include <mutex>
#include <type_traits>

#include "fademem_internal.h"

namespace fademem {

// Work split over G resident workgroups.  Query tiles are numbered
// qg = head * q_tiles + tile within the head, Q of them.  The first
// rounds*G tiles run whole, round k giving tile k*G + g to group g.  Of the
// rem = Q - rounds*G remaining tiles, tile i's keys [0, head_len) go to
// group i (i < rem) and its tail [head_len, tiles) to group
// rem + i / tails_per: the G - rem tail groups each take tails_per
// consecutive tails.  head_len = tiles - tail_len, tail_len =
// (tiles - o (tails_per - 1)) / (tails_per + 1) with o = kSegOverhead key
// tiles per extra segment, so a tail group's tails_per tails, with their
// segment overheads, are no more work than one head part.  Every group starts its parts at the same key
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
constexpr int kWaves = kThreads / 64;
constexpr int kBM = kAttnQueries;  // queries per workgroup
constexpr int kQW = kBM / kWaves;  // queries per wave
constexpr int QB = kQW / 32;       // 32-query blocks per wave
constexpr int kBN = 64;            // keys per tile
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kRescaleBound = 256.0f;  // redo a tile whose weights exceed 2^8
constexpr int kSegOverhead = 2;          // key tiles' worth of time a segment's prologue and epilogue cost
static_assert(QB * 32 == kQW && (QB == 1 || QB == 2), "32-query blocks per wave");

template <int D>
struct Shape {
  static constexpr int CH = D / 8;                 // 16-byte chunks per row
  static constexpr int KB = D / 16;                // k-steps of S^T = K Q^T
  static constexpr int DB = D / 32;                // 32-row blocks of O^T
  static constexpr int RPB = 256 / (2 * D);        // rows per 256 bytes of LDS
  static constexpr int TILE_BYTES = kBN * D * 2;
  static constexpr int LOADS = kBN * CH / kThreads;  // 16-byte loads per lane per tile (per K and V)
  static_assert(LOADS * kThreads == kBN * CH, "tile split");
  static_assert(kBM * D == kWaves * QB * DB * 16 * 64, "scratch slot holds every wave's O registers");
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

// Two weights rounded to bf16 and packed as one B-operand word of P.V.
__device__ __forceinline__ uint32_t round_pair(float p0, float p1) {
  bf16x2 pk;
  pk[0] = (__bf16)p0;
  pk[1] = (__bf16)p1;
  return __builtin_bit_cast(uint32_t, pk);
}

__device__ __forceinline__ float pair_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __builtin_elementwise_maximum(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// A pointer the whole wave holds, moved to scalar registers.
__device__ __forceinline__ const char* uniform_ptr(const char* p) {
  const uint64_t u = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(uint32_t(u));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(uint32_t(u >> 32));
  return reinterpret_cast<const char*>((uint64_t(hi) << 32) | lo);
}

// XCD-aware group index: blocks are dealt to the 8 XCDs round-robin, so
// block b runs on XCD b % 8; give each XCD a contiguous run of groups.
__device__ __forceinline__ int xcd_group(int bid, int groups) {
  const int per = groups / 8, rem = groups % 8;
  const int xcd = bid % 8, local = bid / 8;
  return (xcd < rem) ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
}

// Final output of one lane for one 32-query block: O row (query q_row,
// head h) from the O^T accumulators divided by the row sum, and the row's
// LSE.
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

// Scratch slot layout of a partial result: O registers lane-major,
// [wave][qb][db][r][lane], then m and l per (qb, thread).
template <int D>
__device__ __forceinline__ size_t ws_o_index(int wave, int qb, int db, int r, int lane) {
  return ((size_t((wave * QB + qb) * Shape<D>::DB + db) * 16 + r) * 64 + lane);
}

template <int D, bool WIDE>
__device__ __forceinline__ void attend_bf16_body(const AttendArgs& args, const SkPlan& plan) {
  using S = Shape<D>;
  // Three-deep rings of K and V tile buffers, each a separate LDS object.
  __shared__ __attribute__((aligned(16))) char k_lds0[S::TILE_BYTES];
  __shared__ __attribute__((aligned(16))) char k_lds1[S::TILE_BYTES];
  __shared__ __attribute__((aligned(16))) char k_lds2[S::TILE_BYTES];
  __shared__ __attribute__((aligned(16))) char v_lds0[S::TILE_BYTES];
  __shared__ __attribute__((aligned(16))) char v_lds1[S::TILE_BYTES];
  __shared__ __attribute__((aligned(16))) char v_lds2[S::TILE_BYTES];
  // Entry table: K address of row 0 (head 0) of each exposed entry, and the
  // current chunk as entry n_entries; its V rows are ent_vd[e] bytes from
  // its K rows.
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const char** ent_k = reinterpret_cast<const char**>(smem);
  long long* ent_vd = reinterpret_cast<long long*>(smem + (size_t(args.n_entries) + 1) * sizeof(const char*));

  const int g = xcd_group(blockIdx.x, gridDim.x);
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int l32 = lane & 31;
  const int hh = lane >> 5;

  const int H = args.heads;
  const int n_entries = int(args.n_entries);
  const int N = int(args.tokens_per_block);
  const int cur_tokens = int(args.cur_tokens);
  const int Lk = n_entries * N + cur_tokens;
  const int Lq = int(args.q_tokens);
  const size_t row_bytes = size_t(H) * D * 2;
  const char* k_cur = static_cast<const char*>(args.k_cur);
  const int mem_rows = n_entries * N;

  for (int e = tid; e < n_entries + 1; e += kThreads) {
    const char* kp = k_cur;
    const char* vp = static_cast<const char*>(args.v_cur);
    if (e < n_entries) {
      kp = args.k_base + size_t(args.k_order ? args.k_order[e] : e) * args.k_stride;
      vp = args.v_base + size_t(args.v_order[e]) * args.v_stride;
    }
    ent_k[e] = kp;
    ent_vd[e] = vp - kp;
  }

  // Per-lane constants of the tile loads: load i writes destination chunk
  // q = (i*waves + wave)*64 + lane = row n0, LDS position p; it fetches global
  // chunk p ^ swz(n0) of that row.
  auto ld_row = [&](int i) { return ((i * kWaves + wave) * 64 + lane) / S::CH; };
  auto ld_kch = [&](int i) {
    const int q = (i * kWaves + wave) * 64 + lane;
    return uint32_t(((q % S::CH) ^ kswz<D>(q / S::CH)) * 16);
  };
  auto ld_vch = [&](int i) {
    const int q = (i * kWaves + wave) * 64 + lane;
    return uint32_t(((q % S::CH) ^ vswz<D>(q / S::CH)) * 16);
  };
  // Byte offsets from a tile's first row to this lane's K and V chunks.
  uint32_t ld_koff[S::LOADS], ld_voff[S::LOADS];
#pragma unroll
  for (int i = 0; i < S::LOADS; ++i) {
    ld_koff[i] = uint32_t(size_t(ld_row(i)) * row_bytes) + ld_kch(i);
    ld_voff[i] = uint32_t(size_t(ld_row(i)) * row_bytes) + ld_vch(i);
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

  char* const kbuf[3] = {k_lds0, k_lds1, k_lds2};
  char* const vbuf[3] = {v_lds0, v_lds1, v_lds2};

  // One query tile's key tiles [kt0, kt1); the result goes to the output
  // (slot < 0, the range is the whole key axis) or, partial, to scratch slot
  // `slot`.
  auto segment = [&](int h, int qt, int kt0, int kt1, int slot) {
    const size_t head_off = size_t(h) * D * 2;

    // Q fragments (B operand of S^T = K Q^T): query m = l32 of block qb,
    // d = 16*kb + 8*hh + 0..7.
    bf16x8 qf[QB][S::KB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const int q_row = qt * kBM + wave * kQW + 32 * qb + l32;
      const char* qbase = static_cast<const char*>(args.q) + (size_t(q_row < Lq ? q_row : Lq - 1) * H + h) * D * 2;
#pragma unroll
      for (int kb = 0; kb < S::KB; ++kb)
        qf[qb][kb] = *reinterpret_cast<const bf16x8*>(qbase + (16 * kb + 8 * hh) * 2);
    }

    // Address of the last key's row (rows past the last key load it again).
    const char* last_k;
    long long last_vd;
    if (cur_tokens > 0) {
      last_k = k_cur + size_t(cur_tokens - 1) * row_bytes + head_off;
      last_vd = ent_vd[n_entries];
    } else {
      last_k = ent_k[n_entries - 1] + size_t(N - 1) * row_bytes + head_off;
      last_vd = ent_vd[n_entries - 1];
    }

    // Load stream: the next tile to load starts in entry ld_e at row ld_off
    // (ld_e == n_entries: the current chunk).
    int ld_e, ld_off;
    {
      const int k0 = kt0 * kBN;
      if (k0 < mem_rows) {
        ld_e = k0 / N;
        ld_off = k0 - ld_e * N;
      } else {
        ld_e = n_entries;
        ld_off = k0 - mem_rows;
      }
    }
    // Wave-uniform part of one tile's row addresses (entries of >= 64 rows:
    // rows n < ncross are entry ld_e's rows ld_off + n, the rest are entry
    // ld_e+1's rows n - ncross); advances the stream by one tile.
    struct TileRows {
      const char* base0;
      const char* base1;
      long long vd0, vd1;
      int ncross, nvalid, k0;
    };
    auto tile_rows = [&](int tile) {
      TileRows tr;
      tr.k0 = tile * kBN;
      tr.nvalid = Lk - tr.k0;
      if constexpr (WIDE) {
        const int e1 = ld_e + 1 <= n_entries ? ld_e + 1 : n_entries;
        const bool in_mem0 = ld_e < n_entries;
        tr.ncross = in_mem0 ? N - ld_off : kBN;
        tr.base0 = ent_k[ld_e] + head_off + (long long)ld_off * (long long)row_bytes;
        tr.base1 = ent_k[e1] + head_off - (long long)tr.ncross * (long long)row_bytes;
        tr.vd0 = ent_vd[ld_e];
        tr.vd1 = ent_vd[e1];
        ld_off += kBN;
        if (in_mem0 && ld_off >= N) {
          ld_off -= N;
          ++ld_e;
        }
      }
      return tr;
    };
    // Load i (K and V) of a tile into the given buffers.
    auto load_one = [&](const TileRows& tr, int i, char* kb_lds, char* vb_lds) {
      const char* row;
      long long vd;
      if constexpr (WIDE) {
        const int n = ld_row(i);
        const bool cross = n >= tr.ncross;
        const bool valid = n < tr.nvalid;
        row = valid ? (cross ? tr.base1 : tr.base0) + size_t(n) * row_bytes : last_k;
        vd = valid ? (cross ? tr.vd1 : tr.vd0) : last_vd;
      } else {
        // Entries shorter than a tile: resolve the row on its own.
        const int k = tr.k0 + ld_row(i);
        if (k >= Lk) {
          row = last_k;
          vd = last_vd;
        } else if (k < mem_rows) {
          const int e = k / N;
          row = ent_k[e] + head_off + size_t(k - e * N) * row_bytes;
          vd = ent_vd[e];
        } else {
          row = k_cur + head_off + size_t(k - mem_rows) * row_bytes;
          vd = ent_vd[n_entries];
        }
      }
      const int j = i * kWaves + wave;
      __builtin_amdgcn_global_load_lds(row + ld_kch(i), (LDS_AS void*)(kb_lds + j * 1024), 16, 0, 0);
      __builtin_amdgcn_global_load_lds(row + vd + ld_vch(i), (LDS_AS void*)(vb_lds + j * 1024), 16, 0, 0);
    };
    // All loads of a tile.  A full tile inside one entry (the common case)
    // takes its rows from one wave-uniform base plus the lane's fixed
    // offsets, so its addresses cost no vector instructions.
    auto load_tile = [&](const TileRows& tr, char* kb_lds, char* vb_lds) {
      if constexpr (WIDE) {
        if (tr.ncross >= kBN && tr.nvalid >= kBN) {
          const char* kbase = uniform_ptr(tr.base0);
          const char* vbase = uniform_ptr(tr.base0 + tr.vd0);
#pragma unroll
          for (int i = 0; i < S::LOADS; ++i) {
            const int j = i * kWaves + wave;
            __builtin_amdgcn_global_load_lds(kbase + ld_koff[i], (LDS_AS void*)(kb_lds + j * 1024), 16, 0, 0);
            __builtin_amdgcn_global_load_lds(vbase + ld_voff[i], (LDS_AS void*)(vb_lds + j * 1024), 16, 0, 0);
          }
          return;
        }
      }
#pragma unroll
      for (int i = 0; i < S::LOADS; ++i) load_one(tr, i, kb_lds, vb_lds);
    };
    auto issue_tile = [&](int tile, char* kb_lds, char* vb_lds) { load_tile(tile_rows(tile), kb_lds, vb_lds); };

    // A wave whose queries all lie past the last one (the last query tile
    // of a head is usually partial) does no arithmetic: it issues its share
    // of every tile's loads and meets the same barriers as the other waves
    // (two in the prologue, one per key tile), and leaves no result.
    if (qt * kBM + wave * kQW >= Lq) {
      __syncthreads();
      issue_tile(kt0, kbuf[0], vbuf[0]);
      if (kt0 + 1 < kt1) issue_tile(kt0 + 1, kbuf[1], vbuf[1]);
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      int b = 2;
      for (int t = kt0; t < kt1; ++t) {
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (t + 2 < kt1)
          issue_tile(t + 2, b == 0 ? kbuf[0] : b == 1 ? kbuf[1] : kbuf[2], b == 0 ? vbuf[0] : b == 1 ? vbuf[1] : vbuf[2]);
        b = b == 2 ? 0 : b + 1;
      }
      return;
    }

    f32x16 o[QB][S::DB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
      for (int db = 0; db < S::DB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[qb][db][r] = 0.0f;
    float m_run[QB], l_run[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      m_run[qb] = -INFINITY;  // running (possibly stale) max of raw scores
      l_run[qb] = 0.0f;       // this lane's partial sum of 2^(s*c2 - m_run*c2)
    }

    const int partial_tile = (Lk % kBN) ? (Lk / kBN) : -1;  // the tile with keys >= Lk, if any
    f32x16 s_cur[2][QB];  // S^T of the current tile [nb][qb]
    u32x4 p_cur[4][QB];   // P of the current tile [ks][qb] (bf16 pairs)
    float ps_cur[QB];     // this lane's sum of the current tile's weights so far

    // Softmax without a per-tile row max: a tile's weights are taken against
    // the running max m_run as it stands.  If any weight of a row exceeds
    // 2^8 (seen as the lane's tile sum exceeding 2^8: every weight is at most
    // the sum), the tile is redone against the exact new max and O and l are
    // rescaled; otherwise every weight stays <= 2^8 and the stale m_run
    // cancels in the final normalisation.
    //
    // Score pair pi (0..kPairs-1) of a tile: query block qb = pi/16, rows
    // r, r+1 of accumulator block nb.  Pairs [0, kPairsB) are exponentiated
    // in block B, the rest in the next block A.
    constexpr int kPairs = 16 * QB;
    constexpr int kPairsB = 8 * QB;
    auto exp_pair = [&](const f32x16 (&s)[2][QB], u32x4 (&p)[4][QB], float (&ps)[QB], int pi) {
      const int qb = pi / 16, rr = pi % 16, nb = rr / 8, r = 2 * (rr % 8);
      const float mc = m_run[qb] * c2;
      const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[nb][qb][r], c2, -mc));
      const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[nb][qb][r + 1], c2, -mc));
      ps[qb] = ps[qb] + (p0 + p1);
      const uint32_t w = round_pair(p0, p1);
      asm volatile("" ::"v"(w));  // keep the weight in its pipeline step
      p[2 * nb + (r >> 3)][qb][(r & 7) >> 1] = w;
    };
    // Mask keys >= Lk of a tile to -inf.
    auto mask = [&](int tile, f32x16 (&s)[2][QB]) {
      const int k0 = tile * kBN;
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = k0 + 32 * nb + 8 * (r >> 2) + 4 * hh + (r & 3);
            if (key >= Lk) s[nb][qb][r] = -INFINITY;
          }
    };
    // Row max of a tile's scores (v_maximum3: NaN-propagating, so the raw
    // MFMA results need no canonicalisation), reduced over the lane pair.
    auto row_max = [&](const f32x16 (&s)[2][QB], float (&mx)[QB]) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        float m0 = s[0][qb][0], m1 = s[1][qb][0];
#pragma unroll
        for (int r = 1; r < 15; r += 2) {
          m0 = __builtin_elementwise_maximum(m0, __builtin_elementwise_maximum(s[0][qb][r], s[0][qb][r + 1]));
          m1 = __builtin_elementwise_maximum(m1, __builtin_elementwise_maximum(s[1][qb][r], s[1][qb][r + 1]));
        }
        mx[qb] = pair_max(__builtin_elementwise_maximum(m0, __builtin_elementwise_maximum(m1, __builtin_elementwise_maximum(
                                                                                                 s[0][qb][15], s[1][qb][15]))));
      }
    };
    // S^T of a tile from its K buffer (masked if it is the partial tile).
    auto qk_tile = [&](int tile, const char* kb_lds, f32x16 (&s)[2][QB]) {
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
          for (int r = 0; r < 16; ++r) s[nb][qb][r] = 0.0f;
#pragma unroll
      for (int kb = 0; kb < S::KB; ++kb) {
        const bf16x8 k0 = *reinterpret_cast<const bf16x8*>(kb_lds + k_rd[kb]);
        const bf16x8 k1 = *reinterpret_cast<const bf16x8*>(kb_lds + k_rd[kb] + 32 * D * 2);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
          s[0][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k0, qf[qb][kb], s[0][qb], 0, 0, 0);
          s[1][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k1, qf[qb][kb], s[1][qb], 0, 0, 0);
        }
      }
      if (tile == partial_tile) mask(tile, s);
    };
    // Redo a tile against the exact running max: its scores again from its K
    // buffer, new m_run, rescale O and l, recompute all its weights and the
    // tile sum.
    auto redo_tile = [&](int tile, const char* kb_lds, u32x4 (&p)[4][QB], float (&ps)[QB]) {
      f32x16 s[2][QB];
      qk_tile(tile, kb_lds, s);
      float mx[QB];
      row_max(s, mx);
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const float m_new = __builtin_elementwise_maximum(m_run[qb], mx[qb]);
        const float alpha = __builtin_amdgcn_exp2f((m_run[qb] - m_new) * c2);
        m_run[qb] = m_new;
        l_run[qb] *= alpha;
#pragma unroll
        for (int db = 0; db < S::DB; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[qb][db][r] *= alpha;
        ps[qb] = 0.0f;
      }
#pragma unroll
      for (int pi = 0; pi < kPairs; ++pi) exp_pair(s, p, ps, pi);
    };
    // End of a tile's weights: redo it if a weight grew past 2^8, then add
    // its sum to l.
    auto close_tile = [&](int tile, const char* kb_lds, u32x4 (&p)[4][QB], float (&ps)[QB]) {
      bool grow = false;
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) grow = grow || !(ps[qb] <= kRescaleBound);
      if (__any(grow)) redo_tile(tile, kb_lds, p, ps);
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        l_run[qb] += ps[qb];
      }
    };
    auto read_k = [&](const char* kb_lds, int kb, bf16x8 (&kf)[2]) {
      kf[0] = *reinterpret_cast<const bf16x8*>(kb_lds + k_rd[kb]);
      kf[1] = *reinterpret_cast<const bf16x8*>(kb_lds + k_rd[kb] + 32 * D * 2);
    };
    // V^T fragment of k-step ks, 32-row block db (two transposing reads).
    auto read_v = [&](const char* vb_lds, int ks, int db) {
      bf16x8 a;
#pragma unroll
      for (int second = 0; second < 2; ++second) {
        const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (LDS_AS s16x4*)((LDS_AS const char*)(vb_lds) + v_rd[db] + (16 * ks + 8 * second) * D * 2));
        const bf16x4 vb = __builtin_bit_cast(bf16x4, v);
#pragma unroll
        for (int e = 0; e < 4; ++e) a[4 * second + e] = vb[e];
      }
      return a;
    };
    constexpr int kStepsB = 2 * S::DB;                // block B steps: (ks, pair of 32-row blocks)
    constexpr int kDbPerStep = S::DB * 4 / kStepsB;   // = 2
    constexpr int kPrefetch = 1;                      // steps between an LDS read and its MFMA

    // One pipeline iteration for tile t (ring slot b): boundary, block A,
    // tile t's weight check, block B.  LOAD: tile t+2 exists (its loads are
    // issued); NEXT: tile t+1 exists; maskn: tile t+1 has keys >= Lk.
    auto iteration = [&](int t, auto b_c, auto load_c, auto next_c, bool maskn) {
      constexpr int b = decltype(b_c)::value;
      constexpr bool LOAD = decltype(load_c)::value;
      constexpr bool NEXT = decltype(next_c)::value;
      const char* kb_next = kbuf[(b + 1) % 3];
      const char* vb_cur = vbuf[b];
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();  // tiles t, t+1 landed for every wave; tile t-1's buffers are free
      TileRows tr;
      if constexpr (LOAD) tr = tile_rows(t + 2);

      // Block A: S(t+1) = K(t+1) Q^T, one k-step per step, beside the loads
      // of tile t+2 and the weights of S(t)'s pairs [kPairsB, kPairs).  The
      // LDS reads of step st + kPrefetch are issued in step st (block A's
      // last steps prefetch block B's first V^T fragments).
      f32x16 s_next[2][QB];
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
          for (int r = 0; r < 16; ++r) s_next[nb][qb][r] = 0.0f;
      bf16x8 kring[kPrefetch + 1][2];
      bf16x8 vring[kPrefetch + 1][kDbPerStep];
      if constexpr (NEXT) {
#pragma unroll
        for (int j = 0; j < kPrefetch && j < S::KB; ++j) read_k(kb_next, j, kring[j]);
      }
#pragma unroll
      for (int st = 0; st < S::KB; ++st) {
        if constexpr (NEXT) {
          if (st + kPrefetch < S::KB) read_k(kb_next, st + kPrefetch, kring[(st + kPrefetch) % (kPrefetch + 1)]);
        }
        {
          const int j = st + kPrefetch - S::KB;  // block B step to prefetch
          if (j >= 0 && j < kStepsB) {
#pragma unroll
            for (int d = 0; d < kDbPerStep; ++d)
              vring[j % (kPrefetch + 1)][d] =
                  read_v(vb_cur, j / (S::DB / kDbPerStep), (j % (S::DB / kDbPerStep)) * kDbPerStep + d);
          }
        }
        if constexpr (LOAD) {
          if (st == 0) load_tile(tr, kbuf[(b + 2) % 3], vbuf[(b + 2) % 3]);
        }
        if constexpr (NEXT) {
#pragma unroll
          for (int nb = 0; nb < 2; ++nb)
#pragma unroll
            for (int qb = 0; qb < QB; ++qb)
              s_next[nb][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kring[st % (kPrefetch + 1)][nb], qf[qb][st],
                                                                      s_next[nb][qb], 0, 0, 0);
        }
#pragma unroll
        for (int pi = kPairsB; pi < kPairs; ++pi)
          if (st == (pi - kPairsB) * S::KB / (kPairs - kPairsB)) exp_pair(s_cur, p_cur, ps_cur, pi);
        __builtin_amdgcn_sched_barrier(0);
      }
      close_tile(t, kbuf[b], p_cur, ps_cur);  // tile t's K buffer is refilled only in the next block A
      __builtin_amdgcn_sched_barrier(0);

      // Block B: O += V(t) P(t), two 32-row blocks of one k-step per step,
      // beside the weights of S(t+1)'s pairs [0, kPairsB).
      if constexpr (NEXT) {
        if (maskn) mask(t + 1, s_next);
      }
      u32x4 p_next[4][QB];
      float ps_next[QB];
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) ps_next[qb] = 0.0f;
#pragma unroll
      for (int st = 0; st < kStepsB; ++st) {
        const int ks = st / (S::DB / kDbPerStep), db0 = (st % (S::DB / kDbPerStep)) * kDbPerStep;
        if (st + kPrefetch < kStepsB) {
          const int j = st + kPrefetch;
#pragma unroll
          for (int d = 0; d < kDbPerStep; ++d)
            vring[j % (kPrefetch + 1)][d] =
                read_v(vb_cur, j / (S::DB / kDbPerStep), (j % (S::DB / kDbPerStep)) * kDbPerStep + d);
        }
#pragma unroll
        for (int d = 0; d < kDbPerStep; ++d)
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
            o[qb][db0 + d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                vring[st % (kPrefetch + 1)][d], __builtin_bit_cast(bf16x8, p_cur[ks][qb]), o[qb][db0 + d], 0, 0, 0);
        if constexpr (NEXT) {
#pragma unroll
          for (int pi = 0; pi < kPairsB; ++pi)
            if (st == pi * kStepsB / kPairsB) exp_pair(s_next, p_next, ps_next, pi);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      if constexpr (NEXT) {
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) s_cur[nb][qb] = s_next[nb][qb];
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
          for (int ks = 0; ks < 4; ++ks) p_cur[ks][qb] = p_next[ks][qb];
          ps_cur[qb] = ps_next[qb];
        }
      }
    };

    // Prologue: tiles kt0 and kt0+1 into ring slots 0 and 1; S(kt0), its
    // exact row max and its first kPairsB weights.
    __syncthreads();  // entry table visible; the previous segment's reads of the buffers are done
    issue_tile(kt0, kbuf[0], vbuf[0]);
    if (kt0 + 1 < kt1) issue_tile(kt0 + 1, kbuf[1], vbuf[1]);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    {
      qk_tile(kt0, kbuf[0], s_cur);
      row_max(s_cur, m_run);
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) ps_cur[qb] = 0.0f;
#pragma unroll
      for (int pi = 0; pi < kPairsB; ++pi) exp_pair(s_cur, p_cur, ps_cur, pi);
    }

    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    using T = std::true_type;
    using F = std::false_type;
    int t = kt0;
    while (true) {
      if (t + 2 >= kt1) break;
      iteration(t, I0{}, T{}, T{}, false);
      ++t;
      if (t + 2 >= kt1) break;
      iteration(t, I1{}, T{}, T{}, false);
      ++t;
      if (t + 2 >= kt1) break;
      iteration(t, I2{}, T{}, T{}, false);
      ++t;
    }
    // The last one or two tiles (no loads left to issue).
    if (t + 1 < kt1) {
      const int b = (t - kt0) % 3;
      const bool mk = (t + 1 == partial_tile);
      if (b == 0) iteration(t, I0{}, F{}, T{}, mk);
      else if (b == 1) iteration(t, I1{}, F{}, T{}, mk);
      else iteration(t, I2{}, F{}, T{}, mk);
      ++t;
    }
    {
      const int b = (t - kt0) % 3;
      if (b == 0) iteration(t, I0{}, F{}, F{}, false);
      else if (b == 1) iteration(t, I1{}, F{}, F{}, false);
      else iteration(t, I2{}, F{}, F{}, false);
    }
    // (The last tile's rescale was applied at its boundary.)
    if (slot < 0) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
        store_out<D>(args, o[qb], m_run[qb] * c2, pair_sum(l_run[qb]), qt * kBM + wave * kQW + 32 * qb + l32, h, hh);
    } else {
      float* ws = args.ws + size_t(slot) * attend_slot_floats(D);
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
        for (int db = 0; db < S::DB; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) ws[ws_o_index<D>(wave, qb, db, r, lane)] = o[qb][db][r];
        ws[kBM * D + qb * kThreads + tid] = m_run[qb];
        ws[kBM * D + (QB + qb) * kThreads + tid] = l_run[qb];
      }
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
// (slot i) and tail part (slot rem + i) and writes the output.  The slot
// rows of waves past the last query hold no result; they are read but
// never stored.
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
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int mi = kBM * D + qb * kThreads + tid, li = kBM * D + (QB + qb) * kThreads + tid;
    const float m_max = fmaxf(part[0][mi], part[1][mi]);
    f32x16 o[S::DB];
#pragma unroll
    for (int db = 0; db < S::DB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[db][r] = 0.0f;
    float l_tot = 0.0f;
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const float* ws = part[p];
      const float f = __builtin_amdgcn_exp2f((ws[mi] - m_max) * c2);
      l_tot += f * pair_sum(ws[li]);
#pragma unroll
      for (int db = 0; db < S::DB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] += f * ws[ws_o_index<D>(wave, qb, db, r, lane)];
    }
    store_out<D>(args, o, m_max * c2, l_tot, (qg % plan.q_tiles) * kBM + wave * kQW + 32 * qb + l32,
                 qg / plan.q_tiles, hh);
  }
}

}  // namespace

// Kernels: head dimension, entries of at least one key tile (or shorter).
__global__ __launch_bounds__(kThreads, 1) void attend_bf16_d128(AttendArgs args, SkPlan plan) {
  attend_bf16_body<128, true>(args, plan);
}
__global__ __launch_bounds__(kThreads, 1) void attend_bf16_d64(AttendArgs args, SkPlan plan) {
  attend_bf16_body<64, true>(args, plan);
}
__global__ __launch_bounds__(kThreads, 1) void attend_bf16_d128_short(AttendArgs args, SkPlan plan) {
  attend_bf16_body<128, false>(args, plan);
}
__global__ __launch_bounds__(kThreads, 1) void attend_bf16_d64_short(AttendArgs args, SkPlan plan) {
  attend_bf16_body<64, false>(args, plan);
}
__global__ __launch_bounds__(kThreads) void attend_bf16_merge_d128(AttendArgs args, SkPlan plan) {
  attend_bf16_merge_body<128>(args, plan);
}
__global__ __launch_bounds__(kThreads) void attend_bf16_merge_d64(AttendArgs args, SkPlan plan) {
  attend_bf16_merge_body<64>(args, plan);
}

namespace {

typedef void (*AttnKernel)(AttendArgs, SkPlan);

hipError_t launch_d(AttnKernel kernel, AttnKernel merge, std::once_flag& attr_once, const AttendArgs& a,
                    hipStream_t stream) {
  const int64_t q_tiles64 = (a.q_tokens + kBM - 1) / kBM;
  if (q_tiles64 * a.heads > int64_t(0x7fffffff)) return hipErrorInvalidValue;
  const int64_t lk = a.n_entries * a.tokens_per_block + a.cur_tokens;
  SkPlan plan;
  plan.q_tiles = int(q_tiles64);
  plan.tiles = int((lk + kBN - 1) / kBN);
  const int total = plan.q_tiles * a.heads;
  const size_t shmem = size_t(a.n_entries + 1) * 16;  // entry table; tile buffers are static
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
  {
    // A tail group runs tails_per segments, each with a prologue (two tile
    // loads waited in full) and an epilogue: about kSegOverhead key tiles
    // each, beyond the head part's one.
    const int over = kSegOverhead * (plan.tails_per - 1);
    plan.tail_len = plan.tiles > over ? (plan.tiles - over) / (plan.tails_per + 1) : 0;
  }
  plan.head_len = plan.tiles - plan.tail_len;
  const int launched =
      plan.rounds > 0 ? plan.groups
                      : plan.rem + (plan.tail_len > 0 ? (plan.rem + plan.tails_per - 1) / plan.tails_per : 0);
  hipLaunchKernelGGL(kernel, dim3(launched), dim3(kThreads), shmem, stream, a, plan);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (plan.rem > 0 && plan.tail_len > 0) {
    hipLaunchKernelGGL(merge, dim3(plan.rem), dim3(kThreads), 0, stream, a, plan);
    e = hipGetLastError();
  }
  return e;
}

std::once_flag attr_once[4];

}  // namespace

hipError_t launch_attend_bf16(const AttendArgs& a, hipStream_t stream) {
  const int w = a.tokens_per_block >= kBN ? 1 : 0;
  static const AttnKernel k128[2] = {attend_bf16_d128_short, attend_bf16_d128};
  static const AttnKernel k64[2] = {attend_bf16_d64_short, attend_bf16_d64};
  if (a.head_dim == 128) return launch_d(k128[w], attend_bf16_merge_d128, attr_once[w], a, stream);
  if (a.head_dim == 64) return launch_d(k64[w], attend_bf16_merge_d64, attr_once[2 + w], a, stream);
  return hipErrorInvalidValue;
}

}  // namespace fademem
