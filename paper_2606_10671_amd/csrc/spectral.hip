// Distance-dependent spectral decay (FadeMem Sec. 3.2; supplementary Sec. S2):
// per clip of channel-averaged latent frames z_0..z_T-1 ([H][W] fp32 each),
// the orthonormal 2-D DCT-II D(z_t) = A_H z_t A_W^T of every frame up to the
// largest lag, then for every radial band k (given as a band index per
// coefficient) and lag the Pearson correlation of band k's coefficients of
// frame 0 and of frame lag, averaged over clips:
//   C_k(lag) = mean_clips Pearson(D(z_0)|B_k, D(z_lag)|B_k).
//
// Kernels:
// * dct_basis_kernel -- A_N[k][n] = s_k cos(pi (2n+1) k / (2N)), s_0 =
//   sqrt(1/N), s_k = sqrt(2/N), in fp64, stored fp32;
// * band_order_kernel -- the coefficients grouped by band (a stable
//   counting sort in one block), so each band is a contiguous index list;
// * spectral_fused_kernel (frames up to 64 x 128) -- persistent blocks, each
//   taking an equal contiguous range of the (clip, lag) frames: per frame
//   T = z A_W^T and D = A_H T on the fp32 matrix cores
//   (v_mfma_f32_16x16x4_f32; wave j owns the 16 columns v of tile j), the
//   second product taking T straight from the first one's accumulators,
//   then D written to LDS in band order and reduced per band to the fp64
//   sums S_y, S_yy and S_xy against frame 0's coefficients x (kept in LDS).
//   Frames go in pairs: both transforms are staged, then one band pass
//   sums both (six sums per band), so the band pass's latency is paid once
//   per two frames; no transform ever reaches HBM;
// * clip_mean_kernel -- per clip the Pearson coefficient from those sums
//   (frame 0's own, at lag 0, give S_x and S_xx), then the mean over clips
//   in a fixed order (every call gives the same bits).
// Larger frames take the general path:
// * dct2_kernel -- one block per (clip, run of frames): both bases (as
//   transposes) in LDS once, then per frame z^T in LDS, T = z A_W^T and
//   D = A_H T, each thread computing 4 x 4 output tiles from 16-byte LDS
//   reads (8 FMAs per read); fp32 products and sums; sizes padded to
//   multiples of 4 with zeros;
// * band_corr_kernel -- one block per (clip, lag): each wave takes bands in
//   turn and sums y, y^2 and x y over the band in fp64 (lanes, then a wave
//   reduction), x being frame 0.
#include <math.h>
#include <string.h>

#include <mutex>
#include <vector>

#include "fademem_internal.h"

namespace {

inline size_t rup(size_t x) { return (x + 255) / 256 * 256; }

constexpr int kSpecLdsBytes = 160 * 1024;  // LDS of one workgroup on gfx950
constexpr int kSpecMaxBands = 1024;
constexpr int kSpecMaxLags = 65535;        // grid.y

struct SpecLayout {
  size_t off_ah, off_aw, off_d, off_perm, off_start, off_clip, total;
};

bool spec_layout(int64_t clips, int64_t nlag, int64_t H, int64_t W, int64_t bands, bool fused, SpecLayout* L) {
  const double d_bytes = fused ? 0.0 : double(clips) * double(nlag) * double(H) * double(W) * 4.0;
  const double c_bytes = double(clips) * double(nlag) * double(bands) * 24.0;
  if (d_bytes > 1e15 || c_bytes > 1e15) return false;
  size_t off = 0;
  L->off_ah = off;    off = rup(off + size_t(H * H) * 4);
  L->off_aw = off;    off = rup(off + size_t(W * W) * 4);
  L->off_d = off;     off = rup(off + (fused ? 0 : size_t(clips) * size_t(nlag) * size_t(H * W) * 4));
  L->off_perm = off;  off = rup(off + size_t(H * W) * 4);
  L->off_start = off; off = rup(off + size_t(bands + 1) * 4);
  L->off_clip = off;  off = rup(off + size_t(clips) * size_t(nlag) * size_t(bands) * 24);
  L->total = off;
  return true;
}

int64_t pad4(int64_t x) { return (x + 3) / 4 * 4; }
size_t dct_lds_bytes(int64_t H, int64_t W) {
  const int64_t Hp = pad4(H), Wp = pad4(W);
  return size_t(2 * Hp * Wp + Hp * Hp + Wp * Wp) * 4;
}
constexpr int kDctFramesPerBlock = 8;

__global__ void dct_basis_kernel(float* A, int N) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= N * N) return;
  const int k = i / N, n = i % N;
  const double s = k == 0 ? sqrt(1.0 / N) : sqrt(2.0 / N);
  A[i] = float(s * cos(M_PI * (2.0 * n + 1.0) * double(k) / (2.0 * N)));
}

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kDctThreads = 512;

__global__ __launch_bounds__(kDctThreads) void dct2_kernel(const float* latents, int64_t frames, int nlag, int H, int W,
                                                   const float* AH, const float* AW, float* D) {
  extern __shared__ __attribute__((aligned(16))) float sm[];
  const int Hp = (H + 3) & ~3, Wp = (W + 3) & ~3;
  float* zt = sm;                 // z^T   [Wp][Hp]
  float* ts = zt + Wp * Hp;       // T     [Hp][Wp]
  float* aht = ts + Hp * Wp;      // A_H^T [Hp][Hp]: aht[h][u] = A_H[u][h]
  float* awt = aht + Hp * Hp;     // A_W^T [Wp][Wp]: awt[w][v] = A_W[v][w]
  const int64_t c = blockIdx.x;
  const int tid = threadIdx.x;
  const int HW = H * W;
  for (int i = tid; i < Hp * Hp; i += kDctThreads) {
    const int h = i / Hp, u = i % Hp;
    aht[i] = (h < H && u < H) ? AH[u * H + h] : 0.0f;
  }
  for (int i = tid; i < Wp * Wp; i += kDctThreads) {
    const int w = i / Wp, v = i % Wp;
    awt[i] = (w < W && v < W) ? AW[v * W + w] : 0.0f;
  }
  const int th = Hp / 4, tw = Wp / 4, tiles = th * tw;
  const int t0 = blockIdx.y * kDctFramesPerBlock;
  const int t1 = min(t0 + kDctFramesPerBlock, nlag);
  for (int t = t0; t < t1; ++t) {
    const float* z = latents + (size_t(c) * size_t(frames) + size_t(t)) * size_t(HW);
    __syncthreads();  // the previous frame's reads of zt and ts are done (and the bases are in)
    for (int i = tid; i < Wp * Hp; i += kDctThreads) {
      const int w = i / Hp, h = i % Hp;
      zt[i] = (w < W && h < H) ? z[h * W + w] : 0.0f;
    }
    __syncthreads();
    for (int i = tid; i < tiles; i += kDctThreads) {  // T[h][v] = sum_w z[h][w] A_W[v][w]
      const int h0 = 4 * (i / tw), v0 = 4 * (i % tw);
      f32x4 acc[4] = {};
#pragma unroll 4
      for (int w = 0; w < Wp; ++w) {
        const f32x4 zv = *reinterpret_cast<const f32x4*>(zt + w * Hp + h0);
        const f32x4 av = *reinterpret_cast<const f32x4*>(awt + w * Wp + v0);
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
          for (int b = 0; b < 4; ++b) acc[a][b] = __builtin_fmaf(zv[a], av[b], acc[a][b]);
      }
#pragma unroll
      for (int a = 0; a < 4; ++a) *reinterpret_cast<f32x4*>(ts + (h0 + a) * Wp + v0) = acc[a];
    }
    __syncthreads();
    float* out = D + (size_t(c) * size_t(nlag) + size_t(t)) * size_t(HW);
    for (int i = tid; i < tiles; i += kDctThreads) {  // D[u][v] = sum_h A_H[u][h] T[h][v]
      const int u0 = 4 * (i / tw), v0 = 4 * (i % tw);
      f32x4 acc[4] = {};
#pragma unroll 4
      for (int h = 0; h < Hp; ++h) {
        const f32x4 av = *reinterpret_cast<const f32x4*>(aht + h * Hp + u0);
        const f32x4 tv = *reinterpret_cast<const f32x4*>(ts + h * Wp + v0);
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
          for (int b = 0; b < 4; ++b) acc[a][b] = __builtin_fmaf(av[a], tv[b], acc[a][b]);
      }
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const int u = u0 + a;
        if (u >= H) continue;
#pragma unroll
        for (int b = 0; b < 4; ++b)
          if (v0 + b < W) out[u * W + v0 + b] = acc[a][b];
      }
    }
  }
}

// Exclusive prefix sum over the block (all threads must call it); *total
// gets the sum of every thread's value.
__device__ int block_exclusive_scan(int v, int32_t* wsum, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int x = v;
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  __syncthreads();  // wsum is free
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  int before = 0, all = 0;
  for (int w = 0; w < nw; ++w) {
    const int t = wsum[w];
    if (w < wave) before += t;
    all += t;
  }
  *total = all;
  return before + x - v;
}

// Coefficient indices grouped by band, in index order within a band;
// entries outside [0, bands) are left out.  One block of 1024 threads with
// the band map in LDS: thread t counts band t / C in chunk t % C of the map
// (C = 1024 / bands chunks per band), a block prefix sum gives each (band,
// chunk) its first position, and the thread writes that chunk's indices of
// the band in order.
constexpr int kOrderMaxHW = 40960;
constexpr int kOrderThreads = 1024;
__global__ __launch_bounds__(kOrderThreads) void band_order_kernel(const int32_t* band_of, int HW, int bands,
                                                                   int32_t* perm, int32_t* start) {
  __shared__ int16_t map[kOrderMaxHW];
  __shared__ int32_t wsum[kOrderThreads / 64];
  const int tid = threadIdx.x;
  for (int i = tid; i < HW; i += kOrderThreads) {
    const int b = band_of[i];
    map[i] = int16_t((b >= 0 && b < bands) ? b : -1);
  }
  const int C = kOrderThreads / bands;  // bands <= 1024
  const int b = tid / C, j = tid % C;
  const bool on = b < bands;
  const int len = (HW + C - 1) / C;
  const int i0 = min(HW, j * len), i1 = min(HW, i0 + len);
  __syncthreads();
  int n = 0;
  if (on)
    for (int i = i0; i < i1; ++i) n += (map[i] == b);
  int total;
  int pos = block_exclusive_scan(n, wsum, &total);
  if (on && j == 0) start[b] = pos;
  if (tid == 0) start[bands] = total;
  if (on)
    for (int i = i0; i < i1; ++i)
      if (map[i] == b) perm[pos++] = i;
}

__device__ __forceinline__ double wave_sum(double v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__global__ __launch_bounds__(256) void band_corr_kernel(const float* D, int nlag, int HW, const int32_t* perm,
                                                        const int32_t* start, int bands, double* per_clip) {
  const int64_t c = blockIdx.x;
  const int lag = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const float* x = D + size_t(c) * size_t(nlag) * size_t(HW);
  const float* y = x + size_t(lag) * size_t(HW);
  double* out = per_clip + (size_t(c) * size_t(nlag) + size_t(lag)) * size_t(bands) * 3;
  for (int b = wave; b < bands; b += 4) {
    const int s0 = start[b], s1 = start[b + 1];
    double sy = 0, syy = 0, sxy = 0;
    for (int j = s0 + lane; j < s1; j += 64) {
      const int i = perm[j];
      const double xv = x[i], yv = y[i];
      sy += yv;
      syy += yv * yv;
      sxy += xv * yv;
    }
    sy = wave_sum(sy);
    syy = wave_sum(syy);
    sxy = wave_sum(sxy);
    if (lane == 0) {
      out[3 * b] = sy;
      out[3 * b + 1] = syy;
      out[3 * b + 2] = sxy;
    }
  }
}

// ---- fused path: frames of up to 64 x 128 ------------------------------
constexpr int kFusedThreads = 512;  // 8 waves; wave j owns v-tile j (16 columns)
constexpr int kFusedMaxH = 64, kFusedMaxW = 128;

__host__ __device__ inline int fused_zl_stride(int W) { return (W + 15) / 16 * 16 + 4; }
__host__ __device__ inline int r16(int x) { return (x + 15) / 16 * 16; }

// Byte offsets of the fused kernel's LDS regions.  zl: the frame, [16 HT]
// rows of stride S = 16 n + 4 floats (zero outside H x W), so that the
// 16-byte reads of 16 consecutive rows fall in distinct banks; dl: the
// transform D in band order (at set-up, the inverse of the band order);
// dl2: the second frame of a pair;
// xl: frame 0's coefficients in band order; ahl: A_H as the second
// product's A fragments; sl: the band starts.
struct FusedLds {
  int zl, dl, dl2, xl, ahl, sl, total;
};
__host__ __device__ inline FusedLds fused_lds(int H, int W, int bands) {
  const int HT = (H + 15) / 16;
  FusedLds L;
  int off = 0;
  L.zl = off;  off += r16(16 * HT * fused_zl_stride(W) * 4);
  L.dl = off;  off += r16(H * W * 4 + 4);  // + a spare slot that takes left-out coefficients
  L.dl2 = off; off += r16(H * W * 4 + 4);  // the second frame of a pair
  L.xl = off;  off += r16(H * W * 4);
  L.ahl = off; off += r16(HT * HT * 256 * 4);
  L.sl = off;  off += r16((bands + 1) * 4);
  L.total = off;
  return L;
}

bool fused_fits(int64_t H, int64_t W, int64_t bands) {
  return H <= kFusedMaxH && W <= kFusedMaxW && fused_lds(int(H), int(W), int(bands)).total <= kSpecLdsBytes;
}

// fp64 lane -> lane moves within rows of 16 (DPP), on the two halves.
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  const long long b = __double_as_longlong(v);
  const int lo = __builtin_amdgcn_update_dpp(0, int(b), CTRL, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(0, int(b >> 32), CTRL, 0xf, 0xf, false);
  return __longlong_as_double((static_cast<long long>(hi) << 32) | static_cast<unsigned int>(lo));
}
__device__ __forceinline__ double lane_f64(double v, int l) {
  const long long b = __double_as_longlong(v);
  const int lo = __builtin_amdgcn_readlane(int(b), l), hi = __builtin_amdgcn_readlane(int(b >> 32), l);
  return __longlong_as_double((static_cast<long long>(hi) << 32) | static_cast<unsigned int>(lo));
}
// Sum over the 64 lanes in a fixed order (every lane gets the same bits):
// pairs, quads, eights and sixteens within each row, then the four rows.
__device__ __forceinline__ double wave_total(double v) {
  v += dpp_f64<0xB1>(v);   // quad_perm [1, 0, 3, 2]
  v += dpp_f64<0x4E>(v);   // quad_perm [2, 3, 0, 1]
  v += dpp_f64<0x141>(v);  // row_half_mirror
  v += dpp_f64<0x140>(v);  // row_mirror
  return (lane_f64(v, 0) + lane_f64(v, 16)) + (lane_f64(v, 32) + lane_f64(v, 48));
}

// v_mfma_f32_16x16x4_f32 lane layout (64 lanes, l = lane): A operand
// A[l % 16][l / 16], B operand B[l / 16][l % 16], result element r of lane l
// is C[4 (l / 16) + r][l % 16].  The contraction index k of one step can be
// any 4 values of the summed index, as long as A and B agree:
// * T = z A_W^T, step (q, e): k = w = 16 q + 4 (l / 16) + e, so lane l reads
//   z[h][16 q + 4 (l / 16) .. + 3] with one 16-byte LDS read for 4 steps, and
//   holds B = A_W[v][w] for its own v-tile in registers for the whole run;
// * D = A_H T, step (i, r): k = h = 16 i + 4 (l / 16) + r, which is where
//   element r of lane l of T's tile i already sits: T feeds the second
//   product from its accumulators with no data movement.
// Each lane writes its D values straight to their band-order positions, so
// a band is a contiguous run of dl and xl.  Band b is always reduced by wave
// b % 8, which also keeps frame 0's run for it: that needs no barrier.
template <int HT, int NQ>
__global__ __launch_bounds__(kFusedThreads) void spectral_fused_kernel(const float* latents, int64_t frames, int nlag,
                                                                       int64_t clips, int H, int W, const float* AH,
                                                                       const float* AW, const int32_t* perm,
                                                                       const int32_t* start, int bands,
                                                                       double* per_clip) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const FusedLds L = fused_lds(H, W, bands);
  float* zl = reinterpret_cast<float*>(smem + L.zl);
  float* dl = reinterpret_cast<float*>(smem + L.dl);
  int32_t* inv = reinterpret_cast<int32_t*>(smem + L.dl);  // set-up only
  float* xl = reinterpret_cast<float*>(smem + L.xl);
  float* ahl = reinterpret_cast<float*>(smem + L.ahl);
  int32_t* sl = reinterpret_cast<int32_t*>(smem + L.sl);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int S = fused_zl_stride(W);  // NQ = (W + 15) / 16 quads of 16 columns = v-tiles
  const int HW = H * W;
  const int nperm = start[bands];
  const bool mma = wave < NQ;
  const int vcol = 16 * wave + (lane & 15);

  for (int i = tid; i < 16 * HT * S; i += kFusedThreads) zl[i] = 0.0f;
  for (int i = tid; i < HT * HT * 256; i += kFusedThreads) {  // [a][i][lane][r]
    const int r = i & 3, l = (i >> 2) & 63, ai = i >> 8;
    const int a = ai / HT, it = ai % HT;
    const int u = 16 * a + (l & 15), h = 16 * it + 4 * (l >> 4) + r;
    ahl[i] = (u < H && h < H) ? AH[u * H + h] : 0.0f;
  }
  for (int i = tid; i <= bands; i += kFusedThreads) sl[i] = start[i];
  for (int i = tid; i < HW; i += kFusedThreads) inv[i] = -1;
  f32x4 bw[NQ];  // bw[q][e] = A_W[v][16 q + 4 (l / 16) + e]
#pragma unroll
  for (int q = 0; q < NQ; ++q)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int w = 16 * q + 4 * (lane >> 4) + e;
      bw[q][e] = (mma && vcol < W && w < W) ? AW[vcol * W + w] : 0.0f;
    }
  __syncthreads();
  for (int j = tid; j < nperm; j += kFusedThreads) inv[perm[j]] = j;
  __syncthreads();
  int pos[4 * HT];  // band-order position of result element (a, r) of this lane; HW (spare) if left out
#pragma unroll
  for (int a = 0; a < HT; ++a)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int u = 16 * a + 4 * (lane >> 4) + r;
      const int p = (mma && u < H && vcol < W) ? inv[u * W + vcol] : -1;
      pos[4 * a + r] = p >= 0 ? p : HW;
    }
  // This block's frames: an equal contiguous share of the (clip, lag) order,
  // preceded by frame 0 of its first clip when the share starts past it.
  const int64_t total = clips * int64_t(nlag);
  const int64_t f0 = total * blockIdx.x / gridDim.x, f1 = total * (blockIdx.x + 1) / gridDim.x;
  const int64_t c_first = f0 / nlag;
  const int t_first = int(f0 - c_first * nlag);
  const int64_t njobs = (f1 - f0) + (t_first != 0 ? 1 : 0);
  // Frame loads: W % 4 == 0 as float4 chunks of the contiguous frame (chunk
  // tid + 512 k), else one float per (row, column) with column tid % 128.
  const bool vec = (W & 3) == 0;
  constexpr int kChunks = HT;  // float4 chunks per thread: H W <= 16 HT x 128 = 2048 HT floats
  static_assert(kChunks * kFusedThreads * 4 >= 16 * HT * kFusedMaxW, "chunk count");
  int zoff[kChunks];  // LDS offset of each chunk, or -1
#pragma unroll
  for (int k = 0; k < kChunks; ++k) {
    const int e = 4 * (tid + kFusedThreads * k);
    zoff[k] = (vec && e < HW) ? (e / W) * S + e % W : -1;
  }
  const int cz = tid & 127, rz = tid >> 7;
  f32x4 zr[HT];  // vec: chunk k in zr[k]; else row rz + 4 k in zr[k / 4][k % 4]
  auto load_z = [&](int64_t c, int t) {
    const float* z = latents + (size_t(c) * size_t(frames) + size_t(t)) * size_t(HW);
    if (vec) {
#pragma unroll
      for (int k = 0; k < kChunks; ++k)
        if (zoff[k] >= 0) zr[k] = *reinterpret_cast<const f32x4*>(z + 4 * (tid + kFusedThreads * k));
    } else {
#pragma unroll
      for (int k = 0; k < 4 * HT; ++k) {
        const int h = rz + 4 * k;
        zr[k / 4][k % 4] = (cz < W && h < H) ? z[h * W + cz] : 0.0f;
      }
    }
  };
  auto store_z = [&]() {
    if (vec) {
#pragma unroll
      for (int k = 0; k < kChunks; ++k)
        if (zoff[k] >= 0) *reinterpret_cast<f32x4*>(zl + zoff[k]) = zr[k];
    } else {
#pragma unroll
      for (int k = 0; k < 4 * HT; ++k) {
        const int h = rz + 4 * k;
        if (cz < W && h < H) zl[h * S + cz] = zr[k / 4][k % 4];
      }
    }
  };
  struct Job {
    int64_t c;
    int t;
    bool emit;
  };
  auto next_job = [&](const Job& j) -> Job {
    if (!j.emit) return Job{j.c, t_first, true};
    return j.t + 1 == nlag ? Job{j.c + 1, 0, true} : Job{j.c, j.t + 1, true};
  };
  float* dl2 = reinterpret_cast<float*>(smem + L.dl2);
  auto zfrag = [&](f32x4* a, int q) {
#pragma unroll
    for (int i = 0; i < HT; ++i)
      a[i] = *reinterpret_cast<const f32x4*>(zl + (16 * i + (lane & 15)) * S + 16 * q + 4 * (lane >> 4));
  };  auto products = [&](f32x4 (&dacc)[HT]) {
    if (mma) {
      f32x4 tacc[HT], acur[HT];
#pragma unroll
      for (int i = 0; i < HT; ++i) tacc[i] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        zfrag(acur, q);
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
          for (int i = 0; i < HT; ++i)
            tacc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(acur[i][e], bw[q][e], tacc[i], 0, 0, 0);
      }
#pragma unroll
      for (int a = 0; a < HT; ++a) dacc[a] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int i = 0; i < HT; ++i) {
        f32x4 ah[HT];
#pragma unroll
        for (int a = 0; a < HT; ++a) ah[a] = *reinterpret_cast<const f32x4*>(ahl + ((a * HT + i) * 64 + lane) * 4);
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int a = 0; a < HT; ++a)
            dacc[a] = __builtin_amdgcn_mfma_f32_16x16x4f32(ah[a][r], tacc[i][r], dacc[a], 0, 0, 0);
      }
    }
  };
  auto scatter = [&](float* dst, const f32x4 (&dacc)[HT]) {
    if (mma) {
#pragma unroll
      for (int a = 0; a < HT; ++a)
#pragma unroll
        for (int r = 0; r < 4; ++r) dst[pos[4 * a + r]] = dacc[a][r];
    }
  };
  auto reduce1 = [&](const Job& jb, const float* dsrc) {
    const int64_t c = jb.c;
    const int t = jb.t;
    const bool emit = jb.emit;
    double* out = per_clip + (size_t(c) * size_t(nlag) + size_t(t)) * size_t(bands) * 3;
    for (int b = wave; b < bands; b += kFusedThreads / 64) {
      const int s0 = sl[b], s1 = sl[b + 1];
      double sy = 0, syy = 0, sxy = 0;
      if (t == 0) {  // frame 0 of a clip: its run becomes x
        for (int j = s0 + lane; j < s1; j += 64) {
          const float yf = dsrc[j];
          xl[j] = yf;
          const double y = yf;
          sy += y;
          syy = fma(y, y, syy);
        }
        sy = wave_total(sy);
        syy = wave_total(syy);
        sxy = syy;
      } else {
        int j = s0 + lane;
        for (; j + 192 < s1; j += 256) {  // four elements per lane in flight
          float xf[4], yf[4];
#pragma unroll
          for (int m = 0; m < 4; ++m) {
            xf[m] = xl[j + 64 * m];
            yf[m] = dsrc[j + 64 * m];
          }
#pragma unroll
          for (int m = 0; m < 4; ++m) {
            const double x = xf[m], y = yf[m];
            sy += y;
            syy = fma(y, y, syy);
            sxy = fma(x, y, sxy);
          }
        }
        for (; j < s1; j += 64) {
          const double x = xl[j], y = dsrc[j];
          sy += y;
          syy = fma(y, y, syy);
          sxy = fma(x, y, sxy);
        }
        sy = wave_total(sy);
        syy = wave_total(syy);
        sxy = wave_total(sxy);
      }
      if (emit && lane == 0) {
        out[3 * b] = sy;
        out[3 * b + 1] = syy;
        out[3 * b + 2] = sxy;
      }
    }
  };
  // Two frames of one clip, neither frame 0: one pass over x and both
  // transforms, six sums per band.
  auto reduce2 = [&](const Job& ja, const Job& jb) {
    double* outa = per_clip + (size_t(ja.c) * size_t(nlag) + size_t(ja.t)) * size_t(bands) * 3;
    double* outb = per_clip + (size_t(jb.c) * size_t(nlag) + size_t(jb.t)) * size_t(bands) * 3;
    for (int b = wave; b < bands; b += kFusedThreads / 64) {
      const int s0 = sl[b], s1 = sl[b + 1];
      double sa = 0, saa = 0, sxa = 0, sb = 0, sbb = 0, sxb = 0;
      int j = s0 + lane;
      for (; j + 192 < s1; j += 256) {
        float xf[4], af[4], bf[4];
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          xf[m] = xl[j + 64 * m];
          af[m] = dl[j + 64 * m];
          bf[m] = dl2[j + 64 * m];
        }
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          const double x = xf[m], ya = af[m], yb = bf[m];
          sa += ya;
          saa = fma(ya, ya, saa);
          sxa = fma(x, ya, sxa);
          sb += yb;
          sbb = fma(yb, yb, sbb);
          sxb = fma(x, yb, sxb);
        }
      }
      for (; j < s1; j += 64) {
        const double x = xl[j], ya = dl[j], yb = dl2[j];
        sa += ya;
        saa = fma(ya, ya, saa);
        sxa = fma(x, ya, sxa);
        sb += yb;
        sbb = fma(yb, yb, sbb);
        sxb = fma(x, yb, sxb);
      }
      sa = wave_total(sa);
      saa = wave_total(saa);
      sxa = wave_total(sxa);
      sb = wave_total(sb);
      sbb = wave_total(sbb);
      sxb = wave_total(sxb);
      if (lane == 0) {
        outa[3 * b] = sa;
        outa[3 * b + 1] = saa;
        outa[3 * b + 2] = sxa;
        outb[3 * b] = sb;
        outb[3 * b + 1] = sbb;
        outb[3 * b + 2] = sxb;
      }
    }
  };

  Job ja{c_first, 0, t_first == 0};
  load_z(ja.c, ja.t);
  __syncthreads();  // every lane has read its positions from inv
  store_z();
  __syncthreads();
  for (int64_t k = 0; k < njobs; k += 2) {
    const bool has_b = k + 1 < njobs, has_n = k + 2 < njobs;
    const Job jb = next_job(ja);
    const Job jn = next_job(jb);
    if (has_b) load_z(jb.c, jb.t);
    f32x4 da[HT], db[HT];
    products(da);     // zl holds frame a
    __syncthreads();  // every read of zl, and the previous pair's band sums, are done
    if (has_b) store_z();
    __syncthreads();
    if (has_n) load_z(jn.c, jn.t);
    if (has_b) products(db);  // zl holds frame b
    __syncthreads();
    scatter(dl, da);
    if (has_b) scatter(dl2, db);
    if (has_n) store_z();
    __syncthreads();
    if (has_b && ja.t != 0 && jb.t != 0 && ja.c == jb.c) {
      reduce2(ja, jb);
    } else {
      reduce1(ja, dl);
      if (has_b) reduce1(jb, dl2);
    }
    ja = jn;
  }
}

typedef void (*FusedKernel)(const float*, int64_t, int, int64_t, int, int, const float*, const float*,
                            const int32_t*, const int32_t*, int, double*);
template <int HT>
constexpr FusedKernel kFusedRow[8] = {spectral_fused_kernel<HT, 1>, spectral_fused_kernel<HT, 2>,
                                      spectral_fused_kernel<HT, 3>, spectral_fused_kernel<HT, 4>,
                                      spectral_fused_kernel<HT, 5>, spectral_fused_kernel<HT, 6>,
                                      spectral_fused_kernel<HT, 7>, spectral_fused_kernel<HT, 8>};
FusedKernel fused_kernel(int H, int W) {  // H <= 64, W <= 128
  const int HT = (H + 15) / 16, q = (W + 15) / 16 - 1;
  return HT == 1 ? kFusedRow<1>[q] : HT == 2 ? kFusedRow<2>[q] : HT == 3 ? kFusedRow<3>[q] : kFusedRow<4>[q];
}

// Per clip, band b and lag, the Pearson coefficient from the band sums
// S_y, S_yy, S_xy of frame lag (x = frame 0, whose own sums at lag 0 are
// S_x, S_xx):
//   r = (n S_xy - S_x S_y) / sqrt((n S_xx - S_x^2)(n S_yy - S_y^2)),
// NaN for a band without spread; then the mean over clips into
// corr[band][lag].  Block = 16 consecutive (lag, band) outputs x 16 clip
// groups: group g takes clips g, g + 16, ... in order, then the 16 partial
// sums are added in group order (a fixed order, so every call gives the
// same bits).
constexpr int kMeanOuts = 16, kMeanGroups = 16;
__global__ __launch_bounds__(kMeanOuts * kMeanGroups) void clip_mean_kernel(const double* per_clip,
                                                                           const int32_t* start, int64_t clips,
                                                                           int nlag, int bands, double* corr) {
  __shared__ double part[kMeanGroups][kMeanOuts];
  const int o = threadIdx.x % kMeanOuts, g = threadIdx.x / kMeanOuts;
  const int64_t n_out = int64_t(bands) * nlag;
  const int64_t i = int64_t(blockIdx.x) * kMeanOuts + o;  // i = lag * bands + band
  double s = 0.0;
  if (i < n_out) {
    const int b = int(i % bands);
    const double n = double(start[b + 1] - start[b]);
    for (int64_t c = g; c < clips; c += kMeanGroups) {
      const double* f = per_clip + (size_t(c) * size_t(n_out) + size_t(i)) * 3;
      const double* f0 = per_clip + (size_t(c) * size_t(n_out) + size_t(b)) * 3;  // lag 0
      const double sx = f0[0], sxx = f0[1], sy = f[0], syy = f[1], sxy = f[2];
      const double cov = n * sxy - sx * sy;
      const double vx = n * sxx - sx * sx, vy = n * syy - sy * sy;
      s += cov / sqrt(vx * vy);
    }
  }
  part[g][o] = s;
  __syncthreads();
  if (g == 0 && i < n_out) {
    double t = 0.0;
    for (int k = 0; k < kMeanGroups; ++k) t += part[k][o];
    const int lag = int(i / bands), b = int(i % bands);
    corr[size_t(b) * nlag + lag] = t / double(clips);
  }
}

bool spec_args_ok(int64_t clips, int64_t frames, int32_t height, int32_t width, int32_t bands, int64_t max_lag) {
  if (clips < 1 || clips > int64_t(0x7fffffff) || frames < 1) return false;
  if (max_lag < 0 || max_lag >= frames || max_lag + 1 > kSpecMaxLags) return false;
  if (height < 1 || width < 1 || height > 1024 || width > 1024) return false;
  if (int64_t(height) * width > 40960) return false;
  if (bands < 1 || bands > kSpecMaxBands) return false;
  if (!fused_fits(height, width, bands) && dct_lds_bytes(height, width) > size_t(kSpecLdsBytes)) return false;
  return true;
}

bool is_aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

}  // namespace

// Workspace of the allocation-free entry point: one copy per GPU, in the
// library's code object, held until the process ends.  Host code never
// passes this name to a kernel (on the host it is only a stand-in for the
// symbol): it uses the device address hipGetSymbolAddress returns for the
// current device.
constexpr size_t kStaticScratchBytes = size_t(64) << 20;
static __device__ __align__(256) char scratch[kStaticScratchBytes];

namespace {

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxScratchDevices];  // device address of `scratch` per device, once looked up

// The current device's copy of `scratch` (looked up on the first call on
// that device, with it current).
int static_scratch(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return FADEMEM_EHIP;
  if (dev < 0 || dev >= kMaxScratchDevices) return FADEMEM_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return FADEMEM_EHIP;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return FADEMEM_OK;
}

}  // namespace

extern "C" {

int fademem_spectral_workspace_bytes(int64_t clips, int64_t frames, int32_t height, int32_t width, int32_t bands,
                                     int64_t max_lag, size_t* bytes) {
  if (!bytes || !spec_args_ok(clips, frames, height, width, bands, max_lag)) return FADEMEM_EINVAL;
  SpecLayout L;
  if (!spec_layout(clips, max_lag + 1, height, width, bands, fused_fits(height, width, bands), &L))
    return FADEMEM_EINVAL;
  *bytes = L.total;
  return FADEMEM_OK;
}

int fademem_spectral_corr(const float* latents, int64_t clips, int64_t frames, int32_t height, int32_t width,
                          const int32_t* band_of, int32_t bands, int64_t max_lag, void* workspace,
                          size_t workspace_bytes, double* corr, void* stream) {
  if (!latents || !band_of || !workspace || !corr) return FADEMEM_EINVAL;
  if (!is_aligned(latents, 4) || !is_aligned(band_of, 4) || !is_aligned(workspace, 256) || !is_aligned(corr, 8))
    return FADEMEM_EINVAL;
  if (!spec_args_ok(clips, frames, height, width, bands, max_lag)) return FADEMEM_EINVAL;
  const int nlag = int(max_lag + 1);
  const bool fused = fused_fits(height, width, bands);
  SpecLayout L;
  if (!spec_layout(clips, nlag, height, width, bands, fused, &L)) return FADEMEM_EINVAL;
  if (workspace_bytes < L.total) return FADEMEM_ENOMEM;
  char* ws = static_cast<char*>(workspace);
  float* ah = reinterpret_cast<float*>(ws + L.off_ah);
  float* aw = reinterpret_cast<float*>(ws + L.off_aw);
  float* d = reinterpret_cast<float*>(ws + L.off_d);
  int32_t* perm = reinterpret_cast<int32_t*>(ws + L.off_perm);
  int32_t* start = reinterpret_cast<int32_t*>(ws + L.off_start);
  double* per_clip = reinterpret_cast<double*>(ws + L.off_clip);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const int HW = height * width;
  (void)hipGetLastError();
  hipLaunchKernelGGL(dct_basis_kernel, dim3((height * height + 255) / 256), dim3(256), 0, s, ah, int(height));
  hipLaunchKernelGGL(dct_basis_kernel, dim3((width * width + 255) / 256), dim3(256), 0, s, aw, int(width));
  hipLaunchKernelGGL(band_order_kernel, dim3(1), dim3(kOrderThreads), 0, s, band_of, HW, int(bands), perm, start);
  if (fused) {
    const int lds = fused_lds(height, width, bands).total;
    const FusedKernel fn = fused_kernel(height, width);
    if (lds > 64 * 1024 &&
        hipFuncSetAttribute(reinterpret_cast<const void*>(fn), hipFuncAttributeMaxDynamicSharedMemorySize, lds) !=
            hipSuccess)
      return FADEMEM_EHIP;
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
      return FADEMEM_EHIP;
    const int64_t total = clips * int64_t(nlag);
    const unsigned grid = unsigned(total < cus ? total : cus);  // one block per CU, every block has a frame
    hipLaunchKernelGGL(fn, dim3(grid), dim3(kFusedThreads), size_t(lds), s, latents, frames, nlag, clips,
                       int(height), int(width), ah, aw, perm, start, int(bands), per_clip);
  } else {
    const size_t lds = dct_lds_bytes(height, width);
    if (lds > 64 * 1024) {
      hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(dct2_kernel),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
      if (e != hipSuccess) return FADEMEM_EHIP;
    }
    const unsigned runs = unsigned((nlag + kDctFramesPerBlock - 1) / kDctFramesPerBlock);
    hipLaunchKernelGGL(dct2_kernel, dim3(unsigned(clips), runs), dim3(kDctThreads), lds, s, latents, frames, nlag,
                       int(height), int(width), ah, aw, d);
    hipLaunchKernelGGL(band_corr_kernel, dim3(unsigned(clips), unsigned(nlag)), dim3(256), 0, s, d, nlag, HW, perm,
                       start, int(bands), per_clip);
  }
  const int64_t outs = int64_t(bands) * nlag;
  hipLaunchKernelGGL(clip_mean_kernel, dim3(unsigned((outs + kMeanOuts - 1) / kMeanOuts)),
                     dim3(kMeanOuts * kMeanGroups), 0, s, per_clip, start, clips, nlag, int(bands), corr);
  return hipGetLastError() == hipSuccess ? FADEMEM_OK : FADEMEM_EHIP;
}


// The same analysis with its workspace in the library's static scratch of
// the current device: no allocation, no workspace argument.  Requests whose
// workspace would exceed kStaticScratchBytes are refused before anything is
// enqueued.  Every call on a GPU shares that GPU's scratch: calls that
// overlap on one GPU (other streams, other threads) race.  The kernels write
// every scratch byte they read, so nothing needs clearing between calls.
int fademem_spectral_corr_static(const float* latents, int64_t clips, int64_t frames, int32_t height, int32_t width,
                                 const int32_t* band_of, int32_t bands, int64_t max_lag, double* corr,
                                 void* stream) {
  if (!latents || !band_of || !corr) return FADEMEM_EINVAL;
  if (!spec_args_ok(clips, frames, height, width, bands, max_lag)) return FADEMEM_EINVAL;
  SpecLayout L;
  if (!spec_layout(clips, max_lag + 1, height, width, bands, fused_fits(height, width, bands), &L))
    return FADEMEM_EINVAL;
  if (L.total > kStaticScratchBytes) return FADEMEM_ESCRATCH;
  void* ws = nullptr;
  const int rc = static_scratch(&ws);
  if (rc != FADEMEM_OK) return rc;
  return fademem_spectral_corr(latents, clips, frames, height, width, band_of, bands, max_lag, ws,
                               kStaticScratchBytes, corr, stream);
}

// ---------------------------------------------------------------------------
// Host steps of the analysis (Sec. 3.2, supplementary Sec. S2) on the
// correlation curves: a few dozen numbers, no device work.
// ---------------------------------------------------------------------------

// Radial bands: bands equal-width bins of r(u, v) = sqrt((u/H)^2 + (v/W)^2)
// over [0, max r], the last bin closed, the DC coefficient left out (-1);
// a band's radius is its bin centre.
int fademem_spectral_band_map(int32_t height, int32_t width, int32_t bands, int32_t* band_of, double* centres) {
  if (!band_of || height < 1 || width < 1 || height > 1024 || width > 1024 || bands < 1 || bands > kSpecMaxBands)
    return FADEMEM_EINVAL;
  auto radius = [&](int u, int v) {
    const double a = double(u) / double(height), b = double(v) / double(width);
    return sqrt(a * a + b * b);
  };
  const double r_max = radius(height - 1, width - 1);
  for (int u = 0; u < height; ++u)
    for (int v = 0; v < width; ++v) {
      int32_t k = -1;
      if (u != 0 || v != 0) {
        const double x = floor(radius(u, v) / r_max * double(bands));
        k = x >= double(bands - 1) ? bands - 1 : int32_t(x);
      }
      band_of[size_t(u) * size_t(width) + size_t(v)] = k;
    }
  if (centres)
    for (int k = 0; k < bands; ++k) centres[k] = (double(k) + 0.5) * r_max / double(bands);
  return FADEMEM_OK;
}

// Decorrelation horizon of each band's curve corr[k][0..lags-1]: smooth it
// with a centred moving average over `window` lags (shrinking at the ends);
// the horizon is the first lag >= 1, once the smoothed curve has made at
// least half of its total decay (s[0] - min s), where its next one-lag fall
// is below `drop` times its steepest one-lag fall; -1 if there is none (or
// the curve never falls).
int fademem_spectral_horizons(const double* corr, int32_t bands, int64_t lags, int32_t window, double drop,
                              int64_t* horizon) {
  if (!corr || !horizon || bands < 1 || lags < 1 || lags > (int64_t(1) << 24) || window < 1 || !(drop >= 0.0))
    return FADEMEM_EINVAL;
  std::vector<double> sm;
  try {
    sm.resize(size_t(lags));
  } catch (...) {
    return FADEMEM_ENOMEM;
  }
  const int64_t h = window / 2;
  for (int k = 0; k < bands; ++k) {
    const double* c = corr + size_t(k) * size_t(lags);
    for (int64_t i = 0; i < lags; ++i) {
      const int64_t lo = i - h < 0 ? 0 : i - h, hi = i + h + 1 < lags ? i + h + 1 : lags;
      double sum = 0.0;
      for (int64_t j = lo; j < hi; ++j) sum += c[j];
      sm[size_t(i)] = sum / double(hi - lo);
    }
    double lowest = sm[0], steepest = -INFINITY;
    for (int64_t i = 0; i < lags; ++i) lowest = fmin(lowest, sm[size_t(i)]);
    for (int64_t i = 0; i + 1 < lags; ++i) steepest = fmax(steepest, sm[size_t(i)] - sm[size_t(i) + 1]);
    const double total = sm[0] - lowest;
    horizon[k] = -1;
    if (!(total > 0.0 && steepest > 0.0)) continue;
    for (int64_t lag = 1; lag + 1 < lags; ++lag) {
      if (sm[0] - sm[size_t(lag)] >= 0.5 * total && sm[size_t(lag)] - sm[size_t(lag) + 1] < drop * steepest) {
        horizon[k] = lag;
        break;
      }
    }
  }
  return FADEMEM_OK;
}

// r = a t^(-b) fitted to n points by least squares on r: Gauss-Newton on
// the residuals r_i - a t_i^(-b), started from the straight line through
// (log t, log r); stops when a step changes a and b by less than 1e-14
// relative, or after `iters` steps.
int fademem_spectral_fit(const double* t, const double* r, int64_t n, int32_t iters, double* a_out, double* b_out) {
  if (!t || !r || !a_out || !b_out || n < 2 || iters < 0) return FADEMEM_EINVAL;
  for (int64_t i = 0; i < n; ++i)
    if (!(t[i] > 0.0) || !(r[i] > 0.0) || isinf(t[i]) || isinf(r[i])) return FADEMEM_EINVAL;
  double mx = 0.0, my = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    mx += log(t[i]);
    my += log(r[i]);
  }
  mx /= double(n);
  my /= double(n);
  double sxx = 0.0, sxy = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    const double dx = log(t[i]) - mx, dy = log(r[i]) - my;
    sxx += dx * dx;
    sxy += dx * dy;
  }
  if (!(sxx > 0.0)) return FADEMEM_EINVAL;  // every t equal: the exponent is not determined
  const double slope = sxy / sxx;
  double a = exp(my - slope * mx), b = -slope;
  for (int it = 0; it < iters; ++it) {
    // Normal equations of the linearised problem: J = [df/da, df/db].
    double jaa = 0.0, jab = 0.0, jbb = 0.0, ga = 0.0, gb = 0.0;
    for (int64_t i = 0; i < n; ++i) {
      const double lt = log(t[i]);
      const double f = a * exp(-b * lt);
      const double da = f / a, db = -lt * f, res = r[i] - f;
      jaa += da * da;
      jab += da * db;
      jbb += db * db;
      ga += da * res;
      gb += db * res;
    }
    const double det = jaa * jbb - jab * jab;
    if (!(det != 0.0) || isinf(det)) break;
    const double sa = (jbb * ga - jab * gb) / det, sb = (jaa * gb - jab * ga) / det;
    a += sa;
    b += sb;
    if (fabs(sa) <= 1e-14 * fmax(1.0, fabs(a)) && fabs(sb) <= 1e-14 * fmax(1.0, fabs(b))) break;
  }
  if (!isfinite(a) || !isfinite(b)) return FADEMEM_EINVAL;
  *a_out = a;
  *b_out = b;
  return FADEMEM_OK;
}

}  // extern "C"
