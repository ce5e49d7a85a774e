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
// * dct2_kernel -- one block per (clip, run of frames): both bases (as
//   transposes) in LDS once, then per frame z^T in LDS, T = z A_W^T and
//   D = A_H T, each thread computing 4 x 4 output tiles from 16-byte LDS
//   reads (8 FMAs per read); fp32 products and sums; sizes padded to
//   multiples of 4 with zeros;
// * band_order_kernel -- the coefficients grouped by band (stable counting
//   sort, one thread), so each band is a contiguous index list;
// * band_corr_kernel -- one block per (clip, lag): each wave takes bands in
//   turn, sums x, y, x^2, y^2, xy over the band in fp64 (lanes, then a wave
//   reduction), and writes the Pearson coefficient
//   (n Sxy - Sx Sy) / sqrt((n Sxx - Sx^2)(n Syy - Sy^2));
// * clip_mean_kernel -- the mean over clips, in clip order (deterministic).
#include <math.h>
#include <string.h>

#include "fademem_internal.h"

namespace {

inline size_t rup(size_t x) { return (x + 255) / 256 * 256; }

constexpr int kSpecLdsBytes = 160 * 1024;  // LDS of one workgroup on gfx950
constexpr int kSpecMaxBands = 1024;
constexpr int kSpecMaxLags = 65535;        // grid.y

struct SpecLayout {
  size_t off_ah, off_aw, off_d, off_perm, off_start, off_clip, total;
};

bool spec_layout(int64_t clips, int64_t nlag, int64_t H, int64_t W, int64_t bands, SpecLayout* L) {
  const double d_bytes = double(clips) * double(nlag) * double(H) * double(W) * 4.0;
  const double c_bytes = double(clips) * double(nlag) * double(bands) * 8.0;
  if (d_bytes > 1e15 || c_bytes > 1e15) return false;
  size_t off = 0;
  L->off_ah = off;    off = rup(off + size_t(H * H) * 4);
  L->off_aw = off;    off = rup(off + size_t(W * W) * 4);
  L->off_d = off;     off = rup(off + size_t(clips) * size_t(nlag) * size_t(H * W) * 4);
  L->off_perm = off;  off = rup(off + size_t(H * W) * 4);
  L->off_start = off; off = rup(off + size_t(bands + 1) * 4);
  L->off_clip = off;  off = rup(off + size_t(clips) * size_t(nlag) * size_t(bands) * 8);
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

// Coefficient indices grouped by band, in index order within a band;
// entries outside [0, bands) are left out.  One block of 1024 threads with
// the band map in LDS: thread t takes band t / C in chunk t % C of the map
// (C = chunks per band), counts it, then after a prefix over (band, chunk)
// writes that chunk's indices of that band in order.
constexpr int kOrderMaxHW = 40960;
constexpr int kOrderThreads = 1024;
__global__ __launch_bounds__(kOrderThreads) void band_order_kernel(const int32_t* band_of, int HW, int bands,
                                                                   int32_t* perm, int32_t* start) {
  __shared__ int16_t map[kOrderMaxHW];
  __shared__ int32_t cnt[kOrderThreads];
  const int tid = threadIdx.x;
  for (int i = tid; i < HW; i += kOrderThreads) {
    const int b = band_of[i];
    map[i] = int16_t((b >= 0 && b < bands) ? b : -1);
  }
  const int C = bands >= kOrderThreads ? 1 : kOrderThreads / bands;  // chunks per band
  const int per_round = kOrderThreads / C;                           // bands per round
  const int len = (HW + C - 1) / C;
  for (int b0 = 0; b0 < bands; b0 += per_round) {
    const int b = b0 + tid / C, j = tid % C;
    const bool on = tid / C < per_round && b < bands;
    const int i0 = j * len, i1 = min(HW, i0 + len);
    __syncthreads();
    int n = 0;
    if (on)
      for (int i = i0; i < i1; ++i) n += (map[i] == b);
    cnt[tid] = n;
    __syncthreads();
    if (tid == 0) {
      int acc = b0 == 0 ? 0 : start[b0];
      for (int t = 0; t < per_round * C; ++t) {
        const int bt = b0 + t / C;
        if (bt >= bands) break;
        if (t % C == 0) start[bt] = acc;
        const int m = cnt[t];
        cnt[t] = acc;
        acc += m;
      }
      start[min(bands, b0 + per_round)] = acc;
    }
    __syncthreads();
    if (on) {
      int pos = cnt[tid];
      for (int i = i0; i < i1; ++i)
        if (map[i] == b) perm[pos++] = i;
    }
  }
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
  double* out = per_clip + (size_t(c) * size_t(nlag) + size_t(lag)) * size_t(bands);
  for (int b = wave; b < bands; b += 4) {
    const int s0 = start[b], s1 = start[b + 1];
    double sx = 0, sy = 0, sxx = 0, syy = 0, sxy = 0;
    for (int j = s0 + lane; j < s1; j += 64) {
      const int i = perm[j];
      const double xv = x[i], yv = y[i];
      sx += xv;
      sy += yv;
      sxx += xv * xv;
      syy += yv * yv;
      sxy += xv * yv;
    }
    sx = wave_sum(sx);
    sy = wave_sum(sy);
    sxx = wave_sum(sxx);
    syy = wave_sum(syy);
    sxy = wave_sum(sxy);
    if (lane == 0) {
      const double n = double(s1 - s0);
      const double cov = n * sxy - sx * sy;
      const double vx = n * sxx - sx * sx, vy = n * syy - sy * sy;
      out[b] = cov / sqrt(vx * vy);  // NaN for a band without spread
    }
  }
}

__global__ void clip_mean_kernel(const double* per_clip, int64_t clips, int nlag, int bands, double* corr) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;  // i = band * nlag + lag
  if (i >= int64_t(bands) * nlag) return;
  const int b = int(i / nlag), lag = int(i % nlag);
  double s = 0.0;
  for (int64_t c = 0; c < clips; ++c) s += per_clip[(size_t(c) * nlag + lag) * bands + b];
  corr[i] = s / double(clips);
}

bool spec_args_ok(int64_t clips, int64_t frames, int32_t height, int32_t width, int32_t bands, int64_t max_lag) {
  if (clips < 1 || clips > int64_t(0x7fffffff) || frames < 1) return false;
  if (max_lag < 0 || max_lag >= frames || max_lag + 1 > kSpecMaxLags) return false;
  if (height < 1 || width < 1 || height > 1024 || width > 1024) return false;
  if (int64_t(height) * width > 40960) return false;
  if (dct_lds_bytes(height, width) > size_t(kSpecLdsBytes)) return false;
  if (bands < 1 || bands > kSpecMaxBands) return false;
  return true;
}

bool is_aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

}  // namespace

extern "C" {

int fademem_spectral_workspace_bytes(int64_t clips, int64_t frames, int32_t height, int32_t width, int32_t bands,
                                     int64_t max_lag, size_t* bytes) {
  if (!bytes || !spec_args_ok(clips, frames, height, width, bands, max_lag)) return FADEMEM_EINVAL;
  SpecLayout L;
  if (!spec_layout(clips, max_lag + 1, height, width, bands, &L)) return FADEMEM_EINVAL;
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
  SpecLayout L;
  if (!spec_layout(clips, nlag, height, width, bands, &L)) return FADEMEM_EINVAL;
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
  const int64_t outs = int64_t(bands) * nlag;
  hipLaunchKernelGGL(clip_mean_kernel, dim3(unsigned((outs + 255) / 256)), dim3(256), 0, s, per_clip, clips, nlag,
                     int(bands), corr);
  return hipGetLastError() == hipSuccess ? FADEMEM_OK : FADEMEM_EHIP;
}

}  // extern "C"
