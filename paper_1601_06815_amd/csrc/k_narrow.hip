// Per-bin contraction for layers with few input channels (C <= 4, e.g. an
// RGB first layer), where the three per-bin products of arXiv:1601.06815
// (Section 2 forward, Section 3.2 backward) have a dimension too small for a
// tiled GEMM and the work is bound by streaming the wide spectra through HBM:
//
//   forward          Yhat[f][k][bp]  = sum_{c<C} What[f][c][k] * Xhat[f][c][bp]
//   backward_data    dXhat[f][c][bp] = sum_k conj(What[f][c][k]) * Ghat[f][k][bp]
//   backward_filter  dWhat[s][f][c][k] = sum_{bp in chunk s} conj(Xhat[f][c][bp]) * Ghat[f][k][bp]
//
// The first two give each lane VEC neighbouring tiles of one bin and keep the
// C channel values (or C accumulators) in registers, so every wide spectrum is
// read or written exactly once with 16-byte accesses; the bin's kernel
// spectra are staged in LDS and read as broadcasts. The third gives each wave
// 16 kernels and a chunk of tiles; lanes accumulate C x 16 complex partial
// sums over their tiles and combine them with a reduce-scatter across the
// wave (96 lane exchanges for C = 3 instead of 576 for a full butterfly). The
// partial sums of the chunks are added by the inverse-transform kernel, in a
// fixed order.
//
// With few tiles per bin (B P <= 64, e.g. the single images of the paper's
// sweeps) a lane per tile would leave the workgroup nearly idle and walk all K
// kernels in one dependent chain; the forward and backward_data variants for
// that case spread the kernels over the lanes as well (one workgroup per bin),
// and the backward_filter variant (B P <= 16) gives each lane one kernel.
#include <algorithm>

#include "oaa_internal.hpp"
#include "tile_common.hpp"

namespace oaa {

namespace {

using tile::cmad;

constexpr int kThreads = 256;
constexpr int kKB = 256;       // kernel spectra staged per LDS block
constexpr int kIter = 4;       // groups of VEC tiles per lane (forward, backward_data)
constexpr int kKG = 16;        // kernels per wave (backward_filter)
constexpr int kFewTiles = 64;  // B P up to which the few-tile variants run

__device__ __forceinline__ float2 cmad_conj(float2 a, float2 b, float2 c) {
  // c + conj(a) * b
  return make_float2(fmaf(a.x, b.x, fmaf(a.y, b.y, c.x)), fmaf(a.x, b.y, fmaf(-a.y, b.x, c.y)));
}

template <int VEC>
__device__ __forceinline__ void load_vec(const float2* p, float2 (&v)[VEC]) {
  if constexpr (VEC == 2) {
    const float4 t = *reinterpret_cast<const float4*>(p);
    v[0] = make_float2(t.x, t.y);
    v[1] = make_float2(t.z, t.w);
  } else {
    v[0] = *p;
  }
}

template <int VEC>
__device__ __forceinline__ void store_vec(float2* p, const float2 (&v)[VEC]) {
  if constexpr (VEC == 2) {
    *reinterpret_cast<float4*>(p) = make_float4(v[0].x, v[0].y, v[1].x, v[1].y);
  } else {
    *p = v[0];
  }
}

// forward: A = What [C][K] (lda = K), B = Xhat [C][BP], out [K][BP].
// GemmParams: M = K, N = BP, Kr = C.
template <int CN, int VEC>
__global__ void __launch_bounds__(kThreads) narrow_forward_kernel(GemmParams p) {
  __shared__ float2 ws[CN][kKB];
  const int f = unique_bin(blockIdx.y, p.L);
  const int K = p.M;
  const long BP = p.N;
  const float2* A = p.A + size_t(f) * p.a_fstride;
  const float2* B = p.B + size_t(f) * p.b_fstride;
  float2* O = p.C + size_t(f) * p.c_fstride;
  const long base = (long(blockIdx.x) * kIter * kThreads + threadIdx.x) * VEC;

  float2 x[kIter][CN][VEC];
#pragma unroll
  for (int it = 0; it < kIter; ++it) {
    const long bp = base + long(it) * kThreads * VEC;
    const long bc = bp < BP ? bp : 0;
#pragma unroll
    for (int c = 0; c < CN; ++c) load_vec<VEC>(B + c * p.ldb + bc, x[it][c]);
  }
  for (int k0 = 0; k0 < K; k0 += kKB) {
    const int kb = min(kKB, K - k0);
    __syncthreads();
    for (int i = threadIdx.x; i < CN * kb; i += kThreads) ws[i / kb][i % kb] = A[(i / kb) * p.lda + k0 + i % kb];
    __syncthreads();
    for (int kk = 0; kk < kb; ++kk) {
      float2 w[CN];
#pragma unroll
      for (int c = 0; c < CN; ++c) w[c] = ws[c][kk];
      float2* row = O + size_t(k0 + kk) * p.ldc;
#pragma unroll
      for (int it = 0; it < kIter; ++it) {
        const long bp = base + long(it) * kThreads * VEC;
        float2 y[VEC];
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
          y[v] = make_float2(0.f, 0.f);
#pragma unroll
          for (int c = 0; c < CN; ++c) y[v] = cmad(y[v], w[c], x[it][c][v]);  // y + w * x
        }
        if (bp < BP) store_vec<VEC>(row + bp, y);
      }
    }
  }
}

// backward_data: A = What [C][K] (lda = K), B = Ghat [K][BP], out [C][BP].
// GemmParams: M = C, N = BP, Kr = K.
template <int CN, int VEC>
__global__ void __launch_bounds__(kThreads) narrow_bwd_data_kernel(GemmParams p) {
  __shared__ float2 ws[CN][kKB];
  const int f = unique_bin(blockIdx.y, p.L);
  const int K = p.Kr;
  const long BP = p.N;
  const float2* A = p.A + size_t(f) * p.a_fstride;
  const float2* B = p.B + size_t(f) * p.b_fstride;
  float2* O = p.C + size_t(f) * p.c_fstride;
  const long base = (long(blockIdx.x) * kIter * kThreads + threadIdx.x) * VEC;
  long bc[kIter];
#pragma unroll
  for (int it = 0; it < kIter; ++it) {
    const long bp = base + long(it) * kThreads * VEC;
    bc[it] = bp < BP ? bp : 0;
  }

  float2 acc[kIter][CN][VEC];
#pragma unroll
  for (int it = 0; it < kIter; ++it)
#pragma unroll
    for (int c = 0; c < CN; ++c)
#pragma unroll
      for (int v = 0; v < VEC; ++v) acc[it][c][v] = make_float2(0.f, 0.f);

  for (int k0 = 0; k0 < K; k0 += kKB) {
    const int kb = min(kKB, K - k0);
    __syncthreads();
    for (int i = threadIdx.x; i < CN * kb; i += kThreads) ws[i / kb][i % kb] = A[(i / kb) * p.lda + k0 + i % kb];
    __syncthreads();
#pragma unroll 2
    for (int kk = 0; kk < kb; ++kk) {
      const float2* row = B + size_t(k0 + kk) * p.ldb;
      float2 g[kIter][VEC];
#pragma unroll
      for (int it = 0; it < kIter; ++it) load_vec<VEC>(row + bc[it], g[it]);
#pragma unroll
      for (int c = 0; c < CN; ++c) {
        const float2 w = ws[c][kk];
#pragma unroll
        for (int it = 0; it < kIter; ++it)
#pragma unroll
          for (int v = 0; v < VEC; ++v) acc[it][c][v] = cmad_conj(w, g[it][v], acc[it][c][v]);
      }
    }
  }
#pragma unroll
  for (int it = 0; it < kIter; ++it) {
    const long bp = base + long(it) * kThreads * VEC;
    if (bp < BP) {
#pragma unroll
      for (int c = 0; c < CN; ++c) store_vec<VEC>(O + c * p.ldc + bp, acc[it][c]);
    }
  }
}

// Sum NV floats over the 64 lanes of a wave. On return lanes with bit 0
// clear hold NV/32 totals in a[0 .. NV/32): those of indices
// off + [0, NV/32), off = sum over the halving steps of the lane's bit times
// the half size (returned).
template <int NV>
__device__ __forceinline__ int wave_reduce_scatter(float (&a)[NV], int lane) {
  static_assert(NV % 32 == 0, "reduce-scatter needs a multiple of 32 values");
  int off = 0;
#pragma unroll
  for (int s = 0; s < 5; ++s) {
    const int mask = 32 >> s;
    const int half = NV >> (s + 1);
    const bool hi = (lane & mask) != 0;
#pragma unroll
    for (int j = 0; j < half; ++j) {
      const float lo_v = a[j], hi_v = a[j + half];
      const float send = hi ? lo_v : hi_v;
      const float keep = hi ? hi_v : lo_v;
      a[j] = keep + __shfl_xor(send, mask);
    }
    off += hi ? half : 0;
  }
#pragma unroll
  for (int j = 0; j < NV / 32; ++j) a[j] += __shfl_xor(a[j], 1);
  return off;
}

// backward_filter: A = Xhat [C][BP] (lda = BP), B = Ghat [K][BP] (ldb = BP),
// out partial sums [split][C][K] per bin (ldc = K).
// GemmParams: M = C, N = K, Kr = BP, nsplit chunks of kchunk tiles.
template <int CN, int VEC>
__global__ void __launch_bounds__(kThreads) narrow_bwd_filter_kernel(GemmParams p) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int kbase = (blockIdx.x * (kThreads / 64) + wave) * kKG;
  const int K = p.N;
  if (kbase >= K) return;  // no barrier below: idle waves may leave
  const int f = unique_bin(blockIdx.z, p.L), split = blockIdx.y;
  const long BP = p.Kr;
  const float2* A = p.A + size_t(f) * p.a_fstride;
  const float2* B = p.B + size_t(f) * p.b_fstride;
  const long b0 = long(split) * p.kchunk;
  const long b1 = min(BP, b0 + long(p.kchunk));
  const float2* grow[kKG];
#pragma unroll
  for (int i = 0; i < kKG; ++i) grow[i] = B + size_t(min(kbase + i, K - 1)) * p.ldb;

  float acc[CN * kKG * 2];
#pragma unroll
  for (int j = 0; j < CN * kKG * 2; ++j) acc[j] = 0.f;

  for (long bp = b0 + long(lane) * VEC; bp < b1; bp += 64 * VEC) {
    float2 x[CN][VEC], g[kKG][VEC];
#pragma unroll
    for (int c = 0; c < CN; ++c) load_vec<VEC>(A + c * p.lda + bp, x[c]);
#pragma unroll
    for (int i = 0; i < kKG; ++i) load_vec<VEC>(grow[i] + bp, g[i]);
#pragma unroll
    for (int c = 0; c < CN; ++c)
#pragma unroll
      for (int i = 0; i < kKG; ++i) {
        float2 s = make_float2(acc[(c * kKG + i) * 2], acc[(c * kKG + i) * 2 + 1]);
#pragma unroll
        for (int v = 0; v < VEC; ++v) s = cmad_conj(x[c][v], g[i][v], s);
        acc[(c * kKG + i) * 2] = s.x;
        acc[(c * kKG + i) * 2 + 1] = s.y;
      }
  }
  constexpr int NV = CN * kKG * 2;
  const int off = wave_reduce_scatter<NV>(acc, lane);
  if (lane & 1) return;
  float* out = reinterpret_cast<float*>(p.C + size_t(split) * p.c_sstride + size_t(f) * p.c_fstride);
#pragma unroll
  for (int j = 0; j < NV / 32; ++j) {
    const int idx = off + j;          // float index within the wave's C x 16 complex block
    const int ci = idx >> 1;          // complex index c * 16 + i
    const int c = ci / kKG, i = ci % kKG;
    if (kbase + i < K) out[(size_t(c) * p.ldc + kbase + i) * 2 + (idx & 1)] = acc[j];
  }
}

// Few tiles per bin: lane t takes tile j = t mod NB (NB = 2^nb_log2 >= B P)
// and kernels t / NB + i 256 / NB. Forward: each lane writes its own outputs.
template <int CN>
__global__ void __launch_bounds__(kThreads) narrow_forward_few_kernel(GemmParams p, int nb_log2) {
  const int f = unique_bin(blockIdx.x, p.L);
  const int K = p.M, BP = p.N;
  const int j = threadIdx.x & ((1 << nb_log2) - 1), nk = kThreads >> nb_log2;
  if (j >= BP) return;  // no barrier below
  const float2* A = p.A + size_t(f) * p.a_fstride;
  const float2* B = p.B + size_t(f) * p.b_fstride;
  float2* O = p.C + size_t(f) * p.c_fstride;
  float2 x[CN];
#pragma unroll
  for (int c = 0; c < CN; ++c) x[c] = B[c * p.ldb + j];
#pragma unroll 4
  for (int k = threadIdx.x >> nb_log2; k < K; k += nk) {
    float2 y = make_float2(0.f, 0.f);
#pragma unroll
    for (int c = 0; c < CN; ++c) y = cmad(y, A[c * p.lda + k], x[c]);
    O[size_t(k) * p.ldc + j] = y;
  }
}

// Few tiles per bin, backward_data: each lane sums its kernels for its tile,
// then the 256 / NB lanes of a tile are added in LDS in a fixed order.
template <int CN>
__global__ void __launch_bounds__(kThreads) narrow_bwd_data_few_kernel(GemmParams p, int nb_log2) {
  __shared__ float2 red[CN][kThreads];
  const int f = unique_bin(blockIdx.x, p.L);
  const int K = p.Kr, BP = p.N;
  const int t = threadIdx.x, mask = (1 << nb_log2) - 1, j = t & mask, nk = kThreads >> nb_log2;
  const float2* A = p.A + size_t(f) * p.a_fstride;
  const float2* B = p.B + size_t(f) * p.b_fstride;
  float2* O = p.C + size_t(f) * p.c_fstride;
  float2 acc[CN];
#pragma unroll
  for (int c = 0; c < CN; ++c) acc[c] = make_float2(0.f, 0.f);
  if (j < BP) {
#pragma unroll 4
    for (int k = t >> nb_log2; k < K; k += nk) {
      const float2 g = B[size_t(k) * p.ldb + j];
#pragma unroll
      for (int c = 0; c < CN; ++c) acc[c] = cmad_conj(A[c * p.lda + k], g, acc[c]);
    }
  }
#pragma unroll
  for (int c = 0; c < CN; ++c) red[c][t] = acc[c];
  __syncthreads();
  if (t < (CN << nb_log2) && (t & mask) < BP) {
    const int c = t >> nb_log2, jj = t & mask;
    float2 sum = make_float2(0.f, 0.f);
    for (int q = 0; q < nk; ++q) {
      const float2 v = red[c][(q << nb_log2) + jj];
      sum.x += v.x;
      sum.y += v.y;
    }
    O[c * p.ldc + jj] = sum;
  }
}

// Few tiles per bin (B P <= 16), backward_filter: a lane per kernel walks
// the bin's tiles (one partial sum: no split).
constexpr int kFewTilesFilter = 16;

template <int CN>
__global__ void __launch_bounds__(kThreads) narrow_bwd_filter_few_kernel(GemmParams p) {
  const int k = blockIdx.x * kThreads + threadIdx.x;
  const int K = p.N, BP = p.Kr;
  if (k >= K) return;
  const int f = unique_bin(blockIdx.y, p.L);
  const float2* A = p.A + size_t(f) * p.a_fstride;
  const float2* g = p.B + size_t(f) * p.b_fstride + size_t(k) * p.ldb;
  float2 acc[CN];
#pragma unroll
  for (int c = 0; c < CN; ++c) acc[c] = make_float2(0.f, 0.f);
  for (int bp = 0; bp < BP; ++bp) {
    const float2 gv = g[bp];
#pragma unroll
    for (int c = 0; c < CN; ++c) acc[c] = cmad_conj(A[c * p.lda + bp], gv, acc[c]);
  }
  float2* out = p.C + size_t(f) * p.c_fstride;
#pragma unroll
  for (int c = 0; c < CN; ++c) out[size_t(c) * p.ldc + k] = acc[c];
}

int few_tiles_log2(long BP) {
  int l = 0;
  while ((1L << l) < BP) ++l;
  return l;
}

template <int CN, int VEC>
hipError_t launch_fwd(const GemmParams& p, hipStream_t s) {
  const long per_wg = long(kIter) * kThreads * VEC;
  const unsigned nx = unsigned((long(p.N) + per_wg - 1) / per_wg);
  hipLaunchKernelGGL((narrow_forward_kernel<CN, VEC>), dim3(nx, unsigned(p.F)), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

template <int CN, int VEC>
hipError_t launch_bwd_data(const GemmParams& p, hipStream_t s) {
  const long per_wg = long(kIter) * kThreads * VEC;
  const unsigned nx = unsigned((long(p.N) + per_wg - 1) / per_wg);
  hipLaunchKernelGGL((narrow_bwd_data_kernel<CN, VEC>), dim3(nx, unsigned(p.F)), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

template <int CN, int VEC>
hipError_t launch_bwd_filter(const GemmParams& p, hipStream_t s) {
  const int groups = (p.N + kKG - 1) / kKG;
  const unsigned nx = unsigned((groups + kThreads / 64 - 1) / (kThreads / 64));
  hipLaunchKernelGGL((narrow_bwd_filter_kernel<CN, VEC>), dim3(nx, unsigned(p.nsplit), unsigned(p.F)),
                     dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

// Pair-wide (16-byte) accesses need every row start and chunk start even.
bool pairs_ok(long ld, long chunk, int nsplit) { return ld % 2 == 0 && (nsplit == 1 || chunk % 2 == 0); }

template <int CN>
hipError_t launch_narrow_c(const GemmParams& p, hipStream_t s) {
  const bool few = p.N >= 1 && p.N <= kFewTiles && p.nsplit == 1;
  if (few && p.a_trans && !p.a_conj && !p.b_trans && !p.b_conj) {
    hipLaunchKernelGGL(narrow_forward_few_kernel<CN>, dim3(unsigned(p.F)), dim3(kThreads), 0, s, p,
                       few_tiles_log2(p.N));
    return hipGetLastError();
  }
  if (few && !p.a_trans && p.a_conj && !p.b_trans && !p.b_conj) {
    hipLaunchKernelGGL(narrow_bwd_data_few_kernel<CN>, dim3(unsigned(p.F)), dim3(kThreads), 0, s, p,
                       few_tiles_log2(p.N));
    return hipGetLastError();
  }
  if (p.Kr >= 1 && p.Kr <= kFewTilesFilter && p.nsplit == 1 && !p.a_trans && p.a_conj && p.b_trans && !p.b_conj) {
    hipLaunchKernelGGL(narrow_bwd_filter_few_kernel<CN>, dim3(unsigned((p.N + kThreads - 1) / kThreads), unsigned(p.F)),
                       dim3(kThreads), 0, s, p);
    return hipGetLastError();
  }
  if (p.a_trans && !p.a_conj && !p.b_trans && !p.b_conj) {
    const bool v2 = pairs_ok(p.ldb, 0, 1) && p.ldc % 2 == 0;
    return v2 ? launch_fwd<CN, 2>(p, s) : launch_fwd<CN, 1>(p, s);
  }
  if (!p.a_trans && p.a_conj && !p.b_trans && !p.b_conj) {
    const bool v2 = pairs_ok(p.ldb, 0, 1) && p.ldc % 2 == 0;
    return v2 ? launch_bwd_data<CN, 2>(p, s) : launch_bwd_data<CN, 1>(p, s);
  }
  if (!p.a_trans && p.a_conj && p.b_trans && !p.b_conj) {
    const bool v2 = pairs_ok(p.lda, p.kchunk, p.nsplit) && p.ldb % 2 == 0 && p.Kr % 2 == 0;
    return v2 ? launch_bwd_filter<CN, 2>(p, s) : launch_bwd_filter<CN, 1>(p, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

int narrow_channels(const GemmParams& p) {
  if (p.a_trans && !p.a_conj && !p.b_trans && !p.b_conj) return p.Kr;  // forward: reduction over C
  return p.M;                                                            // backward: output rows are C
}

bool narrow_supported(const GemmParams& p) {
  const int c = narrow_channels(p);
  return c >= 1 && c <= kNarrowMaxC;
}

hipError_t launch_cgemm_narrow(const GemmParams& p, hipStream_t s) {
  switch (narrow_channels(p)) {
    case 1: return launch_narrow_c<1>(p, s);
    case 2: return launch_narrow_c<2>(p, s);
    case 3: return launch_narrow_c<3>(p, s);
    case 4: return launch_narrow_c<4>(p, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace oaa
