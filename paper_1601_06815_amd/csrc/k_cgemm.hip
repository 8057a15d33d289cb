// Per-frequency-bin complex contraction (arXiv:1601.06815, Introduction and
// Section 2: the Hadamard product of block and kernel spectra, summed over the
// C channels of the layer; Section 3.2 for the two backward products).
//
// For every bin f (the unique bins only, see unique_bin) the three passes are
// complex matrix products:
//   forward          Yhat[f]  (K x BP) = What[f]^T   (K x C)  * Xhat[f] (C x BP)
//   backward_data    dXhat[f] (C x BP) = conj What[f] (C x K)  * Ghat[f] (K x BP)
//   backward_filter  dWhat[f] (C x K)  = conj Xhat[f] (C x BP) * Ghat[f]^T (BP x K)
//
// Two implementations share the operand staging: each 256-lane workgroup
// loads a 16-deep slice of the reduction for its output tile from global
// memory into registers with branch-free, clamped addresses (all loads in
// flight at once), stores it to LDS as separate real and imaginary planes,
// and prefetches the next slice while the current one is consumed.
//  * vector ALU: 64 x 64 complex tile, 4 x 4 complex accumulators per lane;
//  * fp32 matrix cores (v_mfma_f32_16x16x4f32): 128 x 128 (or 96 x 128)
//    complex tile per workgroup, double-buffered LDS with one barrier per
//    slice, workgroups renumbered so that tiles sharing operands run on the
//    same XCD; each complex multiply-accumulate of a 16 x 16 x 4 block is four
//    real MFMAs, re += ar*br + (-ai)*bi and im += ar*bi + ai*br.
#include <algorithm>

#include "oaa_internal.hpp"

// Minimum waves per SIMD asked of the register allocator for the
// matrix-core kernel.
#ifndef OAA_WAVES_GEMM
#define OAA_WAVES_GEMM 1
#endif

namespace oaa {

namespace {

constexpr int kThreads = 256;
constexpr int kKC = 16;  // reduction depth of one LDS slice

// A ROWS x kKC slice of an operand whose element (row, k) is stored at
// X[k*ld + row] (ROW_CONTIG) or X[row*ld + k]; loads are coalesced along the
// contiguous index. Out-of-range elements read a valid clamped address and
// are replaced by zero.
template <bool ROW_CONTIG, int ROWS>
struct Slice {
  static constexpr int PER = ROWS * kKC / kThreads;
  float2 v[PER];

  __device__ __forceinline__ static void coords(int e, int& rl, int& kl) {
    if (ROW_CONTIG) {
      rl = e % ROWS;
      kl = e / ROWS;
    } else {
      kl = e % kKC;
      rl = e / kKC;
    }
  }

  __device__ __forceinline__ void load(const float2* X, long ld, int r0, int nrows, int k0, int kend) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      int rl, kl;
      coords(int(threadIdx.x) + kThreads * i, rl, kl);
      const int r = r0 + rl, k = k0 + kl;
      const bool ok = r < nrows && k < kend;
      const int rc = ok ? r : r0, kc = ok ? k : k0;
      const float2 t = ROW_CONTIG ? X[size_t(kc) * ld + rc] : X[size_t(rc) * ld + kc];
      v[i] = ok ? t : make_float2(0.f, 0.f);
    }
  }

  template <int LD>
  __device__ __forceinline__ void store(float (*re)[LD], float (*im)[LD], bool conj) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      int rl, kl;
      coords(int(threadIdx.x) + kThreads * i, rl, kl);
      re[kl][rl] = v[i].x;
      im[kl][rl] = conj ? -v[i].y : v[i].y;
    }
  }
};

struct TileCoords {
  int f, split, m0, n0, k_begin, k_end;
};

template <int TM, int TN>
__device__ __forceinline__ TileCoords tile_coords(const GemmParams& p) {
  TileCoords t;
  t.f = unique_bin(blockIdx.z, p.L);
  t.split = blockIdx.y;
  const int tiles_n = (p.N + TN - 1) / TN;
  t.m0 = (blockIdx.x / tiles_n) * TM;
  t.n0 = (blockIdx.x % tiles_n) * TN;
  t.k_begin = t.split * p.kchunk;
  t.k_end = min(p.Kr, t.k_begin + p.kchunk);
  return t;
}

// ---------------------------------------------------------------------------
// vector-ALU implementation

constexpr int kVM = 64, kVN = 64;

template <bool AT, bool AC, bool BT, bool BC>
__global__ void __launch_bounds__(kThreads) cgemm_valu_kernel(GemmParams p) {
  __shared__ float Asr[kKC][kVM + 4], Asi[kKC][kVM + 4];
  __shared__ float Bsr[kKC][kVN + 4], Bsi[kKC][kVN + 4];
  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;
  const TileCoords tc = tile_coords<kVM, kVN>(p);
  const float2* A = p.A + size_t(tc.f) * p.a_fstride;
  const float2* B = p.B + size_t(tc.f) * p.b_fstride;

  float accr[4][4], acci[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) accr[i][j] = acci[i][j] = 0.f;

  Slice<AT, kVM> sa;
  Slice<!BT, kVN> sb;
  sa.load(A, p.lda, tc.m0, p.M, tc.k_begin, tc.k_end);
  sb.load(B, p.ldb, tc.n0, p.N, tc.k_begin, tc.k_end);
  for (int k0 = tc.k_begin; k0 < tc.k_end; k0 += kKC) {
    sa.template store<kVM + 4>(Asr, Asi, AC);
    sb.template store<kVN + 4>(Bsr, Bsi, BC);
    __syncthreads();
    if (k0 + kKC < tc.k_end) {
      sa.load(A, p.lda, tc.m0, p.M, k0 + kKC, tc.k_end);
      sb.load(B, p.ldb, tc.n0, p.N, k0 + kKC, tc.k_end);
    }
#pragma unroll
    for (int kk = 0; kk < kKC; ++kk) {
      float ar[4], ai[4], br[4], bi[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        ar[i] = Asr[kk][ty + 16 * i];
        ai[i] = Asi[kk][ty + 16 * i];
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        br[j] = Bsr[kk][tx + 16 * j];
        bi[j] = Bsi[kk][tx + 16 * j];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          accr[i][j] = __builtin_fmaf(ar[i], br[j], accr[i][j]);
          accr[i][j] = __builtin_fmaf(-ai[i], bi[j], accr[i][j]);
          acci[i][j] = __builtin_fmaf(ar[i], bi[j], acci[i][j]);
          acci[i][j] = __builtin_fmaf(ai[i], br[j], acci[i][j]);
        }
    }
    __syncthreads();
  }

  float2* Cm = p.C + size_t(tc.f) * p.c_fstride + size_t(tc.split) * p.c_sstride;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = tc.m0 + ty + 16 * i;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int nn = tc.n0 + tx + 16 * j;
      if (m < p.M && nn < p.N) Cm[size_t(m) * p.ldc + nn] = make_float2(accr[i][j], acci[i][j]);
    }
  }
}

// ---------------------------------------------------------------------------
// matrix-core implementation

typedef float floatx4 __attribute__((ext_vector_type(4)));

// Workgroups are dispatched round-robin over the 8 XCDs (each with its own
// L2). Renumber them so that consecutive logical tiles, which share operand
// slices, run on the same XCD at about the same time.
__device__ __forceinline__ unsigned xcd_local_order(unsigned w, unsigned nwg) {
  const unsigned q = nwg / 8, r = nwg % 8, x = w % 8, j = w / 8;
  return x * q + min(x, r) + j;
}

// MB x NB blocks of 16 x 16 per wave, waves in a 2 x 2 grid:
// tile (32*MB) x (32*NB) complex per workgroup.
template <int MB, int NB, bool AT, bool AC, bool BT, bool BC>
__global__ void __launch_bounds__(kThreads, OAA_WAVES_GEMM) cgemm_mfma_kernel(GemmParams p) {
  constexpr int TM = 32 * MB, TN = 32 * NB;
  constexpr int LDA = TM + 16, LDB = TN + 16;  // padded LDS row strides (floats)
  __shared__ float Asr[2][kKC][LDA], Asi[2][kKC][LDA];
  __shared__ float Bsr[2][kKC][LDB], Bsi[2][kKC][LDB];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * 16 * MB, wn = (wave & 1) * 16 * NB;

  // logical tile order: bin, split, row tile, column tile (fastest)
  const unsigned tiles_m = (p.M + TM - 1) / TM, tiles_n = (p.N + TN - 1) / TN;
  const unsigned nwg = gridDim.x;
  unsigned lw = xcd_local_order(blockIdx.x, nwg);
  const int tn = lw % tiles_n;
  lw /= tiles_n;
  const int tm = lw % tiles_m;
  lw /= tiles_m;
  const int split = lw % p.nsplit;
  const int f = unique_bin(int(lw / p.nsplit), p.L);
  const int m0 = tm * TM, n0 = tn * TN;
  const int k_begin = split * p.kchunk;
  const int k_end = min(p.Kr, k_begin + p.kchunk);
  const float2* A = p.A + size_t(f) * p.a_fstride;
  const float2* B = p.B + size_t(f) * p.b_fstride;

  floatx4 accr[MB][NB], acci[MB][NB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      accr[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
      acci[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    }

  const int lr = lane & 15;  // operand row (A) / column (B) within a 16-block
  const int lk = lane >> 4;  // operand reduction index within a 4-step

  Slice<AT, TM> sa;
  Slice<!BT, TN> sb;
  sa.load(A, p.lda, m0, p.M, k_begin, k_end);
  sb.load(B, p.ldb, n0, p.N, k_begin, k_end);
  sa.template store<LDA>(Asr[0], Asi[0], AC);
  sb.template store<LDB>(Bsr[0], Bsi[0], BC);
  __syncthreads();
  int buf = 0;
  for (int k0 = k_begin; k0 < k_end; k0 += kKC) {
    const bool more = k0 + kKC < k_end;
    if (more) {
      sa.load(A, p.lda, m0, p.M, k0 + kKC, k_end);
      sb.load(B, p.ldb, n0, p.N, k0 + kKC, k_end);
    }
#pragma unroll
    for (int ks = 0; ks < kKC; ks += 4) {
      const int kr = ks + lk;
      float ar[MB], ai[MB], nai[MB], br[NB], bi[NB];
#pragma unroll
      for (int i = 0; i < MB; ++i) {
        ar[i] = Asr[buf][kr][wm + 16 * i + lr];
        ai[i] = Asi[buf][kr][wm + 16 * i + lr];
        nai[i] = -ai[i];
      }
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        br[j] = Bsr[buf][kr][wn + 16 * j + lr];
        bi[j] = Bsi[buf][kr][wn + 16 * j + lr];
      }
        // four independent sweeps, so that dependent accumulations are
        // MB*NB instructions apart
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
          for (int j = 0; j < NB; ++j)
            accr[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(ar[i], br[j], accr[i][j], 0, 0, 0);
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
          for (int j = 0; j < NB; ++j)
            acci[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(ar[i], bi[j], acci[i][j], 0, 0, 0);
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
          for (int j = 0; j < NB; ++j)
            accr[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(nai[i], bi[j], accr[i][j], 0, 0, 0);
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
          for (int j = 0; j < NB; ++j)
            acci[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(ai[i], br[j], acci[i][j], 0, 0, 0);
    }
    if (more) {
      sa.template store<LDA>(Asr[buf ^ 1], Asi[buf ^ 1], AC);
      sb.template store<LDB>(Bsr[buf ^ 1], Bsi[buf ^ 1], BC);
    }
    __syncthreads();
    buf ^= 1;
  }

  // 16 x 16 result block: lane holds rows 4*(lane/16) + r, r < 4, of column lane % 16
  float2* Cm = p.C + size_t(f) * p.c_fstride + size_t(split) * p.c_sstride;
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int nn = n0 + wn + 16 * j + lr;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + wm + 16 * i + 4 * lk + r;
        if (m < p.M && nn < p.N) Cm[size_t(m) * p.ldc + nn] = make_float2(accr[i][j][r], acci[i][j][r]);
      }
    }
}

template <int MB, int NB, bool AT, bool AC, bool BT, bool BC>
hipError_t launch_mfma_shape(const GemmParams& p, hipStream_t s) {
  const unsigned tiles = unsigned(((p.M + 32 * MB - 1) / (32 * MB)) * ((p.N + 32 * NB - 1) / (32 * NB)));
  const unsigned nwg = tiles * unsigned(p.nsplit) * unsigned(p.F);
  hipLaunchKernelGGL((cgemm_mfma_kernel<MB, NB, AT, AC, BT, BC>), dim3(nwg), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

// Row tile of 96 when that wastes less than 128 does (e.g. 96 channels).
template <bool AT, bool AC, bool BT, bool BC>
hipError_t launch_mfma(const GemmParams& p, hipStream_t s) {
  const long waste128 = (long)((p.M + 127) / 128) * 128 - p.M;
  const long waste96 = (long)((p.M + 95) / 96) * 96 - p.M;
  if (waste96 < waste128) return launch_mfma_shape<3, 4, AT, AC, BT, BC>(p, s);
  return launch_mfma_shape<4, 4, AT, AC, BT, BC>(p, s);
}

template <int TM, int TN, class Kern>
hipError_t launch(Kern kern, const GemmParams& p, hipStream_t s) {
  const unsigned tiles = unsigned(((p.M + TM - 1) / TM) * ((p.N + TN - 1) / TN));
  hipLaunchKernelGGL(kern, dim3(tiles, unsigned(p.nsplit), unsigned(p.F)), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_cgemm_valu(const GemmParams& p, hipStream_t s) {
  if (p.kchunk % kKC != 0 && p.nsplit > 1) return hipErrorInvalidValue;
  // the three operand orientations the layer uses
  if (p.a_trans && !p.a_conj && !p.b_trans && !p.b_conj)
    return launch<kVM, kVN>(cgemm_valu_kernel<true, false, false, false>, p, s);
  if (!p.a_trans && p.a_conj && !p.b_trans && !p.b_conj)
    return launch<kVM, kVN>(cgemm_valu_kernel<false, true, false, false>, p, s);
  if (!p.a_trans && p.a_conj && p.b_trans && !p.b_conj)
    return launch<kVM, kVN>(cgemm_valu_kernel<false, true, true, false>, p, s);
  return hipErrorInvalidValue;
}

hipError_t launch_cgemm_mfma(const GemmParams& p, hipStream_t s) {
  if (p.kchunk % kKC != 0 && p.nsplit > 1) return hipErrorInvalidValue;
  if (p.a_trans && !p.a_conj && !p.b_trans && !p.b_conj) return launch_mfma<true, false, false, false>(p, s);
  if (!p.a_trans && p.a_conj && !p.b_trans && !p.b_conj) return launch_mfma<false, true, false, false>(p, s);
  if (!p.a_trans && p.a_conj && p.b_trans && !p.b_conj) return launch_mfma<false, true, true, false>(p, s);
  return hipErrorInvalidValue;
}

bool mfma_preferred(const GemmParams& p) { return p.M >= 32 && p.N >= 32 && p.Kr >= 16; }

}  // namespace oaa
