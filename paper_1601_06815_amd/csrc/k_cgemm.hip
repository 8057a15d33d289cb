// Per-frequency-bin complex contraction (arXiv:1601.06815, Introduction and
// Section 2: the Hadamard product of block and kernel spectra, summed over the
// C channels of the layer; Section 3.2 for the two backward products).
//
// For every bin f the three passes are complex matrix products:
//   forward          Yhat[f]  (K x BP) = What[f]^T   (K x C)  * Xhat[f] (C x BP)
//   backward_data    dXhat[f] (C x BP) = conj What[f] (C x K)  * Ghat[f] (K x BP)
//   backward_filter  dWhat[f] (C x K)  = conj Xhat[f] (C x BP) * Ghat[f]^T (BP x K)
// This file holds the vector-ALU implementation: 64 x 64 complex output tile
// per 256-lane workgroup, 4 x 4 complex accumulators per lane, operands staged
// through LDS in 16-deep slices of the reduction.
#include <algorithm>

#include "oaa_internal.hpp"

namespace oaa {

namespace {

constexpr int kTM = 64, kTN = 64, kKC = 16;

template <bool AT, bool AC, bool BT, bool BC>
__global__ void __launch_bounds__(256) cgemm_valu_kernel(GemmParams p) {
  __shared__ float2 As[kKC][kTM + 1];
  __shared__ float2 Bs[kKC][kTN + 1];
  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;
  const int f = blockIdx.z, split = blockIdx.y;
  const int tiles_n = (p.N + kTN - 1) / kTN;
  const int m0 = (blockIdx.x / tiles_n) * kTM, n0 = (blockIdx.x % tiles_n) * kTN;
  const int k_begin = split * p.kchunk;
  const int k_end = min(p.Kr, k_begin + p.kchunk);
  const float2* A = p.A + size_t(f) * p.a_fstride;
  const float2* B = p.B + size_t(f) * p.b_fstride;

  float accr[4][4], acci[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) accr[i][j] = acci[i][j] = 0.f;

  for (int k0 = k_begin; k0 < k_end; k0 += kKC) {
#pragma unroll
    for (int e0 = 0; e0 < kTM * kKC; e0 += 256) {
      const int e = e0 + tid;
      int ml, kl;
      if (AT) { ml = e % kTM; kl = e / kTM; } else { kl = e % kKC; ml = e / kKC; }
      const int m = m0 + ml, kk = k0 + kl;
      float2 v = make_float2(0.f, 0.f);
      if (m < p.M && kk < k_end) v = AT ? A[size_t(kk) * p.lda + m] : A[size_t(m) * p.lda + kk];
      if (AC) v.y = -v.y;
      As[kl][ml] = v;
    }
#pragma unroll
    for (int e0 = 0; e0 < kTN * kKC; e0 += 256) {
      const int e = e0 + tid;
      int nl, kl;
      if (BT) { kl = e % kKC; nl = e / kKC; } else { nl = e % kTN; kl = e / kTN; }
      const int nn = n0 + nl, kk = k0 + kl;
      float2 v = make_float2(0.f, 0.f);
      if (nn < p.N && kk < k_end) v = BT ? B[size_t(nn) * p.ldb + kk] : B[size_t(kk) * p.ldb + nn];
      if (BC) v.y = -v.y;
      Bs[kl][nl] = v;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kKC; ++kk) {
      float2 a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          accr[i][j] = __builtin_fmaf(a[i].x, b[j].x, accr[i][j]);
          accr[i][j] = __builtin_fmaf(-a[i].y, b[j].y, accr[i][j]);
          acci[i][j] = __builtin_fmaf(a[i].x, b[j].y, acci[i][j]);
          acci[i][j] = __builtin_fmaf(a[i].y, b[j].x, acci[i][j]);
        }
    }
    __syncthreads();
  }

  float2* Cm = p.C + size_t(f) * p.c_fstride + size_t(split) * p.c_sstride;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty + 16 * i;
    if (m >= p.M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int nn = n0 + tx + 16 * j;
      if (nn < p.N) Cm[size_t(m) * p.ldc + nn] = make_float2(accr[i][j], acci[i][j]);
    }
  }
}

template <bool AT, bool AC, bool BT, bool BC>
hipError_t launch_valu(const GemmParams& p, hipStream_t s) {
  const unsigned tiles = unsigned(((p.M + kTM - 1) / kTM) * ((p.N + kTN - 1) / kTN));
  hipLaunchKernelGGL((cgemm_valu_kernel<AT, AC, BT, BC>), dim3(tiles, unsigned(p.nsplit), unsigned(p.F)),
                     dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_cgemm_valu(const GemmParams& p, hipStream_t s) {
  if (p.kchunk % kKC != 0 && p.nsplit > 1) return hipErrorInvalidValue;
  // the three operand orientations the layer uses
  if (p.a_trans && !p.a_conj && !p.b_trans && !p.b_conj) return launch_valu<true, false, false, false>(p, s);
  if (!p.a_trans && p.a_conj && !p.b_trans && !p.b_conj) return launch_valu<false, true, false, false>(p, s);
  if (!p.a_trans && p.a_conj && p.b_trans && !p.b_conj) return launch_valu<false, true, true, false>(p, s);
  return hipErrorInvalidValue;
}

hipError_t launch_cgemm_mfma(const GemmParams&, hipStream_t) { return hipErrorNotSupported; }

}  // namespace oaa
