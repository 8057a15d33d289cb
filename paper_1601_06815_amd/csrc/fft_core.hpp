// Register-resident small FFTs for gfx950.
//
// Each lane transforms one whole length-L sequence held in VGPRs (L <= 64);
// every loop below has a compile-time trip count and is fully unrolled, so all
// twiddle factors fold to literal constants and all array indices to register
// names. The 2-D transforms of a tile are built from these 1-D transforms by
// the kernels, with an LDS transpose between the row and the column pass.
//
// Conventions: forward transform X[k] = sum_j x[j] exp(-2 pi i jk/L); inverse
// is the same with +i and no 1/L scaling (the caller scales once).
#pragma once

#include <hip/hip_runtime.h>

#include "twiddle.hpp"

namespace oaa {

__host__ __device__ constexpr int bitrev(int k, int L) {
  int r = 0;
  for (int b = 1; b < L; b <<= 1) {
    r = (r << 1) | (k & 1);
    k >>= 1;
  }
  return r;
}

// (dr + i di) * exp(SIGN * 2 pi i t / L), written to (orr, oi).
template <int L, int SIGN>
__host__ __device__ __forceinline__ void twiddle_mul(int t, float dr, float di, float& orr, float& oi) {
  if (t == 0) {
    orr = dr;
    oi = di;
  } else if (4 * t == L) {  // exp(SIGN * i pi/2) = SIGN * i
    orr = SIGN > 0 ? -di : di;
    oi = SIGN > 0 ? dr : -dr;
  } else {
    const float c = tw::kTable<L>.c[t];
    const float s = SIGN > 0 ? tw::kTable<L>.s[t] : -tw::kTable<L>.s[t];
    orr = __builtin_fmaf(dr, c, -di * s);
    oi = __builtin_fmaf(dr, s, di * c);
  }
}

// In-place radix-2 decimation-in-frequency FFT. Input in natural order; on
// return, coefficient k sits at position bitrev(k, L). ZERO_HI states that
// entries [L/2, L) of the input are zero, which turns the first stage into a
// twiddle multiplication.
template <int L, int SIGN, bool ZERO_HI>
__host__ __device__ __forceinline__ void fft_dif(float (&re)[L], float (&im)[L]) {
#pragma unroll
  for (int half = L / 2; half >= 1; half /= 2) {
#pragma unroll
    for (int base = 0; base < L; base += 2 * half) {
#pragma unroll
      for (int j = 0; j < half; ++j) {
        const int a = base + j;
        const int b = a + half;
        const int t = j * (L / (2 * half));
        float dr, di;
        if (ZERO_HI && half == L / 2) {
          dr = re[a];
          di = im[a];
        } else {
          const float ar = re[a], ai = im[a], br = re[b], bi = im[b];
          re[a] = ar + br;
          im[a] = ai + bi;
          dr = ar - br;
          di = ai - bi;
        }
        twiddle_mul<L, SIGN>(t, dr, di, re[b], im[b]);
      }
    }
  }
}

// Forward real transform of two real rows at once: z = row0 + i*row1 is
// transformed and the Hermitian halves separated. Outputs bins v = 0..L/2 of
// both rows. zr/zi hold the two rows on entry and are clobbered.
template <int L, bool ZERO_HI>
__host__ __device__ __forceinline__ void rfft_pair(float (&zr)[L], float (&zi)[L],
                                          float2 (&X0)[L / 2 + 1], float2 (&X1)[L / 2 + 1]) {
  fft_dif<L, -1, ZERO_HI>(zr, zi);
#pragma unroll
  for (int v = 0; v <= L / 2; ++v) {
    const int pv = bitrev(v, L);
    const int pm = bitrev((L - v) % L, L);
    const float a = zr[pv], b = zi[pv], c = zr[pm], d = zi[pm];
    X0[v] = make_float2(0.5f * (a + c), 0.5f * (b - d));
    X1[v] = make_float2(0.5f * (b + d), 0.5f * (c - a));
  }
}

// Inverse real transform of two rows given by their half spectra A, B
// (bins 0..L/2). Returns L * row0 in zr (natural order after the caller reads
// position bitrev(s, L)) and L * row1 in zi. The imaginary parts of bins 0
// and L/2 are ignored, as for any Hermitian half spectrum.
template <int L>
__host__ __device__ __forceinline__ void irfft_pair(const float2 (&A)[L / 2 + 1], const float2 (&B)[L / 2 + 1],
                                           float (&zr)[L], float (&zi)[L]) {
  zr[0] = A[0].x;
  zi[0] = B[0].x;
  zr[L / 2] = A[L / 2].x;
  zi[L / 2] = B[L / 2].x;
#pragma unroll
  for (int v = 1; v < L / 2; ++v) {
    zr[v] = A[v].x - B[v].y;
    zi[v] = A[v].y + B[v].x;
    zr[L - v] = A[v].x + B[v].y;
    zi[L - v] = B[v].x - A[v].y;
  }
  fft_dif<L, +1, false>(zr, zi);
}

}  // namespace oaa
