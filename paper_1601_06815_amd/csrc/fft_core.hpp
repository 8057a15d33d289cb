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

// (dr + i di) * exp(SIGN * 2 pi i t / L), written to (orr, oi); t in [0, L).
// The quarter turns (t = 0, L/4, L/2, 3L/4) are exchanges and sign flips.
template <int L, int SIGN>
__host__ __device__ __forceinline__ void twiddle_mul(int t, float dr, float di, float& orr, float& oi) {
  if (t == 0) {
    orr = dr;
    oi = di;
  } else if (4 * t == L) {  // exp(SIGN * i pi/2) = SIGN * i
    orr = SIGN > 0 ? -di : di;
    oi = SIGN > 0 ? dr : -dr;
  } else if (2 * t == L) {  // -1
    orr = -dr;
    oi = -di;
  } else if (4 * t == 3 * L) {  // exp(SIGN * 3 i pi/2) = -SIGN * i
    orr = SIGN > 0 ? di : -di;
    oi = SIGN > 0 ? -dr : dr;
  } else {
    const float c = tw::kTable<L>.c[t];
    const float s = SIGN > 0 ? tw::kTable<L>.s[t] : -tw::kTable<L>.s[t];
    orr = __builtin_fmaf(dr, c, -di * s);
    oi = __builtin_fmaf(dr, s, di * c);
  }
}

// In-place decimation-in-frequency FFT. Input in natural order; on return,
// coefficient k sits at position bitrev(k, L). ZERO_HI states that entries
// [L/2, L) of the input are zero.
//
// Stages go in pairs (radix 2^2): the radix-2 stages of half-sizes h and h/2
// take the four elements j, j + h/2, j + h, j + 3h/2 of a block of 2h
// (j < h/2) to the same places as two radix-2 stages would, with
//   d02 = x0 - x2, d13 = x1 - x3, r = exp(SIGN i pi/2) d13 (a quarter turn),
//   x0 + x2 + x1 + x3,  (x0 + x2 - x1 - x3) W^(2t),  (d02 + r) W^t,
//   (d02 - r) W^(3t),  W = exp(SIGN 2 pi i / L), t = j L / (2h),
// i.e. three twiddle products per four points where the two stages take
// four (the quarter turn of the second pair is an exchange). With an odd
// number of stages the last one (h = 1, twiddles 1) is radix 2.
template <int L, int SIGN, bool ZERO_HI>
__host__ __device__ __forceinline__ void fft_dif(float (&re)[L], float (&im)[L]) {
#pragma unroll
  for (int half = L / 2; half >= 2; half /= 4) {
    const int q = half / 2, s = L / (2 * half);
    const bool zh = ZERO_HI && half == L / 2;  // x2 = x3 = 0 in the first pair of stages
#pragma unroll
    for (int base = 0; base < L; base += 2 * half) {
#pragma unroll
      for (int j = 0; j < q; ++j) {
        const int i0 = base + j, i1 = i0 + q, i2 = i0 + half, i3 = i2 + q;
        const int t = j * s;
        const float x0r = re[i0], x0i = im[i0], x1r = re[i1], x1i = im[i1];
        const float x2r = zh ? 0.f : re[i2], x2i = zh ? 0.f : im[i2];
        const float x3r = zh ? 0.f : re[i3], x3i = zh ? 0.f : im[i3];
        const float s02r = x0r + x2r, s02i = x0i + x2i, s13r = x1r + x3r, s13i = x1i + x3i;
        const float d02r = x0r - x2r, d02i = x0i - x2i, d13r = x1r - x3r, d13i = x1i - x3i;
        // r = SIGN i d13
        const float rr = SIGN > 0 ? -d13i : d13i, ri = SIGN > 0 ? d13r : -d13r;
        re[i0] = s02r + s13r;
        im[i0] = s02i + s13i;
        twiddle_mul<L, SIGN>(2 * t, s02r - s13r, s02i - s13i, re[i1], im[i1]);
        twiddle_mul<L, SIGN>(t, d02r + rr, d02i + ri, re[i2], im[i2]);
        twiddle_mul<L, SIGN>(3 * t, d02r - rr, d02i - ri, re[i3], im[i3]);
      }
    }
  }
  // log2 L odd: a last radix-2 stage of half-size 1 (twiddle 1); with
  // L = 2 and ZERO_HI its second input is zero
  if ((L & 0x55555555) == 0) {
#pragma unroll
    for (int a = 0; a < L; a += 2) {
      const float ar = re[a], ai = im[a];
      const float br = (ZERO_HI && L == 2) ? 0.f : re[a + 1], bi = (ZERO_HI && L == 2) ? 0.f : im[a + 1];
      re[a] = ar + br;
      im[a] = ai + bi;
      re[a + 1] = ar - br;
      im[a + 1] = ai - bi;
    }
  }
}

// ---------------------------------------------------------------------------
// Transforms split over a pair of neighbouring lanes (h = lane bit 0), for
// long sides where one lane cannot hold a whole sequence at good occupancy.

// Value of x in the other lane of the pair, via DPP quad permute [1,0,3,2].
__device__ __forceinline__ float pair_swap(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0xB1, 0xF, 0xF, false));
}

// c ? a : b for register-array elements a and b of compile-time index. The
// operands are made opaque first: otherwise the compiler may select the
// index instead of the value and lower the access into a compare-and-select
// over the whole array.
__device__ __forceinline__ float pick(bool c, float a, float b) {
  asm volatile("" : "+v"(a), "+v"(b));
  return c ? a : b;
}

// Length-L transform; lane h holds elements h L/2 + i, i < L/2. The first
// decimation-in-frequency stage pairs element i of lane 0 (a) with element i
// of lane 1 (b): lane 0 keeps a + b, lane 1 (a - b) w^i. Both lanes run the
// same instructions: with the partner's value p, each forms p + sg * own
// (sg = +1 on lane 0, -1 on lane 1) and multiplies by 1 + hf (w^i - 1)
// (hf = 0 on lane 0, 1 on lane 1), so no lane branches or selects. Then each
// lane transforms its half alone. On return lane h holds coefficient 2m + h
// at position bitrev(m, L/2). Both lanes of every pair must execute this
// together.
template <int L, int SIGN>
__device__ __forceinline__ void fft_dif_split(float (&re)[L / 2], float (&im)[L / 2], int h) {
  const float sg = h ? -1.f : 1.f, hf = h ? 1.f : 0.f;
#pragma unroll
  for (int i = 0; i < L / 2; ++i) {
    const float pr = pair_swap(re[i]), pi = pair_swap(im[i]);
    const float dr = __builtin_fmaf(sg, re[i], pr), di = __builtin_fmaf(sg, im[i], pi);
    if (i == 0) {
      re[i] = dr;
      im[i] = di;
    } else {
      const float c = tw::kTable<L>.c[i], sn = SIGN > 0 ? tw::kTable<L>.s[i] : -tw::kTable<L>.s[i];
      const float wr = __builtin_fmaf(hf, c - 1.f, 1.f), wi = hf * sn;
      re[i] = __builtin_fmaf(dr, wr, -di * wi);
      im[i] = __builtin_fmaf(dr, wi, di * wr);
    }
  }
  fft_dif<L / 2, SIGN, false>(re, im);
}

// Same when elements [L/2, L) are zero: both lanes hold elements [0, L/2)
// on entry and no exchange is needed (lane 1 multiplies by w^i).
template <int L, int SIGN>
__device__ __forceinline__ void fft_dif_split_zh(float (&re)[L / 2], float (&im)[L / 2], int h) {
  const float hf = h ? 1.f : 0.f;
#pragma unroll
  for (int i = 1; i < L / 2; ++i) {
    const float c = tw::kTable<L>.c[i], sn = SIGN > 0 ? tw::kTable<L>.s[i] : -tw::kTable<L>.s[i];
    const float wr = __builtin_fmaf(hf, c - 1.f, 1.f), wi = hf * sn;
    const float dr = re[i], di = im[i];
    re[i] = __builtin_fmaf(dr, wr, -di * wi);
    im[i] = __builtin_fmaf(dr, wi, di * wr);
  }
  fft_dif<L / 2, SIGN, false>(re, im);
}

// Inverse real transform of two rows split over a lane pair: getA(v),
// getB(v) return bin v in [0, L/2] of the two half spectra. On return lane h
// holds L * row0[s] in zr and L * row1[s] in zi for s = 2m + h at position
// bitrev(m, L/2). The imaginary parts of bins 0 and L/2 are ignored.
template <int L, int BATCH = 0, class FA, class FB>
__device__ __forceinline__ void irfft_pair_split(FA getA, FB getB, float (&zr)[L / 2], float (&zi)[L / 2], int h) {
  constexpr int H = L / 2;
#pragma unroll
  for (int i = 0; i < H; ++i) {
    // lane 0: z[i]; lane 1: z[H + i], built from bin L - (H + i) = H - i
    const int v = h ? H - i : i;
    const float2 a = getA(v), b = getB(v);
    if (i == 0) {
      zr[0] = a.x;
      zi[0] = b.x;
    } else {
      // lane 0: a.x - b.y, a.y + b.x; lane 1: a.x + b.y, b.x - a.y
      const float sg = h ? 1.f : -1.f;
      zr[i] = __builtin_fmaf(sg, b.y, a.x);
      zi[i] = __builtin_fmaf(-sg, a.y, b.x);
    }
    // (with BATCH, the reads are issued in groups of BATCH elements, which
    // bounds the registers they hold)
    if (BATCH && i % BATCH == BATCH - 1) asm volatile("" ::: "memory");
  }
  fft_dif_split<L, +1>(zr, zi, h);
}

// Inverse column transform split over a lane pair: getU(u) returns row u of
// the column. Columns that hold only rows [0, L/2] of a Hermitian sequence
// (mir) are transformed as rows [0, L/2] with rows 0 and L/2 halved; the
// caller then takes twice the real part. On return lane h holds row 2m + h
// at position bitrev(m, L/2).
template <int L, class FU>
__device__ __forceinline__ void column_inverse_split(FU getU, bool mir, float (&re)[L / 2], float (&im)[L / 2], int h) {
  constexpr int H = L / 2;
#pragma unroll
  for (int i = 0; i < H; ++i) {
    float2 z = getU(h * H + i);
    if (i == 0) {  // rows 0 and L/2
      z.x *= mir ? 0.5f : 1.f;
      z.y *= mir ? 0.5f : 1.f;
    } else if (h == 1 && mir) {  // rows past L/2
      z = make_float2(0.f, 0.f);
    }
    re[i] = z.x;
    im[i] = z.y;
  }
  fft_dif_split<L, +1>(re, im, h);
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
