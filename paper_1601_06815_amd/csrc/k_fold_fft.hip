// Overlap-add of the forward pass carried out in the frequency domain
// (arXiv:1601.06815, Section 2: block results overlap by n-1 and are added).
//
// A shift by n rows multiplies spectrum bin (u, v) by exp(+2 pi i n u / L)
// (written e^{+nu}); since every transform side here satisfies L >= 2n, no
// shifted tile wraps around. Hence the n x n output block (P, Q) is the
// inverse transform, cropped to [0, n)^2, of
//     Y(P,Q) + e^{+nu} Y(P-1,Q) + e^{+nv} Y(P,Q-1) + e^{+n(u+v)} Y(P-1,Q-1),
// the same sum the spatial overlap-add forms, tile by tile.
//
// One workgroup takes one block row of one plane (a run of its tiles): the
// column transforms fold in the block row above (read a second time, mostly
// from L2, since neighbouring workgroups run back to back on one XCD), and the
// row transforms fold in the left neighbour's column transform from LDS.
#include <algorithm>

#include "fft_core.hpp"
#include "oaa_internal.hpp"
#include "tile_common.hpp"

namespace oaa {

namespace {

using namespace tile;

// ---------------------------------------------------------------------------
// Forward output from tile spectra.
//
// One workgroup per (plane, block row, run of tile columns). LDS: zbuf
// [TQ + 1][TS] float2: column transforms (rows [0, L/2]) of tiles q0-1 ..
// q0+nq-1 of the block row, folded along u with the block row above; then
// obuf [n][TQ][n + 1] floats: the block row's output, written to HBM row by
// row with consecutive lanes on consecutive pixels.
template <int L>
__global__ void __launch_bounds__(kMaxThreads, fft_waves<L>(OAA_WAVES_FOLD)) irfft2_fold_crop_kernel(FoldCropParams p) {
  constexpr int V = L / 2 + 1;
  constexpr int RT = L / 2 + 1;
  extern __shared__ float smem[];
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int n = p.n, T = p.T, M = p.M;
  const int TS = odd_at_least(RT * V);
  float2* zbuf = reinterpret_cast<float2*>(smem);
  float* obuf = smem + size_t(p.TQ + 1) * TS * 2;
  const int OS = n | 1;  // obuf stride between tiles, odd
  const unsigned wg = xcd_local_order(blockIdx.x, gridDim.x);
  const int chunk = int(wg % p.nchunk);
  const unsigned rest = wg / p.nchunk;
  const int strip = int(rest % T);
  const unsigned plane = rest / T;
  const int img = int(plane / p.n_ch), ch = int(plane % p.n_ch);
  const int q0 = chunk * p.TQ, nq = min(p.TQ, T - q0);
  const size_t tiles_per_ch = size_t(p.n_img) * T * T;
  const size_t fstride = size_t(p.n_ch) * tiles_per_ch;
  const size_t ustride = size_t(V) * fstride;
  const float2* in = p.src + size_t(ch) * tiles_per_ch + size_t(img) * T * T;
  float* out = p.dst + size_t(plane) * M * M;
  const float scale = 1.0f / float(L * L);

  constexpr bool SPLIT = L >= 64;
  constexpr int HL = L / 2;
  if (SPLIT) {
    for (int task = tid; task < 2 * (nq + 1) * V; task += nthr) {
      const int h = task & 1, base = task >> 1;
      const int qq = base % (nq + 1), v = base / (nq + 1);
      const int Qt = q0 - 1 + qq;
      const bool live = Qt >= 0;
      const bool up = live && strip > 0;
      const float2* cur = in + size_t(strip) * T + (live ? Qt : 0) + size_t(v) * fstride;
      const float2* abv = cur - (up ? T : 0);
      const bool mir = v == 0 || v == L / 2;
      float re[HL], im[HL];
      column_inverse_split<L>(
          [&](int u) {
            const float2 c = cur[u * ustride];
            const float2 a = abv[u * ustride];
            return cmad(live ? c : make_float2(0.f, 0.f), twiddle<L, +1>(n * u), up ? a : make_float2(0.f, 0.f));
          },
          mir, re, im, h);
      const float rs = mir ? 2.f : 1.f, is = mir ? 0.f : 1.f;
      float2* zt = zbuf + qq * TS + v;
#pragma unroll
      for (int m = 0; m < HL; ++m) {
        const int r = 2 * m + h;
        if (r < RT) zt[r * V] = make_float2(re[bitrev(m, HL)] * rs, im[bitrev(m, HL)] * is);
      }
    }
  }
  // column tasks: tile column q0 - 1 + qq (qq = 0 is the halo), bin column v
  for (int task = tid; task < (SPLIT ? 0 : (nq + 1) * V); task += nthr) {
    const int qq = task % (nq + 1), v = task / (nq + 1);
    const int Qt = q0 - 1 + qq;
    const bool live = Qt >= 0;
    const bool up = live && strip > 0;
    const float2* cur = in + size_t(strip) * T + (live ? Qt : 0) + size_t(v) * fstride;
    const float2* abv = cur - (up ? T : 0);
    // Columns v = 0 and v = L/2 hold no products in rows u > L/2: there the
    // folded column h is Hermitian, so with g = h on rows [0, L/2] (rows 0 and
    // L/2 halved) and zero elsewhere, h = g + conj(g mirrored) and the
    // inverse of h is 2 Re(inverse of g).
    const bool mir = v == 0 || v == L / 2;
    const float edge = mir ? 0.5f : 1.f;
    float re[L], im[L];
#pragma unroll
    for (int u = 0; u < L; ++u) {
      const float2 c = cur[u * ustride];
      const float2 a = abv[u * ustride];
      const float2 f = cmad(live ? c : make_float2(0.f, 0.f), twiddle<L, +1>(n * u),
                            up ? a : make_float2(0.f, 0.f));
      if (u > L / 2) {
        re[u] = mir ? 0.f : f.x;
        im[u] = mir ? 0.f : f.y;
      } else if (u == 0 || u == L / 2) {
        re[u] = f.x * edge;
        im[u] = f.y * edge;
      } else {
        re[u] = f.x;
        im[u] = f.y;
      }
    }
    fft_dif<L, +1, false>(re, im);
    const float rs = mir ? 2.f : 1.f, is = mir ? 0.f : 1.f;
    float2* zt = zbuf + qq * TS + v;
#pragma unroll
    for (int r = 0; r < RT; ++r) {
      const int pos = bitrev(r, L);
      zt[r * V] = make_float2(re[pos] * rs, im[pos] * is);
    }
  }
  __syncthreads();
  // fold along v with the left neighbour, inverse row transforms, crop to the
  // tile's n x n output block in LDS
  const int npair = (n + 1) >> 1;
  if (SPLIT) {
    for (int task = tid; task < 2 * npair * nq; task += nthr) {
      const int h = task & 1, base = task >> 1;
      const int q = base % nq, pr = base / nq;
      const int r0 = 2 * pr;
      const float2* za = zbuf + (q + 1) * TS + r0 * V;
      const float2* zb = zbuf + q * TS + r0 * V;
      float zr[HL], zi[HL];
      irfft_pair_split<L>([&](int k) { return cmad(za[k], twiddle<L, +1>(n * k), zb[k]); },
                          [&](int k) { return cmad(za[V + k], twiddle<L, +1>(n * k), zb[V + k]); }, zr, zi, h);
      float* o0 = obuf + (size_t(r0) * nq + q) * OS;
      float* o1 = o0 + size_t(nq) * OS;
      const bool has1 = r0 + 1 < n;
#pragma unroll
      for (int m = 0; m < HL; ++m) {
        const int sx = 2 * m + h;
        if (sx < n) {
          o0[sx] = zr[bitrev(m, HL)] * scale;
          if (has1) o1[sx] = zi[bitrev(m, HL)] * scale;
        }
      }
    }
  }
  for (int task = tid; task < (SPLIT ? 0 : npair * nq); task += nthr) {
    const int q = task % nq, pr = task / nq;
    const int r0 = 2 * pr;
    const float2* za = zbuf + (q + 1) * TS + r0 * V;
    const float2* zb = zbuf + q * TS + r0 * V;
    float2 A[V], Bv[V];
#pragma unroll
    for (int k = 0; k < V; ++k) {
      const float2 t = twiddle<L, +1>(n * k);
      A[k] = cmad(za[k], t, zb[k]);
      Bv[k] = cmad(za[V + k], t, zb[V + k]);  // row n (odd n) is discarded below
    }
    float zr[L], zi[L];
    irfft_pair<L>(A, Bv, zr, zi);
    float* o0 = obuf + (size_t(r0) * nq + q) * OS;
    float* o1 = o0 + size_t(nq) * OS;
    const bool has1 = r0 + 1 < n;
#pragma unroll
    for (int s = 0; s < L / 2; ++s) {
      if (s < n) {
        const int pos = bitrev(s, L);
        o0[s] = zr[pos] * scale;
        if (has1) o1[s] = zi[pos] * scale;
      }
    }
  }
  __syncthreads();
  // the block row's valid output: rows strip*n - off + [0, n), columns
  // q0*n - off + [0, nq*n), both clipped to [0, M)
  const int W = nq * n;
  const int i0 = strip * n - p.off, j0 = q0 * n - p.off;
  const int rb = max(0, -i0), re_ = min(n, M - i0);
  const int cb = max(0, -j0), ce = min(W, M - j0);
  const int wr = ce - cb;
  if (wr <= 0 || re_ <= rb) return;
  for (int e = tid; e < (re_ - rb) * wr; e += nthr) {
    const int r = rb + e / wr, c = cb + e % wr;
    const int q = c / n, s = c - q * n;
    out[size_t(i0 + r) * M + j0 + c] = obuf[(size_t(r) * nq + q) * OS + s];
  }
}

// ---------------------------------------------------------------------------
// Forward output for blocks with 2b > L (support S = b + n - 1 <= L): a block
// result shifted by b would wrap inside L, so the neighbours are added in
// space after the inverse.
//
// One workgroup per (plane, block row P, run of tile columns) with the halo
// column q0 - 1. Column inverses of the block row's tiles (rows [0, b), zc)
// and of the row above (rows [b, S), za); row inverses of those rows, each
// written over its own row's spectrum (S <= L real values in the 2 (L/2 + 1)
// floats of a row); then every output pixel of the block row is the sum, in
// a fixed order, of its tile's value and the overhangs of the left, upper and
// upper-left neighbours.
template <int L>
__global__ void __launch_bounds__(kMaxThreads) irfft2_overlap_crop_kernel(FoldCropParams p) {
  constexpr int V = L / 2 + 1;
  extern __shared__ float smem[];
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int b = p.n, S = p.S, na = S - b, T = p.T, M = p.M;
  const int TQ1 = p.TQ + 1;
  const int TSc = odd_at_least(b * V), TSa = odd_at_least(na * V);
  float2* zc = reinterpret_cast<float2*>(smem);  // [TQ+1][TSc]
  float2* za = zc + size_t(TQ1) * TSc;            // [TQ+1][TSa]
  // real rows after the row inverses: row r of tile qq at float offset
  // 2 (qq TS + r V) of the same array
  const float* sc = reinterpret_cast<const float*>(zc);
  const float* sa = reinterpret_cast<const float*>(za);
  const int SSc = 2 * TSc, SSa = 2 * TSa, RS = 2 * V;
  const unsigned wg = xcd_local_order(blockIdx.x, gridDim.x);
  const int chunk = int(wg % p.nchunk);
  const unsigned rest = wg / p.nchunk;
  const int To = p.To, sh = p.shift;
  const int strip = int(rest % To);
  const unsigned plane = rest / To;
  const int img = int(plane / p.n_ch), ch = int(plane % p.n_ch);
  const int q0 = chunk * p.TQ, nq = min(p.TQ, To - q0);
  const size_t tiles_per_ch = size_t(p.n_img) * T * T;
  const size_t fstride = size_t(p.n_ch) * tiles_per_ch;
  const size_t ustride = size_t(V) * fstride;
  const float2* in = p.src + size_t(ch) * tiles_per_ch + size_t(img) * T * T;
  float* out = p.dst + size_t(plane) * M * M;
  const float scale = 1.0f / float(L * L);

  constexpr bool SPLIT = L >= 64;
  constexpr int HL = L / 2;
  if (SPLIT) {
    for (int task = tid; task < 4 * (nq + 1) * V; task += nthr) {
      const int h = task & 1, base = task >> 1;
      const int qq = base % (nq + 1), rest2 = base / (nq + 1);
      const int v = rest2 % V, part = rest2 / V;
      const int Qt = q0 - 1 + qq, Pt = strip - part;
      const bool live = Qt >= 0 && Qt < T && Pt >= 0 && Pt < T && (part == 0 || na > 0);
      const float2* col = in + size_t(live ? Pt : 0) * T + (live ? Qt : 0) + size_t(v) * fstride;
      const bool mir = v == 0 || v == L / 2;
      float re[HL], im[HL];
      column_inverse_split<L>(
          [&](int u) {
            const float2 z = col[u * ustride];
            return live ? z : make_float2(0.f, 0.f);
          },
          mir, re, im, h);
      const float rs = mir ? 2.f : 1.f, is = mir ? 0.f : 1.f;
#pragma unroll
      for (int m = 0; m < HL; ++m) {
        const int r = (2 * m + h + sh) & (L - 1);
        const float2 val = make_float2(re[bitrev(m, HL)] * rs, im[bitrev(m, HL)] * is);
        if (part == 0) {
          if (r < b) zc[qq * TSc + v + r * V] = val;
        } else {
          if (r >= b && r < S) za[qq * TSa + v + (r - b) * V] = val;
        }
      }
    }
  }
  // column inverses: part 0 = this block row, part 1 = the block row above
  for (int task = tid; task < (SPLIT ? 0 : 2 * (nq + 1) * V); task += nthr) {
    const int qq = task % (nq + 1), rest2 = task / (nq + 1);
    const int v = rest2 % V, part = rest2 / V;
    const int Qt = q0 - 1 + qq, Pt = strip - part;
    const bool live = Qt >= 0 && Qt < T && Pt >= 0 && Pt < T && (part == 0 || na > 0);
    const float2* col = in + size_t(live ? Pt : 0) * T + (live ? Qt : 0) + size_t(v) * fstride;
    // columns v = 0 and v = L/2 hold no products in rows u > L/2 (Hermitian
    // there): inverse of the rows [0, L/2] with rows 0, L/2 halved, twice
    // the real part
    const bool mir = v == 0 || v == L / 2;
    float re[L], im[L];
#pragma unroll
    for (int u = 0; u < L; ++u) {
      const float2 z = col[u * ustride];
      float zr = live ? z.x : 0.f, zi = live ? z.y : 0.f;
      if (u > L / 2) {
        zr = mir ? 0.f : zr;
        zi = mir ? 0.f : zi;
      } else if (u == 0 || u == L / 2) {
        zr *= mir ? 0.5f : 1.f;
        zi *= mir ? 0.5f : 1.f;
      }
      re[u] = zr;
      im[u] = zi;
    }
    fft_dif<L, +1, false>(re, im);
    const float rs = mir ? 2.f : 1.f, is = mir ? 0.f : 1.f;
    // row r of the inverse is row (r + shift) mod L of the tile
    if (part == 0) {
      float2* zt = zc + qq * TSc + v;
#pragma unroll
      for (int r = 0; r < L; ++r) {
        const int rt = (r + sh) & (L - 1);
        if (rt < b) zt[rt * V] = make_float2(re[bitrev(r, L)] * rs, im[bitrev(r, L)] * is);
      }
    } else {
      float2* zt = za + qq * TSa + v;
#pragma unroll
      for (int r = 0; r < L; ++r) {
        const int rt = (r + sh) & (L - 1);
        if (rt >= b && rt < S) zt[(rt - b) * V] = make_float2(re[bitrev(r, L)] * rs, im[bitrev(r, L)] * is);
      }
    }
  }
  __syncthreads();
  // row inverses, two rows per task (a missing partner row is zero)
  const int pc = (b + 1) / 2, pa = (na + 1) / 2;
  if (SPLIT) {
    for (int task = tid; task < 2 * (nq + 1) * (pc + pa); task += nthr) {
      const int h = task & 1, base = task >> 1;
      const int qq = base % (nq + 1), k = base / (nq + 1);
      const bool above = k >= pc;
      const int r0 = 2 * (above ? k - pc : k), rows = above ? na : b;
      const float2* zt = above ? za + qq * TSa + r0 * V : zc + qq * TSc + r0 * V;
      const bool has1 = r0 + 1 < rows;
      float zr[HL], zi[HL];
      irfft_pair_split<L>([&](int v) { return zt[v]; },
                          [&](int v) { return has1 ? zt[V + v] : make_float2(0.f, 0.f); }, zr, zi, h);
      // both lanes have read their bins: the pair's rows may be overwritten
      // once the partner is done too, which the exchange inside the
      // transform guarantees for the lanes of the pair
      float* d0 = reinterpret_cast<float*>(const_cast<float2*>(zt));
#pragma unroll
      for (int m = 0; m < HL; ++m) {
        const int sx = (2 * m + h + sh) & (L - 1);
        if (sx < S) {
          d0[sx] = zr[bitrev(m, HL)] * scale;
          if (has1) d0[RS + sx] = zi[bitrev(m, HL)] * scale;
        }
      }
    }
  }
  for (int task = tid; task < (SPLIT ? 0 : (nq + 1) * (pc + pa)); task += nthr) {
    const int qq = task % (nq + 1), k = task / (nq + 1);
    const bool above = k >= pc;
    const int r0 = 2 * (above ? k - pc : k), rows = above ? na : b;
    const float2* zt = above ? za + qq * TSa + r0 * V : zc + qq * TSc + r0 * V;
    const bool has1 = r0 + 1 < rows;
    float2 A[V], Bv[V];
#pragma unroll
    for (int v = 0; v < V; ++v) {
      A[v] = zt[v];
      Bv[v] = has1 ? zt[V + v] : make_float2(0.f, 0.f);
    }
    float zr[L], zi[L];
    irfft_pair<L>(A, Bv, zr, zi);
    float* d0 = reinterpret_cast<float*>(const_cast<float2*>(zt));  // this task's own two rows
#pragma unroll
    for (int s = 0; s < L; ++s) {
      const int st = (s + sh) & (L - 1);  // column s of the inverse is column st of the tile
      if (st < S) {
        d0[st] = zr[bitrev(s, L)] * scale;
        if (has1) d0[RS + st] = zi[bitrev(s, L)] * scale;
      }
    }
  }
  __syncthreads();
  // output rows strip*b - off + [0, b), columns q0*b - off + [0, nq b), clipped
  const int W = nq * b;
  const int i0 = strip * b - p.off, j0 = q0 * b - p.off;
  const int rb = max(0, -i0), re_ = min(b, M - i0);
  const int cb = max(0, -j0), ce = min(W, M - j0);
  const int wr = ce - cb;
  if (wr <= 0 || re_ <= rb) return;
  for (int e = tid; e < (re_ - rb) * wr; e += nthr) {
    const int r = rb + e / wr, c = cb + e % wr;
    const int q = c / b, s = c - q * b;
    const float* own = sc + (q + 1) * SSc + r * RS;
    const float* left = sc + q * SSc + r * RS;
    float v = own[s];
    if (s < na) v += left[b + s];
    if (r < na) {
      v += sa[(q + 1) * SSa + r * RS + s];
      if (s < na) v += sa[q * SSa + r * RS + b + s];
    }
    out[size_t(i0 + r) * M + j0 + c] = v;
  }
}

// ---------------------------------------------------------------------------
// launchers

template <int L>
hipError_t launch_fold_crop_L(FoldCropParams p, hipStream_t s) {
  constexpr int V = L / 2 + 1;
  if (p.To != p.T || p.shift != 0) return hipErrorInvalidValue;
  const int TS = odd_at_least((L / 2 + 1) * V);
  const size_t zb = size_t(TS) * 8;                 // column transforms of one tile
  const size_t ob = size_t(p.n) * (p.n | 1) * 4;    // output block of one tile
  int tq = std::min<int>(std::min<int>(p.T, OAA_FOLD_TQ_MAX),
                         kLdsBudget > zb ? int((kLdsBudget - zb) / (zb + ob)) : 0);
  if (tq < 1) return hipErrorInvalidConfiguration;
  const int nchunk = (p.T + tq - 1) / tq;
  p.TQ = (p.T + nchunk - 1) / nchunk;
  p.nchunk = nchunk;
  p.SPW = 1;
  p.ngroups = p.T;
  const long planes = long(p.n_img) * p.n_ch;
  const size_t lds = zb * (p.TQ + 1) + ob * p.TQ;
  const int tasks = (L >= 64 ? 2 : 1) * std::max((p.TQ + 1) * V, ((p.n + 1) / 2) * p.TQ);
  const long nwg = planes * p.T * p.nchunk;
  hipLaunchKernelGGL(irfft2_fold_crop_kernel<L>, dim3(unsigned(nwg)), dim3(pick_threads(tasks)), lds, s, p);
  return hipGetLastError();
}

template <int L>
hipError_t launch_overlap_crop_L(FoldCropParams p, hipStream_t s) {
  constexpr int V = L / 2 + 1;
  const int b = p.n, S = p.S, na = S - b;
  if (na < 0 || S > L || 2 * b <= L || p.To < p.T || p.shift < 0 || p.shift >= L) return hipErrorInvalidValue;
  const size_t per_tile = size_t(odd_at_least(b * V) + odd_at_least(na * V)) * 8;
  int tq = std::min<int>(p.To, int(kLdsBudget / per_tile) - 1);
  if (tq < 1) return hipErrorInvalidConfiguration;
  const int nchunk = (p.To + tq - 1) / tq;
  p.TQ = (p.To + nchunk - 1) / nchunk;
  p.nchunk = nchunk;
  const long planes = long(p.n_img) * p.n_ch;
  const size_t lds = per_tile * (p.TQ + 1);
  const int tasks = (L >= 64 ? 2 : 1) * std::max(2 * (p.TQ + 1) * V, (p.TQ + 1) * ((b + 1) / 2 + (na + 1) / 2));
  const long nwg = planes * p.To * p.nchunk;
  hipLaunchKernelGGL(irfft2_overlap_crop_kernel<L>, dim3(unsigned(nwg)), dim3(pick_threads(tasks)), lds, s, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_irfft2_overlap_crop(int L, const FoldCropParams& p, hipStream_t s) {
  switch (L) {
    case 2: return launch_overlap_crop_L<2>(p, s);
    case 4: return launch_overlap_crop_L<4>(p, s);
    case 8: return launch_overlap_crop_L<8>(p, s);
    case 16: return launch_overlap_crop_L<16>(p, s);
    case 32: return launch_overlap_crop_L<32>(p, s);
    case 64: return launch_overlap_crop_L<64>(p, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_irfft2_fold_crop(int L, const FoldCropParams& p, hipStream_t s) {
  switch (L) {
    case 2: return launch_fold_crop_L<2>(p, s);
    case 4: return launch_fold_crop_L<4>(p, s);
    case 8: return launch_fold_crop_L<8>(p, s);
    case 16: return launch_fold_crop_L<16>(p, s);
    case 32: return launch_fold_crop_L<32>(p, s);
    case 64: return launch_fold_crop_L<64>(p, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace oaa
