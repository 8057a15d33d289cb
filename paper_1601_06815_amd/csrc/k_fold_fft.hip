// Overlap by n carried out in the frequency domain (arXiv:1601.06815,
// Section 2: block results overlap by n-1 and are added; Section 3.2: the
// error-propagation convolution works on the overlapping windows of the
// gradient).
//
// A shift by n rows multiplies a spectrum bin (u, v) by exp(-+2 pi i n u / L);
// since every transform side here satisfies L >= 2n, no shifted tile wraps
// around. Hence:
//  * the n x n output block (P, Q) of the forward pass is the inverse
//    transform, cropped to [0, n)^2, of
//        Y(P,Q) + e^{+nu} Y(P-1,Q) + e^{+nv} Y(P,Q-1) + e^{+n(u+v)} Y(P-1,Q-1)
//    (the same sum the spatial overlap-add forms, tile by tile);
//  * the 2n x 2n gradient window (P, Q) starting at (P n, Q n) has spectrum
//        G(P,Q) + e^{-nv} G(P,Q+1) + e^{-nu} G(P+1,Q) + e^{-n(u+v)} G(P+1,Q+1)
//    where G(a, b) is the spectrum of the n x n block (a, b). A window of
//    2n rather than 2n-1 leaves both backward products unchanged: the extra
//    row and column only meet kernel taps beyond n, which are zero.
// (e^{+-nu} stands for exp(+-2 pi i n u / L).)
//
// The window kernel walks down the block rows of one plane, keeping the
// previous block row's folded column in registers (fold along u) and
// prefetching the next block row's input while it transforms the current one;
// the fold along v uses the neighbouring block's row transform in LDS. The
// forward kernel takes one block row per workgroup and reads the row above
// again (from L2: the two workgroups run back to back on one XCD).
#include <algorithm>

#include "fft_core.hpp"
#include "oaa_internal.hpp"
#include "tile_common.hpp"

namespace oaa {

namespace {

using namespace tile;

// ---------------------------------------------------------------------------
// Gradient windows from block spectra.
//
// LDS: img [n + 1][Wp] floats (one block row of the framed plane; row n stays
// zero), zbuf [TQ + 1][TS] float2 (row transforms of the TQ + 1 blocks of
// that block row; blocks are at most L/2 wide, so rows [0, L/2) suffice).
template <int L>
__global__ void __launch_bounds__(kMaxThreads) window_fold_rfft2_kernel(WindowFoldParams p) {
  constexpr int V = L / 2 + 1;
  constexpr int ROWS = L / 2;
  constexpr int PAIRS = (ROWS + 1) / 2;
  extern __shared__ float smem[];
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int n = p.n, T = p.T, H = p.H;
  const int TS = odd_at_least(2 * PAIRS * V);
  const unsigned wg = xcd_local_order(blockIdx.x, gridDim.x);
  const int chunk = int(wg % p.nchunk);
  const unsigned rest = wg / p.nchunk;
  const int grp = int(rest % p.ngroups);
  const unsigned plane = rest / p.ngroups;
  const int img = int(plane / p.n_ch), ch = int(plane % p.n_ch);
  const int q0 = chunk * p.TQ, nq = min(p.TQ, T - q0);
  const int pb = grp * p.SPW, pe = min(T, pb + p.SPW);
  const int nb = nq + 1;  // block columns q0 .. q0 + nq
  const int W = nb * n;
  const int Wp = (p.TQ + 1) * n + L / 2;
  float* img_s = smem;                                                                 // [n+1][Wp]
  float2* zbuf = reinterpret_cast<float2*>(smem + even_floats(size_t(n + 1) * Wp));  // [TQ+1][TS]
  const float* src = p.src + size_t(plane) * H * H;
  const size_t tiles_per_ch = size_t(p.n_img) * T * T;
  const size_t fstride = size_t(p.n_ch) * tiles_per_ch;
  const size_t ustride = size_t(V) * fstride;
  float2* out = p.dst + size_t(ch) * tiles_per_ch + size_t(img) * T * T + q0;

  // column task of this lane: window column Q (block columns Q and Q+1), bin column v
  const bool has_task = tid < nq * V;
  const int Q = tid % nq, v = tid / nq;
  const float2 twv = twiddle<L, -1>(n * v);
  float prev_r[L], prev_i[L];  // folded column of the previous block row

  // block row b of the framed plane: rows b*n - off + [0, n)
  constexpr int PF = L < 16 ? L : 16;
  RowPrefetch<PF> pf;
  const bool use_pf = RowPrefetch<PF>::fits(n, W);
  if (use_pf) pf.load(src, H, pb * n - p.off, q0 * n - p.off, n, W);
  for (int c = tid; c < Wp; c += nthr) img_s[n * Wp + c] = 0.f;
  for (int b = pb; b <= pe; ++b) {
    if (use_pf)
      pf.store(img_s, Wp, n, W);
    else
      stage_rows(img_s, Wp, src, H, b * n - p.off, q0 * n - p.off, n, W);
    __syncthreads();
    if (use_pf && b < pe) pf.load(src, H, (b + 1) * n - p.off, q0 * n - p.off, n, W);
    // row transforms of the nb blocks (n <= L/2 entries per row)
    for (int task = tid; task < PAIRS * nb; task += nthr) {
      const int qb = task % nb, pr = task / nb;
      const int r0 = 2 * pr;
      float2* zt = zbuf + qb * TS + r0 * V;
      if (r0 >= n) {
#pragma unroll
        for (int k = 0; k < 2 * V; ++k) zt[k] = make_float2(0.f, 0.f);
        continue;
      }
      const float* row_a = img_s + r0 * Wp + qb * n;
      const float* row_b = row_a + Wp;  // the zero row when r0 + 1 == n
      float zr[L], zi[L];
#pragma unroll
      for (int s = 0; s < L; ++s) {
        if (s < L / 2) {
          const float a = row_a[s], bb = row_b[s];
          const bool in = s < n;
          zr[s] = in ? a : 0.f;
          zi[s] = in ? bb : 0.f;
        } else {
          zr[s] = 0.f;
          zi[s] = 0.f;
        }
      }
      float2 X0[V], X1[V];
      rfft_pair<L, true>(zr, zi, X0, X1);
#pragma unroll
      for (int k = 0; k < V; ++k) {
        zt[k] = X0[k];
        zt[V + k] = X1[k];
      }
    }
    __syncthreads();
    if (has_task) {
      // fold along v, then transform the column (rows >= L/2 are zero)
      const float2* za = zbuf + Q * TS + v;
      const float2* zb = zbuf + (Q + 1) * TS + v;
      float re[L], im[L];
#pragma unroll
      for (int r = 0; r < L; ++r) {
        if (r < ROWS) {
          const float2 z = cmad(za[r * V], twv, zb[r * V]);
          re[r] = z.x;
          im[r] = z.y;
        } else {
          re[r] = 0.f;
          im[r] = 0.f;
        }
      }
      fft_dif<L, -1, true>(re, im);
      if (b > pb) {
        // window row b-1 = this column's previous value + e^{-nu} * current
        float2* o = out + size_t(b - 1) * T + Q + size_t(v) * fstride;
#pragma unroll
        for (int u = 0; u < L; ++u) {
          const int pos = bitrev(u, L);
          const float2 cur = make_float2(re[pos], im[pos]);
          o[u * ustride] = cmad(make_float2(prev_r[u], prev_i[u]), twiddle<L, -1>(n * u), cur);
        }
      }
#pragma unroll
      for (int u = 0; u < L; ++u) {
        const int pos = bitrev(u, L);
        prev_r[u] = re[pos];
        prev_i[u] = im[pos];
      }
    }
    __syncthreads();  // img and zbuf are refilled by the next block row
  }
}

// ---------------------------------------------------------------------------
// Forward output from tile spectra.
//
// One workgroup per (plane, block row, run of tile columns). LDS: zbuf
// [TQ + 1][TS] float2: column transforms (rows [0, L/2]) of tiles q0-1 ..
// q0+nq-1 of the block row, folded along u with the block row above.
template <int L>
__global__ void __launch_bounds__(kMaxThreads) irfft2_fold_crop_kernel(FoldCropParams p) {
  constexpr int V = L / 2 + 1;
  constexpr int RT = L / 2 + 1;
  extern __shared__ float smem[];
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int n = p.n, T = p.T, M = p.M;
  const int TS = odd_at_least(RT * V);
  float2* zbuf = reinterpret_cast<float2*>(smem);
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

  // column tasks: tile column q0 - 1 + qq (qq = 0 is the halo), bin column v
  for (int task = tid; task < (nq + 1) * V; task += nthr) {
    const int qq = task % (nq + 1), v = task / (nq + 1);
    const int Qt = q0 - 1 + qq;
    const bool live = Qt >= 0;
    const bool up = live && strip > 0;
    const float2* cur = in + size_t(strip) * T + (live ? Qt : 0) + size_t(v) * fstride;
    const float2* abv = cur - (up ? T : 0);
    float re[L], im[L];
#pragma unroll
    for (int u = 0; u < L; ++u) {
      const float2 c = cur[u * ustride];
      const float2 a = abv[u * ustride];
      const float2 f = cmad(live ? c : make_float2(0.f, 0.f), twiddle<L, +1>(n * u),
                            up ? a : make_float2(0.f, 0.f));
      re[u] = f.x;
      im[u] = f.y;
    }
    fft_dif<L, +1, false>(re, im);
    float2* zt = zbuf + qq * TS + v;
#pragma unroll
    for (int r = 0; r < RT; ++r) {
      const int pos = bitrev(r, L);
      zt[r * V] = make_float2(re[pos], im[pos]);
    }
  }
  __syncthreads();
  // fold along v with the left neighbour, inverse row transforms, crop
  const int npair = (n + 1) >> 1;
  for (int task = tid; task < npair * nq; task += nthr) {
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
    const int i0 = strip * n + r0 - p.off;
    const int j0 = (q0 + q) * n - p.off;
    const bool w0 = i0 >= 0 && i0 < M;
    const bool w1 = r0 + 1 < n && i0 + 1 >= 0 && i0 + 1 < M;
#pragma unroll
    for (int s = 0; s < L / 2; ++s) {
      const int j = j0 + s;
      if (s < n && j >= 0 && j < M) {
        const int pos = bitrev(s, L);
        if (w0) out[size_t(i0) * M + j] = zr[pos] * scale;
        if (w1) out[size_t(i0 + 1) * M + j] = zi[pos] * scale;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// launchers

// block-row groups: enough workgroups for the device when planes are few
inline void pick_groups(long planes, int T, int& SPW, int& ngroups) {
  int ng = 1;
  if (planes < 2048) ng = int(std::min<long>(T, (2048 + planes - 1) / planes));
  SPW = (T + ng - 1) / ng;
  ngroups = (T + SPW - 1) / SPW;
}

template <int L>
hipError_t launch_window_L(WindowFoldParams p, hipStream_t s) {
  constexpr int V = L / 2 + 1;
  constexpr int PAIRS = (L / 2 + 1) / 2;
  const int TS = odd_at_least(2 * PAIRS * V);
  auto lds_for = [&](int tq) {
    const size_t Wp = size_t(tq + 1) * p.n + L / 2;
    return even_floats(size_t(p.n + 1) * Wp) * 4 + size_t(TS) * (tq + 1) * 8;
  };
  // one column task per lane (the previous block row stays in its registers)
  int tq_max = kMaxThreads / V;
  int nchunk = (p.T + tq_max - 1) / tq_max;
  while (lds_for((p.T + nchunk - 1) / nchunk) > kLdsBudget && (p.T + nchunk - 1) / nchunk > 1) ++nchunk;
  p.TQ = (p.T + nchunk - 1) / nchunk;
  p.nchunk = (p.T + p.TQ - 1) / p.TQ;
  const size_t lds = lds_for(p.TQ);
  if (lds > kLdsBudget) return hipErrorInvalidConfiguration;
  const long planes = long(p.n_img) * p.n_ch;
  pick_groups(planes, p.T, p.SPW, p.ngroups);
  const int tasks = std::max(p.TQ * V, PAIRS * (p.TQ + 1));
  const long nwg = planes * p.ngroups * p.nchunk;
  hipLaunchKernelGGL(window_fold_rfft2_kernel<L>, dim3(unsigned(nwg)), dim3(pick_threads(tasks)), lds, s, p);
  return hipGetLastError();
}

template <int L>
hipError_t launch_fold_crop_L(FoldCropParams p, hipStream_t s) {
  constexpr int V = L / 2 + 1;
  const int TS = odd_at_least((L / 2 + 1) * V);
  const size_t per_tile = size_t(TS) * 8;
  int tq = std::min<int>(p.T, int(kLdsBudget / per_tile) - 1);
  if (tq < 1) return hipErrorInvalidConfiguration;
  const int nchunk = (p.T + tq - 1) / tq;
  p.TQ = (p.T + nchunk - 1) / nchunk;
  p.nchunk = nchunk;
  p.SPW = 1;
  p.ngroups = p.T;
  const long planes = long(p.n_img) * p.n_ch;
  const size_t lds = per_tile * (p.TQ + 1);
  const int tasks = std::max((p.TQ + 1) * V, ((p.n + 1) / 2) * p.TQ);
  const long nwg = planes * p.T * p.nchunk;
  hipLaunchKernelGGL(irfft2_fold_crop_kernel<L>, dim3(unsigned(nwg)), dim3(pick_threads(tasks)), lds, s, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_window_fold_rfft2(int L, const WindowFoldParams& p, hipStream_t s) {
  switch (L) {
    case 2: return launch_window_L<2>(p, s);
    case 4: return launch_window_L<4>(p, s);
    case 8: return launch_window_L<8>(p, s);
    case 16: return launch_window_L<16>(p, s);
    case 32: return launch_window_L<32>(p, s);
    case 64: return launch_window_L<64>(p, s);
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
