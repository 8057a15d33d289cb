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
// obuf [n][TQ n + 1] floats: the block row's output, written to HBM row by
// row with consecutive lanes on consecutive pixels.
// O32: spectrum bins are addressed as 32-bit lane offsets from a wave-uniform
// row base (V fstride * 8 < 2^32) and output pixels as 32-bit offsets from
// the plane (M * M * 4 < 2^32), with no 64-bit arithmetic per access.
template <int L, bool O32>
__global__ void __launch_bounds__(kMaxThreads, fft_waves<L>(OAA_WAVES_FOLD)) irfft2_fold_crop_kernel(FoldCropParams p) {
  constexpr int V = L / 2 + 1;
  constexpr int RT = L / 2 + 1;
  extern __shared__ float smem[];
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int n = p.n, T = p.T, M = p.M;
  const int TS = odd_at_least(RT * V);
  float2* zbuf = reinterpret_cast<float2*>(smem);
  float* obuf = smem + size_t(p.TQ + 1) * TS * 2;
  const int OWp = (p.TQ * n) | 1;  // obuf row stride, odd
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
    const float2* abv = up ? cur - T : cur;
    // Columns v = 0 and v = L/2 hold no products in rows u > L/2: there the
    // folded column h is Hermitian, so with g = h on rows [0, L/2] (rows 0 and
    // L/2 halved) and zero elsewhere, h = g + conj(g mirrored) and the
    // inverse of h is 2 Re(inverse of g).
    const bool mir = v == 0 || v == L / 2;
    const float edge = mir ? 0.5f : 1.f;
    // lane offsets of this tile and of the one above (itself when there is
    // none: both are read unconditionally, the unused one is zeroed)
    const unsigned oc = unsigned((size_t(v) * fstride + size_t(strip) * T + (live ? Qt : 0)) * 8u);
    const unsigned oa = up ? oc - unsigned(T) * 8u : oc;
    const float2* bu = in;
    float re[L], im[L];
#pragma unroll
    for (int u = 0; u < L; ++u) {
      float2 c, a;
      if (O32) {
        c = load_at(bu, oc);
        a = load_at(bu, oa);
        advance_uniform(bu, ustride);
      } else {
        c = cur[u * ustride];
        a = abv[u * ustride];
      }
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
      float* o0 = obuf + size_t(r0) * OWp + q * n;
      float* o1 = o0 + OWp;
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
    float* o0 = obuf + size_t(r0) * OWp + q * n;
    float* o1 = o0 + OWp;
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
  // lanes over columns in rows of a power-of-two width (no division)
  const int lw = 32 - __builtin_clz(unsigned(wr - 1) | 1u), cw = 1 << lw;
  for (int e = tid; e < (re_ - rb) << lw; e += nthr) {
    const int r = rb + (e >> lw), c = cb + (e & (cw - 1));
    if (c >= ce) continue;
    const float val = obuf[size_t(r) * OWp + c];
    if (O32)
      store_at(out, unsigned((i0 + r) * M + j0 + c) * 4u, val);
    else
      out[size_t(i0 + r) * M + j0 + c] = val;
  }
}

// ---------------------------------------------------------------------------
// Forward output, RB whole block rows per workgroup (L <= 32, 2b <= L).
//
// The R = RB T tiles of block rows P0 .. P0 + RB - 1 are consecutive, and so
// are the tiles above them, so every load instruction reads runs of R
// consecutive tiles of one bin (128 bytes from R = 16 on). Lane (t, k)
// folds packed column k of tile t with the tile above it (e^{+b u}, in the
// frequency domain) and inverts it; the row pass folds along v with the left
// neighbour (e^{+b v}), inverts pairs of rows and crops to b x b; the block
// rows are then written out row by row.
//
// Packed column k = 0 carries the real columns v = 0 and v = L/2 as
// h0[u] + i h1[u], rows u > L/2 rebuilt from the conjugates of rows L - u
// (those bins are not stored); both parts of its inverse are real.
//
// LDS: zrow [R][ZT] float2 (rows [0, b) of the folded column inverses, L/2
// packed slots per row, ZT = b L/2 + 1), then obuf [RB b][T b + 1] floats.
template <int L>
__global__ void __launch_bounds__(kMaxThreads) irfft2_fold_runs_kernel(FoldCropParams p) {
  constexpr int V = L / 2 + 1, HB = L / 2;
  extern __shared__ float smem[];
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int b = p.n, T = p.T, M = p.M, RB = p.RB, R = RB * T;
  const int ZT = b * HB + 1;
  float2* zrow = reinterpret_cast<float2*>(smem);
  const int OW = T * b, OWp = OW | 1;
  float* obuf = smem + size_t(R) * ZT * 2;
  const unsigned wg = xcd_local_order(blockIdx.x, gridDim.x);
  const int grp = int(wg % p.ngroups);
  const unsigned plane = wg / p.ngroups;
  const int P0 = grp * RB, rbh = min(RB, T - P0);  // block rows of this workgroup
  const int img = int(plane / p.n_ch), ch = int(plane % p.n_ch);
  const size_t tiles_per_ch = size_t(p.n_img) * T * T;
  const size_t fstride = size_t(p.n_ch) * tiles_per_ch;
  const float2* in = p.src + size_t(ch) * tiles_per_ch + size_t(img) * T * T;
  float* out = p.dst + size_t(plane) * M * M;
  const float scale = 1.0f / float(L * L);
  const float2 zero2 = make_float2(0.f, 0.f);

  // column pass
  {
    const int t = tid % R, k = tid / R;
    if (k < HB && t < rbh * T) {
      const bool up = P0 + t / T > 0;
      // bin (u, v) of tile P0 T + t at the wave-uniform row base in + u V
      // fstride plus the lane offset (v fstride + P0 T + t) * 8, below
      // V fstride * 8 < 2^32 (checked by the launcher); the tile above is T
      // tiles earlier (itself when there is none, then zeroed)
      const unsigned lo = unsigned((size_t(k) * fstride + size_t(P0) * T + t) * 8u);
      const unsigned la = up ? lo - unsigned(T) * 8u : lo;
      float re[L], im[L];
      const float2* bu = in;
      if (k == 0) {
        const unsigned lh = unsigned(size_t(HB) * fstride * 8u);
        float2 h0[V], h1[V];
#pragma unroll
        for (int u = 0; u <= L / 2; ++u) {
          const float2 tw = twiddle<L, +1>(b * u);
          const float2 c0 = load_at(bu, lo), a0 = load_at(bu, la);
          const float2 c1 = load_at(bu, lo + lh), a1 = load_at(bu, la + lh);
          h0[u] = cmad(c0, tw, up ? a0 : zero2);
          h1[u] = cmad(c1, tw, up ? a1 : zero2);
          advance_uniform(bu, size_t(V) * fstride);
        }
        // z[u] = h0[u] + i h1[u], h[L - u] = conj h[u]
#pragma unroll
        for (int u = 0; u < L; ++u) {
          const int m = u <= L / 2 ? u : L - u;
          const float sgn = u <= L / 2 ? 1.f : -1.f;
          re[u] = h0[m].x - sgn * h1[m].y;
          im[u] = sgn * h0[m].y + h1[m].x;
        }
      } else {
#pragma unroll
        for (int u = 0; u < L; ++u) {
          const float2 c = load_at(bu, lo), a = load_at(bu, la);
          const float2 f = cmad(c, twiddle<L, +1>(b * u), up ? a : zero2);
          re[u] = f.x;
          im[u] = f.y;
          advance_uniform(bu, size_t(V) * fstride);
        }
      }
      fft_dif<L, +1, false>(re, im);
      float2* zt = zrow + size_t(t) * ZT + k;
#pragma unroll
      for (int r = 0; r < L / 2; ++r) {
        const int pos = bitrev(r, L);
        if (r < b) zt[r * HB] = make_float2(re[pos], im[pos]);
      }
    }
  }
  __syncthreads();
  // row pass: fold along v with the left neighbour, inverse row transforms
  // of row pairs, crop to the block
  const int npair = (b + 1) / 2;
  for (int task = tid; task < rbh * T * npair; task += nthr) {
    const int tt = task % (rbh * T), pr = task / (rbh * T);
    const int i = tt / T, q = tt % T;
    const int r0 = 2 * pr;
    const bool has1 = r0 + 1 < b;
    const bool left = q > 0;
    const float2* za = zrow + size_t(tt) * ZT + r0 * HB;
    const float2* zl = zrow + size_t(left ? tt - 1 : tt) * ZT + r0 * HB;
    const int rb1 = has1 ? HB : 0;  // row r0 + 1, or r0 again when b is odd
    float2 A[V], Bv[V];
    {
      const float2 a0 = za[0], b0 = za[rb1];
      const float2 l0 = left ? zl[0] : zero2, m0 = left ? zl[rb1] : zero2;
      // slot 0: (bin 0, bin L/2) of a row, both real; e^{+b v} is 1 at v = 0
      // and (-1)^b at v = L/2
      const float sg = (b & 1) ? -1.f : 1.f;
      A[0] = make_float2(a0.x + l0.x, 0.f);
      A[L / 2] = make_float2(a0.y + sg * l0.y, 0.f);
      Bv[0] = make_float2(b0.x + m0.x, 0.f);
      Bv[L / 2] = make_float2(b0.y + sg * m0.y, 0.f);
    }
#pragma unroll
    for (int v = 1; v < HB; ++v) {
      const float2 tw = twiddle<L, +1>(b * v);
      A[v] = cmad(za[v], tw, left ? zl[v] : zero2);
      Bv[v] = cmad(za[rb1 + v], tw, left ? zl[rb1 + v] : zero2);
    }
    float zr[L], zi[L];
    irfft_pair<L>(A, Bv, zr, zi);
    float* o0 = obuf + size_t(i * b + r0) * OWp + q * b;
    float* o1 = o0 + OWp;
#pragma unroll
    for (int s2 = 0; s2 < L / 2; ++s2) {
      if (s2 < b) {
        const int pos = bitrev(s2, L);
        o0[s2] = zr[pos] * scale;
        if (has1) o1[s2] = zi[pos] * scale;
      }
    }
  }
  __syncthreads();
  // plane rows P0 b - off + [0, rbh b), clipped to [0, M); lanes over columns
  // in rows of a power-of-two width (no division)
  const int i0 = P0 * b - p.off, j0 = -p.off;
  const int rb = max(0, -i0), re_ = min(rbh * b, M - i0);
  const int cb = max(0, -j0), ce = min(OW, M - j0);
  const int wr = ce - cb;
  if (wr <= 0 || re_ <= rb) return;
  const int lw = 32 - __builtin_clz(unsigned(wr - 1) | 1u), cw = 1 << lw;
  for (int e = tid; e < (re_ - rb) << lw; e += nthr) {
    const int r = rb + (e >> lw), c = cb + (e & (cw - 1));
    if (c < ce) store_at(out, unsigned((i0 + r) * M + j0 + c) * 4u, obuf[size_t(r) * OWp + c]);
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
// O32: bins read at 32-bit lane offsets from wave-uniform row bases and
// output pixels written at 32-bit offsets from the plane (launcher checks).
template <int L, bool O32>
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
    const unsigned lo = unsigned((size_t(v) * fstride + size_t(live ? Pt : 0) * T + (live ? Qt : 0)) * 8u);
    const float2* bu = in;
    // columns v = 0 and v = L/2 hold no products in rows u > L/2 (Hermitian
    // there): inverse of the rows [0, L/2] with rows 0, L/2 halved, twice
    // the real part
    const bool mir = v == 0 || v == L / 2;
    float re[L], im[L];
#pragma unroll
    for (int u = 0; u < L; ++u) {
      const float2 z = O32 ? load_at(bu, lo) : col[u * ustride];
      if (O32) advance_uniform(bu, ustride);
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
  // lanes over columns in rows of a power-of-two width; column / b by a
  // reciprocal multiply (c < TQ b, which the LDS budget keeps below 2^13)
  const int lw = 32 - __builtin_clz(unsigned(wr - 1) | 1u), cw = 1 << lw;
  const SmallDiv div_b(b);
  for (int e = tid; e < (re_ - rb) << lw; e += nthr) {
    const int r = rb + (e >> lw), c = cb + (e & (cw - 1));
    if (c >= ce) continue;
    const int q = div_b(c), s = c - q * b;
    const float* own = sc + (q + 1) * SSc + r * RS;
    const float* left = sc + q * SSc + r * RS;
    float v = own[s];
    if (s < na) v += left[b + s];
    if (r < na) {
      v += sa[(q + 1) * SSa + r * RS + s];
      if (s < na) v += sa[q * SSa + r * RS + b + s];
    }
    if (O32)
      store_at(out, unsigned((i0 + r) * M + j0 + c) * 4u, v);
    else
      out[size_t(i0 + r) * M + j0 + c] = v;
  }
}

// ---------------------------------------------------------------------------
// Same result as irfft2_overlap_crop_kernel (2b > L, L <= 32). A workgroup
// takes SPW consecutive block rows of a plane and walks down them, RB per
// step.
//
// A step inverts the tiles of tile rows P .. P + RB - 1 (RB T consecutive
// tiles, so every load instruction reads runs of RB T tiles of one bin) and
// keeps rows and columns [0, S) of each inverse. Output block (P, Q) sums its
// own tile, the overhang of its left neighbour, and the overhangs of the two
// tiles above it: from LDS inside the step, and for the step's first block
// row from a carry that the previous step left: the overhang rows of its last
// tile row, already summed along the row. A workgroup that does not start at
// block row 0 first inverts the tile row above its first block row, for the
// carry alone. Each tile is thus loaded and inverted once, plus once more
// per group boundary; the per-block-row kernel does both twice.
//
// LDS: zb [RB T][TSz] float2, TSz = S V rounded up to odd (column inverses,
// rows [0, S) at stride V; after the row inverses row r of tile t holds S
// reals from float 2 (t TSz + r V)), then carry [2][S - b][To b] floats.
// Bins are read at 32-bit lane offsets and output pixels written at 32-bit
// offsets (the launcher checks both fit).
template <int L>
__global__ void __launch_bounds__(kMaxThreads) irfft2_overlap_rows_kernel(FoldCropParams p) {
  constexpr int V = L / 2 + 1;
  extern __shared__ float smem[];
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int b = p.n, S = p.S, na = S - b, T = p.T, To = p.To, M = p.M, RB = p.RB, sh = p.shift;
  const int TSz = odd_at_least(S * V), CW = To * b;
  float2* zb = reinterpret_cast<float2*>(smem);
  const float* zr = smem;  // the same array, read as real rows
  float* carry = smem + size_t(RB) * T * TSz * 2;
  const unsigned wg = xcd_local_order(blockIdx.x, gridDim.x);
  const int grp = int(wg % p.ngroups);
  const unsigned plane = wg / p.ngroups;
  const int Pb = grp * p.SPW, Pe = min(To, Pb + p.SPW);  // output block rows of this workgroup
  const int img = int(plane / p.n_ch), ch = int(plane % p.n_ch);
  const size_t tiles_per_ch = size_t(p.n_img) * T * T;
  const size_t fstride = size_t(p.n_ch) * tiles_per_ch;
  const size_t ustride = size_t(V) * fstride;
  const float2* in = p.src + size_t(ch) * tiles_per_ch + size_t(img) * T * T;
  float* out = p.dst + size_t(plane) * M * M;
  const float scale = 1.0f / float(L * L);
  // lanes over output columns in rows of a power-of-two width; divisions by
  // b through a reciprocal multiply (operands below To b and RB b, < 2^16)
  const int lw = 32 - __builtin_clz(unsigned(CW - 1) | 1u), cw = 1 << lw;
  const SmallDiv div_b(b);
  // real value at row r, column s of tile (row pl of the step, column q)
  auto at = [&](int pl, int q, int r, int s) { return zr[2 * ((pl * T + q) * TSz + r * V) + s]; };
  // overhang rows [b, S) of tile row pl at output column c = q b + s: its own
  // tile and the left neighbour's overhang columns
  auto overhang = [&](int pl, int q, int s, int rr) {
    float v = q < T ? at(pl, q, b + rr, s) : 0.f;
    if (s < na && q > 0) v += at(pl, q - 1, b + rr, b + s);
    return v;
  };
  for (int e = tid; e < na * CW; e += nthr) carry[e] = 0.f;  // nothing above block row 0
  int cur = 0;
  // step at tile row P0: tile rows P0 .. P0 + tr - 1, output block rows
  // P0 .. P0 + orow - 1; the first step of a later group is the tile row
  // above the group (Pb - 1), with no output rows
  for (int P0 = Pb > 0 ? Pb - 1 : 0; P0 < Pe;) {
    const bool halo = P0 < Pb;
    const int tr = halo ? 1 : max(0, min(RB, T - P0));  // tile rows of this step
    const int orow = halo ? 0 : min(RB, Pe - P0);       // output block rows of this step
    const int nt = tr * T;
    // column inverses; columns v = 0 and v = L/2 hold no bins in rows
    // u > L/2 (Hermitian there): inverse of rows [0, L/2] with rows 0 and L/2
    // halved, twice the real part
    for (int task = tid; task < nt * V; task += nthr) {
      const int t = task % nt, v = task / nt;
      const unsigned lo = unsigned((size_t(v) * fstride + size_t(P0) * T + t) * 8u);
      const bool mir = v == 0 || v == L / 2;
      const float2* bu = in;
      float re[L], im[L];
#pragma unroll
      for (int u = 0; u < L; ++u) {
        float2 z = make_float2(0.f, 0.f);
        if (u <= L / 2 || !mir) z = load_at(bu, lo);
        advance_uniform(bu, ustride);
        if (u == 0 || u == L / 2) {
          z.x *= mir ? 0.5f : 1.f;
          z.y *= mir ? 0.5f : 1.f;
        }
        re[u] = z.x;
        im[u] = z.y;
      }
      fft_dif<L, +1, false>(re, im);
      const float rs = mir ? 2.f : 1.f, is = mir ? 0.f : 1.f;
      float2* zt = zb + t * TSz + v;
      // row r of the inverse is row (r + shift) mod L of the tile
#pragma unroll
      for (int r = 0; r < L; ++r) {
        const int rt = (r + sh) & (L - 1);
        if (rt < S) zt[rt * V] = make_float2(re[bitrev(r, L)] * rs, im[bitrev(r, L)] * is);
      }
    }
    __syncthreads();
    // row inverses of row pairs, written over the pair's own spectrum rows
    const int ps = (S + 1) / 2;
    for (int task = tid; task < nt * ps; task += nthr) {
      const int t = task % nt, r0 = 2 * (task / nt);
      const bool has1 = r0 + 1 < S;
      float2* zt = zb + t * TSz + r0 * V;
      float2 A[V], Bv[V];
#pragma unroll
      for (int v = 0; v < V; ++v) {
        A[v] = zt[v];
        Bv[v] = has1 ? zt[V + v] : make_float2(0.f, 0.f);
      }
      float xr[L], xi[L];
      irfft_pair<L>(A, Bv, xr, xi);
      float* d0 = reinterpret_cast<float*>(zt);
#pragma unroll
      for (int s2 = 0; s2 < L; ++s2) {
        const int st = (s2 + sh) & (L - 1);  // column s2 of the inverse is column st of the tile
        if (st < S) {
          d0[st] = xr[bitrev(s2, L)] * scale;
          if (has1) d0[2 * V + st] = xi[bitrev(s2, L)] * scale;
        }
      }
    }
    __syncthreads();
    // output block rows P0 .. P0 + orow - 1: pixel (P b - off + rr, c - off)
    const float* cin = carry + cur * na * CW;
    for (int e = tid; e < (orow * b) << lw; e += nthr) {
      const int r = e >> lw, c = e & (cw - 1);
      if (c >= CW) continue;
      const int pl = div_b(r), rr = r - pl * b;
      const int q = div_b(c), s = c - q * b;
      const int i = (P0 + pl) * b - p.off + rr, j = c - p.off;
      if (i < 0 || i >= M || j < 0 || j >= M) continue;
      float v = 0.f;
      if (pl < tr) {
        if (q < T) v = at(pl, q, rr, s);
        if (s < na && q > 0) v += at(pl, q - 1, rr, b + s);
      }
      if (rr < na) v += pl == 0 ? cin[rr * CW + c] : (pl - 1 < tr ? overhang(pl - 1, q, s, rr) : 0.f);
      store_at(out, unsigned(i * M + j) * 4u, v);
    }
    // carry of the next step: the overhang rows of this step's last tile row
    // (the next step starts right below it whenever there is one)
    const int next = halo ? Pb : P0 + RB;
    if (next < Pe) {
      float* cn = carry + (cur ^ 1) * na * CW;
      for (int e = tid; e < na << lw; e += nthr) {
        const int rr = e >> lw, c = e & (cw - 1);
        if (c >= CW) continue;
        const int q = div_b(c), s = c - q * b;
        cn[rr * CW + c] = tr > 0 ? overhang(tr - 1, q, s, rr) : 0.f;
      }
      cur ^= 1;
    }
    __syncthreads();
    P0 = next;
  }
}

// ---------------------------------------------------------------------------
// launchers

template <int L>
hipError_t launch_fold_crop_L(FoldCropParams p, hipStream_t s) {
  constexpr int V = L / 2 + 1;
  if (p.To != p.T || p.shift != 0) return hipErrorInvalidValue;
  const long planes = long(p.n_img) * p.n_ch;
  // Runs of whole block rows for L = 16 and 32 (at L <= 8 the transforms are
  // too short to repay the packed columns), with 32-bit lane offsets.
  if constexpr (L >= 16 && L <= 32) if (OAA_FOLD_RUNS && 2 * p.n <= L && size_t(p.M) * p.M * 4 < (size_t(1) << 32) &&
      size_t(V) * size_t(p.n_ch) * p.n_img * p.T * p.T * 8 < (size_t(1) << 32)) {
    // whole block rows, RB of them per workgroup: runs of at least 16 tiles
    // where the lanes allow, every column task on a lane of its own
    constexpr int HB = L / 2;
    const int rb = std::min(std::max(1, (16 + p.T - 1) / p.T), std::max(1, kMaxThreads / (p.T * HB)));
    const int R = rb * p.T;
    const size_t lds = size_t(R) * (p.n * HB + 1) * 8 + size_t(rb * p.n) * ((p.T * p.n) | 1) * 4;
    if (R * HB <= kMaxThreads && lds <= kLdsRowsBudget) {
      p.RB = rb;
      p.ngroups = (p.T + rb - 1) / rb;
      auto kern = irfft2_fold_runs_kernel<L>;
      const hipError_t e = allow_lds(kern, kLdsRowsBudget);
      if (e != hipSuccess) return e;
      const int nthr = pick_threads(std::max(R * HB, R * ((p.n + 1) / 2)));
      hipLaunchKernelGGL(kern, dim3(unsigned(planes * p.ngroups)), dim3(nthr), lds, s, p);
      return hipGetLastError();
    }
  }
  const int TS = odd_at_least((L / 2 + 1) * V);
  const size_t zb = size_t(TS) * 8;                 // column transforms of one tile
  const size_t ob = size_t(p.n) * (p.n + 1) * 4;    // output block of one tile (and padding)
  int tq = std::min<int>(std::min<int>(p.T, OAA_FOLD_TQ_MAX),
                         kLdsBudget > zb ? int((kLdsBudget - zb) / (zb + ob)) : 0);
  if (tq < 1) return hipErrorInvalidConfiguration;
  const int nchunk = (p.T + tq - 1) / tq;
  p.TQ = (p.T + nchunk - 1) / nchunk;
  p.nchunk = nchunk;
  p.SPW = 1;
  p.ngroups = p.T;
  const size_t lds = zb * (p.TQ + 1) + size_t(p.n) * ((p.TQ * p.n) | 1) * 4;
  const int tasks = (L >= 64 ? 2 : 1) * std::max((p.TQ + 1) * V, ((p.n + 1) / 2) * p.TQ);
  const long nwg = planes * p.T * p.nchunk;
  const bool o32 = size_t(V) * size_t(p.n_ch) * p.n_img * p.T * p.T * 8 < (size_t(1) << 32) &&
                   size_t(p.M) * p.M * 4 < (size_t(1) << 32);
  auto kern = o32 ? irfft2_fold_crop_kernel<L, true> : irfft2_fold_crop_kernel<L, false>;
  hipLaunchKernelGGL(kern, dim3(unsigned(nwg)), dim3(pick_threads(tasks)), lds, s, p);
  return hipGetLastError();
}

template <int L>
hipError_t launch_overlap_crop_L(FoldCropParams p, hipStream_t s) {
  constexpr int V = L / 2 + 1;
  const int b = p.n, S = p.S, na = S - b;
  if (na < 0 || S > L || 2 * b <= L || p.To < p.T || p.shift < 0 || p.shift >= L) return hipErrorInvalidValue;
  const long planes = long(p.n_img) * p.n_ch;
  // a workgroup per plane, RB block rows per step: runs of at least 16 tiles
  // where LDS allows (L >= 4: below, the rows are too short to matter)
  if constexpr (L >= 4 && L <= 32) if (OAA_OVERLAP_ROWS && p.To <= p.T + 1 && size_t(p.M) * p.M * 4 < (size_t(1) << 32) &&
      size_t(V) * size_t(p.n_ch) * p.n_img * p.T * p.T * 8 < (size_t(1) << 32) && long(p.To) * b < 65536) {
    const size_t tsz = size_t(odd_at_least(S * V)) * 8;
    const size_t cbytes = size_t(2) * na * p.To * b * 4;
    auto lds_for = [&](int rb) { return size_t(rb) * p.T * tsz + cbytes; };
    int rb = std::min(std::max(1, (16 + p.T - 1) / p.T), p.To);
    while (rb > 1 && lds_for(rb) > kLdsBudget) --rb;
    // measured: faster on enough planes to fill the GPU, with several block
    // rows per step or at L <= 16; one L = 32 row per step, or a few hundred
    // planes (the paper's single-image sweeps), run faster through the
    // per-block-row kernel, which keeps more workgroups in flight
    if (planes >= 1024 && (rb >= 2 || L <= 16) && lds_for(rb) <= kLdsBudget && long(rb) * b < 65536) {
      p.RB = rb;
      // groups of block rows so that there are about OAA_OVERLAP_MIN_WG
      // workgroups (one tile row more is inverted per group)
      const int steps = (p.To + rb - 1) / rb;
      const long ng = std::min<long>(steps, std::max<long>(1, (OAA_OVERLAP_MIN_WG + planes - 1) / planes));
      p.SPW = int((steps + ng - 1) / ng) * rb;
      p.ngroups = (p.To + p.SPW - 1) / p.SPW;
      const int nt = rb * p.T;
      const int nthr = pick_threads(std::max(nt * V, nt * ((S + 1) / 2)));
      hipLaunchKernelGGL(irfft2_overlap_rows_kernel<L>, dim3(unsigned(planes * p.ngroups)), dim3(nthr), lds_for(rb), s, p);
      return hipGetLastError();
    }
  }
  const size_t per_tile = size_t(odd_at_least(b * V) + odd_at_least(na * V)) * 8;
  int tq = std::min<int>(std::min<int>(p.To, OAA_OVERLAP_TQ_MAX), int(kLdsBudget / per_tile) - 1);
  if (tq < 1) return hipErrorInvalidConfiguration;
  const int nchunk = (p.To + tq - 1) / tq;
  p.TQ = (p.To + nchunk - 1) / nchunk;
  p.nchunk = nchunk;
  const size_t lds = per_tile * (p.TQ + 1);
  const int tasks = (L >= 64 ? 2 : 1) * std::max(2 * (p.TQ + 1) * V, (p.TQ + 1) * ((b + 1) / 2 + (na + 1) / 2));
  const long nwg = planes * p.To * p.nchunk;
  const bool o32 = size_t(V) * size_t(p.n_ch) * p.n_img * p.T * p.T * 8 < (size_t(1) << 32) &&
                   size_t(p.M) * p.M * 4 < (size_t(1) << 32);
  auto kern = o32 ? irfft2_overlap_crop_kernel<L, true> : irfft2_overlap_crop_kernel<L, false>;
  hipLaunchKernelGGL(kern, dim3(unsigned(nwg)), dim3(pick_threads(tasks)), lds, s, p);
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
