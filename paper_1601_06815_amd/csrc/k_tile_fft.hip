// Tiling + zero-padding + 2-D real FFT of blocks and windows, and the
// inverse transforms with crop (arXiv:1601.06815, Section 2: block division,
// padding, per-block transforms; Section 3.2: the two backward convolutions).
//
// Forward: one workgroup handles a run of consecutive tiles along one block
// row of one plane. The plane rows that the run covers are staged in LDS with
// coalesced loads; pass 1 (one lane per pair of tile rows) transforms rows,
// pass 2 (one lane per tile column) transforms columns and writes the spectra
// bin-major with consecutive tiles at consecutive addresses.
// Gradient windows (and input blocks taken as windows of side and pitch b):
// one workgroup walks down the window rows of a plane, several per step for
// L <= 32 with the rows read straight from memory (window_rows_rfft2_kernel),
// one per step with a ring of 2n input rows in LDS for L = 64
// (window_rfft2_kernel).
// Inverse with crop (error propagation, weight gradient): the two passes in
// the opposite order, keeping the top-left n x n of every tile. The forward
// inverse with overlap-add is in k_fold_fft.hip.
//
// LDS intermediates are stored tile-major with an odd per-tile stride (in
// complex elements), so every index inside a tile is a compile-time offset
// and consecutive tiles fall in different banks.
#include <algorithm>

#include "fft_core.hpp"
#include "oaa_internal.hpp"
#include "tile_common.hpp"

namespace oaa {

namespace {

using namespace tile;

// ---------------------------------------------------------------------------
// Pass bodies with each transform split over a lane pair (h = lane bit 0),
// used for L = 64 where a whole sequence per lane would need ~270 VGPRs.

// Two real rows (row_a, row_b; entries s >= R, and s >= L/2 under ZH, are
// zero) -> their half spectra, bins v of zt[v] and zt[V + v]. Lane h writes
// the bins of its parity.
template <int L, bool ZH>
__device__ __forceinline__ void row_pair_split(const float* row_a, const float* row_b, int R, bool has_b,
                                               float2* zt, int h) {
  constexpr int H = L / 2, V = L / 2 + 1;
  float zr[H], zi[H];
#pragma unroll
  for (int i = 0; i < H; ++i) {
    const int s = ZH ? i : h * H + i;
    const bool in = s < R;
    const float a = row_a[s], b = row_b[s];
    zr[i] = in ? a : 0.f;
    zi[i] = in && has_b ? b : 0.f;
  }
  if (ZH)
    fft_dif_split_zh<L, -1>(zr, zi, h);
  else
    fft_dif_split<L, -1>(zr, zi, h);
  // lane h holds Z[2m + h]; bin v pairs Z[v] with Z[L - v] (same parity)
#pragma unroll
  for (int m = 0; m <= H / 2; ++m) {
    const int ps = bitrev(m, H);
    const int p0 = bitrev(m == 0 ? 0 : H - m, H);   // partner of v = 2m (lane 0)
    const int p1 = bitrev(H - 1 - (m < H / 2 ? m : 0), H);  // partner of v = 2m + 1 (lane 1)
    const float a = zr[ps], b = zi[ps];
    const float c = pick(h, zr[p1], zr[p0]), d = pick(h, zi[p1], zi[p0]);
    const int v = 2 * m + h;
    if (h == 0 || m < H / 2) {
      zt[v] = make_float2(0.5f * (a + c), 0.5f * (b - d));
      zt[V + v] = make_float2(0.5f * (b + d), 0.5f * (c - a));
    }
  }
}

// Complex column (rows [0, ROWS) of zt at stride V, zero beyond) -> forward
// transform, coefficient U stored at o[U * ustride]; lane h stores U of its parity.
template <int L, bool ZH>
__device__ __forceinline__ void column_split_store(const float2* zt, int ROWS, float2* o, size_t ustride, int h) {
  constexpr int H = L / 2, V = L / 2 + 1;
  float re[H], im[H];
#pragma unroll
  for (int i = 0; i < H; ++i) {
    const int r = ZH ? i : h * H + i;
    const float2 z = zt[(r < ROWS ? r : 0) * V];
    re[i] = r < ROWS ? z.x : 0.f;
    im[i] = r < ROWS ? z.y : 0.f;
  }
  if (ZH)
    fft_dif_split_zh<L, -1>(re, im, h);
  else
    fft_dif_split<L, -1>(re, im, h);
#pragma unroll
  for (int m = 0; m < H; ++m) {
    const int pos = bitrev(m, H);
    o[size_t(2 * m + h) * ustride] = make_float2(re[pos], im[pos]);
  }
}

// ---------------------------------------------------------------------------
// Forward: windows -> spectra
//
// LDS: img [R + 1][Wp] floats (row R stays zero), then zbuf [TQ][TS] float2,
// TS >= ROWS * V (rounded up to whole row pairs) odd, ROWS = L/2 when
// windows fill at most half a tile (ZH), else L. Row r of tile q's row transform is at zbuf[q * TS + r * V + v].
template <int L, bool ZH>
__global__ void __launch_bounds__(kMaxThreads, fft_waves<L>(OAA_WAVES_TILE)) tile_rfft2_kernel(TileFwdParams p) {
  constexpr int V = L / 2 + 1;
  constexpr int ROWS = ZH ? L / 2 : L;
  constexpr int S = ZH ? L / 2 : L;         // row entries that may be nonzero
  constexpr int PAIRS = (ROWS + 1) / 2;     // row pairs covering rows [0, ROWS)
  extern __shared__ float smem[];
  const int tid = threadIdx.x, nthr = blockDim.x;
  const unsigned wg = xcd_local_order(blockIdx.x, gridDim.x);
  const int chunk = int(wg % p.nchunk);
  const unsigned rest = wg / p.nchunk;
  const int R = p.R, pitch = p.pitch;
  int strip, img, ch, q0, nq;
  if (p.gather) {  // kernels q0 .. q0+nq-1 of channel ch, side by side
    strip = 0;
    img = 0;
    ch = int(rest);
    q0 = chunk * p.TQ;
    nq = min(p.TQ, p.n_img - q0);
  } else {  // tiles q0 .. q0+nq-1 of block row `strip` of plane (img, ch)
    strip = int(rest % p.T);
    const unsigned plane = rest / p.T;
    img = int(plane / p.n_ch);
    ch = int(plane % p.n_ch);
    q0 = chunk * p.TQ;
    nq = min(p.TQ, p.T - q0);
  }
  const int W = (nq - 1) * pitch + R;
  const int Wp = bank_stride((p.TQ - 1) * pitch + R + L);  // reads past W stay inside the row
  const int TS = odd_at_least(2 * PAIRS * V);
  float* img_s = smem;                                                                 // [R+1][Wp]
  float2* zbuf = reinterpret_cast<float2*>(smem + even_floats(size_t(R + 1) * Wp));  // [TQ][TS]

  if (p.gather) {
    const size_t pstride = size_t(p.n_ch) * p.H * p.H;
    const float* src = p.src + size_t(q0) * pstride + size_t(ch) * p.H * p.H;
    for (int e = tid; e < nq * R * R; e += nthr) {
      const int q = e / (R * R), rs = e - q * R * R;
      const int r = rs / R, c = rs - r * R;
      img_s[r * Wp + q * pitch + c] = src[size_t(q) * pstride + rs];
    }
    // pitch == R: the row has no gaps; clear what the row reads may touch past W
    for (int e = tid; e < R * (Wp - W); e += nthr) img_s[(e / (Wp - W)) * Wp + W + e % (Wp - W)] = 0.f;
  } else {
    const float* src = p.src + (size_t(img) * p.n_ch + ch) * p.H * p.H;
    stage_rows(img_s, Wp, src, p.H, strip * pitch - p.off, q0 * pitch - p.off, R, W);
  }
  for (int c = tid; c < Wp; c += nthr) img_s[R * Wp + c] = 0.f;
  __syncthreads();

  constexpr bool SPLIT = L >= 64;
  // pass 1: real rows, two per lane (row R is the zero row); pairs past the
  // window write zero rows, so pass 2 reads every row unconditionally
  if (SPLIT) {
    for (int task = tid; task < 2 * PAIRS * nq; task += nthr) {
      const int h = task & 1, base = task >> 1;
      const int q = base % nq, pr = base / nq;
      const int r0 = 2 * pr;
      float2* zt = zbuf + q * TS + r0 * V;
      if (r0 >= R) {
        for (int v = h; v < 2 * V; v += 2) zt[v] = make_float2(0.f, 0.f);
        continue;
      }
      const float* row_a = img_s + r0 * Wp + q * pitch;
      row_pair_split<L, ZH>(row_a, row_a + Wp, R, true, zt, h);
    }
  }
  for (int task = tid; task < (SPLIT ? 0 : PAIRS * nq); task += nthr) {
    const int q = task % nq, pr = task / nq;
    const int r0 = 2 * pr;
    float2* zt = zbuf + q * TS + r0 * V;
    if (r0 >= R) {
#pragma unroll
      for (int v = 0; v < 2 * V; ++v) zt[v] = make_float2(0.f, 0.f);
      continue;
    }
    const float* row_a = img_s + r0 * Wp + q * pitch;
    const float* row_b = row_a + Wp;
    float zr[L], zi[L];
#pragma unroll
    for (int s = 0; s < L; ++s) {
      if (s < S) {
        const float a = row_a[s], b = row_b[s];
        const bool in = s < R;
        zr[s] = in ? a : 0.f;
        zi[s] = in ? b : 0.f;
      } else {
        zr[s] = 0.f;
        zi[s] = 0.f;
      }
    }
    float2 X0[V], X1[V];
    rfft_pair<L, ZH>(zr, zi, X0, X1);
#pragma unroll
    for (int v = 0; v < V; ++v) {
      zt[v] = X0[v];
      zt[V + v] = X1[v];
    }
  }
  __syncthreads();

  // pass 2: complex columns, bin-major stores
  const size_t tiles_per_ch = size_t(p.n_img) * p.T * p.T;
  const size_t fstride = size_t(p.n_ch) * tiles_per_ch;
  const size_t ustride = size_t(V) * fstride;
  float2* out = p.dst + size_t(ch) * tiles_per_ch + size_t(img) * p.T * p.T + size_t(strip) * p.T + q0;
  if (SPLIT) {
    for (int task = tid; task < 2 * V * nq; task += nthr) {
      const int h = task & 1, base = task >> 1;
      const int q = base % nq, v = base / nq;
      column_split_store<L, ZH>(zbuf + q * TS + v, ROWS, out + size_t(v) * fstride + q, ustride, h);
    }
  }
  for (int task = tid; task < (SPLIT ? 0 : V * nq); task += nthr) {
    const int q = task % nq, v = task / nq;
    const float2* zt = zbuf + q * TS + v;
    float re[L], im[L];
#pragma unroll
    for (int r = 0; r < L; ++r) {
      if (r < ROWS) {
        const float2 z = zt[r * V];
        re[r] = z.x;
        im[r] = z.y;
      } else {
        re[r] = 0.f;
        im[r] = 0.f;
      }
    }
    fft_dif<L, -1, ZH>(re, im);
    float2* o = out + size_t(v) * fstride + q;
#pragma unroll
    for (int u = 0; u < L; ++u) {
      const int pos = bitrev(u, L);
      o[u * ustride] = make_float2(re[pos], im[pos]);
    }
  }
}

// ---------------------------------------------------------------------------
// Gradient windows: window (P, Q) is the S x S region of the framed plane
// (plane rows/cols shifted by -off) starting at (P n, Q n), n the window
// pitch and S <= 2n. A workgroup walks down the window rows [pb, pe) of one
// plane for a run of window columns. Consecutive window rows share input
// rows, so the input sits in a ring of 2n rows in LDS (framed row a in ring
// row a mod 2n) and only the n new rows are loaded per step, prefetched into
// registers while the current windows are transformed.
//
// LDS: ring [2n][Wp] floats, then zbuf [TQ][TS] float2 (row transforms,
// rows [0, ROWS)).
template <int L, bool ZH>
__global__ void __launch_bounds__(kMaxThreads, fft_waves<L>(OAA_WAVES_WINDOW)) window_rfft2_kernel(WindowParams p) {
  constexpr int V = L / 2 + 1;
  constexpr int ROWS = ZH ? L / 2 : L;
  constexpr int S = ZH ? L / 2 : L;
  constexpr int PAIRS = (ROWS + 1) / 2;
  constexpr int PF = L < 16 ? L : 16;
  extern __shared__ float smem[];
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int n = p.n, T = p.T, H = p.H, R = 2 * n, SW = p.S;
  const int TS = odd_at_least(2 * PAIRS * V);
  const unsigned wg = xcd_local_order(blockIdx.x, gridDim.x);
  const int chunk = int(wg % p.nchunk);
  const unsigned rest = wg / p.nchunk;
  const int grp = int(rest % p.ngroups);
  const unsigned plane = rest / p.ngroups;
  const int img = int(plane / p.n_ch), ch = int(plane % p.n_ch);
  const int q0 = chunk * p.TQ, nq = min(p.TQ, T - q0);
  const int pb = grp * p.SPW, pe = min(T, pb + p.SPW);
  const int W = (nq - 1) * n + SW;             // framed columns [q0 n, q0 n + W) the windows cover
  const int Wp = bank_stride((p.TQ - 1) * n + L);  // window reads stay inside the row
  float* ring = smem;                                                               // [2n][Wp]
  float2* zbuf = reinterpret_cast<float2*>(smem + even_floats(size_t(R) * Wp));  // [TQ][TS]
  const float* src = p.src + size_t(plane) * H * H;
  const size_t tiles_per_ch = size_t(p.n_img) * T * T;
  const size_t fstride = size_t(p.n_ch) * tiles_per_ch;
  const size_t ustride = size_t(V) * fstride;
  float2* out_base = p.dst + size_t(ch) * tiles_per_ch + size_t(img) * T * T + q0;
  const int col0 = q0 * n - p.off;

  // ring rows of window row pb: framed rows [pb n, pb n + 2n); clear the padding
  for (int i = tid; i < R * Wp; i += nthr) ring[i] = 0.f;
  __syncthreads();
  {
    const int a0 = pb * n, s0 = a0 % R;
    // rows a0 .. a0+2n-1 land in ring rows s0 .. (wrapping at 2n)
    stage_rows(ring + s0 * Wp, Wp, src, H, a0 - p.off, col0, R - s0, W);
    if (s0 > 0) stage_rows(ring, Wp, src, H, a0 + (R - s0) - p.off, col0, s0, W);
  }
  RowPrefetch<PF> pf;
  // (L = 64: the registers are worth more to the split transforms)
  const bool use_pf = L <= 32 && OAA_WINDOW_PREFETCH && RowPrefetch<PF>::fits(n, W);

  for (int P = pb; P < pe; ++P) {
    const int a0 = P * n;
    const int slot0 = a0 % R;
    __syncthreads();
    const bool next = P + 1 < pe;
    if (next && use_pf) pf.load(src, H, a0 + R - p.off, col0, n, W);
    // pass 1: window rows two at a time; pairs past the window write zero rows
    constexpr bool SPLIT = L >= 64;
    if (SPLIT) {
      for (int task = tid; task < 2 * PAIRS * nq; task += nthr) {
        const int h = task & 1, base = task >> 1;
        const int q = base % nq, pr = base / nq;
        const int r0 = 2 * pr;
        float2* zt = zbuf + q * TS + r0 * V;
        if (r0 >= SW) {
          for (int k = h; k < 2 * V; k += 2) zt[k] = make_float2(0.f, 0.f);
          continue;
        }
        int sa = slot0 + r0;
        if (sa >= R) sa -= R;
        int sb = sa + 1;
        if (sb >= R) sb -= R;
        row_pair_split<L, ZH>(ring + sa * Wp + q * n, ring + sb * Wp + q * n, SW, r0 + 1 < SW, zt, h);
      }
    }
    for (int task = tid; task < (SPLIT ? 0 : PAIRS * nq); task += nthr) {
      const int q = task % nq, pr = task / nq;
      const int r0 = 2 * pr;
      float2* zt = zbuf + q * TS + r0 * V;
      if (r0 >= SW) {
#pragma unroll
        for (int k = 0; k < 2 * V; ++k) zt[k] = make_float2(0.f, 0.f);
        continue;
      }
      const bool has_b = r0 + 1 < SW;  // row r0 + 1 inside the window
      int sa = slot0 + r0;
      if (sa >= R) sa -= R;
      int sb = sa + 1;
      if (sb >= R) sb -= R;
      const float* row_a = ring + sa * Wp + q * n;
      const float* row_b = ring + sb * Wp + q * n;
      float zr[L], zi[L];
#pragma unroll
      for (int s = 0; s < L; ++s) {
        if (s < S) {
          const float x0 = row_a[s], x1 = row_b[s];
          const bool in = s < SW;
          zr[s] = in ? x0 : 0.f;
          zi[s] = in && has_b ? x1 : 0.f;
        } else {
          zr[s] = 0.f;
          zi[s] = 0.f;
        }
      }
      float2 X0[V], X1[V];
      rfft_pair<L, ZH>(zr, zi, X0, X1);
#pragma unroll
      for (int k = 0; k < V; ++k) {
        zt[k] = X0[k];
        zt[V + k] = X1[k];
      }
    }
    __syncthreads();
    // the ring rows of framed rows [a0, a0 + n) (ring rows [slot0, slot0 + n),
    // slot0 being 0 or n) are free now: bring in framed rows [a0 + 2n, a0 + 3n)
    if (next) {
      if (use_pf)
        pf.store(ring + slot0 * Wp, Wp, n, W);
      else
        stage_rows(ring + slot0 * Wp, Wp, src, H, a0 + R - p.off, col0, n, W);
    }
    // pass 2: complex columns, bin-major stores of window row P
    float2* out = out_base + size_t(P) * T;
    if (SPLIT) {
      for (int task = tid; task < 2 * V * nq; task += nthr) {
        const int h = task & 1, base = task >> 1;
        const int q = base % nq, v = base / nq;
        column_split_store<L, ZH>(zbuf + q * TS + v, ROWS, out + size_t(v) * fstride + q, ustride, h);
      }
    }
    for (int task = tid; task < (SPLIT ? 0 : V * nq); task += nthr) {
      const int q = task % nq, v = task / nq;
      const float2* zt = zbuf + q * TS + v;
      float re[L], im[L];
#pragma unroll
      for (int r = 0; r < L; ++r) {
        if (r < ROWS) {
          const float2 z = zt[r * V];
          re[r] = z.x;
          im[r] = z.y;
        } else {
          re[r] = 0.f;
          im[r] = 0.f;
        }
      }
      fft_dif<L, -1, ZH>(re, im);
      float2* o = out + size_t(v) * fstride + q;
#pragma unroll
      for (int u = 0; u < L; ++u) {
        const int pos = bitrev(u, L);
        o[u * ustride] = make_float2(re[pos], im[pos]);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Windows -> spectra, several window rows per step (L <= 32).
//
// Windows of neighbouring window rows share S - n framed rows, and the row
// transform of a framed row is the same for every window containing it. A
// step transforms the (rw - 1) n + S framed rows of rw window rows once per
// window column, then runs the column transforms of all rw x nq windows.
// When a workgroup holds whole rows of T windows, the rw T windows of a step
// are consecutive tiles, and each spectrum bin is written as one run of rw T
// complex values (the launcher picks rw for runs of at least 16, 128 bytes).
//
// The row transforms read the plane from memory through a buffer resource
// over it (elements outside the plane read as zero, so the framing and the
// zero padding cost no branches); LDS holds only the transformed rows, and
// more workgroups share a CU. (Staging the rows in LDS first, with the next
// step's rows prefetched into registers, measured slower.)
//
// Transformed rows are stored packed, L/2 complex slots per row: slot 0 holds
// the two real bins v = 0 and v = L/2 as (re, im), slots 1 .. L/2-1 the bins
// in between. The column transform of slot 0 is one complex transform of the
// two real columns v = 0 and v = L/2, separated afterwards by symmetry; it
// stores their bins u <= L/2 only, since bins (L - u, v) of these columns
// are their conjugates and nothing reads them. Every lane then stores about
// L values.
//
// FULL: the window side is exactly L (L/2 under ZH), so no window entry
// needs masking.
//
// LDS: zbuf [TQ][TS] float2, TS >= NA L/2 odd, NA = (RW - 1) n + S_MAX
// rounded up to even.
template <int L, bool ZH, bool FULL>
__global__ void __launch_bounds__(kMaxThreads, 2) window_rows_rfft2_kernel(WindowParams p) {
  constexpr int V = L / 2 + 1;
  constexpr int HB = L / 2;                 // packed slots per transformed row
  constexpr int S_MAX = ZH ? L / 2 : L;     // window side bound the transforms assume
  extern __shared__ float smem[];
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int n = p.n, T = p.T, H = p.H, SW = p.S, RW = p.RW;
  const int NA = ((RW - 1) * n + S_MAX + 1) & ~1;
  const int TS = odd_at_least(NA * HB);
  const unsigned wg = xcd_local_order(blockIdx.x, gridDim.x);
  const int chunk = int(wg % p.nchunk);
  const unsigned rest = wg / p.nchunk;
  const int grp = int(rest % p.ngroups);
  const unsigned plane = rest / p.ngroups;
  const int img = int(plane / p.n_ch), ch = int(plane % p.n_ch);
  const int q0 = chunk * p.TQ, nq = min(p.TQ, T - q0);
  const int pb = grp * p.SPW, pe = min(T, pb + p.SPW);
  float2* zbuf = reinterpret_cast<float2*>(smem);  // [TQ][TS]
  const float* src = p.src + size_t(plane) * H * H;
  const __amdgpu_buffer_rsrc_t rs = buffer_resource(src, unsigned(H) * unsigned(H) * 4u);
  const size_t tiles_per_ch = size_t(p.n_img) * T * T;
  const size_t fstride = size_t(p.n_ch) * tiles_per_ch;
  float2* out_base = p.dst + size_t(ch) * tiles_per_ch + size_t(img) * T * T + q0;
  const int col0 = q0 * n - p.off;

  for (int P0 = pb; P0 < pe; P0 += RW) {
    const int rw = min(RW, pe - P0);
    // pass 1: the step's framed rows two at a time, plane rows prow0 + r0
    // and prow0 + r0 + 1, columns col0 + q n + s
    const int NR = (rw - 1) * n + SW, prow0 = P0 * n - p.off;
    for (int task = tid; task < ((NR + 1) / 2) * nq; task += nthr) {
      const int q = task % nq, r0 = 2 * (task / nq);
      const bool has_b = r0 + 1 < NR;
      const int ga = prow0 + r0, gc = col0 + q * n;
      float zr[L], zi[L];
#pragma unroll
      for (int s = 0; s < L; ++s) {
        if (s < S_MAX) {
          const bool cok = unsigned(gc + s) < unsigned(H) && (FULL || s < SW);
          const bool aok = cok && unsigned(ga) < unsigned(H);
          const bool bok = cok && has_b && unsigned(ga + 1) < unsigned(H);
          zr[s] = buffer_load_f1(rs, aok ? unsigned(ga * H + gc + s) * 4u : kOutOfRange);
          zi[s] = buffer_load_f1(rs, bok ? unsigned((ga + 1) * H + gc + s) * 4u : kOutOfRange);
        } else {
          zr[s] = 0.f;
          zi[s] = 0.f;
        }
      }
      float2 X0[V], X1[V];
      rfft_pair<L, ZH>(zr, zi, X0, X1);
      float2* zt = zbuf + q * TS + r0 * HB;
      zt[0] = make_float2(X0[0].x, X0[L / 2].x);
      zt[HB] = make_float2(X1[0].x, X1[L / 2].x);
#pragma unroll
      for (int k = 1; k < HB; ++k) {
        zt[k] = X0[k];
        zt[HB + k] = X1[k];
      }
    }
    __syncthreads();
    // pass 2: column transforms of the rw x nq windows; lanes run over the
    // window columns, then the window rows, so that a store instruction
    // covers consecutive tiles of one bin
    for (int task = tid; task < HB * rw * nq; task += nthr) {
      const int q = task % nq, r2 = task / nq;
      const int w = r2 % rw, k = r2 / rw;
      const float2* zt = zbuf + q * TS + (w * n) * HB + k;
      float re[L], im[L];
#pragma unroll
      for (int r = 0; r < L; ++r) {
        if (r < S_MAX) {
          const float2 z = zt[r * HB];
          const bool in = FULL || r < SW;
          re[r] = in ? z.x : 0.f;
          im[r] = in ? z.y : 0.f;
        } else {
          re[r] = 0.f;
          im[r] = 0.f;
        }
      }
      fft_dif<L, -1, ZH>(re, im);
      // bin (u, v) of this window at obase + u V fstride (wave-uniform) plus
      // the lane's byte offset (v fstride + w T + q) * 8, below V fstride * 8
      // < 2^32 (checked by the launcher)
      float2* obase = out_base + size_t(P0) * T;
      const unsigned lo = unsigned((size_t(k) * fstride + size_t(w) * T + q) * 8u);
      if (k == 0) {
        // Z = C0 + i C1 with C0, C1 the Hermitian spectra of columns 0, L/2:
        // C0[u] = (Z[u] + conj Z[-u]) / 2, C1[u] = (Z[u] - conj Z[-u]) / (2i)
        const unsigned lh = lo + unsigned(size_t(L / 2) * fstride * 8u);
        float2* bu = obase;
#pragma unroll
        for (int u = 0; u <= L / 2; ++u) {
          const int pu = bitrev(u, L), pm = bitrev((L - u) % L, L);
          const float ar = re[pu], ai = im[pu], br = re[pm], bi = im[pm];
          store_at(bu, lo, make_float2(0.5f * (ar + br), 0.5f * (ai - bi)));
          store_at(bu, lh, make_float2(0.5f * (ai + bi), 0.5f * (br - ar)));
          advance_uniform(bu, size_t(V) * fstride);
        }
      } else {
        float2* bu = obase;
#pragma unroll
        for (int u = 0; u < L; ++u) {
          const int pu = bitrev(u, L);
          store_at(bu, lo, make_float2(re[pu], im[pu]));
          advance_uniform(bu, size_t(V) * fstride);
        }
      }
    }
    __syncthreads();  // zbuf free for the next step
  }
}

// ---------------------------------------------------------------------------
// Inverse column pass shared by the inverse kernels: for the tiles at
// in[q], q < nq (bin f at in[q + f * fstride], plus nsplit - 1 partial sums
// spaced split_stride apart), transform every column v and keep rows
// [0, ROWS) at zbuf[q * TS + r * V + v].
// O32: bins addressed as 32-bit lane offsets (v fstride + q) * 8 from
// wave-uniform row bases (the caller checks V fstride * 8 < 2^32).
template <int L, int ROWS, bool O32>
__device__ __forceinline__ void inverse_columns(const float2* in, size_t fstride, int nsplit,
                                                size_t split_stride, int nq, int TS, float2* zbuf) {
  constexpr int V = L / 2 + 1;
  const size_t ustride = size_t(V) * fstride;
  for (int task = threadIdx.x; task < V * nq; task += blockDim.x) {
    const int q = task % nq, v = task / nq;
    const float2* col = in + q + size_t(v) * fstride;
    const unsigned lo = unsigned((size_t(v) * fstride + q) * 8u);
    float re[L], im[L];
    const float2* bu = in;
#pragma unroll
    for (int u = 0; u < L; ++u) {
      const float2 z = O32 ? load_at(bu, lo) : col[u * ustride];
      if (O32) advance_uniform(bu, ustride);
      re[u] = z.x;
      im[u] = z.y;
    }
    for (int s = 1; s < nsplit; ++s) {
      const float2* cs = col + s * split_stride;
      const float2* bs = in + s * split_stride;
#pragma unroll
      for (int u = 0; u < L; ++u) {
        const float2 z = O32 ? load_at(bs, lo) : cs[u * ustride];
        if (O32) advance_uniform(bs, ustride);
        re[u] += z.x;
        im[u] += z.y;
      }
    }
    // Columns v = 0 and v = L/2 hold no products in rows u > L/2: there the
    // column h is Hermitian, so with g = h on rows [0, L/2] (rows 0 and L/2
    // halved) and zero elsewhere, the inverse of h is 2 Re(inverse of g).
    const bool mir = v == 0 || v == L / 2;
#pragma unroll
    for (int u = 0; u < L; ++u) {
      if (u > L / 2) {
        re[u] = mir ? 0.f : re[u];
        im[u] = mir ? 0.f : im[u];
      } else if (u == 0 || u == L / 2) {
        re[u] *= mir ? 0.5f : 1.f;
        im[u] *= mir ? 0.5f : 1.f;
      }
    }
    fft_dif<L, +1, false>(re, im);
    const float rs = mir ? 2.f : 1.f, is = mir ? 0.f : 1.f;
    float2* zt = zbuf + q * TS + v;
#pragma unroll
    for (int r = 0; r < ROWS; ++r) {
      const int pos = bitrev(r, L);
      zt[r * V] = make_float2(re[pos] * rs, im[pos] * is);
    }
  }
}


// ---------------------------------------------------------------------------
// Inverse + top-left n x n crop, scattered to the blocks of the output planes.
// A workgroup takes TQ consecutive tiles of one channel (they may span block
// rows and images), so its spectrum reads are contiguous.
template <int L, bool FULL, bool O32>
__global__ void __launch_bounds__(kMaxThreads, fft_waves<L>(OAA_WAVES_CROP)) irfft2_crop_kernel(CropParams p) {
  constexpr int V = L / 2 + 1;
  constexpr int RT = FULL ? L : L / 2;  // rows kept from the column transforms (>= n)
  extern __shared__ float smem[];
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int n = p.n, H = p.H, org = p.origin;
  const int TS = odd_at_least((RT + 1) * V);
  const int OS = n | 1;  // obuf stride between tiles, odd
  float2* zbuf = reinterpret_cast<float2*>(smem);                   // [TQ][TS]
  float* obuf = smem + size_t(p.TQ) * TS * 2;                       // [n][TQ][OS]
  int* tbase = reinterpret_cast<int*>(obuf + size_t(n) * p.TQ * OS);  // [TQ] x 3
  const unsigned wg = xcd_local_order(blockIdx.x, gridDim.x);
  const int chunk = int(wg % p.nchunk);
  const int ch = int(wg / p.nchunk);
  const int P = p.T * p.T;
  const int tiles = p.n_img * P;
  const int t0 = chunk * p.TQ;
  const int nq = min(p.TQ, tiles - t0);
  const size_t fstride = size_t(p.n_ch) * tiles;
  // per tile: offset of its block in the output plane set, valid rows and columns
  for (int q = tid; q < nq; q += nthr) {
    const int t = t0 + q;
    const int img = t / P, pp = t - img * P;
    const int prow = pp / p.T, qcol = pp - prow * p.T;
    tbase[q] = prow * n * H + qcol * n;
    tbase[p.TQ + q] = img;
    tbase[2 * p.TQ + q] = (min(n, H - prow * n) << 16) | min(n, H - qcol * n);
  }
  constexpr bool SPLIT = L >= 64;
  const float scale = 1.0f / float(L * L);
  const int npair = (n + 1) >> 1;
  if (SPLIT) {
    constexpr int HL = L / 2;
    const float2* in = p.src + size_t(ch) * tiles + t0;
    const size_t ustride = size_t(V) * fstride;
    for (int task = tid; task < 2 * V * nq; task += nthr) {
      const int h = task & 1, base = task >> 1;
      const int q = base % nq, v = base / nq;
      const float2* col = in + q + size_t(v) * fstride;
      float re[HL], im[HL];
      column_inverse_split<L>(
          [&](int u) {
            float2 z = col[u * ustride];
            for (int sp = 1; sp < p.nsplit; ++sp) {
              const float2 t = col[sp * p.split_stride + u * ustride];
              z.x += t.x;
              z.y += t.y;
            }
            return z;
          },
          v == 0 || v == L / 2, re, im, h);
      const bool mir = v == 0 || v == L / 2;
      const float rs = mir ? 2.f : 1.f, is = mir ? 0.f : 1.f;
      float2* zt = zbuf + q * TS + v;
#pragma unroll
      for (int m = 0; m < HL; ++m) {
        const int r = 2 * m + h;
        if (r < RT) zt[r * V] = make_float2(re[bitrev(m, HL)] * rs, im[bitrev(m, HL)] * is);
      }
    }
    __syncthreads();
    for (int task = tid; task < 2 * npair * nq; task += nthr) {
      const int h = task & 1, base = task >> 1;
      const int q = base % nq, pr = base / nq;
      const int r0 = 2 * pr;
      const float2* za = zbuf + q * TS + ((org + r0) & (L - 1)) * V;
      const float2* zb = zbuf + q * TS + ((org + r0 + 1) & (L - 1)) * V;
      const bool has1 = r0 + 1 < n;
      float zr[HL], zi[HL];
      irfft_pair_split<L>([&](int v) { return za[v]; },
                          [&](int v) { return has1 ? zb[v] : make_float2(0.f, 0.f); }, zr, zi, h);
      float* o0 = obuf + (size_t(r0) * p.TQ + q) * OS;
      float* o1 = o0 + size_t(p.TQ) * OS;
#pragma unroll
      for (int m = 0; m < HL; ++m) {
        const int sx = (2 * m + h - org) & (L - 1);  // column 2m + h of the inverse
        if (sx < n) {
          o0[sx] = zr[bitrev(m, HL)] * scale;
          if (has1) o1[sx] = zi[bitrev(m, HL)] * scale;
        }
      }
    }
  } else {
    inverse_columns<L, RT, O32>(p.src + size_t(ch) * tiles + t0, fstride, p.nsplit, p.split_stride, nq, TS, zbuf);
  }
  __syncthreads();
  for (int task = tid; task < (SPLIT ? 0 : npair * nq); task += nthr) {
    const int q = task % nq, pr = task / nq;
    const int r0 = 2 * pr;
    const float2* za = zbuf + q * TS + ((org + r0) & (L - 1)) * V;
    const float2* zb = zbuf + q * TS + ((org + r0 + 1) & (L - 1)) * V;
    const bool has1 = r0 + 1 < n;
    float2 A[V], Bv[V];
#pragma unroll
    for (int v = 0; v < V; ++v) {
      A[v] = za[v];
      Bv[v] = has1 ? zb[v] : make_float2(0.f, 0.f);  // no row n for odd n
    }
    float zr[L], zi[L];
    irfft_pair<L>(A, Bv, zr, zi);
    float* o0 = obuf + (size_t(r0) * p.TQ + q) * OS;
    float* o1 = o0 + size_t(p.TQ) * OS;
#pragma unroll
    for (int s = 0; s < (FULL ? L : L / 2); ++s) {
      const int c = (s - org) & (L - 1);  // column s of the inverse is kept column c
      if (c < n) {
        const int pos = bitrev(s, L);
        o0[c] = zr[pos] * scale;
        if (has1) o1[c] = zi[pos] * scale;
      }
    }
  }
  __syncthreads();
  // row r of every tile, tiles in order: neighbouring tiles of a block row
  // are neighbours in the output row (n * nq * n < 2^16: launcher)
  const SmallDiv div_n(n), div_nq(nq);
  for (int e = tid; e < n * nq * n; e += nthr) {
    const int rest = div_n(e), s = e - rest * n;
    const int r = div_nq(rest), q = rest - r * nq;
    const int lim = tbase[2 * p.TQ + q];
    if (r < (lim >> 16) && s < (lim & 0xffff)) {
      float* o = p.dst + (size_t(tbase[p.TQ + q]) * p.n_ch + ch) * H * H;
      o[tbase[q] + r * H + s] = obuf[(size_t(r) * p.TQ + q) * OS + s];
    }
  }
}

// ---------------------------------------------------------------------------
// launchers

template <int L, bool ZH>
hipError_t launch_fwd_L(TileFwdParams p, hipStream_t s) {
  constexpr int V = L / 2 + 1;
  constexpr int ROWS = ZH ? L / 2 : L;
  constexpr int PAIRS = (ROWS + 1) / 2;
  const int TS = odd_at_least(2 * PAIRS * V);
  auto lds_for = [&](int tq) {
    const size_t Wp = size_t(bank_stride((tq - 1) * p.pitch + p.R + L));
    return even_floats(size_t(p.R + 1) * Wp) * 4 + size_t(TS) * tq * 8;
  };
  // tiles along a row: a block row of T tiles, or (gather) the n_img kernels
  const int run = p.gather ? p.n_img : p.T;
  const int tq_max = p.gather ? 16 : OAA_FWD_TQ_MAX;  // 16 kernels: 128-byte spectrum stores
  int nchunk = (run + tq_max - 1) / tq_max;
  while (nchunk < run && lds_for((run + nchunk - 1) / nchunk) > kLdsBudget) ++nchunk;
  p.TQ = (run + nchunk - 1) / nchunk;
  p.nchunk = (run + p.TQ - 1) / p.TQ;
  const size_t lds = lds_for(p.TQ);
  if (lds > kLdsBudget) return hipErrorInvalidConfiguration;
  const int tasks = (L >= 64 ? 2 : 1) * std::max(PAIRS * p.TQ, V * p.TQ);
  const long nwg = p.gather ? long(p.n_ch) * p.nchunk : long(p.n_img) * p.n_ch * p.T * p.nchunk;
  hipLaunchKernelGGL((tile_rfft2_kernel<L, ZH>), dim3(unsigned(nwg)), dim3(pick_threads(tasks)), lds, s, p);
  return hipGetLastError();
}

template <int L, bool ZH>
hipError_t launch_window_L(WindowParams p, hipStream_t s) {
  constexpr int V = L / 2 + 1;
  constexpr int ROWS = ZH ? L / 2 : L;
  constexpr int PAIRS = (ROWS + 1) / 2;
  const long planes = long(p.n_img) * p.n_ch;
  // 32-bit lane offsets: within a plane, and within one row u of the bins
  const size_t fstride = size_t(p.n_ch) * p.n_img * p.T * p.T;
  if constexpr (L <= 32) if (OAA_WINDOW_ROWS && size_t(p.H) * p.H * 4 < (size_t(1) << 31) &&
      size_t(V) * fstride * 8 < (size_t(1) << 32)) {
    // whole rows of windows per workgroup, rw of them per step so that a
    // step's windows make runs of at least 16 tiles, within the LDS limit
    constexpr int HB = L / 2;
    auto lds_rows = [&](int tq, int rw) {
      const int na = ((rw - 1) * p.n + ROWS + 1) & ~1;
      return size_t(odd_at_least(na * HB)) * tq * 8;
    };
    int nchunk = (p.T + OAA_WINDOW_TQ_MAX - 1) / OAA_WINDOW_TQ_MAX;
    while (nchunk < p.T && lds_rows((p.T + nchunk - 1) / nchunk, 1) > kLdsRowsBudget) ++nchunk;
    p.TQ = (p.T + nchunk - 1) / nchunk;
    p.nchunk = (p.T + p.TQ - 1) / p.TQ;
    // window rows per step: the fewest whose run of rw T tiles is a multiple
    // of 16 (whole 128-byte lines, e.g. two rows of 8), else as many as lengthen
    // the run towards OAA_WINDOW_MIN_RUN, while the LDS of a workgroup stays
    // within OAA_WINDOW_GROW_LDS
    int rw = 1;
    if (p.nchunk == 1) {
      int ra = 0;
      for (int r = 1; r <= p.T && r * p.T <= 64 && !ra; ++r)
        if ((r * p.T) % 16 == 0) ra = r;
      if (ra && lds_rows(p.TQ, ra) <= OAA_WINDOW_GROW_LDS)
        rw = ra;
      else
        while (rw * p.T < OAA_WINDOW_MIN_RUN && rw < p.T && lds_rows(p.TQ, rw + 1) <= OAA_WINDOW_GROW_LDS) ++rw;
    }
    p.RW = rw;
    const size_t lds = lds_rows(p.TQ, rw);
    if (lds > kLdsRowsBudget) return hipErrorInvalidConfiguration;
    int ng = 1;
    if (planes < 2048) ng = int(std::min<long>((p.T + rw - 1) / rw, (2048 + planes - 1) / planes));
    p.SPW = ((p.T + ng - 1) / ng + rw - 1) / rw * rw;
    p.ngroups = (p.T + p.SPW - 1) / p.SPW;
    const int na = ((rw - 1) * p.n + ROWS + 1) & ~1;
    const int nthr = pick_threads(std::max(na / 2 * p.TQ, HB * rw * p.TQ));
    auto kern = p.S == ROWS ? window_rows_rfft2_kernel<L, ZH, true> : window_rows_rfft2_kernel<L, ZH, false>;
    const hipError_t e = allow_lds(kern, kLdsRowsBudget);
    if (e != hipSuccess) return e;
    const long nwg = planes * p.ngroups * p.nchunk;
    hipLaunchKernelGGL(kern, dim3(unsigned(nwg)), dim3(nthr), lds, s, p);
    return hipGetLastError();
  }
  const int TS = odd_at_least(2 * PAIRS * V);
  auto lds_for = [&](int tq) {
    const size_t Wp = size_t(bank_stride((tq - 1) * p.n + L));
    return even_floats(size_t(2 * p.n) * Wp) * 4 + size_t(TS) * tq * 8;
  };
  int nchunk = (p.T + OAA_WINDOW_TQ_MAX - 1) / OAA_WINDOW_TQ_MAX;
  while (nchunk < p.T && lds_for((p.T + nchunk - 1) / nchunk) > kLdsBudget) ++nchunk;
  p.TQ = (p.T + nchunk - 1) / nchunk;
  p.nchunk = (p.T + p.TQ - 1) / p.TQ;
  p.RW = 1;
  const size_t lds = lds_for(p.TQ);
  if (lds > kLdsBudget) return hipErrorInvalidConfiguration;
  int ng = 1;
  if (planes < 2048) ng = int(std::min<long>(p.T, (2048 + planes - 1) / planes));
  p.SPW = (p.T + ng - 1) / ng;
  p.ngroups = (p.T + p.SPW - 1) / p.SPW;
  const int tasks = (L >= 64 ? 2 : 1) * std::max(PAIRS * p.TQ, V * p.TQ);
  const long nwg = planes * p.ngroups * p.nchunk;
  hipLaunchKernelGGL((window_rfft2_kernel<L, ZH>), dim3(unsigned(nwg)), dim3(pick_threads(tasks)), lds, s, p);
  return hipGetLastError();
}

template <int L, bool FULL>
hipError_t launch_crop_LF(CropParams p, hipStream_t s) {
  constexpr int V = L / 2 + 1;
  constexpr int RT = FULL ? L : L / 2;
  const int TS = odd_at_least((RT + 1) * V);
  // column transforms, output block and three tile descriptors per tile
  const size_t per_tile = size_t(TS) * 8 + size_t(p.n) * (p.n | 1) * 4 + 3 * 4;
  const long tiles = long(p.n_img) * p.T * p.T;
  // runs of consecutive tiles (128-byte reads) within OAA_CROP_LDS bytes of
  // LDS, so that several workgroups share a CU (fewer, longer runs measured
  // slower), shortened to keep about 2048 workgroups when there are few tiles
  // (the weight gradient)
  long tq = std::min<long>(long(std::min<size_t>(kLdsBudget, OAA_CROP_LDS) / per_tile), OAA_CROP_TQ_MAX);
  if (tq < 1) tq = 1;
  const long want = (long(p.n_ch) * tiles + 2047) / 2048;
  if (want < tq) tq = std::max<long>(want, 1);
  if (tq > tiles) tq = tiles;
  if (long(p.n) * p.n * tq >= 65536) tq = std::max<long>(1, 65535 / (long(p.n) * p.n));
  const long nchunk = (tiles + tq - 1) / tq;
  p.TQ = int((tiles + nchunk - 1) / nchunk);
  p.nchunk = int(nchunk);
  const size_t lds = per_tile * p.TQ;
  const int tasks = (L >= 64 ? 2 : 1) * std::max(V * p.TQ, ((p.n + 1) / 2) * p.TQ);
  const long nwg = long(p.n_ch) * p.nchunk;
  const bool o32 = OAA_CROP_O32 && size_t(V) * size_t(p.n_ch) * p.n_img * p.T * p.T * 8 < (size_t(1) << 32);
  auto kern = o32 ? irfft2_crop_kernel<L, FULL, true> : irfft2_crop_kernel<L, FULL, false>;
  hipLaunchKernelGGL(kern, dim3(unsigned(nwg)), dim3(pick_threads(tasks)), lds, s, p);
  return hipGetLastError();
}

// blocks of more than L/2 rows need every row of the column transforms
template <int L>
hipError_t launch_crop_L(const CropParams& p, hipStream_t s) {
  if (p.origin < 0 || p.origin >= L || p.n > L) return hipErrorInvalidValue;
  // the kept rows [origin, origin + n) (mod L) within the first half, or all rows
  if (p.origin + p.n > L / 2) return launch_crop_LF<L, true>(p, s);
  return launch_crop_LF<L, false>(p, s);
}

}  // namespace

hipError_t launch_tile_rfft2(int L, const TileFwdParams& p, hipStream_t s) {
  const bool zh = 2 * p.R <= L;
  switch (L) {
    case 2: return zh ? launch_fwd_L<2, true>(p, s) : launch_fwd_L<2, false>(p, s);
    case 4: return zh ? launch_fwd_L<4, true>(p, s) : launch_fwd_L<4, false>(p, s);
    case 8: return zh ? launch_fwd_L<8, true>(p, s) : launch_fwd_L<8, false>(p, s);
    case 16: return zh ? launch_fwd_L<16, true>(p, s) : launch_fwd_L<16, false>(p, s);
    case 32: return zh ? launch_fwd_L<32, true>(p, s) : launch_fwd_L<32, false>(p, s);
    case 64: return zh ? launch_fwd_L<64, true>(p, s) : launch_fwd_L<64, false>(p, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_window_rfft2(int L, const WindowParams& p, hipStream_t s) {
  if (p.S > 2 * p.n || p.S > L || p.S < 1) return hipErrorInvalidValue;
  const bool zh = 2 * p.S <= L;
  switch (L) {
    case 2: return zh ? launch_window_L<2, true>(p, s) : launch_window_L<2, false>(p, s);
    case 4: return zh ? launch_window_L<4, true>(p, s) : launch_window_L<4, false>(p, s);
    case 8: return zh ? launch_window_L<8, true>(p, s) : launch_window_L<8, false>(p, s);
    case 16: return zh ? launch_window_L<16, true>(p, s) : launch_window_L<16, false>(p, s);
    case 32: return zh ? launch_window_L<32, true>(p, s) : launch_window_L<32, false>(p, s);
    case 64: return zh ? launch_window_L<64, true>(p, s) : launch_window_L<64, false>(p, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_irfft2_crop(int L, const CropParams& p, hipStream_t s) {
  switch (L) {
    case 2: return launch_crop_L<2>(p, s);
    case 4: return launch_crop_L<4>(p, s);
    case 8: return launch_crop_L<8>(p, s);
    case 16: return launch_crop_L<16>(p, s);
    case 32: return launch_crop_L<32>(p, s);
    case 64: return launch_crop_L<64>(p, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace oaa
