// Transforms of side L = 64 and 128 (arXiv:1601.06815, Section 2: block
// division, zero padding, the per-block transforms and the overlap-add of the
// block results; Section 3.3 for the transform sides of large kernels), as
// used for large blocks (b up to L - n + 1) and large kernels.
//
// A workgroup keeps the intermediate of TQ tiles in LDS (17 KB per tile at
// L = 64, so one workgroup of up to nine tiles per CU) and walks over groups
// of TQ consecutive tiles of one channel:
//  * forward: pass 1 transforms the column pairs (s, s + L/2) of every window
//    along its rows, lanes over consecutive columns so that the loads of a
//    row are coalesced, and keeps rows u <= L/2 of the two real columns'
//    spectra (rows past L/2 are their conjugates); pass 2 transforms each of
//    those rows along the columns and writes bins (u, v) and (L - u, v) of
//    the half spectrum with lanes over the group's tiles, so that a store
//    instruction writes runs of TQ consecutive tiles of a bin. Consecutive
//    groups run on one XCD at about the same time, so the runs that
//    neighbouring groups write into a bin meet in that XCD's L2;
//  * inverse: pass 1 inverts the columns v <= L/2 (loads in runs of TQ
//    tiles), pass 2 inverts row pairs to real rows, pass 3 writes the kept
//    part of each tile (crop) or the overlap-added plane. At L = 64 teams of
//    workgroups of one XCD take neighbouring groups together, each team
//    walking a contiguous range, so that the 128-byte lines that those
//    groups' runs share come from HBM once; at L = 128 a workgroup walks a
//    contiguous range of groups.
// At L = 64 a lane holds a whole 64-point sequence, and the two halves of the
// workgroup alternate between transforming a group and loading the next into
// their registers (big_rfft2_lane_kernel, big_irfft2_lane_kernel). At
// L = 128, and for forward launches of few groups, each L-point transform is
// split over a pair of neighbouring lanes (fft_dif_split, L/2 complex values
// per lane) and the whole workgroup transforms a group; the forward loads the
// next group into registers while the current group's second pass runs.
#include <algorithm>
#include <type_traits>

#include "fft_core.hpp"
#include "oaa_internal.hpp"
#include "tile_common.hpp"

namespace oaa {

namespace {

using namespace tile;

constexpr size_t kBigLds = 160 * 1024;  // LDS of one CU

// Tiles per group at L = 64 (overridable at build time for tuning sweeps).
#ifndef OAA_BIG_TQ
#define OAA_BIG_TQ 8
#endif

template <int L>
struct Big {
  static constexpr int H2 = L / 2, V = L / 2 + 1;
  // forward LDS row stride (complex): columns [0, L/2) then, one slot on,
  // columns [L/2, L)
  static constexpr int RS = L + 2;
  // inverse LDS row stride (complex): L/2 slots, slot 0 holding the real
  // columns 0 and L/2 as (re, im), plus one slot of padding
  static constexpr int RI = H2 + 1;
  static constexpr int TQ_MAX = L == 64 ? 9 : 2;  // tiles per group (LDS)
  static constexpr int SIDE_MAX = L == 64 ? 3 : 1;  // blocks per side of a one-group plane
};

// threads of a lane-pair forward workgroup: eight waves, which leaves a lane
// 256 registers; L per tile, one task per thread with the register prefetch,
// else threads loop over the tasks
template <int L, bool PF>
constexpr int big_threads() {
  return 512;
}
// threads of an inverse workgroup: eight waves (a lane's registers capped
// at 256)
constexpr int kBigInvThreads = 512;

// LDS per tile (complex elements, odd)
template <int L>
__host__ __device__ inline int fwd_tile_stride() {
  return odd_at_least(Big<L>::H2 * Big<L>::RS);
}
template <int L>
__host__ __device__ inline int inv_tile_stride(int KR) {
  return odd_at_least(KR * Big<L>::RI);
}
// LDS per tile of the one-lane L = 64 kernels (complex elements): the 32 x 66
// (forward) or 64 x 33 (inverse) slots, padded to 3 mod 32, so that tile
// bases fall 6 four-byte banks apart. A wave's lanes over (tile, LDS row) in
// the forward's second pass, and over (tile, column) or (tile, row pair) in
// the inverse's passes, then spread over the banks; at the odd stride 1 mod
// 32, neighbouring tiles fell 2 banks apart, on the banks of the next row or
// column (measured at the large-kernel layer: forward inverse 0.621 ->
// 0.615 ms).
__host__ __device__ constexpr int lane_tile_stride() {
  constexpr int n = 64 * Big<64>::RI;
  static_assert(n == 32 * Big<64>::RS, "both directions hold 2112 complex per tile");
  return n + ((3 - n % 32) + 32) % 32;
}

// first group of this workgroup; groups advance by gridDim.x (a multiple of
// 8), and the workgroups of one XCD take consecutive groups
__device__ __forceinline__ long first_group() {
  const unsigned nwg = gridDim.x;
  return long(blockIdx.x % 8) * (nwg / 8) + blockIdx.x / 8;
}

// The groups a workgroup takes: g, g + step, ... below end. Interleaved
// (consecutive groups on the workgroups of one XCD at about the same time)
// or, with `contig`, a contiguous range per workgroup (the workgroups of one
// XCD holding consecutive ranges). The forward transforms walk interleaved;
// the L = 128 inverse walks contiguous ranges (at L = 64 that was 0.99 ->
// 0.93 ms against interleaved for the large-kernel forward inverse).
struct GroupWalk {
  long g, end, step;
};
__device__ __forceinline__ GroupWalk group_walk(long ngroups, bool contig) {
  const long w = first_group();
  if (contig) {
    const long nwg = gridDim.x, R = (ngroups + nwg - 1) / nwg;
    return {w * R, min(ngroups, (w + 1) * R), 1};
  }
  return {w, ngroups, long(gridDim.x)};
}

// Teams of S workgroups of one XCD (consecutive first_group numbers; nwg is
// a multiple of 8 S, else S is 1) take S consecutive groups at a time, and
// each team walks a contiguous range. The runs of S neighbouring groups in a
// bin share 128-byte lines, which the first of them to read one brings into
// the XCD's L2 for the others, read at about the same time. A line shared by
// groups a workgroup takes one after the other is gone from L2 by the next
// group (a workgroup's group reads 2050 bins), so a contiguous walk with S = 1
// reads each such line again. A team of a whole XCD on one channel at a time
// (S = 32, like the interleaved walk) crowds all XCDs onto a few channels'
// bins and was slower. Measured at the large-kernel layer (groups of one
// nine-tile plane in the forward overlap-add, of 8 tiles = 64 bytes in the
// crops): forward inverse 0.675 / 0.625 / 0.622 / 0.694 ms at S = 1, 4, 8,
// 16; the crops 0.224 -> 0.217 and 0.151 -> 0.142 ms at S = 2, where a pair
// of groups covers one line.
__device__ __forceinline__ GroupWalk group_walk_team(long ngroups, int S0) {
  const long w = first_group(), nwg = gridDim.x;
  const long S = nwg % (8 * S0) == 0 ? S0 : 1;
  const long R = (ngroups + nwg - 1) / nwg, team = w / S, s = w % S;
  return {team * R * S + s, min(ngroups, (team + 1) * R * S), S};
}

// ---------------------------------------------------------------------------
// forward: windows of planes -> half spectra
//
// Pass 1: z = x[., j] + i x[., j + L/2] along the rows; the real columns'
// spectra are C_j[u] = (Z[u] + conj Z[-u]) / 2, C_{j+L/2}[u] =
// (Z[u] - conj Z[-u]) / (2i), Hermitian in u, so rows u <= L/2 suffice; rows
// 0 and L/2 are real and share LDS row 0 as (re, im). Pass 2: rows u in
// [1, L/2) along the columns give bins (u, v), v <= L/2, and (L - u, v) =
// conj X[u][L - v], 0 < v < L/2 (the other bins of rows past L/2 are
// conjugates that nothing reads); the packed row gives rows 0 and L/2 by the
// same separation as pass 1.
template <int L, bool O32, bool PF>
__global__ void __launch_bounds__((big_threads<L, PF>())) big_rfft2_kernel(BigFwdParams p) {
  constexpr int H2 = Big<L>::H2, V = Big<L>::V, RS = Big<L>::RS;
  static_assert(L >= 64, "the pass-1 lanes of one tile must fill whole waves");
  extern __shared__ float smem[];
  float2* lds = reinterpret_cast<float2*>(smem);
  const int TSZ = fwd_tile_stride<L>();
  const int tid = threadIdx.x, h = tid & 1;
  const int P = p.T * p.T, tpc = p.n_img * P;
  const size_t bs = p.bs;
  const long ngroups = long(p.n_ch) * p.ngrp;
  // pass 1: tile q1, columns j and j + L/2, rows [h L/2, h L/2 + L/2); a
  // wave holds one tile (lane = h + 2 (j + (L/2) q1))
  const int j = (tid >> 1) % H2, q1 = (tid >> 1) / H2;
  // pass 2: tile q2 (fastest), LDS row u
  const int q2 = (tid >> 1) % p.TQ, u = (tid >> 1) / p.TQ;
  float zr[H2], zi[H2];

  // part 0: columns j (zr), 1: columns j + L/2 (zi), 2: both
  auto load = [&](long gg, int part) {
    const int ch = int(gg / p.ngrp), t0 = int(gg % p.ngrp) * p.TQ;
    const int nq = min(p.TQ, tpc - t0);
    if (q1 >= nq) return;
    const int t = t0 + q1, img = t / P, pp = t - img * P;
    const int pr = pp / p.T, qc = pp - pr * p.T;
    const float* plane = p.src + (size_t(img) * p.n_ch + ch) * size_t(p.H) * size_t(p.H);
    const __amdgpu_buffer_rsrc_t rs = buffer_resource(plane, unsigned(p.H) * unsigned(p.H) * 4u);
    const int gr0 = pr * p.pitch - p.off + h * H2;
    const int ca = qc * p.pitch - p.off + j, cb = ca + H2;
    const bool oka = j < p.S && unsigned(ca) < unsigned(p.H);
    const bool okb = j + H2 < p.S && unsigned(cb) < unsigned(p.H);
    const int lim = p.S - h * H2;  // rows of this half inside the window
#pragma unroll
    for (int i = 0; i < H2; ++i) {
      const int gr = gr0 + i;
      const bool okr = i < lim && unsigned(gr) < unsigned(p.H);
      if (part != 1) zr[i] = buffer_load_f1(rs, okr && oka ? unsigned(gr * p.H + ca) * 4u : kOutOfRange);
      if (part != 0) zi[i] = buffer_load_f1(rs, okr && okb ? unsigned(gr * p.H + cb) * 4u : kOutOfRange);
    }
  };

  const GroupWalk wk = group_walk(ngroups, false);
  long g = wk.g;
  if (PF && g < wk.end) load(g, 2);
  for (; g < wk.end; g += wk.step) {
    const int ch = int(g / p.ngrp), t0 = int(g % p.ngrp) * p.TQ;
    const int nq = min(p.TQ, tpc - t0);
    if (!PF) load(g, 2);
    if (q1 < nq) {
      fft_dif_split<L, -1>(zr, zi, h);  // lane h: Z[2m + h] at bitrev(m)
      float2* bq = lds + q1 * TSZ;
#pragma unroll
      for (int m = 1; m < H2 / 2; ++m) {  // u = 2m + h in [2, L/2), with u = 1 below
        const int uu = 2 * m + h;
        const int ps = bitrev(m, H2);
        const int p0 = bitrev(H2 - m, H2), p1 = bitrev(H2 - m - 1, H2);  // -uu for h = 0, 1
        const float a = zr[ps], b = zi[ps];
        const float c = pick(h, zr[p1], zr[p0]), d = pick(h, zi[p1], zi[p0]);
        bq[uu * RS + j] = make_float2(0.5f * (a + c), 0.5f * (b - d));
        bq[uu * RS + H2 + 1 + j] = make_float2(0.5f * (b + d), 0.5f * (c - a));
      }
      // m = 0: u = 0 (lane 0) and u = 1 (lane 1, partner L - 1 at m = L/2 - 1);
      // lane 0 also holds u = L/2 at m = L/4
      const float a0 = zr[0], b0 = zi[0];
      if (h) {
        const int pl = bitrev(H2 - 1, H2);
        const float c = zr[pl], d = zi[pl];
        bq[RS + j] = make_float2(0.5f * (a0 + c), 0.5f * (b0 - d));
        bq[RS + H2 + 1 + j] = make_float2(0.5f * (b0 + d), 0.5f * (c - a0));
      } else {
        const int ph = bitrev(H2 / 2, H2);
        bq[j] = make_float2(a0, zr[ph]);
        bq[H2 + 1 + j] = make_float2(b0, zi[ph]);
      }
    }
    // The next group's windows load during pass 2, in two halves: a lane's
    // 64 loads exceed the 63 vector memory instructions a wave can have in
    // flight, and issued at once they stall the wave (and queue this pass's
    // stores behind them). Half goes out before the barrier, half after it
    // (measured at the large-kernel layer, gradient windows: all 64 after
    // the barrier 0.69 ms, all before it 0.66 ms, split 0.56 ms).
    const bool nxt = PF && g + wk.step < wk.end;
    if (nxt) load(g + wk.step, 0);
    __syncthreads();
    if (nxt) load(g + wk.step, 1);
    if (q2 < nq && u < H2) {
      const float2* row = lds + q2 * TSZ + u * RS + h * (H2 + 1);
      float re[H2], im[H2];
#pragma unroll
      for (int i = 0; i < H2; ++i) {
        const float2 z = row[i];
        re[i] = z.x;
        im[i] = z.y;
      }
      fft_dif_split<L, -1>(re, im, h);  // lane h: Y[2m + h] at bitrev(m)
      const int t = t0 + q2;
      const size_t tb = size_t(ch) * p.cs + size_t(t / p.run) * p.rs + size_t(t % p.run);
      // bins (r, v) for v = 2m + h: element (r V + h) bs + tb + m (2 bs)
      auto put = [&](int r, int m, float2 val) {
        if (O32) {
          store_at(p.dst, unsigned(((size_t(r) * V + h) * bs + tb) * 8u) + unsigned(m) * unsigned(2 * bs * 8u), val);
        } else {
          p.dst[(size_t(r) * V + h) * bs + tb + size_t(2 * m) * bs] = val;
        }
      };
      if (u > 0) {
#pragma unroll
        for (int m = 0; m <= H2 / 2; ++m) {
          const int v = 2 * m + h, ps = bitrev(m, H2);
          if (v <= H2) put(u, m, make_float2(re[ps], im[ps]));
          if (v >= 1 && v < H2) {
            const int q0i = bitrev((H2 - m) % H2, H2), q1i = bitrev(H2 - m - 1, H2);
            const float xr = pick(h, re[q1i], re[q0i]), xi = pick(h, im[q1i], im[q0i]);
            put(L - u, m, make_float2(xr, -xi));
          }
        }
      } else {
        // packed row: Y = X[0] + i X[L/2] (both Hermitian in v)
#pragma unroll
        for (int m = 0; m <= H2 / 2; ++m) {
          const int v = 2 * m + h, ps = bitrev(m, H2);
          if (v > H2) continue;
          const int q0i = bitrev((H2 - m) % H2, H2), q1i = bitrev((H2 - m - 1 + H2) % H2, H2);
          const float a = re[ps], b = im[ps];
          const float c = pick(h, re[q1i], re[q0i]), d = pick(h, im[q1i], im[q0i]);
          put(0, m, make_float2(0.5f * (a + c), 0.5f * (b - d)));
          put(H2, m, make_float2(0.5f * (b + d), 0.5f * (c - a)));
        }
      }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// forward at L = 64 with a whole 64-point sequence per lane: a lane
// transforms one column pair (j, j + L/2) of a window along its rows (pass
// 1), then one LDS row along the columns (pass 2). The separations, the LDS
// layout and the bins written are those of the kernel above; without the
// first stage across a lane pair a transform takes about 0.7 of the vector
// instructions. The 32 tasks per tile and pass of a group of eight tiles fill
// four waves, half the workgroup, and the halves alternate: while one
// transforms group i, the other loads the windows of group i + 1 into its
// registers, so the loads have a whole group's passes to arrive. A half's
// pass 2 works in the registers that held its windows.
//
// A wave holds the column pairs of two tiles, possibly of two images, and a
// buffer resource must be the same for the whole wave: the window rows come
// through one resource per group, over the planes of channel ch of the
// group's images. WIDE: spans of the planes or spectra past 32-bit offsets,
// through 64-bit addresses.
template <bool WIDE>
__global__ void __launch_bounds__(512) big_rfft2_lane_kernel(BigFwdParams p) {
  constexpr int L = 64, H2 = L / 2, V = L / 2 + 1, RS = Big<L>::RS;
  extern __shared__ float smem[];
  float2* lds = reinterpret_cast<float2*>(smem);
  const int TSZ = lane_tile_stride();
  const int tid = threadIdx.x, TQ = p.TQ;
  const int half = tid >> 8, ht = tid & 255;  // half of the workgroup (four waves), thread in it
  const int P = p.T * p.T, tpc = p.n_img * P;
  const size_t bs = p.bs;
  const long ngroups = long(p.n_ch) * p.ngrp;
  const size_t HH = size_t(p.H) * p.H, istride = size_t(p.n_ch) * HH;  // floats per plane, per image
  // this thread's tasks: pass 1 tile q1, column pair j (lanes over consecutive
  // columns: coalesced window rows); pass 2 tile q2, LDS row u (lanes over
  // the tiles: runs of consecutive tiles of a bin)
  const int q1 = ht / H2, j = ht % H2, q2 = ht % TQ, u = ht / TQ;
  float zr[L], zi[L];

  // the windows of group g: columns j and j + L/2 of tile q1 as
  // z = x[., j] + i x[., j + L/2]
  auto fetch = [&](long g) {
    const int ch = int(g / p.ngrp), t0 = int(g % p.ngrp) * TQ;
    const int nq = min(TQ, tpc - t0);
    if (q1 >= nq) return;
    const int img0 = t0 / P, img1 = (t0 + nq - 1) / P;
    const float* base = p.src + (size_t(img0) * p.n_ch + ch) * HH;
    const __amdgpu_buffer_rsrc_t rs =
        buffer_resource(base, WIDE ? 0u : unsigned((size_t(img1 - img0) * istride + HH) * 4));
    const int t = t0 + q1, img = t / P, pp = t - img * P;
    const int pr = pp / p.T, qc = pp - pr * p.T;
    const int gr0 = pr * p.pitch - p.off;
    const int ca = qc * p.pitch - p.off + j, cb = ca + H2;
    const bool oka = j < p.S && unsigned(ca) < unsigned(p.H);
    const bool okb = j + H2 < p.S && unsigned(cb) < unsigned(p.H);
    const unsigned pb = unsigned(size_t(img - img0) * istride);  // this tile's plane in rs (elements)
    const float* plane = p.src + (size_t(img) * p.n_ch + ch) * HH;
#pragma unroll
    for (int i = 0; i < L; ++i) {
      const int gr = gr0 + i;
      const bool okr = i < p.S && unsigned(gr) < unsigned(p.H);
      if (WIDE) {
        zr[i] = okr && oka ? plane[size_t(gr) * p.H + ca] : 0.f;
        zi[i] = okr && okb ? plane[size_t(gr) * p.H + cb] : 0.f;
      } else {
        zr[i] = buffer_load_f1(rs, okr && oka ? (pb + unsigned(gr * p.H + ca)) * 4u : kOutOfRange);
        zi[i] = buffer_load_f1(rs, okr && okb ? (pb + unsigned(gr * p.H + cb)) * 4u : kOutOfRange);
      }
    }
  };
  // pass 1 on the fetched windows: the real columns' spectra
  // C_j[u] = (Z[u] + conj Z[L - u]) / 2, C_{j+L/2}[u] = (Z[u] - conj Z[L - u]) / (2i),
  // rows u <= L/2; rows 0 and L/2 (real) share LDS row 0 as (re, im)
  auto columns = [&]() {
    fft_dif<L, -1, false>(zr, zi);  // Z[k] at position bitrev(k)
    float2* bq = lds + (q1 * TSZ + j);
#pragma unroll
    for (int v = 1; v < H2; ++v) {
      const float a = zr[bitrev(v, L)], b = zi[bitrev(v, L)];
      const float c = zr[bitrev(L - v, L)], d = zi[bitrev(L - v, L)];
      bq[v * RS] = make_float2(0.5f * (a + c), 0.5f * (b - d));
      bq[v * RS + H2 + 1] = make_float2(0.5f * (b + d), 0.5f * (c - a));
    }
    bq[0] = make_float2(zr[0], zr[bitrev(H2, L)]);
    bq[H2 + 1] = make_float2(zi[0], zi[bitrev(H2, L)]);
  };
  // pass 2: LDS row u of tile q2 along the columns; bins (u, v), v <= L/2,
  // and (L - u, v) = conj X[u][L - v], 0 < v < L/2; the packed row 0 gives
  // rows 0 and L/2 by the separation of pass 1
  auto row = [&](int ch, int t0) {
    const float2* zrow = lds + (q2 * TSZ + u * RS);
#pragma unroll
    for (int c = 0; c < H2; ++c) {
      const float2 a = zrow[c], b = zrow[H2 + 1 + c];
      zr[c] = a.x;
      zi[c] = a.y;
      zr[H2 + c] = b.x;
      zi[H2 + c] = b.y;
    }
    fft_dif<L, -1, false>(zr, zi);  // Y[v] at position bitrev(v)
    const int t = t0 + q2;
    const size_t tb = size_t(ch) * p.cs + size_t(t / p.run) * p.rs + size_t(t % p.run);
    auto put = [&](int r, int v, float2 val) {
      if (!WIDE) {
        store_at(p.dst, unsigned((size_t(r) * V * bs + tb) * 8u) + unsigned(v) * unsigned(bs * 8u), val);
      } else {
        p.dst[(size_t(r) * V + v) * bs + tb] = val;
      }
    };
    if (u > 0) {
#pragma unroll
      for (int v = 0; v <= H2; ++v) put(u, v, make_float2(zr[bitrev(v, L)], zi[bitrev(v, L)]));
#pragma unroll
      for (int v = 1; v < H2; ++v) put(L - u, v, make_float2(zr[bitrev(L - v, L)], -zi[bitrev(L - v, L)]));
    } else {
#pragma unroll
      for (int v = 0; v <= H2; ++v) {
        const float a = zr[bitrev(v, L)], b = zi[bitrev(v, L)];
        const float c = zr[bitrev((L - v) % L, L)], d = zi[bitrev((L - v) % L, L)];
        put(0, v, make_float2(0.5f * (a + c), 0.5f * (b - d)));
        put(H2, v, make_float2(0.5f * (b + d), 0.5f * (c - a)));
      }
    }
  };

  const GroupWalk wk = group_walk(ngroups, false);
  if (half == 0 && wk.g < wk.end) fetch(wk.g);
  int turn = 0;  // the half whose windows are in registers for this group
  for (long g = wk.g; g < wk.end; g += wk.step, turn ^= 1) {
    const int ch = int(g / p.ngrp), t0 = int(g % p.ngrp) * TQ;
    const int nq = min(TQ, tpc - t0);
    const bool mine = half == turn;
    if (mine) {
      if (q1 < nq) columns();
    } else if (g + wk.step < wk.end) {
      fetch(g + wk.step);
    }
    __syncthreads();
    if (mine && q2 < nq && u < H2) row(ch, t0);
    __syncthreads();
  }
}

// Output of a group that is one whole plane, from its real tiles in LDS (tile
// q at float offset 2 q TSZ, row r of a tile at 2 r RI): output pixel (i, j)
// is framed pixel (i + off, j + off), the sum of at most two tiles per side,
// added in a fixed order. A wave per output row, lanes over the columns. Each
// lane's column offsets in the (at most two) tiles covering its columns, with
// 0/1 weights, are taken once per plane, so that the reads of a row need no
// per-lane branch; the tile rows covering a row are the same for the whole
// wave. RAW: rows and columns are at their inverse index r, kept index
// (r + rot) mod L, and hold L^2 times the values; else at kept index, scaled.
template <int L, bool RAW>
__device__ __forceinline__ void overlap_plane_out(const BigInvParams& p, const float* ldf, int TSZ, int ch, int t0,
                                                  int wave, int lane, int nwave) {
  constexpr int RI = Big<L>::RI;
  const int H = p.H, KR = p.KR, P = p.T * p.T;
  // stored index of kept index k
  auto at = [&](int k) { return RAW ? (k - p.rot) & (L - 1) : k; };
  const float wt = RAW ? 1.0f / float(L * L) : 1.0f;
  const int img = t0 / P, T = p.T, b = p.pitch;
  float* out = p.dst + (size_t(img) * p.n_ch + ch) * H * H;
  const SmallDiv div_b(b);
  constexpr int MCH = (L * Big<L>::SIDE_MAX + 63) / 64;  // H < T b <= L T
  int o0[MCH], o1[MCH];
  float m0[MCH], m1[MCH];
  int ln = lane;  // opaque: the offsets are not kept across the group loop
  asm volatile("" : "+v"(ln));
#pragma unroll
  for (int k = 0; k < MCH; ++k) {
    const int jx = ln + 64 * k, c = jx + p.off, Q1 = div_b(c), ca1 = c - Q1 * b;
    const bool in = jx < H;
    const bool v1 = in && Q1 < T, v0 = in && Q1 >= 1 && Q1 - 1 < T && ca1 + b < KR;
    o0[k] = v0 ? (Q1 - 1) * TSZ * 2 + at(ca1 + b) : 0;
    o1[k] = v1 ? Q1 * TSZ * 2 + at(ca1) : 0;
    m0[k] = v0 ? 1.f : 0.f;
    m1[k] = v1 ? 1.f : 0.f;
  }
  const int nch = (H + 63) / 64;
  for (int i = wave; i < H; i += nwave) {
    const int a = i + p.off, P1 = div_b(a), ra1 = a - P1 * b;
    // tile rows covering framed row a: P1 (row ra1) and P1 - 1 (row ra1 + b)
    const bool r1 = P1 < T, r0 = P1 >= 1 && P1 - 1 < T && ra1 + b < KR;
    const float* l1 = ldf + (r1 ? 2 * (P1 * T * TSZ + at(ra1) * RI) : 0);
    const float* l0 = ldf + (r0 ? 2 * ((P1 - 1) * T * TSZ + at(ra1 + b) * RI) : 0);
    const float w0 = r0 ? wt : 0.f, w1 = r1 ? wt : 0.f;
    float* orow = out + size_t(i) * H;
    float acc[MCH];
#pragma unroll
    for (int k = 0; k < MCH; ++k) {
      if (k >= nch) break;
      const float t0v = __builtin_fmaf(m0[k], l0[o0[k]], m1[k] * l0[o1[k]]);
      const float t1v = __builtin_fmaf(m0[k], l1[o0[k]], m1[k] * l1[o1[k]]);
      acc[k] = __builtin_fmaf(w0, t0v, w1 * t1v);
    }
#pragma unroll
    for (int k = 0; k < MCH; ++k) {
      if (k >= nch) break;
      const int jx = lane + 64 * k;
      if (jx < H) orow[jx] = acc[k];
    }
  }
}

// ---------------------------------------------------------------------------
// inverse: half spectra -> kept part of every tile (crop), or the plane the
// tiles overlap-add to
//
// Pass 1 inverts column w of every tile, w < L/2; column 0 carries the real
// columns 0 and L/2 together as h0[u] + i h1[u] (rows past L/2 rebuilt as the
// conjugates of rows L - u, which are not stored), so its inverse holds both
// real columns. Row r of the inverse becomes kept row (r + rot) mod L. Pass 2
// inverts pairs of kept rows to real rows, written over their own storage;
// column s becomes kept column (s + rot) mod L.
// MODE: the kernel's pass 3 (0 crop, 1 overlap-add of one-group planes, 2
// tiles to the scratch), fixed per instance so that each carries only the
// registers of its own output code.
template <int L, bool O32, int MODE>
__global__ void __launch_bounds__(kBigInvThreads) big_irfft2_kernel(BigInvParams p) {
  constexpr int H2 = Big<L>::H2, V = Big<L>::V, RI = Big<L>::RI;
  extern __shared__ float smem[];
  float2* lds = reinterpret_cast<float2*>(smem);
  const float* ldf = smem;
  const int KR = p.KR, rot = p.rot;
  const int TSZ = inv_tile_stride<L>(KR);
  const int tid = threadIdx.x, nthr = blockDim.x, h = tid & 1;
  const int P = p.T * p.T, tpc = p.n_img * P;
  const size_t fstride = size_t(p.n_ch) * tpc;
  const long ngroups = long(p.n_ch) * p.ngrp;
  const int npair = (KR + 1) / 2;
  const float scale = 1.0f / float(L * L);
  // tasks of passes 1 and 2: h + 2 (q + TQ w), tile q fastest; w is the
  // column (pass 1) or the row pair (pass 2); threads loop over the tasks
  float zr[H2], zi[H2];

  // Column w of tile q, rows [h L/2, h L/2 + L/2), summed over the split
  // partial spectra. Bins are read at a lane offset that steps by one row of
  // bins per element; the offset is made opaque first, so that the addresses
  // of all elements are not precomputed and kept across the group loop.
  using off_t = typename std::conditional<O32, unsigned, size_t>::type;
  auto at = [&](const float2* base, off_t e) { return O32 ? load_at(base, unsigned(e) * 8u) : base[e]; };
  auto load = [&](int ch, int t0, int q, int w) {
    const size_t tb = size_t(ch) * tpc + t0 + q;
    const off_t row = off_t(size_t(V) * fstride);
#pragma unroll
    for (int i = 0; i < H2; ++i) {
      zr[i] = 0.f;
      zi[i] = 0.f;
    }
    for (int sp = 0; sp < p.nsplit; ++sp) {
      const float2* base = p.src + size_t(sp) * p.split_stride;
      if (w > 0) {
        off_t e = off_t((size_t(h) * H2 * V + w) * fstride + tb);
        if (O32) asm volatile("" : "+v"(e));
#pragma unroll
        for (int i = 0; i < H2; ++i) {
          const float2 z = at(base, e);
          e += row;
          zr[i] += z.x;
          zi[i] += z.y;
        }
      } else {
        // columns 0 and L/2 together: rows u <= L/2 give b0 + i b1; rows
        // u > L/2 (lane 1, i > 0) conj b0 + i conj b1 of row L - u. Lane 0
        // walks rows 0, 1, ..., lane 1 rows L/2, L/2 - 1, ...
        off_t e = off_t(size_t(h) * H2 * V * fstride + tb);
        if (O32) asm volatile("" : "+v"(e));
        const off_t half = off_t(size_t(H2) * fstride);
#pragma unroll
        for (int i = 0; i < H2; ++i) {
          const float2 b0 = at(base, e), b1 = at(base, e + half);
          if (h) e -= row; else e += row;
          const bool mirror = h && i > 0;
          zr[i] += mirror ? b0.x + b1.y : b0.x - b1.y;
          zi[i] += mirror ? b1.x - b0.y : b0.y + b1.x;
        }
      }
    }
  };
  // pass 1 of one task: column inverse; row r becomes kept row (r + rot) mod L
  auto column = [&](int q, int w) {
    fft_dif_split<L, +1>(zr, zi, h);  // lane h: row 2m + h at bitrev(m)
    int qo = q * TSZ + w, ro = h + rot;  // opaque: see load
    asm volatile("" : "+v"(qo), "+v"(ro));
    float2* bq = lds + qo;
#pragma unroll
    for (int m = 0; m < H2; ++m) {
      const int rr = (2 * m + ro) & (L - 1);
      if (rr < KR) bq[rr * RI] = make_float2(zr[bitrev(m, H2)], zi[bitrev(m, H2)]);
    }
  };
  // pass 2 of one task: kept rows 2w, 2w + 1 to real rows, written over their
  // own storage; column s becomes kept column (s + rot) mod L. Lane 0 takes
  // bins 0, 1, ..., L/2 - 1 of both rows, lane 1 bins L/2, L/2 - 1, ..., 1
  // (bins 0 and L/2 being the parts of slot 0); the addresses step by one
  // slot per element from opaque starting values, and a missing second row
  // reads the first again and is zeroed, so that neither the compiler's
  // precomputed addresses nor a branch per element hold registers.
  auto rows = [&](int q, int w) {
    const int r0 = 2 * w;
    const bool has1 = r0 + 1 < KR;
    int zo = q * TSZ + r0 * RI, co = h + rot, st = h ? -1 : 1, db = has1 ? RI : 0;
    asm volatile("" : "+v"(zo), "+v"(co), "+v"(st), "+v"(db));
    const float2* za = lds + zo;
    const float keep1 = has1 ? 1.f : 0.f, sg = h ? 1.f : -1.f;
    float xr[H2], xi[H2];
    {
      const float2 a0 = za[0], b0 = za[db];
      xr[0] = h ? a0.y : a0.x;
      xi[0] = keep1 * (h ? b0.y : b0.x);
    }
    int o = h ? H2 - 1 : 1;
#pragma unroll
    for (int i = 1; i < H2; ++i) {
      const float2 a = za[o], bb = za[o + db];
      o += st;
      // lane 0: a.x - b.y, a.y + b.x; lane 1: a.x + b.y, b.x - a.y
      xr[i] = __builtin_fmaf(sg * keep1, bb.y, a.x);
      xi[i] = __builtin_fmaf(-sg, a.y, keep1 * bb.x);
      if (i % 8 == 7) asm volatile("" ::: "memory");  // bounds the reads in flight
    }
    fft_dif_split<L, +1>(xr, xi, h);  // lane h: L row0[s], L row1[s] at s = 2m + h, position bitrev(m)
    float* d0 = smem + 2 * zo;
#pragma unroll
    for (int m = 0; m < H2; ++m) {
      const int cc = (2 * m + co) & (L - 1);
      if (cc < KR) {
        d0[cc] = xr[bitrev(m, H2)] * scale;
        if (has1) d0[2 * RI + cc] = xi[bitrev(m, H2)] * scale;
      }
    }
  };

  const GroupWalk wk = group_walk(ngroups, true);
  for (long g = wk.g; g < wk.end; g += wk.step) {
    const int ch = int(g / p.ngrp), t0 = int(g % p.ngrp) * p.TQ;
    const int nq = min(p.TQ, tpc - t0);
    for (int task = tid; task < L * p.TQ; task += nthr) {
      const int q = (task >> 1) % p.TQ, w = (task >> 1) / p.TQ;
      if (q >= nq) continue;
      load(ch, t0, q, w);
      column(q, w);
    }
    __syncthreads();
    for (int task = tid; task < 2 * npair * p.TQ; task += nthr) {
      const int q = (task >> 1) % p.TQ, w = (task >> 1) / p.TQ;
      if (q < nq) rows(q, w);
    }
    __syncthreads();
    const int H = p.H;
    const int wave = tid >> 6, lane = tid & 63, nwave = nthr >> 6;
    if (MODE == 2) {
      // kept KR x KR of every tile to the scratch, tile after tile
      float* ob = p.tiles + (size_t(ch) * tpc + t0) * KR * KR;
      const SmallDiv div_k(KR);
      for (int qq = wave; qq < nq; qq += nwave) {
        const float* lt = ldf + 2 * qq * TSZ;
        float* ot = ob + size_t(qq) * KR * KR;
        for (int e = lane; e < KR * KR; e += 64) {
          const int rr = div_k(e), cc = e - rr * KR;
          ot[e] = lt[2 * rr * RI + cc];
        }
      }
    } else if (MODE == 0) {
      // kept KR x KR of every tile to its block: a wave per tile (decoded
      // once, wave-uniform), lanes over the block in row order
      const SmallDiv div_k(KR);
      for (int qq = wave; qq < nq; qq += nwave) {
        const int t = t0 + qq, img = t / P, pp = t - img * P;
        const int pr = pp / p.T, qc = pp - pr * p.T;
        const int nrow = min(KR, H - pr * p.pitch), ncol = min(KR, H - qc * p.pitch);
        float* oblk = p.dst + ((size_t(img) * p.n_ch + ch) * H + pr * p.pitch) * H + qc * p.pitch;
        const float* lt = ldf + 2 * qq * TSZ;
        for (int e = lane; e < KR * nrow; e += 64) {
          const int rr = div_k(e), cc = e - rr * KR;
          if (cc < ncol) oblk[rr * H + cc] = lt[2 * rr * RI + cc];
        }
      }
    } else {
      overlap_plane_out<L, false>(p, ldf, TSZ, ch, t0, wave, lane, nwave);
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// inverse at L = 64 with a whole 64-point sequence per lane: a lane inverts
// one column of a tile (pass 1), then one pair of rows (pass 2), in 128
// registers, where the kernel above splits each sequence over a lane pair.
// No first stage runs across a pair (about 0.7 of the vector instructions
// per transform). The 32 tasks per tile and pass of a group of eight tiles
// fill four waves, half the workgroup, and the halves alternate: while one
// transforms group i, the other loads the columns of group i + 1 into its
// registers, which then have passes 2 and 3 of group i to arrive. A nine-tile
// plane has 32 tasks per pass past the half's 256; the loading half runs
// them (loading their columns itself) before it loads the next group.
// Pass 3, the output, takes all eight waves.
//
// Rows and columns stay in LDS at their inverse index r (kept index
// (r + rot) mod L), in tiles of L x (L/2 + 1) slots, so that every LDS
// address is a compile-time offset from the task's base; passes 1 and 2
// write every row and column (skipping the ones nothing reads, under
// conditions that are uniform, makes the compiler keep more of the
// transform's values live across the stores, and spill), pass 2 runs on the
// row pairs that hold kept rows only, and the output pass applies the
// rotation and the 1/L^2 scale. MODE as for the kernel above; SPLIT: more
// than one partial spectrum to sum (the weight gradient's split), loaded in
// batches of 16 rows so that the partial sums and the loads in flight fit
// the registers.
template <bool O32, int MODE, bool SPLIT>
__global__ void __launch_bounds__(512) big_irfft2_lane_kernel(BigInvParams p) {
  constexpr int L = 64, H2 = L / 2, V = L / 2 + 1, RI = Big<L>::RI, HALF = 256;
  extern __shared__ float smem[];
  float2* lds = reinterpret_cast<float2*>(smem);
  const float* ldf = smem;
  const int KR = p.KR, rot = p.rot, TQ = p.TQ;
  const int TSZ = lane_tile_stride();
  const int tid = threadIdx.x;
  const int half = tid >> 8, ht = tid & (HALF - 1);  // half of the workgroup (four waves), thread in it
  const int P = p.T * p.T, tpc = p.n_img * P;
  const size_t fstride = size_t(p.n_ch) * tpc;
  const long ngroups = long(p.n_ch) * p.ngrp;
  // the stored rows (k - rot) mod L of kept rows k < KR are a cyclic run
  // from s0; the row pairs w0, w0 + 1, ... (mod L/2) cover it
  const int s0 = (L - rot) & (L - 1), w0 = s0 >> 1, npair = min(H2, ((s0 & 1) + KR + 1) >> 1);
  const int ntask1 = H2 * TQ, ntask2 = npair * TQ;  // tasks of passes 1 and 2 (tile fastest)
  using off_t = typename std::conditional<O32, unsigned, size_t>::type;
  auto at = [&](const float2* base, off_t e) { return O32 ? load_at(base, unsigned(e) * 8u) : base[e]; };
  float re[L], im[L];  // a lane's sequence: loaded columns, then the pass's working values

  // column w of tile q into re/im (summed over the partial spectra); column
  // 0 carries the real columns 0 and L/2 together as h0[u] + i h1[u], rows
  // past L/2 rebuilt as the conjugates of rows L - u (not stored)
  auto fetch = [&](int ch, int t0, int q, int w) __attribute__((always_inline)) {
    const size_t tb = size_t(ch) * tpc + t0 + q;
    const off_t row = off_t(size_t(V) * fstride);
    // rows [u0, u0 + NU) of one partial: assigned (first) or added
    auto gather = [&](const float2* base, int u0c, auto nu, auto first) __attribute__((always_inline)) {
      constexpr int NU = decltype(nu)::value;
      constexpr bool FIRST = decltype(first)::value;
      const int u0 = u0c;
      if (w > 0) {
        off_t e = off_t((size_t(u0) * V + w) * fstride + tb);
        if (O32) asm volatile("" : "+v"(e));
#pragma unroll
        for (int i = 0; i < NU; ++i) {
          const float2 z = at(base, e);
          e += row;
          re[u0 + i] = FIRST ? z.x : re[u0 + i] + z.x;
          im[u0 + i] = FIRST ? z.y : im[u0 + i] + z.y;
        }
      } else {
        // rows u <= L/2 of columns 0 and L/2 give rows u and L - u
        off_t e = off_t(size_t(u0) * V * fstride + tb);
        if (O32) asm volatile("" : "+v"(e));
        const off_t hoff = off_t(size_t(H2) * fstride);
#pragma unroll
        for (int i = 0; i < NU; ++i) {
          const int u = u0 + i;
          if (u > H2) break;
          const float2 b0 = at(base, e), b1 = at(base, e + hoff);
          e += row;
          re[u] = FIRST ? b0.x - b1.y : re[u] + (b0.x - b1.y);
          im[u] = FIRST ? b0.y + b1.x : im[u] + (b0.y + b1.x);
          if (u > 0 && u < H2) {
            re[L - u] = FIRST ? b0.x + b1.y : re[L - u] + (b0.x + b1.y);
            im[L - u] = FIRST ? b1.x - b0.y : im[L - u] + (b1.x - b0.y);
          }
        }
      }
    };
    if constexpr (!SPLIT) {
      gather(p.src, 0, std::integral_constant<int, L>{}, std::true_type{});
    } else {
      // column 0 reads rows [0, L/2] only, which the first three batches
      // cover (the fourth then reads nothing)
#pragma unroll
      for (int u0 = 0; u0 < L; u0 += 16) {
        gather(p.src, u0, std::integral_constant<int, 16>{}, std::true_type{});
        for (int sp = 1; sp < p.nsplit; ++sp)
          gather(p.src + size_t(sp) * p.split_stride, u0, std::integral_constant<int, 16>{}, std::false_type{});
        asm volatile("" ::: "memory");
      }
    }
  };
  // pass 1 on the fetched column w of tile q
  auto column = [&](int q, int w) __attribute__((always_inline)) {
    fft_dif<L, +1, false>(re, im);  // row r at position bitrev(r)
    float2* bq = lds + (q * TSZ + w);
#pragma unroll
    for (int r = 0; r < L; ++r) bq[r * RI] = make_float2(re[bitrev(r, L)], im[bitrev(r, L)]);
  };
  // pass 2: rows 2w, 2w + 1 to L^2 times their real rows, written over their
  // own storage (slot 0 of a row holds its bins 0 and L/2 as (re, im))
  auto rows = [&](int q, int w) __attribute__((always_inline)) {
    float2* za = lds + (q * TSZ + 2 * w * RI);
    {
      const float2 a0 = za[0], b0 = za[RI];
      re[0] = a0.x;
      im[0] = b0.x;
      re[H2] = a0.y;
      im[H2] = b0.y;
    }
#pragma unroll
    for (int v = 1; v < H2; ++v) {
      const float2 a = za[v], bb = za[RI + v];
      re[v] = a.x - bb.y;
      im[v] = a.y + bb.x;
      re[L - v] = a.x + bb.y;
      im[L - v] = bb.x - a.y;
    }
    fft_dif<L, +1, false>(re, im);  // L^2 row0[s] in re, L^2 row1[s] in im, at position bitrev(s)
    float* d0 = reinterpret_cast<float*>(za);
#pragma unroll
    for (int s = 0; s < L; ++s) {
      d0[s] = re[bitrev(s, L)];
      d0[2 * RI + s] = im[bitrev(s, L)];
    }
  };
  // pass 3, MODE 0 and 2: the kept KR x KR of every tile, scaled, to its
  // block (0) or to the scratch, tile after tile (2); a wave per tile
  // (decoded once, wave-uniform), lanes over the block in row order
  auto crop = [&](int ch, int t0, int nq, int wave, int lane, int nwave, auto rotated) {
    constexpr bool ROT = decltype(rotated)::value;
    const float scale = 1.0f / float(L * L);
    const SmallDiv div_k(KR);
    for (int qq = wave; qq < nq; qq += nwave) {
      const float* lt = ldf + 2 * qq * TSZ;
      int nrow = KR, ncol = KR;
      float* ob;
      int ostride;
      if (MODE == 0) {
        const int t = t0 + qq, img = t / P, pp = t - img * P;
        const int pr = pp / p.T, qc = pp - pr * p.T;
        nrow = min(KR, p.H - pr * p.pitch);
        ncol = min(KR, p.H - qc * p.pitch);
        ob = p.dst + ((size_t(img) * p.n_ch + ch) * p.H + pr * p.pitch) * p.H + qc * p.pitch;
        ostride = p.H;
      } else {
        ob = p.tiles + ((size_t(ch) * tpc + t0 + qq) * KR) * KR;
        ostride = KR;
      }
      for (int e = lane; e < KR * nrow; e += 64) {
        const int rr = div_k(e), cc = e - rr * KR;
        const int sr = ROT ? (rr - rot) & (L - 1) : rr, sc = ROT ? (cc - rot) & (L - 1) : cc;
        if (cc < ncol) ob[rr * ostride + cc] = lt[2 * sr * RI + sc] * scale;
      }
    }
  };

  const GroupWalk wk = group_walk_team(ngroups, MODE == 1 ? 8 : 2);
  const int wave = tid >> 6, lane = tid & 63, nwave = blockDim.x >> 6;
  // this half's first task of a group: tile ht % TQ, column ht / TQ
  auto prefetch = [&](long g) __attribute__((always_inline)) {
    const int ch = int(g / p.ngrp), t0 = int(g % p.ngrp) * TQ;
    if (ht < ntask1 && ht % TQ < min(TQ, tpc - t0)) fetch(ch, t0, ht % TQ, ht / TQ);
  };
  if (half == 0 && wk.g < wk.end) prefetch(wk.g);
  int turn = 0;  // the half whose columns are in registers for this group
  for (long g = wk.g; g < wk.end; g += wk.step, turn ^= 1) {
    const int ch = int(g / p.ngrp), t0 = int(g % p.ngrp) * TQ;
    const int nq = min(TQ, tpc - t0);
    const bool mine = half == turn;
    if (mine) {
      if (ht < ntask1 && ht % TQ < nq) column(ht % TQ, ht / TQ);
    } else {
      for (int k = HALF + ht; k < ntask1; k += HALF) {
        if (k % TQ >= nq) continue;
        fetch(ch, t0, k % TQ, k / TQ);
        column(k % TQ, k / TQ);
      }
    }
    __syncthreads();
    if (mine) {
      if (ht < ntask2 && ht % TQ < nq) rows(ht % TQ, (w0 + ht / TQ) & (H2 - 1));
    } else {
      for (int k = HALF + ht; k < ntask2; k += HALF)
        if (k % TQ < nq) rows(k % TQ, (w0 + k / TQ) & (H2 - 1));
      if (g + wk.step < wk.end) prefetch(g + wk.step);
    }
    __syncthreads();
    if (MODE == 1) {
      overlap_plane_out<L, true>(p, ldf, TSZ, ch, t0, wave, lane, nwave);
    } else if (rot == 0) {
      crop(ch, t0, nq, wave, lane, nwave, std::false_type{});
    } else {
      crop(ch, t0, nq, wave, lane, nwave, std::true_type{});
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// overlap-add of tiles kept in the scratch (planes of more tiles than a
// workgroup holds): output pixel (i, j) of plane (img, ch) is the sum, in a
// fixed order, of the kept elements of the at most two tiles per side whose
// kept range covers framed pixel (i + off, j + off). A workgroup per (plane,
// run of rows), lanes over the columns.
__global__ void __launch_bounds__(256) overlap_gather_kernel(BigInvParams p, int rows_per_wg, int nrg) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const unsigned wg = xcd_local_order(blockIdx.x, gridDim.x);
  const int rg = int(wg % unsigned(nrg));
  const unsigned plane = wg / unsigned(nrg);
  const int img = int(plane / unsigned(p.n_ch)), ch = int(plane % unsigned(p.n_ch));
  const int H = p.H, T = p.T, b = p.pitch, KR = p.KR, P = T * T;
  const size_t tile_elems = size_t(KR) * KR;
  const float* tb = p.tiles + (size_t(ch) * p.n_img * P + size_t(img) * P) * tile_elems;
  float* out = p.dst + size_t(plane) * H * H;
  const SmallDiv div_b(b);
  const int i0 = rg * rows_per_wg, i1 = min(H, i0 + rows_per_wg);
  for (int i = i0 + wave; i < i1; i += 4) {
    const int a = i + p.off, P1 = div_b(a), ra1 = a - P1 * b;
    const bool r1 = P1 < T, r0 = P1 >= 1 && P1 - 1 < T && ra1 + b < KR;
    for (int jx = lane; jx < H; jx += 64) {
      const int c = jx + p.off, Q1 = div_b(c), ca1 = c - Q1 * b;
      const bool c1 = Q1 < T, c0 = Q1 >= 1 && Q1 - 1 < T && ca1 + b < KR;
      float acc = 0.f;
      if (r0 && c0) acc += tb[size_t((P1 - 1) * T + Q1 - 1) * tile_elems + (ra1 + b) * KR + ca1 + b];
      if (r0 && c1) acc += tb[size_t((P1 - 1) * T + Q1) * tile_elems + (ra1 + b) * KR + ca1];
      if (r1 && c0) acc += tb[size_t(P1 * T + Q1 - 1) * tile_elems + ra1 * KR + ca1 + b];
      if (r1 && c1) acc += tb[size_t(P1 * T + Q1) * tile_elems + ra1 * KR + ca1];
      out[size_t(i) * H + jx] = acc;
    }
  }
}

// ---------------------------------------------------------------------------
// launchers

int cu_count() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (!cached[dev]) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) cus = 256;
    cached[dev] = cus;
  }
  return cached[dev];
}

// Waves of these kernels resident on a CU: every instance takes more than 128
// registers per lane, which leaves two waves on each of the four SIMDs.
constexpr int kBigWavesPerCu = 8;

// Persistent grid: whole rounds over the 8 XCDs, as many workgroups as are
// resident (by LDS and by registers), at most one per group.
unsigned persistent_grid(long ngroups, size_t lds, int nthr) {
  const long by_lds = long(kBigLds / std::max<size_t>(lds, 1));
  const long by_waves = kBigWavesPerCu / std::max(1, (nthr + 63) / 64);
  const long per_cu = std::max<long>(1, std::min(by_lds, by_waves));
  long nwg = std::min<long>(per_cu * cu_count(), (ngroups + 7) / 8 * 8);
  nwg = std::max<long>(8, nwg / 8 * 8);
  return unsigned(nwg);
}

// tiles per group: runs of eight (64-byte segments of a bin) at L = 64, or
// whole planes where fewer fit; two at L = 128
template <int L>
int group_tiles(int P, long tpc) {
  int tq = L == 64 ? OAA_BIG_TQ : 2;
  if (P > 1 && P < tq) tq = P * (tq / P);
  return int(std::max<long>(1, std::min<long>(tq, tpc)));
}

template <int L, bool PF>
hipError_t launch_big_fwd_LP(const BigFwdParams& p, size_t lds, long ngroups, hipStream_t s) {
  constexpr int V = Big<L>::V;
  // one past the largest element the layout addresses
  const long tpc = long(p.n_img) * p.T * p.T;
  const size_t end = size_t(L * V - 1) * p.bs + size_t(p.n_ch - 1) * p.cs + size_t((tpc - 1) / p.run) * p.rs +
                     size_t(std::min<long>(p.run, tpc));
  const bool o32 = end * 8 < (size_t(1) << 32);
  auto kern = o32 ? big_rfft2_kernel<L, true, PF> : big_rfft2_kernel<L, false, PF>;
  const hipError_t e = allow_lds(kern, kBigLds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(persistent_grid(ngroups, lds, L * p.TQ)), dim3(L * p.TQ), lds, s, p);
  return hipGetLastError();
}

template <int L>
hipError_t launch_big_fwd_L(BigFwdParams p, hipStream_t s) {
  if (p.S < 1 || p.S > L || p.T < 1 || p.H < 1 || size_t(p.H) * p.H * 4 >= (size_t(1) << 31))
    return hipErrorInvalidValue;
  const int P = p.T * p.T;
  const long tpc = long(p.n_img) * P;
  if (tpc < 1 || tpc > 0x7fffffffL) return hipErrorInvalidValue;
  if (p.run == 0) {
    p.run = int(tpc);
    p.rs = 0;
    p.bs = size_t(p.n_ch) * size_t(tpc);
    p.cs = size_t(tpc);
  }
  if (p.run < 1) return hipErrorInvalidValue;
  p.TQ = group_tiles<L>(P, tpc);
  p.ngrp = int((tpc + p.TQ - 1) / p.TQ);
  const size_t lds = size_t(fwd_tile_stride<L>()) * p.TQ * 8;
  // one task per thread (group_tiles keeps L TQ within a workgroup)
  if (lds > kBigLds || L * p.TQ > big_threads<L, true>()) return hipErrorInvalidConfiguration;
  const long ngroups = long(p.n_ch) * p.ngrp;
  // at L = 64 the alternating halves need two groups or more per workgroup
  // (one per CU) to overlap anything; smaller launches take the lane pairs
  // (measured at the 224 x 224 RGB layer: kernel spectra, 24 groups, 0.017
  // against 0.025 ms)
  if constexpr (L == 64) {
    if (ngroups < 2L * cu_count()) return launch_big_fwd_LP<L, true>(p, lds, ngroups, s);
    constexpr int V = Big<L>::V;
    const size_t end = size_t(L * V - 1) * p.bs + size_t(p.n_ch - 1) * p.cs + size_t((tpc - 1) / p.run) * p.rs +
                       size_t(std::min<long>(p.run, tpc));
    // the planes one group's windows read: tiles of at most TQ images
    const size_t span = (size_t(p.TQ - 1) * p.n_ch + 1) * size_t(p.H) * p.H * 4;
    const bool narrow = end * 8 < (size_t(1) << 32) && span < size_t(kOutOfRange);
    auto kern = narrow ? big_rfft2_lane_kernel<false> : big_rfft2_lane_kernel<true>;
    const hipError_t e = allow_lds(kern, kBigLds);
    if (e != hipSuccess) return e;
    const size_t lane_lds = size_t(lane_tile_stride()) * p.TQ * 8;
    if (lane_lds > kBigLds) return hipErrorInvalidConfiguration;
    constexpr int nthr = 512;  // two halves of four waves: 32 TQ <= 256 tasks per pass
    hipLaunchKernelGGL(kern, dim3(persistent_grid(ngroups, lane_lds, nthr)), dim3(nthr), lane_lds, s, p);
    return hipGetLastError();
  } else {
    return launch_big_fwd_LP<L, false>(p, lds, ngroups, s);
  }
}

template <int L, int MODE>
hipError_t launch_big_inv_LM(const BigInvParams& p, size_t lds, long ngroups, hipStream_t s) {
  constexpr int V = Big<L>::V;
  const bool o32 =
      (size_t(L) * V * size_t(p.n_ch) * size_t(p.n_img) * p.T * p.T + size_t(p.nsplit - 1) * p.split_stride) * 8 <
      (size_t(1) << 32);
  auto kern = o32 ? big_irfft2_kernel<L, true, MODE> : big_irfft2_kernel<L, false, MODE>;
  const hipError_t e = allow_lds(kern, kBigLds);
  if (e != hipSuccess) return e;
  const int nthr = std::min(L * p.TQ, kBigInvThreads);
  hipLaunchKernelGGL(kern, dim3(persistent_grid(ngroups, lds, nthr)), dim3(nthr), lds, s, p);
  return hipGetLastError();
}

template <int L>
hipError_t launch_big_inv_LS(const BigInvParams& p, size_t lds, long ngroups, hipStream_t s) {
  switch (p.overlap) {
    case 0: return launch_big_inv_LM<L, 0>(p, lds, ngroups, s);
    case 1: return launch_big_inv_LM<L, 1>(p, lds, ngroups, s);
    case 2: return launch_big_inv_LM<L, 2>(p, lds, ngroups, s);
    default: return hipErrorInvalidValue;
  }
}

// L = 64: one sequence per lane, tiles of whole L x (L/2 + 1) slots
template <bool O32>
hipError_t launch_big_inv_lane_O(const BigInvParams& p, size_t lds, long ngroups, hipStream_t s) {
  void (*kern)(BigInvParams) = nullptr;
  if (p.overlap == 0)
    kern = p.nsplit > 1 ? big_irfft2_lane_kernel<O32, 0, true> : big_irfft2_lane_kernel<O32, 0, false>;
  else if (p.nsplit == 1)  // the overlap-add of forward spectra: one partial
    kern = p.overlap == 1 ? big_irfft2_lane_kernel<O32, 1, false> : big_irfft2_lane_kernel<O32, 2, false>;
  if (!kern) return hipErrorInvalidValue;
  const hipError_t e = allow_lds(kern, kBigLds);
  if (e != hipSuccess) return e;
  constexpr int nthr = 512;
  hipLaunchKernelGGL(kern, dim3(persistent_grid(ngroups, lds, nthr)), dim3(nthr), lds, s, p);
  return hipGetLastError();
}

hipError_t launch_big_inv_lane(const BigInvParams& p, long ngroups, hipStream_t s) {
  constexpr int L = 64;
  const size_t lds = size_t(lane_tile_stride()) * p.TQ * 8;
  if (lds > kBigLds || p.TQ > Big<L>::TQ_MAX) return hipErrorInvalidConfiguration;
  const size_t tpc = size_t(p.n_img) * p.T * p.T;
  const bool o32 = (size_t(L) * Big<L>::V * size_t(p.n_ch) * tpc + size_t(p.nsplit - 1) * p.split_stride) * 8 <
                   (size_t(1) << 32);
  return o32 ? launch_big_inv_lane_O<true>(p, lds, ngroups, s) : launch_big_inv_lane_O<false>(p, lds, ngroups, s);
}

template <int L>
hipError_t launch_big_inv_L(BigInvParams p, hipStream_t s) {
  if (p.KR < 1 || p.KR > L || p.rot < 0 || p.rot >= L || p.T < 1 || p.H < 1 || p.nsplit < 1 ||
      p.H >= 65536 || size_t(p.H) * p.H >= (size_t(1) << 31))
    return hipErrorInvalidValue;
  const int P = p.T * p.T;
  const long tpc = long(p.n_img) * P;
  if (tpc < 1 || tpc > 0x7fffffffL) return hipErrorInvalidValue;
  bool two_step = false;
  if (p.overlap) {
    if (p.pitch < 1 || p.off < 0 || p.H + p.off >= 65536) return hipErrorInvalidValue;
    if (P <= Big<L>::TQ_MAX) {
      p.TQ = P;  // one plane per group
    } else {
      // keep every tile's KR x KR in the scratch, then add in a second kernel
      if (!p.tiles || long(p.KR) * p.KR >= 65536) return hipErrorInvalidValue;
      two_step = true;
      p.overlap = 2;
      p.TQ = group_tiles<L>(P, tpc);
    }
  } else {
    if (p.pitch != p.KR) return hipErrorInvalidValue;
    p.TQ = group_tiles<L>(P, tpc);
    if (long(p.KR) * p.KR * p.TQ >= 65536) return hipErrorInvalidValue;
  }
  p.ngrp = int((tpc + p.TQ - 1) / p.TQ);
  const size_t lds = size_t(inv_tile_stride<L>(p.KR)) * p.TQ * 8;
  if (lds > kBigLds) return hipErrorInvalidConfiguration;
  const long ngroups = long(p.n_ch) * p.ngrp;
  hipError_t e = hipSuccess;
  if constexpr (L == 64) {
    e = launch_big_inv_lane(p, ngroups, s);
  } else {
    e = launch_big_inv_LS<L>(p, lds, ngroups, s);
  }
  if (e != hipSuccess || !two_step) return e;
  // second step: about 8 rows per workgroup
  const int rows = 8, nrg = (p.H + rows - 1) / rows;
  const long nwg = long(p.n_img) * p.n_ch * nrg;
  if (nwg > 0x7fffffffL) return hipErrorInvalidValue;
  hipLaunchKernelGGL(overlap_gather_kernel, dim3(unsigned(nwg)), dim3(256), 0, s, p, rows, nrg);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_big_rfft2(int L, const BigFwdParams& p, hipStream_t s) {
  switch (L) {
    case 64: return launch_big_fwd_L<64>(p, s);
    case 128: return launch_big_fwd_L<128>(p, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_big_irfft2(int L, const BigInvParams& p, hipStream_t s) {
  switch (L) {
    case 64: return launch_big_inv_L<64>(p, s);
    case 128: return launch_big_inv_L<128>(p, s);
    default: return hipErrorInvalidValue;
  }
}

bool big_overlap_supported(int L, int T) {
  if (L == 64) return T * T <= Big<64>::TQ_MAX;
  if (L == 128) return T * T <= Big<128>::TQ_MAX;
  return false;
}

}  // namespace oaa
