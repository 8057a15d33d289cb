// Fused few-channel passes at transform side 64 (arXiv:1601.06815, Section 2:
// block division, zero padding, the block transforms, the per-bin products,
// the inverse transforms and the overlap-add; Section 3.2: the error
// propagation and the weight gradient).
//
// With few input channels (C <= 4) the per-bin contraction is a handful of
// multiply-adds, and the unfused passes spend their time moving its operands
// and results through HBM: the forward product spectra (K per block) and the
// gradient window spectra (K per block) are many times the size of the
// layer's own inputs and outputs. Here the contraction runs inside the
// transform kernels, on spectra held in LDS, and neither of those spectra is
// ever stored:
//  * forward: a workgroup owns Kg output planes of one image and walks its
//    block rows. Per block row it forms the T Kg product spectra from the
//    row's input block spectra and the Kg kernel spectra, inverts them, and
//    overlap-adds the blocks of the row; the n - 1 rows that the next block
//    row adds to are carried in LDS, so every output row is written once;
//  * error propagation: a workgroup owns two blocks. It transforms the
//    gradient windows of four kernels at a time, accumulates conj(W) G over
//    all kernels in registers (per bin and input channel), then inverts the
//    C results of each block and writes the blocks of dx;
//  * weight gradient: a workgroup owns Kf kernels and a range of block rows.
//    It transforms their gradient windows, accumulates conj(X) G over the
//    range in registers and writes one partial sum per range; the inverse of
//    the unfused pass adds the ranges in a fixed order.
// Spectra are held per tile as 64 x 33 bins (f = u * 33 + v) in LDS slots of
// 2113 complex elements, eight slots per workgroup (one workgroup per CU).
// The input block spectra come in runs of a block row (the T blocks of each
// bin and channel together) and the kernel spectra kernel by kernel, bins
// contiguous, so that the lanes of a wave, one bin each, read their operands
// from a few whole cache lines.
#include <algorithm>

#include "fft_core.hpp"
#include "oaa_internal.hpp"
#include "tile_common.hpp"

namespace oaa {

namespace {

using namespace tile;

constexpr int kL = 64, kH = 32, kV = 33;
constexpr int kRS = kL + 2;            // forward pass-1 row stride (complex)
constexpr int kSlot = 2113;            // complex per slot: 32 x 66 and 64 x 33 fit; odd
constexpr int kPos = kL * kV;          // bin positions
constexpr size_t kLdsMax = 160 * 1024;

// A workgroup holds NS slots (4 or 8) and runs 64 NS threads: a lane pair
// per column of every slot. Four slots (68 KB) let two workgroups share a CU,
// so that one's loads and barriers overlap the other's arithmetic; eight serve
// planes of more than four blocks per side.
template <int NS>
struct Fz {
  static constexpr int threads = 64 * NS;
  static constexpr int pos_iter = (kPos + threads - 1) / threads;
  static constexpr size_t slot_bytes = size_t(NS) * kSlot * 8;
};

// Workgroup barrier for LDS traffic only: the waves' LDS accesses are
// complete when it returns; their global stores need not be (nothing in
// these kernels reads back what the workgroup wrote to global memory).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Bins (u, v) with u > 32 and v in {0, 32} are conjugates of stored bins and
// are neither stored nor read.
__device__ __forceinline__ bool bin_used(int f) {
  const int u = f / kV, v = f - u * kV;
  return u <= kH || (v != 0 && v != kH);
}

__device__ __forceinline__ float2 cmul(float2 a, float2 b) {
  return make_float2(__builtin_fmaf(a.x, b.x, -a.y * b.y), __builtin_fmaf(a.x, b.y, a.y * b.x));
}
// acc + conj(a) b
__device__ __forceinline__ float2 cmac_conj(float2 acc, float2 a, float2 b) {
  return make_float2(__builtin_fmaf(a.x, b.x, __builtin_fmaf(a.y, b.y, acc.x)),
                     __builtin_fmaf(a.x, b.y, __builtin_fmaf(-a.y, b.x, acc.y)));
}
// acc + a b
__device__ __forceinline__ float2 cmac(float2 acc, float2 a, float2 b) {
  return make_float2(__builtin_fmaf(a.x, b.x, __builtin_fmaf(-a.y, b.y, acc.x)),
                     __builtin_fmaf(a.x, b.y, __builtin_fmaf(a.y, b.x, acc.y)));
}

// First item of this workgroup; items advance by gridDim.x (a multiple of
// 8), and the workgroups of one XCD take consecutive items.
__device__ __forceinline__ long first_item() {
  const unsigned nwg = gridDim.x;
  return long(blockIdx.x % 8) * (nwg / 8) + blockIdx.x / 8;
}

// Forward pass 1 of the S x S window at (r0, c0) of an H x H plane (zero
// outside the plane and past S), zero-padded to 64 x 64: lane pair j
// transforms z = x[., j] + i x[., j + 32] along the rows; the real columns'
// spectra are C_j[u] = (Z[u] + conj Z[-u]) / 2 and C_{j+32}[u] =
// (Z[u] - conj Z[-u]) / (2i), Hermitian in u, so rows u <= 32 are kept:
// row u at u * 66 (columns [0, 32), then one slot on, [32, 64)), rows 0 and
// 32 sharing row 0 as (re, im). The plane must be the same in every lane
// of the wave.
__device__ __forceinline__ void fwd_columns(float2* bq, const float* plane, int H, int r0, int c0, int S, int j,
                                            int h) {
  float zr[kH], zi[kH];
  const __amdgpu_buffer_rsrc_t rs = buffer_resource(plane, unsigned(H) * unsigned(H) * 4u);
  // lane values are made opaque once per call: otherwise the compiler keeps
  // every element's offset in a register across the caller's loops
  int gr = r0 + h * kH, ca = c0 + j, lim = S - h * kH;
  asm volatile("" : "+v"(gr), "+v"(ca), "+v"(lim));
  const int cb = ca + kH;
  const bool oka = j < S && unsigned(ca) < unsigned(H);
  const bool okb = j + kH < S && unsigned(cb) < unsigned(H);
  unsigned ro = unsigned(gr * H + ca) * 4u;  // byte offset of (row gr, column ca)
  const unsigned rstep = unsigned(H) * 4u, cbo = unsigned(kH) * 4u;
#pragma unroll
  for (int i = 0; i < kH; ++i) {
    const bool okr = i < lim && unsigned(gr + i) < unsigned(H);
    zr[i] = buffer_load_f1(rs, okr && oka ? ro : kOutOfRange);
    zi[i] = buffer_load_f1(rs, okr && okb ? ro + cbo : kOutOfRange);
    ro += rstep;
  }
  fft_dif_split<kL, -1>(zr, zi, h);  // lane h: Z[2m + h] at bitrev(m)
#pragma unroll
  for (int m = 1; m < kH / 2; ++m) {  // u = 2m + h in [2, 32), with u = 1 below
    const int uu = 2 * m + h;
    const int ps = bitrev(m, kH);
    const int p0 = bitrev(kH - m, kH), p1 = bitrev(kH - m - 1, kH);  // -uu for h = 0, 1
    const float a = zr[ps], b = zi[ps];
    const float c = pick(h, zr[p1], zr[p0]), d = pick(h, zi[p1], zi[p0]);
    bq[uu * kRS + j] = make_float2(0.5f * (a + c), 0.5f * (b - d));
    bq[uu * kRS + kH + 1 + j] = make_float2(0.5f * (b + d), 0.5f * (c - a));
  }
  // m = 0: u = 0 (lane 0) and u = 1 (lane 1, partner 63 at m = 31); lane 0
  // also holds u = 32 at m = 16
  const float a0 = zr[0], b0 = zi[0];
  if (h) {
    const int pl = bitrev(kH - 1, kH);
    const float c = zr[pl], d = zi[pl];
    bq[kRS + j] = make_float2(0.5f * (a0 + c), 0.5f * (b0 - d));
    bq[kRS + kH + 1 + j] = make_float2(0.5f * (b0 + d), 0.5f * (c - a0));
  } else {
    const int ph = bitrev(kH / 2, kH);
    bq[j] = make_float2(a0, zr[ph]);
    bq[kH + 1 + j] = make_float2(b0, zi[ph]);
  }
}

// Forward pass 2, read half: row u of pass 1 (lane h: columns [32h, 32h+32)).
__device__ __forceinline__ void fwd_row_read(const float2* bq, int u, int h, float (&re)[kH], float (&im)[kH]) {
  int o = u * kRS + h * (kH + 1);
  asm volatile("" : "+v"(o));
  const float2* row = bq + o;
#pragma unroll
  for (int i = 0; i < kH; ++i) {
    const float2 z = row[i];
    re[i] = z.x;
    im[i] = z.y;
  }
}

// Forward pass 2, transform and write half: rows u in [1, 32) give bins
// (u, v), v <= 32, and (64 - u, v) = conj X[u][64 - v] for 0 < v < 32; the
// packed row u = 0 gives rows 0 and 32 (both Hermitian in v) by the same
// separation as pass 1. Bins go to the slot as bq[r * 33 + v]. Every lane
// of the workgroup must have read its row before any lane writes.
__device__ __forceinline__ void fwd_row_write(float2* bq, int u, int h, float (&re)[kH], float (&im)[kH]) {
  fft_dif_split<kL, -1>(re, im, h);  // lane h: Y[2m + h] at bitrev(m)
  if (u > 0) {
    int oa = u * kV + h, ob = (kL - u) * kV + h;  // bins (u, h) and (64 - u, h)
    asm volatile("" : "+v"(oa), "+v"(ob));
    float2* ba = bq + oa;
    float2* bb = bq + ob;
#pragma unroll
    for (int m = 0; m <= kH / 2; ++m) {
      const int v = 2 * m + h, ps = bitrev(m, kH);
      if (v <= kH) ba[2 * m] = make_float2(re[ps], im[ps]);
      if (v >= 1 && v < kH) {
        const int q0i = bitrev((kH - m) % kH, kH), q1i = bitrev(kH - m - 1, kH);
        const float xr = pick(h, re[q1i], re[q0i]), xi = pick(h, im[q1i], im[q0i]);
        bb[2 * m] = make_float2(xr, -xi);
      }
    }
  } else {
#pragma unroll
    for (int m = 0; m <= kH / 2; ++m) {
      const int v = 2 * m + h, ps = bitrev(m, kH);
      if (v > kH) continue;
      const int q0i = bitrev((kH - m) % kH, kH), q1i = bitrev((kH - m - 1 + kH) % kH, kH);
      const float a = re[ps], b = im[ps];
      const float c = pick(h, re[q1i], re[q0i]), d = pick(h, im[q1i], im[q0i]);
      bq[v] = make_float2(0.5f * (a + c), 0.5f * (b - d));
      bq[kH * kV + v] = make_float2(0.5f * (b + d), 0.5f * (c - a));
    }
  }
}

// Inverse pass 1 of column w of the bins in a slot (in place): columns 0 and
// 32 go together as h0[u] + i h1[u] (rows past 32 rebuilt as the conjugates
// of rows 64 - u), so that slot 0 of each row ends up holding both real
// columns. Row r of the inverse becomes kept row (r + rot) mod 64, rows
// [0, KR) kept, at bq[row * 33 + w].
__device__ __forceinline__ void inv_column(float2* bq, int w, int h, int KR, int rot) {
  float zr[kH], zi[kH];
  if (w > 0) {
    int o = h * kH * kV + w;  // opaque per call (see fwd_columns)
    asm volatile("" : "+v"(o));
    const float2* col = bq + o;
#pragma unroll
    for (int i = 0; i < kH; ++i) {
      const float2 z = col[i * kV];
      zr[i] = z.x;
      zi[i] = z.y;
    }
  } else {
    // lane 0 walks rows 0, 1, ..., lane 1 rows 32, 31, ... (the mirrors of
    // rows 32, 33, ...)
    int o = h * kH * kV, st = h ? -kV : kV;
    asm volatile("" : "+v"(o), "+v"(st));
#pragma unroll
    for (int i = 0; i < kH; ++i) {
      const float2 b0 = bq[o], b1 = bq[o + kH];
      o += st;
      const bool mirror = h && i > 0;
      zr[i] = mirror ? b0.x + b1.y : b0.x - b1.y;
      zi[i] = mirror ? b1.x - b0.y : b0.y + b1.x;
    }
  }
  fft_dif_split<kL, +1>(zr, zi, h);  // lane h: row 2m + h at bitrev(m)
  int ro = h + rot, cw = w;
  asm volatile("" : "+v"(ro), "+v"(cw));
#pragma unroll
  for (int m = 0; m < kH; ++m) {
    const int rr = (2 * m + ro) & (kL - 1);
    if (rr < KR) bq[rr * kV + cw] = make_float2(zr[bitrev(m, kH)], zi[bitrev(m, kH)]);
  }
}

// Inverse pass 2: kept rows 2w and 2w + 1 of a slot (complex offset `so`) to
// real rows, scaled, written over their own storage as floats (row r at
// floats 2 (so + r * 33) + column); column s becomes kept column
// (s + rot) mod 64.
__device__ __forceinline__ void inv_rows(float* smem, int so, int w, int h, int KR, int rot, float scale) {
  const int r0 = 2 * w;
  const bool has1 = r0 + 1 < KR;
  // Row bins: lane 0 takes bins 0, 1, ..., 31 of both rows, lane 1 bins 32,
  // 31, ..., 1; bins 0 and 32 are the two parts of slot 0. A missing second
  // row reads the first again and is zeroed.
  int zo = so + r0 * kV, co = h + rot, st = h ? -1 : 1, db = has1 ? kV : 0;
  asm volatile("" : "+v"(zo), "+v"(co), "+v"(st), "+v"(db));
  const float2* za = reinterpret_cast<const float2*>(smem) + zo;
  const float keep1 = has1 ? 1.f : 0.f, sg = h ? 1.f : -1.f;
  float xr[kH], xi[kH];
  {
    const float2 a0 = za[0], b0 = za[db];
    xr[0] = h ? a0.y : a0.x;
    xi[0] = keep1 * (h ? b0.y : b0.x);
  }
  int o = h ? kH - 1 : 1;
#pragma unroll
  for (int i = 1; i < kH; ++i) {
    const float2 a = za[o], b = za[o + db];
    o += st;
    // lane 0: a.x - b.y, a.y + b.x; lane 1: a.x + b.y, b.x - a.y
    xr[i] = __builtin_fmaf(sg * keep1, b.y, a.x);
    xi[i] = __builtin_fmaf(-sg, a.y, keep1 * b.x);
    if (i % 8 == 7) asm volatile("" ::: "memory");  // bounds the reads in flight
  }
  fft_dif_split<kL, +1>(xr, xi, h);  // lane h: L row0[s], L row1[s] at s = 2m + h, position bitrev(m)
  float* d0 = smem + 2 * zo;
#pragma unroll
  for (int m = 0; m < kH; ++m) {
    const int cc = (2 * m + co) & (kL - 1);
    if (cc < KR) {
      d0[cc] = xr[bitrev(m, kH)] * scale;
      if (has1) d0[2 * kV + cc] = xi[bitrev(m, kH)] * scale;
    }
  }
}

// Forward pass 2 over the first ns of NS slots (32 NS lane pairs: slot
// fastest, 32 rows), with the barrier between the reads and the writes.
template <int NS>
__device__ __forceinline__ void fwd_rows_all(float2* lds, int ns) {
  const int tid = threadIdx.x, h = tid & 1, pr = tid >> 1;
  const int s = pr % NS, u = pr / NS;
  const bool act = s < ns;
  float re[kH], im[kH];
  if (act) fwd_row_read(lds + s * kSlot, u, h, re, im);
  lds_barrier();
  if (act) fwd_row_write(lds + s * kSlot, u, h, re, im);
}

// Inverse passes 1 and 2 of the first ns slots, keeping KR rows and columns.
template <int NS>
__device__ __forceinline__ void inverse_all(float* smem, int ns, int KR, int rot) {
  const int tid = threadIdx.x, h = tid & 1, pr = tid >> 1;
  float2* lds = reinterpret_cast<float2*>(smem);
  {
    const int q = pr / kH, w = pr % kH;  // a wave per slot
    if (q < ns) inv_column(lds + q * kSlot, w, h, KR, rot);
  }
  lds_barrier();
  const int npair = (KR + 1) / 2;
  const float scale = 1.0f / float(kL * kL);
  for (int task = pr; task < ns * npair; task += Fz<NS>::threads / 2) {
    const int q = task % ns, w = task / ns;
    inv_rows(smem, q * kSlot, w, h, KR, rot, scale);
  }
}

// ---------------------------------------------------------------------------
// forward

template <int C, int KG, int NS>
__global__ void __launch_bounds__(Fz<NS>::threads) fused_fwd_kernel(FusedFwdParams p) {
  constexpr int TMAX = NS / KG, NT = Fz<NS>::threads, PI = Fz<NS>::pos_iter;
  // chunks of 64 output columns: M < T b <= 64 T <= 64 TMAX
  constexpr int MCH = TMAX;
  extern __shared__ float smem[];
  float2* lds = reinterpret_cast<float2*>(smem);
  float* carry = smem + 2 * NS * kSlot;  // [KG][n - 1][M]
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  constexpr int nwave = NT / 64;
  const int T = p.T, b = p.b, KR = p.KR, nov = KR - b, M = p.M, off = p.off;
  const long nitems = long(p.B) * p.ngrp;
  const SmallDiv div_b(b);
  for (long it = first_item(); it < nitems; it += gridDim.x) {
    const int img = int(it / p.ngrp), k0 = int(it % p.ngrp) * KG;
    const int nk = min(KG, p.K - k0), ns = nk * T;
    for (int r = 0; r < T; ++r) {
      // products of the block row's spectra with the kernels': slot ks T + q
      const float2* xrow = p.xs + size_t(img * T + r) * C * kPos * T;
      int ft = tid;  // opaque: the bins' addresses are not kept across the passes
      asm volatile("" : "+v"(ft));
#pragma unroll
      for (int i5 = 0; i5 < PI; ++i5) {
        // two bins' operands in flight at a time (registers). The loads are
        // unconditional (indices clamped into the operands), so that they
        // issue together rather than one per branch
        if (i5 % 2 == 0) asm volatile("" ::: "memory");
        const int f = ft + i5 * NT, fl = min(f, kPos - 1);
        float2 xv[C][TMAX], wv[C][KG];
#pragma unroll
        for (int c = 0; c < C; ++c) {
#pragma unroll
          for (int q = 0; q < TMAX; ++q) xv[c][q] = xrow[(size_t(c) * kPos + fl) * T + min(q, T - 1)];
#pragma unroll
          for (int ks = 0; ks < KG; ++ks) wv[c][ks] = p.ws[(size_t(k0 + min(ks, nk - 1)) * C + c) * kPos + fl];
        }
        if (f >= kPos || !bin_used(f)) continue;
#pragma unroll
        for (int ks = 0; ks < KG; ++ks) {
          if (ks >= nk) continue;
#pragma unroll
          for (int q = 0; q < TMAX; ++q) {
            if (q >= T) continue;
            float2 acc = cmul(wv[0][ks], xv[0][q]);
#pragma unroll
            for (int c = 1; c < C; ++c) acc = cmac(acc, wv[c][ks], xv[c][q]);
            lds[(ks * T + q) * kSlot + f] = acc;
          }
        }
      }
      lds_barrier();
      inverse_all<NS>(smem, ns, KR, 0);
      lds_barrier();
      // Framed row a = r b + ra of the block row is output row a - off, the
      // sum of the blocks of this row covering each column (at most two, in
      // column order) and, for ra < n - 1, the carried rows of the block row
      // above (added first). Rows ra >= b are carried to the next block row
      // (or written, after the last one).
      // per lane, for each chunk of 64 output columns: the float offsets of
      // its column in the (at most two) blocks that cover it, -1 if none
      // (offsets 0 and weight 0 where no block covers it, so that the reads
      // need no branch)
      int o0[MCH], o1[MCH];
      float m0[MCH], m1[MCH];
#pragma unroll
      for (int ch = 0; ch < MCH; ++ch) {
        const int j = lane + 64 * ch, cf = j + off, Q1 = div_b(cf), ca1 = cf - Q1 * b;
        const bool in = j < M;
        const bool v0 = in && Q1 >= 1 && Q1 - 1 < T && ca1 + b < KR, v1 = in && Q1 < T;
        o0[ch] = v0 ? 2 * (Q1 - 1) * kSlot + ca1 + b : 0;
        o1[ch] = v1 ? 2 * Q1 * kSlot + ca1 : 0;
        m0[ch] = v0 ? 1.f : 0.f;
        m1[ch] = v1 ? 1.f : 0.f;
      }
      const int nch = (M + 63) / 64;
      for (int task = wave; task < nk * b; task += nwave) {
        const int ks = task / b, ra = task - ks * b;
        const int i = r * b + ra - off;
        if (i < 0 || i >= M) continue;
        const bool add_carry = r > 0 && ra < nov;
        const float* lrow = smem + 2 * (ks * T * kSlot + ra * kV);
        const float* crow = add_carry ? carry + (ks * nov + ra) * M : lrow;  // (weight 0 then)
        float* orow = p.y + ((size_t(img) * p.K + k0 + ks) * M + i) * size_t(M);
        const float cw = add_carry ? 1.f : 0.f;
        float acc[MCH];
#pragma unroll
        for (int ch = 0; ch < MCH; ++ch) {
          if (ch >= nch) break;
          const int j = min(lane + 64 * ch, M - 1);
          acc[ch] = __builtin_fmaf(cw, crow[j], __builtin_fmaf(m0[ch], lrow[o0[ch]], m1[ch] * lrow[o1[ch]]));
        }
        // the output is written once and not read here: non-temporal stores
        // keep it from evicting the spectra the other items of this image
        // and kernel read (measured at the 224 x 224 RGB layer: 0.78 ->
        // 0.72 ms)
#pragma unroll
        for (int ch = 0; ch < MCH; ++ch) {
          if (ch >= nch) break;
          const int j = lane + 64 * ch;
          if (j < M) __builtin_nontemporal_store(acc[ch], orow + j);
        }
      }
      lds_barrier();  // the carry has been read
      const bool last = r == T - 1;
      for (int task = wave; task < nk * nov; task += nwave) {
        const int ks = task / nov, rb = task - ks * nov, ra = b + rb;
        const int i = r * b + ra - off;
        if (last && (i < 0 || i >= M)) continue;
        const float* lrow = smem + 2 * (ks * T * kSlot + ra * kV);
        float* crow = carry + (ks * nov + rb) * M;
        float* orow = p.y + ((size_t(img) * p.K + k0 + ks) * M + (last ? i : 0)) * size_t(M);
        float acc[MCH];
#pragma unroll
        for (int ch = 0; ch < MCH; ++ch) {
          if (ch >= nch) break;
          acc[ch] = __builtin_fmaf(m0[ch], lrow[o0[ch]], m1[ch] * lrow[o1[ch]]);
        }
#pragma unroll
        for (int ch = 0; ch < MCH; ++ch) {
          if (ch >= nch) break;
          const int j = lane + 64 * ch;
          if (j < M) {
            if (last)
              __builtin_nontemporal_store(acc[ch], orow + j);
            else
              crow[j] = acc[ch];
          }
        }
      }
      lds_barrier();
    }
  }
}

// ---------------------------------------------------------------------------
// error propagation

// TQ = NS / 4 blocks per item, the gradient windows of four kernels each per
// chunk.
template <int C, int NS>
__global__ void __launch_bounds__(Fz<NS>::threads) fused_bwd_data_kernel(FusedBwdDataParams p) {
  constexpr int TQ = NS / 4, NT = Fz<NS>::threads, PI = Fz<NS>::pos_iter;
  extern __shared__ float smem[];
  float2* lds = reinterpret_cast<float2*>(smem);
  const int tid = threadIdx.x, h = tid & 1, pr = tid >> 1, wave = tid >> 6, lane = tid & 63;
  constexpr int nwave = NT / 64;
  const int T = p.T, P = T * T, b = p.b, N = p.N, M = p.M;
  const long BP = long(p.B) * P;
  const long nitems = (BP + TQ - 1) / TQ;
  const int nkc = (p.K + 3) / 4;
  const SmallDiv div_b(b);
  for (long it = first_item(); it < nitems; it += gridDim.x) {
    const long t0 = TQ * it;
    const int nt = int(min<long>(TQ, BP - t0));
    float2 acc[PI][TQ][C];
#pragma unroll
    for (int i5 = 0; i5 < PI; ++i5)
#pragma unroll
      for (int tq = 0; tq < TQ; ++tq)
#pragma unroll
        for (int c = 0; c < C; ++c) acc[i5][tq][c] = make_float2(0.f, 0.f);
    for (int kc = 0; kc < nkc; ++kc) {
      const int k0 = kc * 4, nk = min(4, p.K - k0);
      {
        // gradient windows: slot ks TQ + tq, a wave per slot
        const int s = pr / kH, j = pr % kH, ks = s / TQ, tq = s - ks * TQ;
        if (ks < nk && tq < nt) {
          const long t = t0 + tq;
          const int img = int(t / P), pp = int(t - long(img) * P);
          const int prow = pp / T, qc = pp - prow * T;
          const float* plane = p.g + (size_t(img) * p.K + k0 + ks) * size_t(M) * M;
          fwd_columns(lds + s * kSlot, plane, M, prow * b - p.off, qc * b - p.off, p.S, j, h);
        }
      }
      lds_barrier();
      fwd_rows_all<NS>(lds, NS);  // inactive slots hold unread values
      lds_barrier();
      // dXhat[tq][c] += conj(W[k][c]) Ghat[k][tq] over the chunk's kernels
      int ft = tid;
      asm volatile("" : "+v"(ft));
#pragma unroll
      for (int i5 = 0; i5 < PI; ++i5) {
        if (i5 % 2 == 0) asm volatile("" ::: "memory");
        const int f = ft + i5 * NT, fl = min(f, kPos - 1);
        float2 wv[C][4];
#pragma unroll
        for (int c = 0; c < C; ++c)
#pragma unroll
          for (int ks = 0; ks < 4; ++ks) wv[c][ks] = p.ws[(size_t(k0 + min(ks, nk - 1)) * C + c) * kPos + fl];
        if (f >= kPos || !bin_used(f)) continue;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          if (ks >= nk) continue;
#pragma unroll
          for (int tq = 0; tq < TQ; ++tq) {
            if (tq >= nt) continue;
            const float2 gv = lds[(ks * TQ + tq) * kSlot + f];
#pragma unroll
            for (int c = 0; c < C; ++c) acc[i5][tq][c] = cmac_conj(acc[i5][tq][c], wv[c][ks], gv);
          }
        }
      }
      lds_barrier();
    }
    // the blocks' input-gradient spectra to slots tq C + c, inverted
#pragma unroll
    for (int i5 = 0; i5 < PI; ++i5) {
      const int f = tid + i5 * NT;
      if (f >= kPos || !bin_used(f)) continue;
#pragma unroll
      for (int tq = 0; tq < TQ; ++tq)
#pragma unroll
        for (int c = 0; c < C; ++c)
          if (tq < nt) lds[(tq * C + c) * kSlot + f] = acc[i5][tq][c];
    }
    lds_barrier();
    inverse_all<NS>(smem, nt * C, b, 0);
    lds_barrier();
    // kept b x b of each block to dx: a wave per slot, lanes over the block
    for (int qq = wave; qq < nt * C; qq += nwave) {
      const int tq = qq / C, c = qq - tq * C;
      const long t = t0 + tq;
      const int img = int(t / P), pp = int(t - long(img) * P);
      const int prow = pp / T, qc = pp - prow * T;
      const int nrow = min(b, N - prow * b), ncol = min(b, N - qc * b);
      float* oblk = p.dx + ((size_t(img) * C + c) * N + size_t(prow) * b) * N + size_t(qc) * b;
      const float* lt = smem + 2 * qq * kSlot;
      for (int e = lane; e < b * nrow; e += 64) {
        const int rr = div_b(e), cc = e - rr * b;
        if (cc < ncol) oblk[size_t(rr) * N + cc] = lt[2 * rr * kV + cc];
      }
    }
    lds_barrier();
  }
}

// ---------------------------------------------------------------------------
// weight gradient

template <int C, int KF, int NS>
__global__ void __launch_bounds__(Fz<NS>::threads) fused_bwd_filter_kernel(FusedBwdFilterParams p) {
  constexpr int TMAX = NS / KF, NT = Fz<NS>::threads, PI = Fz<NS>::pos_iter;
  extern __shared__ float smem[];
  float2* lds = reinterpret_cast<float2*>(smem);
  const int tid = threadIdx.x, h = tid & 1, pr = tid >> 1;
  const int T = p.T, b = p.b, M = p.M, K = p.K;
  const long nrows = long(p.B) * T;
  const long nitems = long(p.nkg) * p.nsplit;
  for (long it = first_item(); it < nitems; it += gridDim.x) {
    const int kg = int(it % p.nkg), sp = int(it / p.nkg);
    const int k0 = kg * KF, nk = min(KF, K - k0), ns = nk * T;
    const long R0 = long(sp) * p.rows_per_split, R1 = min(nrows, R0 + p.rows_per_split);
    float2 acc[PI][KF][C];
#pragma unroll
    for (int i5 = 0; i5 < PI; ++i5)
#pragma unroll
      for (int ks = 0; ks < KF; ++ks)
#pragma unroll
        for (int c = 0; c < C; ++c) acc[i5][ks][c] = make_float2(0.f, 0.f);
    for (long R = R0; R < R1; ++R) {
      const int img = int(R / T), prow = int(R - long(img) * T);
      {
        // gradient windows of the block row: slot ks T + q, a wave per slot
        const int s = pr / kH, j = pr % kH;
        if (s < ns) {
          const int ks = s / T, q = s - ks * T;
          const float* plane = p.g + (size_t(img) * K + k0 + ks) * size_t(M) * M;
          fwd_columns(lds + s * kSlot, plane, M, prow * b - p.off, q * b - p.off, p.S, j, h);
        }
      }
      lds_barrier();
      fwd_rows_all<NS>(lds, ns);
      lds_barrier();
      // dWhat[k][c] += conj(Xhat[c][q]) Ghat[k][q] over the row's blocks
      const float2* xrow = p.xs + size_t(R) * C * kPos * T;
      int ft = tid;
      asm volatile("" : "+v"(ft));
#pragma unroll
      for (int i5 = 0; i5 < PI; ++i5) {
        if (i5 % 2 == 0) asm volatile("" ::: "memory");
        const int f = ft + i5 * NT, fl = min(f, kPos - 1);
        float2 xv[C][TMAX];
#pragma unroll
        for (int c = 0; c < C; ++c)
#pragma unroll
          for (int q = 0; q < TMAX; ++q) xv[c][q] = xrow[(size_t(c) * kPos + fl) * T + min(q, T - 1)];
        if (f >= kPos || !bin_used(f)) continue;
#pragma unroll
        for (int ks = 0; ks < KF; ++ks) {
          if (ks >= nk) continue;
#pragma unroll
          for (int q = 0; q < TMAX; ++q) {
            if (q >= T) continue;
            const float2 gv = lds[(ks * T + q) * kSlot + f];
#pragma unroll
            for (int c = 0; c < C; ++c) acc[i5][ks][c] = cmac_conj(acc[i5][ks][c], xv[c][q], gv);
          }
        }
      }
      lds_barrier();
    }
    // partial sum of this range of block rows: [split][F][C][K]
#pragma unroll
    for (int i5 = 0; i5 < PI; ++i5) {
      const int f = tid + i5 * NT;
      if (f >= kPos || !bin_used(f)) continue;
#pragma unroll
      for (int c = 0; c < C; ++c)
#pragma unroll
        for (int ks = 0; ks < KF; ++ks)
          if (ks < nk) p.part[((size_t(sp) * kPos + f) * C + c) * K + k0 + ks] = acc[i5][ks][c];
    }
  }
}

// ---------------------------------------------------------------------------
// launchers

int fused_cu_count() {
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

// as many workgroups as are resident (LDS-bound), whole rounds over the 8
// XCDs, at most one per item
unsigned fused_grid(long items, size_t lds) {
  const long per_cu = std::max<long>(1, long(kLdsMax / std::max<size_t>(lds, 1)));
  long nwg = std::min<long>(per_cu * fused_cu_count(), (items + 7) / 8 * 8);
  nwg = std::max<long>(8, nwg / 8 * 8);
  return unsigned(nwg);
}

bool planes_ok(long n_planes, int H) {
  return H >= 1 && H < 46341 && size_t(H) * H * 4 < (size_t(1) << 31) && n_planes >= 1;
}

// Slots per workgroup: the forward takes four where the blocks of a row fit
// them (two workgroups per CU measured a little faster); the backward
// kernels take eight, so that a chunk of gradient windows covers two blocks
// (error propagation) or two kernels (weight gradient), which halves the
// reads of the kernel or input spectra (measured at the 224 x 224 RGB layer:
// 0.59 against 0.63 ms and 0.59 against 1.14 ms).
#ifndef OAA_FUSED_FWD_SLOTS
#define OAA_FUSED_FWD_SLOTS 4
#endif
int fused_slots(int T) { return T <= OAA_FUSED_FWD_SLOTS ? OAA_FUSED_FWD_SLOTS : 8; }
constexpr int kBwdSlots = 8;

// output planes (forward) or kernels (weight gradient) per item: T g <= NS
int group_for(int T, int ns) {
  if (T < 1 || T > ns) return 0;
  return 4 * T <= ns ? 4 : (2 * T <= ns ? 2 : 1);
}

template <int C, int KG, int NS>
hipError_t launch_fwd_CKN(const FusedFwdParams& p, size_t lds, hipStream_t s) {
  auto kern = fused_fwd_kernel<C, KG, NS>;
  const hipError_t e = allow_lds(kern, kLdsMax);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(fused_grid(long(p.B) * p.ngrp, lds)), dim3(Fz<NS>::threads), lds, s, p);
  return hipGetLastError();
}

template <int C>
hipError_t launch_fwd_C(const FusedFwdParams& p, int ns, size_t lds, hipStream_t s) {
  if (ns == 8) return p.Kg == 1 ? launch_fwd_CKN<C, 1, 8>(p, lds, s) : hipErrorInvalidValue;
  switch (p.Kg) {
    case 1: return launch_fwd_CKN<C, 1, 4>(p, lds, s);
    case 2: return launch_fwd_CKN<C, 2, 4>(p, lds, s);
    case 4: return launch_fwd_CKN<C, 4, 4>(p, lds, s);
    default: return hipErrorInvalidValue;
  }
}

template <int C, int NS>
hipError_t launch_bwd_data_CN(const FusedBwdDataParams& p, hipStream_t s) {
  auto kern = fused_bwd_data_kernel<C, NS>;
  const hipError_t e = allow_lds(kern, kLdsMax);
  if (e != hipSuccess) return e;
  const long BP = long(p.B) * p.T * p.T;
  constexpr int TQ = NS / 4;
  hipLaunchKernelGGL(kern, dim3(fused_grid((BP + TQ - 1) / TQ, Fz<NS>::slot_bytes)), dim3(Fz<NS>::threads),
                     Fz<NS>::slot_bytes, s, p);
  return hipGetLastError();
}

template <int C, int KF, int NS>
hipError_t launch_bwd_filter_CKN(const FusedBwdFilterParams& p, hipStream_t s) {
  auto kern = fused_bwd_filter_kernel<C, KF, NS>;
  const hipError_t e = allow_lds(kern, kLdsMax);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(fused_grid(long(p.nkg) * p.nsplit, Fz<NS>::slot_bytes)), dim3(Fz<NS>::threads),
                     Fz<NS>::slot_bytes, s, p);
  return hipGetLastError();
}

template <int C>
hipError_t launch_bwd_filter_C(const FusedBwdFilterParams& p, hipStream_t s) {
  switch (p.Kf) {
    case 1: return launch_bwd_filter_CKN<C, 1, 8>(p, s);
    case 2: return launch_bwd_filter_CKN<C, 2, 8>(p, s);
    case 4: return launch_bwd_filter_CKN<C, 4, 8>(p, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

int fused_group(int T) { return group_for(T, fused_slots(T)); }

int fused_filter_split(int B, int K, int T, int items) {
  const long kf = group_for(T, kBwdSlots);
  if (kf == 0) return 0;
  const long nkg = (K + kf - 1) / kf, rows = long(B) * T;
  return int(std::max(1L, std::min(rows, (items + nkg - 1) / nkg)));
}

size_t fused_forward_lds(int T, int n, int M) {
  const int ns = fused_slots(T), kg = group_for(T, ns);
  return size_t(ns) * kSlot * 8 + size_t(kg) * size_t(n - 1) * size_t(M) * 4;
}

bool fused_supported(int L, int C, int N, int n, int b, int T) {
  if (L != kL || C < 1 || C > kFusedMaxC || n < 1 || b < 1 || b + n - 1 > kL) return false;
  if (fused_group(T) == 0) return false;
  const int M = N - n + 1;
  if (M < 1 || !planes_ok(1, N)) return false;
  if (T != (N + b - 1) / b) return false;
  return fused_forward_lds(T, n, M) <= kLdsMax;
}

hipError_t launch_fused_forward(FusedFwdParams p, int C, hipStream_t s) {
  if (p.B < 1 || p.K < 1 || p.T < 1 || p.b < 1 || p.M < 1 || p.KR != p.b + p.off || p.KR > kL ||
      !planes_ok(long(p.B) * p.K, p.M))
    return hipErrorInvalidValue;
  const int ns = fused_slots(p.T);
  p.Kg = group_for(p.T, ns);
  if (p.Kg == 0) return hipErrorInvalidValue;
  p.ngrp = (p.K + p.Kg - 1) / p.Kg;
  const size_t lds = fused_forward_lds(p.T, p.off + 1, p.M);
  if (lds > kLdsMax) return hipErrorInvalidConfiguration;
  switch (C) {
    case 1: return launch_fwd_C<1>(p, ns, lds, s);
    case 2: return launch_fwd_C<2>(p, ns, lds, s);
    case 3: return launch_fwd_C<3>(p, ns, lds, s);
    case 4: return launch_fwd_C<4>(p, ns, lds, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_fused_bwd_data(const FusedBwdDataParams& p, int C, hipStream_t s) {
  if (p.B < 1 || p.K < 1 || p.T < 1 || p.b < 1 || p.b > kL || p.S < 1 || p.S > kL || p.off < 0 ||
      !planes_ok(long(p.B) * p.K, p.M) || !planes_ok(long(p.B) * C, p.N))
    return hipErrorInvalidValue;
  if (p.T > kBwdSlots) return hipErrorInvalidValue;
  switch (C) {
    case 1: return launch_bwd_data_CN<1, kBwdSlots>(p, s);
    case 2: return launch_bwd_data_CN<2, kBwdSlots>(p, s);
    case 3: return launch_bwd_data_CN<3, kBwdSlots>(p, s);
    case 4: return launch_bwd_data_CN<4, kBwdSlots>(p, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_fused_bwd_filter(FusedBwdFilterParams p, int C, hipStream_t s) {
  if (p.B < 1 || p.K < 1 || p.T < 1 || p.b < 1 || p.S < 1 || p.S > kL || p.off < 0 || p.nsplit < 1 ||
      !planes_ok(long(p.B) * p.K, p.M))
    return hipErrorInvalidValue;
  p.Kf = group_for(p.T, kBwdSlots);
  if (p.Kf == 0) return hipErrorInvalidValue;
  p.nkg = (p.K + p.Kf - 1) / p.Kf;
  const long nrows = long(p.B) * p.T;
  p.rows_per_split = int((nrows + p.nsplit - 1) / p.nsplit);
  switch (C) {
    case 1: return launch_bwd_filter_C<1>(p, s);
    case 2: return launch_bwd_filter_C<2>(p, s);
    case 3: return launch_bwd_filter_C<3>(p, s);
    case 4: return launch_bwd_filter_C<4>(p, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace oaa
