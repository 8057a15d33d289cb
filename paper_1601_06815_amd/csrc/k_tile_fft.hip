// Tiling + zero-padding + 2-D real FFT of blocks and windows, and the
// inverse transforms with overlap-add or crop (arXiv:1601.06815, Section 2:
// block division, padding, per-block transforms, overlap by n-1 and add).
//
// One workgroup handles a run of consecutive tiles along one block row of one
// plane. Forward: the rows of the plane that the run covers are staged in LDS
// with coalesced loads; pass 1 (one lane per pair of tile rows) transforms
// rows, pass 2 (one lane per tile column) transforms columns and writes the
// spectra bin-major with consecutive tiles in consecutive addresses. Inverse:
// the same two passes in the opposite order; the overlap-add accumulates
// whole block rows in LDS and writes each finished output row once.
#include <algorithm>

#include "fft_core.hpp"
#include "oaa_internal.hpp"

namespace oaa {

namespace {

constexpr int kMaxThreads = 256;
constexpr size_t kLdsBudget = 60 * 1024;

inline int pick_threads(int tasks) {
  int t = ((tasks + 63) / 64) * 64;
  return t < 64 ? 64 : (t > kMaxThreads ? kMaxThreads : t);
}

__host__ __device__ inline size_t even_floats(size_t n) { return (n + 1) & ~size_t(1); }

// ---------------------------------------------------------------------------
// Forward: windows -> spectra
template <int L, bool ZH>
__global__ void __launch_bounds__(kMaxThreads) tile_rfft2_kernel(TileFwdParams p) {
  constexpr int V = L / 2 + 1;
  extern __shared__ float smem[];
  const int tid = threadIdx.x, nthr = blockDim.x;
  const long wg = blockIdx.x;
  const int chunk = int(wg % p.nchunk);
  const long rest = wg / p.nchunk;
  const int strip = int(rest % p.T);
  const long plane = rest / p.T;
  const int img = int(plane / p.n_ch), ch = int(plane % p.n_ch);
  const int q0 = chunk * p.TQ;
  const int nq = min(p.TQ, p.T - q0);
  const int R = p.R, pitch = p.pitch;
  const int W = (nq - 1) * pitch + R;
  float* img_s = smem;                                                      // [R][W]
  float2* zbuf = reinterpret_cast<float2*>(smem + even_floats(size_t(R) * W));  // [R][V][TQ]

  const float* src = p.src + size_t(plane) * p.H * p.H;
  const int row0 = strip * pitch - p.off, col0 = q0 * pitch - p.off;
  for (int idx = tid; idx < R * W; idx += nthr) {
    const int r = idx / W, c = idx - r * W;
    const int gr = row0 + r, gc = col0 + c;
    float val = 0.f;
    if (gr >= 0 && gr < p.H && gc >= 0 && gc < p.H) val = src[size_t(gr) * p.H + gc];
    img_s[idx] = val;
  }
  __syncthreads();

  // pass 1: real rows, two per lane
  const int npair = (R + 1) >> 1;
  for (int task = tid; task < npair * nq; task += nthr) {
    const int q = task % nq, pr = task / nq;
    const int r0 = 2 * pr, r1 = r0 + 1;
    const bool has1 = r1 < R;
    const float* row_a = img_s + r0 * W + q * pitch;
    const float* row_b = row_a + W;
    float zr[L], zi[L];
#pragma unroll
    for (int s = 0; s < L; ++s) {
      if (ZH && s >= L / 2) {
        zr[s] = 0.f;
        zi[s] = 0.f;
      } else {
        const bool in = s < R;
        zr[s] = in ? row_a[s] : 0.f;
        zi[s] = (in && has1) ? row_b[s] : 0.f;
      }
    }
    float2 X0[V], X1[V];
    rfft_pair<L, ZH>(zr, zi, X0, X1);
#pragma unroll
    for (int v = 0; v < V; ++v) {
      zbuf[(r0 * V + v) * p.TQ + q] = X0[v];
      if (has1) zbuf[(r1 * V + v) * p.TQ + q] = X1[v];
    }
  }
  __syncthreads();

  // pass 2: complex columns, bin-major stores
  const size_t tiles_per_ch = size_t(p.n_img) * p.T * p.T;
  const size_t fstride = size_t(p.n_ch) * tiles_per_ch;
  float2* out = p.dst + size_t(ch) * tiles_per_ch + size_t(img) * p.T * p.T + size_t(strip) * p.T + q0;
  for (int task = tid; task < V * nq; task += nthr) {
    const int q = task % nq, v = task / nq;
    float re[L], im[L];
#pragma unroll
    for (int r = 0; r < L; ++r) {
      float2 z = make_float2(0.f, 0.f);
      if (!(ZH && r >= L / 2) && r < R) z = zbuf[(r * V + v) * p.TQ + q];
      re[r] = z.x;
      im[r] = z.y;
    }
    fft_dif<L, -1, ZH>(re, im);
#pragma unroll
    for (int u = 0; u < L; ++u) {
      const int pos = bitrev(u, L);
      out[size_t(u * V + v) * fstride + q] = make_float2(re[pos], im[pos]);
    }
  }
}

// ---------------------------------------------------------------------------
// Inverse column pass shared by the two inverse kernels: spectra of tiles
// [q0, q0+nq) of block row `strip` -> zbuf rows [0, R).
template <int L>
__device__ __forceinline__ void inverse_columns(const float2* in, size_t fstride, int nsplit,
                                                size_t split_stride, int nq, int TQ, int R,
                                                float2* zbuf) {
  constexpr int V = L / 2 + 1;
  for (int task = threadIdx.x; task < V * nq; task += blockDim.x) {
    const int q = task % nq, v = task / nq;
    const float2* col = in + q;
    float re[L], im[L];
#pragma unroll
    for (int u = 0; u < L; ++u) {
      float2 z = col[size_t(u * V + v) * fstride];
      for (int s = 1; s < nsplit; ++s) {
        const float2 t = col[s * split_stride + size_t(u * V + v) * fstride];
        z.x += t.x;
        z.y += t.y;
      }
      re[u] = z.x;
      im[u] = z.y;
    }
    fft_dif<L, +1, false>(re, im);
#pragma unroll
    for (int r = 0; r < L; ++r) {
      if (r < R) {
        const int pos = bitrev(r, L);
        zbuf[(r * V + v) * TQ + q] = make_float2(re[pos], im[pos]);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Inverse + overlap-add + valid crop
template <int L>
__global__ void __launch_bounds__(kMaxThreads) irfft2_overlap_add_kernel(OverlapAddParams p) {
  constexpr int V = L / 2 + 1;
  extern __shared__ float smem[];
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int n = p.n, T = p.T, M = p.M, R = 2 * n - 1;
  const int Wacc = T * n + n - 1;
  float* acc = smem;                                                          // [R][Wacc]
  float2* zbuf = reinterpret_cast<float2*>(smem + even_floats(size_t(R) * Wacc));  // [R][V][TQ]
  const long wg = blockIdx.x;
  const int grp = int(wg % p.ngroups);
  const long plane = wg / p.ngroups;
  const int img = int(plane / p.n_ch), ch = int(plane % p.n_ch);
  const int pb = grp * p.SPW, pe = min(T, pb + p.SPW);
  const size_t tiles_per_ch = size_t(p.n_img) * T * T;
  const size_t fstride = size_t(p.n_ch) * tiles_per_ch;
  const float2* in = p.src + size_t(ch) * tiles_per_ch + size_t(img) * T * T;
  float* out = p.dst + size_t(plane) * M * M;
  const float scale = 1.0f / float(L * L);

  for (int i = tid; i < R * Wacc; i += nthr) acc[i] = 0.f;
  __syncthreads();

  // block row pb-1 is recomputed (not written) to supply the rows that
  // overlap into block row pb
  for (int strip = (pb > 0 ? pb - 1 : 0); strip < pe; ++strip) {
    for (int q0 = 0; q0 < T; q0 += p.TQ) {
      const int nq = min(p.TQ, T - q0);
      inverse_columns<L>(in + size_t(strip) * T + q0, fstride, 1, 0, nq, p.TQ, R, zbuf);
      __syncthreads();
      // rows, in two passes over tiles of even and odd block column so that
      // the overlapping tiles of one pass never touch the same pixel
      for (int parity = 0; parity < 2; ++parity) {
        const int first = (parity - q0) & 1;
        const int cnt = nq > first ? (nq - first + 1) / 2 : 0;
        for (int task = tid; task < n * cnt; task += nthr) {
          const int j = task % cnt, pr = task / cnt;
          const int q = first + 2 * j;
          const int r0 = 2 * pr, r1 = r0 + 1;
          const bool has1 = r1 < R;
          float2 A[V], Bv[V];
#pragma unroll
          for (int v = 0; v < V; ++v) {
            A[v] = zbuf[(r0 * V + v) * p.TQ + q];
            Bv[v] = has1 ? zbuf[(r1 * V + v) * p.TQ + q] : make_float2(0.f, 0.f);
          }
          float zr[L], zi[L];
          irfft_pair<L>(A, Bv, zr, zi);
          float* d0 = acc + r0 * Wacc + (q0 + q) * n;
#pragma unroll
          for (int s = 0; s < L; ++s) {
            if (s < R) {
              const int pos = bitrev(s, L);
              d0[s] += zr[pos] * scale;
              if (has1) d0[Wacc + s] += zi[pos] * scale;
            }
          }
        }
        __syncthreads();
      }
    }
    if (strip >= pb) {
      for (int idx = tid; idx < n * M; idx += nthr) {
        const int r = idx / M, j = idx - r * M;
        const int i = strip * n + r - (n - 1);
        if (i >= 0 && i < M) out[size_t(i) * M + j] = acc[r * Wacc + j + n - 1];
      }
    }
    __syncthreads();
    for (int idx = tid; idx < (n - 1) * Wacc; idx += nthr) acc[idx] = acc[n * Wacc + idx];
    __syncthreads();
    for (int idx = tid; idx < n * Wacc; idx += nthr) acc[(n - 1) * Wacc + idx] = 0.f;
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Inverse + top-left n x n crop, scattered to the blocks of the output planes
template <int L>
__global__ void __launch_bounds__(kMaxThreads) irfft2_crop_kernel(CropParams p) {
  constexpr int V = L / 2 + 1;
  extern __shared__ float smem[];
  const int tid = threadIdx.x, nthr = blockDim.x;
  float2* zbuf = reinterpret_cast<float2*>(smem);  // [n][V][TQ]
  const long wg = blockIdx.x;
  const int chunk = int(wg % p.nchunk);
  const long rest = wg / p.nchunk;
  const int strip = int(rest % p.T);
  const long plane = rest / p.T;
  const int img = int(plane / p.n_ch), ch = int(plane % p.n_ch);
  const int q0 = chunk * p.TQ;
  const int nq = min(p.TQ, p.T - q0);
  const int n = p.n, H = p.H;
  const size_t tiles_per_ch = size_t(p.n_img) * p.T * p.T;
  const size_t fstride = size_t(p.n_ch) * tiles_per_ch;
  const float2* in =
      p.src + size_t(ch) * tiles_per_ch + size_t(img) * p.T * p.T + size_t(strip) * p.T + q0;
  inverse_columns<L>(in, fstride, p.nsplit, p.split_stride, nq, p.TQ, n, zbuf);
  __syncthreads();
  float* out = p.dst + size_t(plane) * H * H;
  const float scale = 1.0f / float(L * L);
  const int npair = (n + 1) >> 1;
  for (int task = tid; task < npair * nq; task += nthr) {
    const int q = task % nq, pr = task / nq;
    const int r0 = 2 * pr, r1 = r0 + 1;
    const bool has1 = r1 < n;
    float2 A[V], Bv[V];
#pragma unroll
    for (int v = 0; v < V; ++v) {
      A[v] = zbuf[(r0 * V + v) * p.TQ + q];
      Bv[v] = has1 ? zbuf[(r1 * V + v) * p.TQ + q] : make_float2(0.f, 0.f);
    }
    float zr[L], zi[L];
    irfft_pair<L>(A, Bv, zr, zi);
    const int gr0 = strip * n + r0, gc0 = (q0 + q) * n;
#pragma unroll
    for (int s = 0; s < L; ++s) {
      if (s < n && gc0 + s < H) {
        const int pos = bitrev(s, L);
        if (gr0 < H) out[size_t(gr0) * H + gc0 + s] = zr[pos] * scale;
        if (has1 && gr0 + 1 < H) out[size_t(gr0 + 1) * H + gc0 + s] = zi[pos] * scale;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// launchers

template <int L, bool ZH>
hipError_t launch_fwd_L(TileFwdParams p, hipStream_t s) {
  constexpr int V = L / 2 + 1;
  auto lds_for = [&](int tq) {
    const size_t W = size_t(tq - 1) * p.pitch + p.R;
    return even_floats(size_t(p.R) * W) * 4 + size_t(p.R) * V * tq * 8;
  };
  int nchunk = 1;
  while (nchunk < p.T && lds_for((p.T + nchunk - 1) / nchunk) > kLdsBudget) ++nchunk;
  p.TQ = (p.T + nchunk - 1) / nchunk;
  p.nchunk = (p.T + p.TQ - 1) / p.TQ;
  const size_t lds = lds_for(p.TQ);
  if (lds > kLdsBudget) return hipErrorInvalidConfiguration;
  const int tasks = std::max(((p.R + 1) / 2) * p.TQ, V * p.TQ);
  const long nwg = long(p.n_img) * p.n_ch * p.T * p.nchunk;
  hipLaunchKernelGGL((tile_rfft2_kernel<L, ZH>), dim3(unsigned(nwg)), dim3(pick_threads(tasks)), lds, s, p);
  return hipGetLastError();
}

template <int L>
hipError_t launch_oa_L(OverlapAddParams p, hipStream_t s) {
  constexpr int V = L / 2 + 1;
  const int R = 2 * p.n - 1;
  const size_t acc_bytes = even_floats(size_t(R) * (size_t(p.T) * p.n + p.n - 1)) * 4;
  const size_t per_tile = size_t(R) * V * 8;
  size_t budget = kLdsBudget;
  if (acc_bytes + per_tile > budget) budget = 160 * 1024;  // gfx950: 160 KiB per workgroup
  if (acc_bytes + per_tile > budget) return hipErrorInvalidConfiguration;
  int tq = int(std::min<size_t>(p.T, (budget - acc_bytes) / per_tile));
  const int nchunk = (p.T + tq - 1) / tq;
  p.TQ = (p.T + nchunk - 1) / nchunk;
  p.nchunk = nchunk;
  const long planes = long(p.n_img) * p.n_ch;
  int ngroups = 1;
  if (planes < 2048) ngroups = int(std::min<long>(p.T, (2048 + planes - 1) / planes));
  p.SPW = (p.T + ngroups - 1) / ngroups;
  p.ngroups = (p.T + p.SPW - 1) / p.SPW;
  const size_t lds = acc_bytes + per_tile * p.TQ;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&irfft2_overlap_add_kernel<L>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (e != hipSuccess) return e;
  }
  const int tasks = std::max(V * p.TQ, p.n * ((p.TQ + 1) / 2));
  hipLaunchKernelGGL(irfft2_overlap_add_kernel<L>, dim3(unsigned(planes * p.ngroups)),
                     dim3(pick_threads(tasks)), lds, s, p);
  return hipGetLastError();
}

template <int L>
hipError_t launch_crop_L(CropParams p, hipStream_t s) {
  constexpr int V = L / 2 + 1;
  const size_t per_tile = size_t(p.n) * V * 8;
  int tq = int(std::min<size_t>(p.T, kLdsBudget / per_tile));
  const int nchunk = (p.T + tq - 1) / tq;
  p.TQ = (p.T + nchunk - 1) / nchunk;
  p.nchunk = nchunk;
  const size_t lds = per_tile * p.TQ;
  const int tasks = std::max(V * p.TQ, ((p.n + 1) / 2) * p.TQ);
  const long nwg = long(p.n_img) * p.n_ch * p.T * p.nchunk;
  hipLaunchKernelGGL(irfft2_crop_kernel<L>, dim3(unsigned(nwg)), dim3(pick_threads(tasks)), lds, s, p);
  return hipGetLastError();
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

hipError_t launch_irfft2_overlap_add(int L, const OverlapAddParams& p, hipStream_t s) {
  switch (L) {
    case 2: return launch_oa_L<2>(p, s);
    case 4: return launch_oa_L<4>(p, s);
    case 8: return launch_oa_L<8>(p, s);
    case 16: return launch_oa_L<16>(p, s);
    case 32: return launch_oa_L<32>(p, s);
    case 64: return launch_oa_L<64>(p, s);
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
