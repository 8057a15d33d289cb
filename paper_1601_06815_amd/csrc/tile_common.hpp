// Device helpers shared by the tile transform kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <mutex>
#include <set>
#include <utility>

#include "buffer_io.hpp"
#include "fft_core.hpp"

// Launch-shape defaults (tiles per workgroup along a block row, register
// prefetch of the next rows); overridable at build time for tuning sweeps.
#ifndef OAA_WINDOW_TQ_MAX
#define OAA_WINDOW_TQ_MAX 64
#endif
#ifndef OAA_WINDOW_ROWS
#define OAA_WINDOW_ROWS 1
#endif
// Consecutive tiles a step of the several-rows window transform aims for
// where no run of whole 128-byte lines is within reach, and the LDS per
// workgroup it may grow to for them (measured: runs of 69 tiles at first224
// cut its gradient windows from 1.17 to 0.92 ms, runs of 28 the overlap-save
// input windows at large128 from 0.33 to 0.30 ms; at large128's T = 8,
// runs of 24 tiles were slower than the line-aligned runs of 16).
#ifndef OAA_WINDOW_MIN_RUN
#define OAA_WINDOW_MIN_RUN 48
#endif
#ifndef OAA_WINDOW_GROW_LDS
#define OAA_WINDOW_GROW_LDS 81920
#endif
#ifndef OAA_WINDOW_PREFETCH
#define OAA_WINDOW_PREFETCH 1
#endif
#ifndef OAA_FOLD_RUNS
#define OAA_FOLD_RUNS 1
#endif
#ifndef OAA_FOLD_TQ_MAX
#define OAA_FOLD_TQ_MAX 64
#endif
#ifndef OAA_OVERLAP_ROWS
#define OAA_OVERLAP_ROWS 1
#endif
#ifndef OAA_OVERLAP_MIN_WG
#define OAA_OVERLAP_MIN_WG 4096
#endif
#ifndef OAA_OVERLAP_TQ_MAX
#define OAA_OVERLAP_TQ_MAX 64
#endif
#ifndef OAA_FWD_TQ_MAX
#define OAA_FWD_TQ_MAX 64
#endif
#ifndef OAA_CROP_O32
#define OAA_CROP_O32 1
#endif
#ifndef OAA_CROP_TQ_MAX
#define OAA_CROP_TQ_MAX 64
#endif
// LDS per workgroup of the inverse with crop (40 KB: four per CU)
#ifndef OAA_CROP_LDS
#define OAA_CROP_LDS 40960
#endif

// Minimum waves per SIMD asked of the register allocator, per transform
// kernel, for L <= 32 (1: no constraint). L = 64 always takes what it needs.
#ifndef OAA_WAVES_TILE
#define OAA_WAVES_TILE 1
#endif
#ifndef OAA_WAVES_WINDOW
#define OAA_WAVES_WINDOW 1
#endif
#ifndef OAA_WAVES_FOLD
#define OAA_WAVES_FOLD 1
#endif
#ifndef OAA_WAVES_CROP
#define OAA_WAVES_CROP 1
#endif

namespace oaa {
namespace tile {

template <int L>
constexpr int fft_waves(int want) { return L <= 32 ? want : 1; }

constexpr int kMaxThreads = 256;
constexpr size_t kLdsBudget = 60 * 1024;
// LDS of the kernels that transform several window rows per step (at most:
// two workgroups per CU)
constexpr size_t kLdsRowsBudget = 80 * 1024;
// Lets a kernel take up to `bytes` of dynamic LDS (beyond 64 KB) on the
// current device; set once per kernel and device (kernels of one signature
// share the function type, so the record is kept per kernel address).
template <class Kern>
hipError_t allow_lds(Kern kern, size_t bytes) {
  static std::mutex mu;
  static std::set<std::pair<const void*, int>> done;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const void* fn = reinterpret_cast<const void*>(kern);
  std::lock_guard<std::mutex> lock(mu);
  if (!done.count({fn, dev})) {
    e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, int(bytes));
    if (e != hipSuccess) return e;
    done.insert({fn, dev});
  }
  return hipSuccess;
}

inline int pick_threads(int tasks) {
  int t = ((tasks + 63) / 64) * 64;
  return t < 64 ? 64 : (t > kMaxThreads ? kMaxThreads : t);
}

__host__ __device__ inline int odd_at_least(int v) { return v | 1; }
// Smallest row stride >= w that is 1 mod 32 (words): lanes that read the same
// column of different LDS rows then fall in different banks.
__host__ __device__ inline int bank_stride(int w) { return w + ((33 - (w & 31)) & 31); }
__host__ __device__ inline size_t even_floats(size_t n) { return (n + 1) & ~size_t(1); }

// Workgroups are dispatched round-robin over the 8 XCDs, each with its own L2.
// Renumber them so that logically consecutive workgroups (neighbouring tiles,
// which share cache lines of their inputs and outputs) run on the same XCD at
// about the same time.
__device__ __forceinline__ unsigned xcd_local_order(unsigned w, unsigned nwg) {
  const unsigned q = nwg / 8, r = nwg % 8, x = w % 8, j = w / 8;
  return x * q + min(x, r) + j;
}

// Copy rows [row0, row0+R) x columns [col0, col0+W) of an H x H plane into
// LDS rows of stride Wp (zero outside the plane). Lanes are laid out along
// the columns; each lane issues up to kUnroll independent loads (clamped to a
// valid address when out of range) before storing any of them.
constexpr int kUnroll = 8;

__device__ __forceinline__ void stage_rows(float* dst, int Wp, const float* src, int H, int row0, int col0,
                                           int R, int W) {
  const int nthr = blockDim.x, tid = threadIdx.x;
  const int Wt = W < nthr ? W : nthr;
  const int rstep = nthr / Wt;
  const int cl = tid % Wt, rl = tid / Wt;
  if (rl >= rstep) return;
  for (int c = cl; c < W; c += Wt) {
    const int gc = col0 + c;
    const bool col_ok = gc >= 0 && gc < H;
    for (int rb = rl; rb < R; rb += kUnroll * rstep) {
      float v[kUnroll];
#pragma unroll
      for (int j = 0; j < kUnroll; ++j) {
        const int r = rb + j * rstep;
        const int gr = row0 + r;
        const bool ok = col_ok && r < R && gr >= 0 && gr < H;
        const float t = src[ok ? size_t(gr) * H + gc : 0];
        v[j] = ok ? t : 0.f;
      }
#pragma unroll
      for (int j = 0; j < kUnroll; ++j) {
        const int r = rb + j * rstep;
        if (r < R) dst[r * Wp + c] = v[j];
      }
    }
  }
}

// Loads and stores of global memory at byte offset `boff` from a
// wave-uniform base: the compiler then addresses with the base in scalar
// registers and a 32-bit lane offset, with no 64-bit arithmetic per access.
// The global address space is spelled out, since a generic pointer (one
// rebuilt from integers, say) would compile to flat accesses, which also
// count as LDS operations in the wave's wait counters.
template <class T>
using global_t = __attribute__((address_space(1))) T;
typedef float f2_native __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float2 load_at(const float2* base, unsigned boff) {
  const f2_native t = *(const global_t<f2_native>*)((const global_t<char>*)(base) + boff);
  return make_float2(t.x, t.y);
}
__device__ __forceinline__ float load_at(const float* base, unsigned boff) {
  return *(const global_t<float>*)((const global_t<char>*)(base) + boff);
}
__device__ __forceinline__ void store_at(float2* base, unsigned boff, float2 v) {
  *(global_t<f2_native>*)((global_t<char>*)(base) + boff) = f2_native{v.x, v.y};
}
__device__ __forceinline__ void store_at(float* base, unsigned boff, float v) {
  *(global_t<float>*)((global_t<char>*)(base) + boff) = v;
}

// x / d for 0 <= x < 2^16 and 0 < d < 2^16 without a division: for d >= 2,
// m = floor((2^32 - 1) / d) + 1 lies in (2^32 / d, 2^32 / d + 1], so x m / 2^32
// exceeds x / d by less than x / 2^32 < 1 / d and its floor is x / d. d = 1
// (where m would be 2^32) is taken apart.
struct SmallDiv {
  int d;
  unsigned m;
  __device__ __forceinline__ explicit SmallDiv(int d_) : d(d_), m(d_ > 1 ? 0xffffffffu / unsigned(d_) + 1u : 0u) {}
  __device__ __forceinline__ int operator()(int x) const { return d > 1 ? int(__umulhi(unsigned(x), m)) : x; }
};

// Advances a wave-uniform pointer by `step` elements. The empty asm keeps
// the pointer in one scalar register pair: without it the compiler
// precomputes the addresses of a whole unrolled loop and runs out of scalar
// registers.
template <class T>
__device__ __forceinline__ void advance_uniform(T*& ptr, size_t step) {
  const unsigned long long a = reinterpret_cast<unsigned long long>(ptr + step);
  unsigned lo = __builtin_amdgcn_readfirstlane(unsigned(a));
  unsigned hi = __builtin_amdgcn_readfirstlane(unsigned(a >> 32));
  asm volatile("" : "+s"(lo), "+s"(hi));
  ptr = reinterpret_cast<T*>((static_cast<unsigned long long>(hi) << 32) | lo);
}

// Register copy of rows [row0, row0+R) x columns [col0, col0+W) of an H x H
// plane (zero outside), for W <= lanes: lane t holds column t % W of rows
// t / W + j * (lanes / W), j < MAXE. Loaded early and stored to LDS later,
// so the loads of the next rows overlap the work on the current ones.
template <int MAXE>
struct RowPrefetch {
  float v[MAXE];

  // whether R x W fits this scheme with blockDim.x lanes
  __device__ __forceinline__ static bool fits(int R, int W) {
    const int nthr = blockDim.x;
    if (W > nthr) return false;
    const int rstep = nthr / W;
    return (R + rstep - 1) / rstep <= MAXE;
  }

  __device__ __forceinline__ void load(const float* src, int H, int row0, int col0, int R, int W) {
    const int nthr = blockDim.x, tid = threadIdx.x;
    const int rstep = nthr / W, c = tid % W, rl = tid / W;
    const int gc = col0 + c;
    const bool col_ok = rl < rstep && gc >= 0 && gc < H;
#pragma unroll
    for (int j = 0; j < MAXE; ++j) {
      const int r = rl + j * rstep;
      const int gr = row0 + r;
      const bool ok = col_ok && r < R && gr >= 0 && gr < H;
      const float t = src[ok ? size_t(gr) * H + gc : 0];
      v[j] = ok ? t : 0.f;
    }
  }

  __device__ __forceinline__ void store(float* dst, int Wp, int R, int W) const {
    const int nthr = blockDim.x, tid = threadIdx.x;
    const int rstep = nthr / W, c = tid % W, rl = tid / W;
    if (rl >= rstep) return;
#pragma unroll
    for (int j = 0; j < MAXE; ++j) {
      const int r = rl + j * rstep;
      if (r < R) dst[r * Wp + c] = v[j];
    }
  }
};

// e^{SIGN * 2 pi i k / L} for any integer k (table lookup; a wave-uniform k
// becomes a scalar load)
template <int L, int SIGN>
__device__ __forceinline__ float2 twiddle(int k) {
  const int m = k & (L - 1);
  const float s = tw::kTable<L>.s[m];
  return make_float2(tw::kTable<L>.c[m], SIGN > 0 ? s : -s);
}

// a + b * c (complex)
__device__ __forceinline__ float2 cmad(float2 a, float2 b, float2 c) {
  return make_float2(__builtin_fmaf(b.x, c.x, __builtin_fmaf(-b.y, c.y, a.x)),
                     __builtin_fmaf(b.x, c.y, __builtin_fmaf(b.y, c.x, a.y)));
}

}  // namespace tile
}  // namespace oaa
