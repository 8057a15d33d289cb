// Per-frequency-bin complex contraction (arXiv:1601.06815, Introduction and
// Section 2: the Hadamard product of block and kernel spectra, summed over the
// C channels of the layer; Section 3.2 for the two backward products).
//
// For every bin f (the unique bins only, see unique_bin) the three passes are
// complex matrix products:
//   forward          Yhat[f]  (K x BP) = What[f]^T   (K x C)  * Xhat[f] (C x BP)
//   backward_data    dXhat[f] (C x BP) = conj What[f] (C x K)  * Ghat[f] (K x BP)
//   backward_filter  dWhat[f] (C x K)  = conj Xhat[f] (C x BP) * Ghat[f]^T (BP x K)
// and, to compose two stacked layers in the frequency domain (Conclusion),
//   W12hat[f] (C x K) = W1hat[f] (C x J) * W2hat[f] (J x K).
//
// Two implementations, both staging 16-deep slices of the reduction for one
// output tile through LDS as separate real and imaginary planes, with the
// next slice loaded into registers while the current one is consumed:
//  * vector ALU: 64 x 64 complex tile per 256-lane workgroup, 4 x 4 complex
//    accumulators per lane, four real multiply-adds per complex one;
//  * fp32 matrix cores (v_mfma_f32_16x16x4f32): 128 x 64 (or 96 x 64, or
//    64 x 96) complex tile per workgroup, persistent workgroups walking the
//    tiles in XCD-local rounds, operands read through buffer resources, LDS
//    slices laid out so that one 16-byte read serves four matrix-core steps,
//    and three real products per complex multiply-add (Gauss's form).
#include <algorithm>

#include "buffer_io.hpp"
#include "oaa_internal.hpp"

// Minimum waves per SIMD asked of the register allocator for the
// matrix-core kernel, and its 16-column blocks per wave (tile width / 32);
// overridable at build time for tuning sweeps.
#ifndef OAA_WAVES_GEMM
#define OAA_WAVES_GEMM 2
#endif
#ifndef OAA_GEMM_NB
#define OAA_GEMM_NB 2
#endif
// Matrix-core step of a slice after which the next slice goes to LDS (0..3).
#ifndef OAA_GEMM_STORE_STEP
#define OAA_GEMM_STORE_STEP 2
#endif

namespace oaa {

namespace {

constexpr int kThreads = 256;
constexpr int kKC = 16;  // reduction depth of one LDS slice

// A ROWS x kKC slice of an operand whose element (row, k) is stored at
// X[k*ld + row] (ROW_CONTIG) or X[row*ld + k]; loads are coalesced along the
// contiguous index. Out-of-range elements read a valid clamped address and
// are replaced by zero.
template <bool ROW_CONTIG, int ROWS>
struct Slice {
  static constexpr int PER = ROWS * kKC / kThreads;
  float2 v[PER];

  __device__ __forceinline__ static void coords(int e, int& rl, int& kl) {
    if (ROW_CONTIG) {
      rl = e % ROWS;
      kl = e / ROWS;
    } else {
      kl = e % kKC;
      rl = e / kKC;
    }
  }

  __device__ __forceinline__ void load(const float2* X, long ld, int r0, int nrows, int k0, int kend) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      int rl, kl;
      coords(int(threadIdx.x) + kThreads * i, rl, kl);
      const int r = r0 + rl, k = k0 + kl;
      const bool ok = r < nrows && k < kend;
      const int rc = ok ? r : r0, kc = ok ? k : k0;
      const float2 t = ROW_CONTIG ? X[size_t(kc) * ld + rc] : X[size_t(rc) * ld + kc];
      v[i] = ok ? t : make_float2(0.f, 0.f);
    }
  }

  template <int LD>
  __device__ __forceinline__ void store(float (*re)[LD], float (*im)[LD], bool conj) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      int rl, kl;
      coords(int(threadIdx.x) + kThreads * i, rl, kl);
      re[kl][rl] = v[i].x;
      im[kl][rl] = conj ? -v[i].y : v[i].y;
    }
  }
};

struct TileCoords {
  int f, split, m0, n0, k_begin, k_end;
};

template <int TM, int TN>
__device__ __forceinline__ TileCoords tile_coords(const GemmParams& p) {
  TileCoords t;
  t.f = unique_bin(blockIdx.z, p.L);
  t.split = blockIdx.y;
  const int tiles_n = (p.N + TN - 1) / TN;
  t.m0 = (blockIdx.x / tiles_n) * TM;
  t.n0 = (blockIdx.x % tiles_n) * TN;
  t.k_begin = t.split * p.kchunk;
  t.k_end = min(p.Kr, t.k_begin + p.kchunk);
  return t;
}

// ---------------------------------------------------------------------------
// vector-ALU implementation

constexpr int kVM = 64, kVN = 64;

template <bool AT, bool AC, bool BT, bool BC>
__global__ void __launch_bounds__(kThreads) cgemm_valu_kernel(GemmParams p) {
  __shared__ float Asr[kKC][kVM + 4], Asi[kKC][kVM + 4];
  __shared__ float Bsr[kKC][kVN + 4], Bsi[kKC][kVN + 4];
  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;
  const TileCoords tc = tile_coords<kVM, kVN>(p);
  const float2* A = p.A + size_t(tc.f) * p.a_fstride;
  const float2* B = p.B + size_t(tc.f) * p.b_fstride;

  float accr[4][4], acci[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) accr[i][j] = acci[i][j] = 0.f;

  Slice<AT, kVM> sa;
  Slice<!BT, kVN> sb;
  sa.load(A, p.lda, tc.m0, p.M, tc.k_begin, tc.k_end);
  sb.load(B, p.ldb, tc.n0, p.N, tc.k_begin, tc.k_end);
  for (int k0 = tc.k_begin; k0 < tc.k_end; k0 += kKC) {
    sa.template store<kVM + 4>(Asr, Asi, AC);
    sb.template store<kVN + 4>(Bsr, Bsi, BC);
    __syncthreads();
    if (k0 + kKC < tc.k_end) {
      sa.load(A, p.lda, tc.m0, p.M, k0 + kKC, tc.k_end);
      sb.load(B, p.ldb, tc.n0, p.N, k0 + kKC, tc.k_end);
    }
#pragma unroll
    for (int kk = 0; kk < kKC; ++kk) {
      float ar[4], ai[4], br[4], bi[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        ar[i] = Asr[kk][ty + 16 * i];
        ai[i] = Asi[kk][ty + 16 * i];
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        br[j] = Bsr[kk][tx + 16 * j];
        bi[j] = Bsi[kk][tx + 16 * j];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          accr[i][j] = __builtin_fmaf(ar[i], br[j], accr[i][j]);
          accr[i][j] = __builtin_fmaf(-ai[i], bi[j], accr[i][j]);
          acci[i][j] = __builtin_fmaf(ar[i], bi[j], acci[i][j]);
          acci[i][j] = __builtin_fmaf(ai[i], br[j], acci[i][j]);
        }
    }
    __syncthreads();
  }

  float2* Cm = p.C + size_t(tc.f) * p.c_fstride + size_t(tc.split) * p.c_sstride;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = tc.m0 + ty + 16 * i;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int nn = tc.n0 + tx + 16 * j;
      if (m < p.M && nn < p.N) Cm[size_t(m) * p.ldc + nn] = make_float2(accr[i][j], acci[i][j]);
    }
  }
}

// ---------------------------------------------------------------------------
// matrix-core implementation

typedef float floatx4 __attribute__((ext_vector_type(4)));

// LDS layout of an operand slice: [row][k'] with separate real and imaginary
// planes, k' = (k % 4) * (kKC / 4) + k / 4. The matrix-core step s of a slice
// uses reduction index k = 4 s + (lane / 16), so one 16-byte read gives a
// lane its values for all four steps of a slice. Rows are padded to kLdk
// floats, which keeps those reads and the stores below free of bank
// conflicts (at most two-way for k-contiguous operands).
constexpr int kLdk = kKC + 4;
__device__ __forceinline__ constexpr int kperm(int k) { return (k % 4) * (kKC / 4) + k / 4; }

// One operand's ROWS x kKC slices, read through a buffer resource over one
// bin's matrix; element (row, k) is at k*ld + row (ROW_CONTIG) or row*ld + k.
// Per tile, each lane computes the byte offsets of its elements relative to
// the slice start (an offset past the resource for rows outside the matrix,
// which the hardware reads as zero); per slice only a scalar offset changes.
//  * ROW_CONTIG: lane t < G*ROWS (G = 256 / ROWS, 2 or 4) takes row t % ROWS
//    and reduction indices t / ROWS + G i; loads are coalesced along rows,
//    and each lane's values form runs of four in k', stored with 16-byte
//    writes. The resource ends at the tile's reduction bound.
//  * k-contiguous: lane t takes k = t % kKC of rows t / kKC + (256/kKC) i;
//    loads are coalesced along k; elements past the reduction bound are
//    redirected out of range per slice.
template <bool ROW_CONTIG, int ROWS>
struct Operand {
  static constexpr int G = ROW_CONTIG ? (kThreads / ROWS >= 4 ? 4 : 2) : 1;
  static constexpr int PER = ROW_CONTIG ? kKC / G : ROWS * kKC / kThreads;
  static_assert(!ROW_CONTIG || (ROWS == 64 || ROWS == 96 || ROWS == 128), "row tile");
  unsigned voff[PER];
  float2 v[PER];
  int kl;  // k-contiguous: this lane's reduction index within a slice

  __device__ __forceinline__ bool active() const {
    return !ROW_CONTIG || int(threadIdx.x) < G * ROWS;
  }

  __device__ __forceinline__ void set_tile(int r0, int nrows, unsigned ld) {
    const int t = threadIdx.x;
    if (ROW_CONTIG) {
      const int r = r0 + t % ROWS, kg = t / ROWS;
      const bool ok = r < nrows && active();
#pragma unroll
      for (int i = 0; i < PER; ++i) voff[i] = ok ? (unsigned(kg + G * i) * ld + unsigned(r)) * 8u : kOutOfRange;
    } else {
      kl = t % kKC;
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int r = r0 + t / kKC + (kThreads / kKC) * i;
        voff[i] = r < nrows ? (unsigned(r) * ld + unsigned(kl)) * 8u : kOutOfRange;
      }
    }
  }

  // slice starting at reduction index k0 of a tile whose reduction ends at
  // ke, from a matrix of `elems` elements at base. The resource starts at the
  // slice, so that the hardware's range check sees only the lane offsets.
  __device__ __forceinline__ void load(const float2* base, size_t elems, unsigned ld, int k0, int ke) {
    if (ROW_CONTIG) {
      const __amdgpu_buffer_rsrc_t rs = buffer_resource(base + size_t(k0) * ld, unsigned(ke - k0) * ld * 8u);
#pragma unroll
      for (int i = 0; i < PER; ++i)
        v[i] = buffer_load_f2(rs, voff[i]);
    } else {
      const __amdgpu_buffer_rsrc_t rs = buffer_resource(base + k0, unsigned(elems - size_t(k0)) * 8u);
      const bool kok = kl < ke - k0;
#pragma unroll
      for (int i = 0; i < PER; ++i)
        v[i] = buffer_load_f2(rs, kok ? voff[i] : kOutOfRange);
    }
  }

  __device__ __forceinline__ void store(float (*re)[kLdk], float (*im)[kLdk], bool conj) const {
    const int t = threadIdx.x;
    if (ROW_CONTIG) {
      if (!active()) return;
      const int r = t % ROWS, kg = t / ROWS;
      // values i = q + (4/G) m, m < 4, share k % 4 = (kg + G q) % 4 and have k / 4 = m + const
#pragma unroll
      for (int q = 0; q < 4 / G; ++q) {
        const int kp = kperm(kg + G * q);
        floatx4 xr, xi;
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          xr[m] = v[q + (4 / G) * m].x;
          xi[m] = conj ? -v[q + (4 / G) * m].y : v[q + (4 / G) * m].y;
        }
        *reinterpret_cast<floatx4*>(&re[r][kp]) = xr;
        *reinterpret_cast<floatx4*>(&im[r][kp]) = xi;
      }
    } else {
      const int kp = kperm(kl);
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int r = t / kKC + (kThreads / kKC) * i;
        re[r][kp] = v[i].x;
        im[r][kp] = conj ? -v[i].y : v[i].y;
      }
    }
  }
};

// One output tile of the logical tile sequence: bin, split, row tile, column
// tile (fastest).
struct MfmaTile {
  int f, split, m0, n0, kb, ke;
};

template <int TM, int TN>
__device__ __forceinline__ MfmaTile mfma_tile(const GemmParams& p, unsigned t, unsigned tiles_m, unsigned tiles_n) {
  MfmaTile c;
  c.n0 = int(t % tiles_n) * TN;
  t /= tiles_n;
  c.m0 = int(t % tiles_m) * TM;
  t /= tiles_m;
  c.split = int(t % unsigned(p.nsplit));
  c.f = unique_bin(int(t / unsigned(p.nsplit)), p.L);
  c.kb = c.split * p.kchunk;
  c.ke = min(p.Kr, c.kb + p.kchunk);
  return c;
}

// Persistent matrix-core contraction. MB x NB blocks of 16 x 16 per wave,
// waves in a 2 x 2 grid: tile (32*MB) x (32*NB) complex per workgroup. The
// grid (a multiple of 8 workgroups) walks the logical tile sequence in
// rounds; in each round the workgroups of one XCD take consecutive tiles, so
// that tiles sharing operand slices share that XCD's L2. Each workgroup
// streams the reduction slices of all its tiles through one double-buffered
// LDS pipeline: the first slice of its next tile is loaded while the last
// slice of the current one is multiplied.
//
// Each complex multiply-add uses three real products (Gauss): with
// p1 = sum ar br, p2 = sum ai bi and p3 = sum (ar + ai)(br + bi), the result
// is re = p1 - p2, im = p3 - p1 - p2.
template <int MB, int NB, bool AT, bool AC, bool BT, bool BC>
__global__ void __launch_bounds__(kThreads, OAA_WAVES_GEMM) cgemm_mfma_kernel(GemmParams p, unsigned ntiles) {
  constexpr int TM = 32 * MB, TN = 32 * NB;
  __shared__ __attribute__((aligned(16))) float Asr[2][TM][kLdk], Asi[2][TM][kLdk];
  __shared__ __attribute__((aligned(16))) float Bsr[2][TN][kLdk], Bsi[2][TN][kLdk];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * 16 * MB, wn = (wave & 1) * 16 * NB;
  const int lr = lane & 15;  // operand row (A) / column (B) within a 16-block
  const int lk = lane >> 4;  // reduction index within a matrix-core step

  const unsigned tiles_m = (p.M + TM - 1) / TM, tiles_n = (p.N + TN - 1) / TN;
  const unsigned nwg = gridDim.x;
  unsigned ct = (blockIdx.x % 8) * (nwg / 8) + blockIdx.x / 8;  // this workgroup's first tile
  if (ct >= ntiles) return;
  MfmaTile cur = mfma_tile<TM, TN>(p, ct, tiles_m, tiles_n);
  int ck = cur.kb;
  // load cursor: one slice ahead of the compute cursor
  unsigned lt = ct;
  MfmaTile nx = cur;
  int lkk = ck;

  Operand<AT, TM> sa;
  Operand<!BT, TN> sb;
  auto set_tile = [&](const MfmaTile& t) {
    sa.set_tile(t.m0, p.M, unsigned(p.lda));
    sb.set_tile(t.n0, p.N, unsigned(p.ldb));
  };
  auto load_slice = [&](const MfmaTile& t, int k0) {
    sa.load(p.A + size_t(t.f) * p.a_fstride, p.a_fstride, unsigned(p.lda), k0, t.ke);
    sb.load(p.B + size_t(t.f) * p.b_fstride, p.b_fstride, unsigned(p.ldb), k0, t.ke);
  };
  auto advance = [&](unsigned& t, MfmaTile& c, int& k, bool reload) {
    k += kKC;
    if (k >= c.ke) {
      t += nwg;
      if (t < ntiles) {
        c = mfma_tile<TM, TN>(p, t, tiles_m, tiles_n);
        k = c.kb;
        if (reload) set_tile(c);
      }
    }
  };

  set_tile(nx);
  load_slice(nx, lkk);
  sa.store(Asr[0], Asi[0], AC);
  sb.store(Bsr[0], Bsi[0], BC);
  advance(lt, nx, lkk, true);
  __syncthreads();

  floatx4 p1[MB][NB], p2[MB][NB], p3[MB][NB];
  auto zero = [&]() {
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        p1[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
        p2[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
        p3[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
      }
  };
  zero();

  int buf = 0;
  for (;;) {
    const bool more = lt < ntiles;
    if (more) load_slice(nx, lkk);
    floatx4 Ar[MB], Ai[MB], Br[NB], Bi[NB];
#pragma unroll
    for (int i = 0; i < MB; ++i) {
      Ar[i] = *reinterpret_cast<const floatx4*>(&Asr[buf][wm + 16 * i + lr][4 * lk]);
      Ai[i] = *reinterpret_cast<const floatx4*>(&Asi[buf][wm + 16 * i + lr][4 * lk]);
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      Br[j] = *reinterpret_cast<const floatx4*>(&Bsr[buf][wn + 16 * j + lr][4 * lk]);
      Bi[j] = *reinterpret_cast<const floatx4*>(&Bsi[buf][wn + 16 * j + lr][4 * lk]);
    }
    // The wave issues its matrix-core products at raised priority, so that
    // the arbiter keeps them flowing while the other waves of the SIMD load
    // and store; the next slice goes to LDS half way through (the buffer it
    // overwrites was released by the previous barrier).
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      if (s == OAA_GEMM_STORE_STEP && more) {
        sa.store(Asr[buf ^ 1], Asi[buf ^ 1], AC);
        sb.store(Bsr[buf ^ 1], Bsi[buf ^ 1], BC);
      }
      float as[MB], bs[NB];
#pragma unroll
      for (int i = 0; i < MB; ++i) as[i] = Ar[i][s] + Ai[i][s];
#pragma unroll
      for (int j = 0; j < NB; ++j) bs[j] = Br[j][s] + Bi[j][s];
      // three independent sweeps, so that dependent accumulations are
      // MB*NB instructions apart
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j)
          p1[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(Ar[i][s], Br[j][s], p1[i][j], 0, 0, 0);
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j)
          p3[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(as[i], bs[j], p3[i][j], 0, 0, 0);
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j)
          p2[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(Ai[i][s], Bi[j][s], p2[i][j], 0, 0, 0);
    }
    __builtin_amdgcn_s_setprio(0);
    if (ck + kKC >= cur.ke) {
      // 16 x 16 result block: lane holds rows 4*(lane/16) + r, r < 4, of column
      // lane % 16; each bin's matrix is under 2^28 elements (32-bit offsets)
      float2* Cm = p.C + size_t(cur.f) * p.c_fstride + size_t(cur.split) * p.c_sstride;
      const unsigned ldc = unsigned(p.ldc);
      const int mb = cur.m0 + wm + 4 * lk, nb = cur.n0 + wn + lr;
      auto result = [&](int i, int j, int r) {
        return make_float2(p1[i][j][r] - p2[i][j][r], p3[i][j][r] - p1[i][j][r] - p2[i][j][r]);
      };
      if (cur.m0 + TM <= p.M && cur.n0 + TN <= p.N) {
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            float2* row = Cm + unsigned(mb + 16 * i + r) * ldc + unsigned(nb);
#pragma unroll
            for (int j = 0; j < NB; ++j) row[16 * j] = result(i, j, r);
          }
      } else {
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int m = mb + 16 * i + r;
            float2* row = Cm + unsigned(m) * ldc + unsigned(nb);
#pragma unroll
            for (int j = 0; j < NB; ++j)
              if (m < p.M && nb + 16 * j < p.N) row[16 * j] = result(i, j, r);
          }
      }
      zero();
    }
    __syncthreads();
    if (!more) break;
    buf ^= 1;
    advance(ct, cur, ck, false);
    advance(lt, nx, lkk, true);
  }
}

// Workgroups per CU and CU count of the current device for one kernel
// instantiation, queried once per device.
template <class Kern>
hipError_t resident_groups(Kern kern, unsigned& groups) {
  static int cached[64] = {0};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  if (cached[dev] == 0) {
    int cus = 0, per_cu = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, kThreads, 0);
    if (e != hipSuccess) return e;
    cached[dev] = (per_cu < 1 ? 1 : per_cu) * (cus < 1 ? 1 : cus);
  }
  groups = unsigned(cached[dev]);
  return hipSuccess;
}

template <int MB, int NB, bool AT, bool AC, bool BT, bool BC>
hipError_t launch_mfma_shape(const GemmParams& p, hipStream_t s) {
  const unsigned long long tiles = (unsigned long long)((p.M + 32 * MB - 1) / (32 * MB)) *
                                   ((p.N + 32 * NB - 1) / (32 * NB)) * unsigned(p.nsplit) * unsigned(p.F);
  if (tiles == 0) return hipSuccess;
  if (tiles > 0xffffffffull) return hipErrorInvalidValue;
  auto kern = cgemm_mfma_kernel<MB, NB, AT, AC, BT, BC>;
  unsigned groups = 0;
  hipError_t e = resident_groups(kern, groups);
  if (e != hipSuccess) return e;
  unsigned long long nwg = groups < tiles ? groups : tiles;
  nwg = (nwg + 7) / 8 * 8;  // whole rounds over the 8 XCDs
  hipLaunchKernelGGL(kern, dim3(unsigned(nwg)), dim3(kThreads), 0, s, p, unsigned(tiles));
  return hipGetLastError();
}

// Row tile of 96 when that wastes less than 128 does (e.g. 96 channels).
// Where the rows are a multiple of 64 and 96-wide column tiles waste less
// than 64-wide ones, 64 x 96 tiles (e.g. the large-kernel layer's forward
// product: 288 tiles per bin, the fifth 64-wide column tile half empty;
// 0.89 -> 0.86 ms). A 96 x 96 tile would need more than the 256 registers
// of two workgroups per CU.
template <bool AT, bool AC, bool BT, bool BC>
hipError_t launch_mfma(const GemmParams& p, hipStream_t s) {
  const long waste128 = (long)((p.M + 127) / 128) * 128 - p.M;
  const long waste96 = (long)((p.M + 95) / 96) * 96 - p.M;
  const long wasteN64 = (long)((p.N + 63) / 64) * 64 - p.N;
  const long wasteN96 = (long)((p.N + 95) / 96) * 96 - p.N;
  if (p.M % 64 == 0 && wasteN96 < wasteN64) return launch_mfma_shape<2, 3, AT, AC, BT, BC>(p, s);
  if (waste96 < waste128) return launch_mfma_shape<3, OAA_GEMM_NB, AT, AC, BT, BC>(p, s);
  return launch_mfma_shape<4, OAA_GEMM_NB, AT, AC, BT, BC>(p, s);
}

template <int TM, int TN, class Kern>
hipError_t launch(Kern kern, const GemmParams& p, hipStream_t s) {
  const unsigned tiles = unsigned(((p.M + TM - 1) / TM) * ((p.N + TN - 1) / TN));
  hipLaunchKernelGGL(kern, dim3(tiles, unsigned(p.nsplit), unsigned(p.F)), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_cgemm_valu(const GemmParams& p, hipStream_t s) {
  if (p.kchunk % kKC != 0 && p.nsplit > 1) return hipErrorInvalidValue;
  // the three operand orientations of the layer's passes, and the plain
  // product that composes two layers' kernel spectra
  if (p.a_trans && !p.a_conj && !p.b_trans && !p.b_conj)
    return launch<kVM, kVN>(cgemm_valu_kernel<true, false, false, false>, p, s);
  if (!p.a_trans && p.a_conj && !p.b_trans && !p.b_conj)
    return launch<kVM, kVN>(cgemm_valu_kernel<false, true, false, false>, p, s);
  if (!p.a_trans && p.a_conj && p.b_trans && !p.b_conj)
    return launch<kVM, kVN>(cgemm_valu_kernel<false, true, true, false>, p, s);
  if (!p.a_trans && !p.a_conj && !p.b_trans && !p.b_conj)  // kernel spectra of two stacked layers
    return launch<kVM, kVN>(cgemm_valu_kernel<false, false, false, false>, p, s);
  return hipErrorInvalidValue;
}

hipError_t launch_cgemm_mfma(const GemmParams& p, hipStream_t s) {
  if (p.kchunk % kKC != 0 && p.nsplit > 1) return hipErrorInvalidValue;
  if (!mfma_fits(p)) return hipErrorInvalidValue;
  if (p.a_trans && !p.a_conj && !p.b_trans && !p.b_conj) return launch_mfma<true, false, false, false>(p, s);
  if (!p.a_trans && p.a_conj && !p.b_trans && !p.b_conj) return launch_mfma<false, true, false, false>(p, s);
  if (!p.a_trans && p.a_conj && p.b_trans && !p.b_conj) return launch_mfma<false, true, true, false>(p, s);
  if (!p.a_trans && !p.a_conj && !p.b_trans && !p.b_conj) return launch_mfma<false, false, false, false>(p, s);
  return hipErrorInvalidValue;
}

// The matrix-core path reads each bin's operands through 32-bit byte offsets.
bool mfma_fits(const GemmParams& p) {
  const size_t lim = size_t(1) << 28;
  return p.a_fstride < lim && p.b_fstride < lim && p.c_fstride < lim && size_t(p.M) * size_t(p.ldc) < lim;
}

bool mfma_preferred(const GemmParams& p) { return p.M >= 32 && p.N >= 32 && p.Kr >= 16 && mfma_fits(p); }

}  // namespace oaa
