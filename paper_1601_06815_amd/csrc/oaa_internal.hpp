// Kernel parameter blocks and launchers shared by the host plan code and the
// HIP kernels. Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>

namespace oaa {

// Spectrum layout used by every kernel: complex64 [F][n_ch][n_img * P],
// bin f = u * (L/2+1) + v, tile index within an image = P_row * T + Q_col.

// Zero-padded windows of a stack of square planes -> spectra.
// Window (P, Q) of plane (img, ch) has element (r, s), r, s < R, equal to
// plane[P*pitch + r - off][Q*pitch + s - off] (0 outside the plane); it is
// placed at [0,R)^2 of an L x L tile and transformed.
struct TileFwdParams {
  const float* src;  // [n_img][n_ch][H][H]
  float2* dst;       // [F][n_ch][n_img * T * T]
  int n_img, n_ch;
  int H;             // plane side
  int pitch;         // block pitch (the kernel side n)
  int off;           // window origin offset in the padded frame
  int R;             // window side
  int T;             // blocks per side
  int TQ;            // tiles per workgroup chunk along a block row
  int nchunk;        // ceil(T / TQ)
  int gather;        // 1: kernel planes (T = 1, R = H): a workgroup takes TQ
                     // consecutive images (kernels) of one channel
};

// Spectra (optionally the sum of `nsplit` partial spectra spaced
// `split_stride` elements apart) -> inverse transform -> the n x n window of
// each tile whose rows and columns start at `origin` (taken modulo L) written
// to block (P, Q) of dst[n_img][n_ch][H][H] at (P n, Q n), clipped to H.
struct CropParams {
  const float2* src;  // [nsplit][F][n_ch][n_img * T * T]
  int nsplit;
  size_t split_stride;
  float* dst;         // [n_img][n_ch][H][H]
  int n_img, n_ch;
  int H, n, T;
  int origin;         // first kept row and column of a tile, in [0, L)
  int TQ, nchunk;
};

// Gradient windows: window (P, Q) is the 2n x 2n region of the plane starting
// at row P*n - off, column Q*n - off (zero outside the plane); its spectrum
// goes to dst like TileFwdParams'.
struct WindowParams {
  const float* src;  // [n_img][n_ch][H][H]
  float2* dst;       // [F][n_ch][n_img * T * T]
  int n_img, n_ch;
  int H, n, off, T;  // n: window pitch b
  int S;             // window side, in [b + n_kernel - 1, min(2b, L)]
  int TQ, nchunk;    // window columns per workgroup, ceil(T / TQ)
  int SPW, ngroups;  // window rows per workgroup, ceil(T / SPW)
  int RW;            // window rows transformed together (set by the launcher)
};

// Forward output through folded tile spectra: output block (P, Q) covers
// rows P*n - off + [0, n) and columns Q*n - off + [0, n) of dst[n_img][n_ch][M][M].
struct FoldCropParams {
  const float2* src;  // [F][n_ch][n_img * T * T]
  float* dst;         // [n_img][n_ch][M][M]
  int n_img, n_ch;
  int M, n, off, T;   // n: block pitch b (block side); off: n_kernel - 1
  int S;              // support of a block result, b + n_kernel - 1 (<= L)
  int To;             // output blocks per side (T, or T + 1 when the last
                      // tiles' overhang reaches past T b)
  int shift;          // each tile is the inverse transform circularly shifted
                      // down and right by `shift` (0 for the forward pass)
  int TQ, nchunk, SPW, ngroups;
  int RB;             // block rows per workgroup or per step (set by the launcher)
};

// Batched complex matrix product, one problem per frequency bin f:
//   Cmat[f] (M x N) = op(A[f]) (M x Kr) * op(B[f]) (Kr x N)
// A element (m, kk) is at A + f*a_fstride + (a_trans ? kk*lda + m : m*lda + kk),
// conjugated when a_conj; likewise B element (kk, n) at
// B + f*b_fstride + (b_trans ? n*ldb + kk : kk*ldb + n). With nsplit > 1 the
// reduction is split into ranges of kchunk and split s writes its partial
// product to Cmat + s*c_sstride.
// Frequency bins of the half spectrum: f = u * (L/2 + 1) + v, u < L, v <= L/2.
// In the columns v = 0 and v = L/2 the spectrum of a real tile is Hermitian
// in u, so bin (u, v) with u > L/2 is the conjugate of bin (L - u, v). The
// contractions compute only the other unique_bins(L) bins (the products stay
// Hermitian there); the inverse transforms read the mirrored bins instead.
__host__ __device__ inline int unique_bins(int L) {
  return (L / 2 + 1) * (L / 2 + 1) + (L / 2 - 1) * (L / 2 - 1);
}
// The fp-th computed bin: all of rows u <= L/2, then v in [1, L/2) of the rest.
__host__ __device__ inline int unique_bin(int fp, int L) {
  const int V = L / 2 + 1, head = (L / 2 + 1) * V;
  if (fp < head) return fp;
  const int t = fp - head, w = L / 2 - 1;
  return (L / 2 + 1 + t / w) * V + 1 + t % w;
}

struct GemmParams {
  const float2* A;
  const float2* B;
  float2* C;
  int M, N, Kr;
  long lda, ldb, ldc;
  size_t a_fstride, b_fstride, c_fstride;
  int nsplit, kchunk;
  size_t c_sstride;
  int F;              // bins computed: unique_bins(L)
  int L;              // transform side
  bool a_trans, a_conj, b_trans, b_conj;
};

// Large transform sides (L = 64, 128), k_big_fft.hip. Tiles of one channel
// are numbered t = img * T * T + P * T + Q; a workgroup transforms TQ
// consecutive tiles of one channel at a time.
//
// Forward: tile t is the S x S window of plane (img, ch) of src whose
// rows and columns start at P * pitch - off and Q * pitch - off (zero outside
// the plane), zero-padded to L x L. Kernel spectra are the case T = 1,
// pitch = S = H (tile t = kernel t).
//
// dst layout: element (bin f, ch, tile t) at f bs + ch cs + (t / run) rs +
// t % run. run = 0 (the launcher's default) is [F][n_ch][n_img T T]; the
// fused few-channel passes use runs of the T blocks of a block row
// (run = T, rs = n_ch F T, bs = T, cs = F T) and of four kernels.
struct BigFwdParams {
  const float* src;  // [n_img][n_ch][H][H]
  float2* dst;
  int n_img, n_ch;
  int H, pitch, off, S, T;
  int run;
  size_t bs, cs, rs;
  int TQ, ngrp;      // tiles per group, groups per channel (launcher)
};

// Inverse: the (optionally split-summed) spectra of each tile -> L x L
// inverse transform, row and column r of which become index (r + rot) mod L;
// indices [0, KR) are kept.
//  * crop (overlap = 0): kept element (a, c) of tile (img, P, Q) goes to
//    dst[img][ch][P * pitch + a][Q * pitch + c] (inside the H x H plane);
//  * overlap-add (overlap = 1): output pixel (i, j) of the H x H plane is the
//    sum over tiles (P, Q) with 0 <= i + off - P pitch < KR (and likewise in
//    j) of their kept element (i + off - P pitch, j + off - Q pitch). Where a
//    plane's tiles fit one workgroup (big_overlap_supported) a group is a
//    whole plane; otherwise the kept KR x KR of every tile goes to `tiles`
//    ([n_ch][n_img T T][KR][KR] floats, overlap_tile_bytes) and a second
//    kernel adds them.
struct BigInvParams {
  const float2* src;  // [nsplit][F][n_ch][n_img * T * T]
  int nsplit;
  size_t split_stride;
  float* dst;         // [n_img][n_ch][H][H]
  float* tiles;       // overlap-add scratch for planes of many tiles (or NULL)
  int n_img, n_ch;
  int H, pitch, off, T;
  int KR, rot, overlap;
  int TQ, ngrp;       // launcher
};
hipError_t launch_big_rfft2(int L, const BigFwdParams& p, hipStream_t s);
hipError_t launch_big_irfft2(int L, const BigInvParams& p, hipStream_t s);
// Whether launch_big_irfft2 overlap-adds planes of T x T tiles in one
// workgroup (else it needs the `tiles` scratch).
bool big_overlap_supported(int L, int T);
// Bytes of that scratch for n_planes planes of T x T tiles keeping KR x KR.
inline size_t overlap_tile_bytes(long n_planes, int T, int KR) {
  return size_t(n_planes) * T * T * KR * KR * 4;
}

// Fused few-channel passes at L = 64 (k_fused.hip): the contraction over
// C <= kFusedMaxC channels (forward, weight gradient) or over the kernels
// (error propagation) inside the transform kernels, so that neither the
// forward product spectra nor the gradient window spectra are stored. Input
// block spectra come in runs of a block row: element (bin f, channel c, block
// (P, Q) of image img) at ((img T + P) C + c) F T + f T + Q; kernel spectra
// kernel by kernel, bins contiguous: (f, c, k) at (k C + c) F + f
// (F = 64 * 33 bin positions f = u * 33 + v).
constexpr int kFusedMaxC = 4;
struct FusedFwdParams {
  const float2* xs;  // input block spectra, runs of a block row
  const float2* ws;  // kernel spectra [K][C][F]
  float* y;          // [B][K][M][M]
  int B, K, M, T, b, KR, off;  // blocks b x b at pitch b, results KR = b + n - 1, off = n - 1
  int Kg, ngrp;      // output planes per workgroup item, items per image (launcher)
};
struct FusedBwdDataParams {
  const float* g;    // [B][K][M][M]
  const float2* ws;  // kernel spectra [K][C][F]
  float* dx;         // [B][C][N][N]
  int B, K, N, M, T, b, off, S;  // gradient windows: S x S at (P b - off, Q b - off)
};
struct FusedBwdFilterParams {
  const float* g;     // [B][K][M][M]
  const float2* xs;   // input block spectra, runs of a block row
  float2* part;       // [nsplit][F][C][K] partial sums of the weight-gradient spectra
  int B, K, M, T, b, off, S;
  int nsplit;         // ranges of block rows
  int Kf, nkg, rows_per_split;  // launcher
};
// Output planes (forward) or kernels (weight gradient) a workgroup item
// takes for T blocks per side: T x group tiles fit the workgroup's LDS slots
// (four, or eight for T > 4); 0 if T > 8.
int fused_group(int T);
// Ranges of block rows of the fused weight gradient for about `items`
// workgroup items (kernel groups x ranges); 0 if the layer is not fused.
int fused_filter_split(int B, int K, int T, int items);
// Whether the fused passes take an overlap-add layer of this tiling.
bool fused_supported(int L, int C, int N, int n, int b, int T);
hipError_t launch_fused_forward(FusedFwdParams p, int C, hipStream_t s);
hipError_t launch_fused_bwd_data(const FusedBwdDataParams& p, int C, hipStream_t s);
hipError_t launch_fused_bwd_filter(FusedBwdFilterParams p, int C, hipStream_t s);

hipError_t launch_tile_rfft2(int L, const TileFwdParams& p, hipStream_t s);
hipError_t launch_irfft2_crop(int L, const CropParams& p, hipStream_t s);
hipError_t launch_window_rfft2(int L, const WindowParams& p, hipStream_t s);
hipError_t launch_irfft2_fold_crop(int L, const FoldCropParams& p, hipStream_t s);
// Same result for blocks larger than L/2 (where the frequency-domain fold
// would wrap): inverse transforms, then the overlap-add in space.
hipError_t launch_irfft2_overlap_crop(int L, const FoldCropParams& p, hipStream_t s);
hipError_t launch_cgemm_valu(const GemmParams& p, hipStream_t s);
hipError_t launch_cgemm_mfma(const GemmParams& p, hipStream_t s);
// Streaming contraction for few input channels (C <= kNarrowMaxC), for the
// three orientations above; the weight-gradient form writes nsplit partial
// sums like the tiled kernels.
constexpr int kNarrowMaxC = 4;
hipError_t launch_cgemm_narrow(const GemmParams& p, hipStream_t s);
bool narrow_supported(const GemmParams& p);
// Shape rule of the automatic choice between the tiled contractions.
bool mfma_preferred(const GemmParams& p);
// Whether the matrix-core engine can address its operands and result with
// 32-bit offsets (each bin's matrices under 2^28 complex elements).
bool mfma_fits(const GemmParams& p);

}  // namespace oaa
