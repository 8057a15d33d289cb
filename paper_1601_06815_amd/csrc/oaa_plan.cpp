// Host side of the C ABI declared in include/oaa.h: plan geometry, argument
// validation, workspace layout, and the order of kernel launches for each
// pass of the overlap-and-add convolution (arXiv:1601.06815, Section 2 for
// the forward pass, Section 3.2 for the two backward convolutions).
#include "oaa.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "oaa_internal.hpp"

// Block tiles (the input with overlap-add, the gradient with overlap-save)
// go through the window transform (window side = pitch = b) where its
// several-rows-per-step kernel pays: fewer than 16 blocks per row (the block
// transform's runs of one block row are shorter than 128 bytes), and at
// L = 32 only for blocks of exactly L/2 (other sides take its masked,
// register-heavy variant).
#ifndef OAA_BLOCKS_AS_WINDOWS
#define OAA_BLOCKS_AS_WINDOWS 1
#endif

// Transform sides from which the tile-group kernels of k_big_fft.hip take
// every transform, and from which their two-step overlap-add (tile results
// through a scratch) serves planes of more tiles than a workgroup holds
// (overridable at build time for comparisons).
#ifndef OAA_BIG_MIN_L
#define OAA_BIG_MIN_L 64
#endif
#ifndef OAA_TWO_STEP_MIN_L
#define OAA_TWO_STEP_MIN_L 128
#endif


// Weight-gradient split: enough partial products that the tiled contraction
// has at least this many tiles, a little over two rounds of its 512 resident
// workgroups. More partial sums balance the rounds better but cost the
// inverse one more read of the whole weight-gradient spectrum each: measured,
// 1152 gives the 56 x 56 layer 8 (11 cost 0.03 ms more) and the large-kernel
// layer at L = 64 one (2 took 0.79 against 0.75 ms for the contraction, and
// 0.19 ms more per step); overridable at build time for sweeps.
#ifndef OAA_SPLIT_TILES
#define OAA_SPLIT_TILES 1152
#endif

// Workgroup items the fused weight gradient aims for (one per CU of a
// 256-CU device): the kernel groups times the ranges of block rows. Each
// range is one more partial sum for the inverse to read and add (measured at
// the 224 x 224 RGB layer: 16 ranges cost its inverse 0.19 ms, 8 ranges
// 0.09 ms, for the same contraction time).
#ifndef OAA_FUSED_ITEMS
#define OAA_FUSED_ITEMS 256
#endif

// Tiles (B T^2) from which the library takes the fused passes by default: the
// fused error propagation gives a workgroup two tiles and walks all K kernels
// for them, so fewer than one pair per CU leaves the device mostly idle (a
// single 64 x 64 image with 100 kernels of 17 x 17: 0.32 ms for the fused
// error propagation against 0.05 ms for the unfused stages).
#ifndef OAA_FUSED_MIN_TILES
#define OAA_FUSED_MIN_TILES 512
#endif

struct oaa_plan_s {
  int B, C, K, N, n;
  int method;  // oaa_method_t
  int b;  // block pitch (block side); the paper's tiling has b = n; the hop
          // L - n + 1 for overlap-save
  int M, T, P, L, F;
  int split, kchunk;
  size_t off[4];
  size_t size[4];
  size_t tiles_off;  // overlap-add scratch after the regions (0 bytes if unused)
  size_t tiles_size;
  size_t ws_bytes;
  char* ws;
  size_t ws_bound;
  bool w_valid, x_valid, g_valid;
  oaa_contraction_t contraction;
  // fused few-channel passes: possible for this tiling, in use, and the
  // ranges of block rows of their weight gradient
  bool fused_ok, fused_auto, fused;
  int fsplit;
  // per-stage timing: event pairs recorded around launches
  bool timing;
  std::vector<hipEvent_t> event_pool;
  struct Rec {
    int stage;
    hipEvent_t start, stop;
  };
  std::vector<Rec> records;
};

bool blocks_as_windows(const oaa_plan_s* p) {
  return OAA_BLOCKS_AS_WINDOWS && p->T < 16 && (p->L <= 16 || 2 * p->b == p->L);
}

namespace {

thread_local std::string g_detail;

oaa_status_t fail(oaa_status_t st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

oaa_status_t fail(oaa_status_t st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_detail = buf;
  return st;
}

constexpr size_t kAlign = 256;
constexpr unsigned long long kMaxElems = 1ull << 60;
constexpr int kMaxSide = 128;   // largest transform side
constexpr int kMaxKernel = 64;  // largest kernel side (2n - 1 <= kMaxSide)
constexpr long long kMaxInt = 0x7fffffffll;

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

int pow2_at_least(int v) {
  int L = 2;
  while (L < v) L *= 2;
  return L;
}

oaa_status_t check_plan(oaa_plan_t plan, bool need_ws) {
  if (!plan) return fail(OAA_ERR_INVALID_ARG, "plan is NULL");
  if (need_ws && !plan->ws)
    return fail(OAA_ERR_NO_WORKSPACE, "no workspace bound (need %zu bytes)", plan->ws_bytes);
  return OAA_OK;
}

oaa_status_t hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return OAA_OK;
  return fail(OAA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// What one pass runs against: the plan, the device memory its spectra live in
// (the bound workspace, or the library's static scratch for the
// allocation-free entry point), and the stream. `own` is true for the bound
// workspace: only then are launches timed and cached spectra recorded.
struct Ctx {
  oaa_plan_t p;
  char* ws;
  hipStream_t s;
  bool own;
};

float2* region(const Ctx& cx, int r) { return reinterpret_cast<float2*>(cx.ws + cx.p->off[r]); }

hipError_t take_event(oaa_plan_t p, hipEvent_t* ev) {
  if (!p->event_pool.empty()) {
    *ev = p->event_pool.back();
    p->event_pool.pop_back();
    return hipSuccess;
  }
  return hipEventCreate(ev);
}

// Run one launch; when timing is on, bracket it with events on stream s.
template <class Fn>
oaa_status_t timed(const Ctx& cx, oaa_stage_t stage, const char* what, Fn&& launch) {
  oaa_plan_t p = cx.p;
  hipStream_t s = cx.s;
  if (!cx.own || !p->timing) return hip_status(launch(), what);
  hipEvent_t a = nullptr, b = nullptr;
  hipError_t e = take_event(p, &a);
  if (e == hipSuccess) e = take_event(p, &b);
  if (e == hipSuccess) e = hipEventRecord(a, s);
  if (e != hipSuccess) {
    if (a) p->event_pool.push_back(a);
    if (b) p->event_pool.push_back(b);
    return hip_status(e, "timing event");
  }
  e = launch();
  if (e == hipSuccess) e = hipEventRecord(b, s);
  if (e != hipSuccess) {
    p->event_pool.push_back(a);
    p->event_pool.push_back(b);
    return hip_status(e, what);
  }
  p->records.push_back({int(stage), a, b});
  return OAA_OK;
}

bool big_side(const oaa_plan_s* p) { return p->L >= OAA_BIG_MIN_L; }

// Forward transform of S x S windows starting every `pitch` at -off in the
// H x H planes of src (n_img x n_ch of them, T x T windows each) into `dst`.
oaa_status_t big_forward(const Ctx& cx, oaa_stage_t stage, const char* what, const float* src, float2* dst,
                         int n_img, int n_ch, int H, int pitch, int off, int S, int T, int run = 0, size_t bs = 0,
                         size_t cs = 0, size_t rs = 0) {
  oaa::BigFwdParams b{};
  b.run = run;
  b.bs = bs;
  b.cs = cs;
  b.rs = rs;
  b.src = src;
  b.dst = dst;
  b.n_img = n_img;
  b.n_ch = n_ch;
  b.H = H;
  b.pitch = pitch;
  b.off = off;
  b.S = S;
  b.T = T;
  return timed(cx, stage, what, [&] { return oaa::launch_big_rfft2(cx.p->L, b, cx.s); });
}

// Inverse transform of the spectra at src (nsplit partial sums spaced
// split_stride apart) of n_img x n_ch planes of T x T tiles; row and column r
// of each inverse become index (r + rot) mod L, of which [0, KR) are kept and
// either written to block (P, Q) at (P pitch, Q pitch) of the H x H output
// planes (overlap false) or overlap-added there, pixel (i, j) being framed
// pixel (i + off, j + off) (overlap true).
oaa_status_t big_inverse(const Ctx& cx, oaa_stage_t stage, const char* what, const float2* src, int nsplit,
                         size_t split_stride, float* dst, int n_img, int n_ch, int H, int pitch, int off, int T, int KR,
                         int rot, bool overlap) {
  oaa::BigInvParams b{};
  b.src = src;
  b.nsplit = nsplit;
  b.split_stride = split_stride;
  b.dst = dst;
  b.tiles = cx.p->tiles_size ? reinterpret_cast<float*>(cx.ws + cx.p->tiles_off) : nullptr;
  b.n_img = n_img;
  b.n_ch = n_ch;
  b.H = H;
  b.pitch = pitch;
  b.off = off;
  b.T = T;
  b.KR = KR;
  b.rot = rot;
  b.overlap = overlap ? 1 : 0;
  return timed(cx, stage, what, [&] { return oaa::launch_big_irfft2(cx.p->L, b, cx.s); });
}

oaa_status_t filter_spectra(const Ctx& cx, const float* w, int K, int C, int n, float2* dst);

oaa_status_t run_filter_fft(const Ctx& cx, const float* w) {
  oaa_plan_t p = cx.p;
  if (p->fused) {
    // kernel by kernel, bins contiguous: (f, c, k) at (k C + c) F + f
    const size_t F = p->F, C = p->C;
    oaa_status_t st = big_forward(cx, OAA_STAGE_W_SPECTRUM, "kernel spectra", w, region(cx, OAA_REGION_W_SPECTRUM),
                                  p->K, p->C, p->n, p->n, 0, p->n, 1, 1, 1, F, C * F);
    if (st == OAA_OK && cx.own) p->w_valid = true;
    return st;
  }
  oaa_status_t st = filter_spectra(cx, w, p->K, p->C, p->n, region(cx, OAA_REGION_W_SPECTRUM));
  if (st == OAA_OK && cx.own) p->w_valid = true;
  return st;
}

// Spectra [F][C][K] at the plan's L of K x C kernels w[k][c] of side n
// (n <= L), zero-padded: the unfused kernel-spectra layout.
oaa_status_t filter_spectra(const Ctx& cx, const float* w, int K, int C, int n, float2* dst) {
  oaa_plan_t p = cx.p;
  hipStream_t s = cx.s;
  if (big_side(p))  // kernels as single-tile planes w[k][c]
    return big_forward(cx, OAA_STAGE_W_SPECTRUM, "kernel spectra", w, dst, K, C, n, n, 0, n, 1);
  oaa::TileFwdParams t{};
  t.src = w;
  t.dst = dst;
  t.n_img = K;
  t.n_ch = C;
  t.H = n;
  t.pitch = n;
  t.off = 0;
  t.R = n;
  t.T = 1;
  t.gather = 1;
  return timed(cx, OAA_STAGE_W_SPECTRUM, "kernel spectra", [&] { return oaa::launch_tile_rfft2(p->L, t, s); });
}

// Scratch of the two layers' spectra for kernel_chain: W1hat [F][C][J], then
// W2hat [F][J][K], each 256-byte aligned.
size_t chain_scratch_bytes(const oaa_plan_s* p, int J) {
  return align_up(size_t(p->F) * p->C * J * 8) + align_up(size_t(p->F) * J * p->K * 8);
}

// Kernel spectra of two stacked layers, x -> conv(., w1) -> conv(., w2) with
// nothing between them (the Conclusion's convolution layers as products in
// the frequency domain): w1 [J][C][n1][n1] and w2 [K][J][n2][n2] are
// transformed at the plan's L, and per bin W12hat[c][k] = sum_j
// W1hat[c][j] W2hat[j][k] is written as the plan's kernel spectra. W12hat is
// the spectrum of the full convolution of the two kernels summed over j, a
// kernel of side n1 + n2 - 1 = n.
oaa_status_t kernel_chain(const Ctx& cx, const float* w1, int J, int n1, const float* w2, int n2, char* scratch) {
  oaa_plan_t p = cx.p;
  float2* w1h = reinterpret_cast<float2*>(scratch);
  float2* w2h = reinterpret_cast<float2*>(scratch + align_up(size_t(p->F) * p->C * J * 8));
  if (oaa_status_t st = filter_spectra(cx, w1, J, p->C, n1, w1h)) return st;
  if (oaa_status_t st = filter_spectra(cx, w2, p->K, J, n2, w2h)) return st;
  oaa::GemmParams g{};
  g.A = w1h;
  g.B = w2h;
  g.C = region(cx, OAA_REGION_W_SPECTRUM);
  g.M = p->C; g.N = p->K; g.Kr = J;
  g.lda = J; g.ldb = p->K; g.ldc = p->K;
  g.a_fstride = size_t(p->C) * J;
  g.b_fstride = size_t(J) * p->K;
  g.c_fstride = size_t(p->C) * p->K;
  g.nsplit = 1; g.kchunk = J; g.c_sstride = 0;
  g.F = oaa::unique_bins(p->L);
  g.L = p->L;
  g.a_trans = false; g.a_conj = false; g.b_trans = false; g.b_conj = false;
  oaa_status_t st = timed(cx, OAA_STAGE_W_SPECTRUM, "kernel spectra of two stacked layers", [&] {
    return oaa::mfma_preferred(g) ? oaa::launch_cgemm_mfma(g, cx.s) : oaa::launch_cgemm_valu(g, cx.s);
  });
  if (st == OAA_OK && cx.own) p->w_valid = true;
  return st;
}

oaa_status_t run_input_fft(const Ctx& cx, const float* x) {
  oaa_plan_t p = cx.p;
  hipStream_t s = cx.s;
  if (p->fused) {
    // runs of a block row: (f, c, block (P, Q) of img) at ((img T + P) C + c) F T + f T + Q
    const size_t F = p->F, C = p->C, T = p->T;
    oaa_status_t st = big_forward(cx, OAA_STAGE_X_SPECTRUM, "input block spectra", x,
                                  region(cx, OAA_REGION_X_SPECTRUM), p->B, p->C, p->N, p->b, 0, p->b, p->T, p->T, T,
                                  F * T, C * F * T);
    if (st == OAA_OK && cx.own) p->x_valid = true;
    return st;
  }
  if (big_side(p)) {
    // overlap-save: L x L windows every h; overlap-add: b x b blocks
    const bool oas = p->method == OAA_METHOD_OVERLAP_SAVE;
    oaa_status_t st = big_forward(cx, OAA_STAGE_X_SPECTRUM, oas ? "input window spectra" : "input block spectra", x,
                                  region(cx, OAA_REGION_X_SPECTRUM), p->B, p->C, p->N, p->b, 0, oas ? p->L : p->b,
                                  p->T);
    if (st == OAA_OK && cx.own) p->x_valid = true;
    return st;
  }
  if (p->method == OAA_METHOD_OVERLAP_SAVE) {
    // L x L windows of x starting every h = L - n + 1
    oaa::WindowParams t{};
    t.src = x;
    t.dst = region(cx, OAA_REGION_X_SPECTRUM);
    t.n_img = p->B;
    t.n_ch = p->C;
    t.H = p->N;
    t.n = p->b;
    t.S = p->L;
    t.off = 0;
    t.T = p->T;
    oaa_status_t st = timed(cx, OAA_STAGE_X_SPECTRUM, "input window spectra",
                            [&] { return oaa::launch_window_rfft2(p->L, t, s); });
    if (st == OAA_OK && cx.own) p->x_valid = true;
    return st;
  }
  oaa_status_t st;
  if (blocks_as_windows(p)) {
    // b x b blocks as windows of side b at pitch b
    oaa::WindowParams t{};
    t.src = x;
    t.dst = region(cx, OAA_REGION_X_SPECTRUM);
    t.n_img = p->B;
    t.n_ch = p->C;
    t.H = p->N;
    t.n = p->b;
    t.S = p->b;
    t.off = 0;
    t.T = p->T;
    st = timed(cx, OAA_STAGE_X_SPECTRUM, "input block spectra",
               [&] { return oaa::launch_window_rfft2(p->L, t, s); });
  } else {
    oaa::TileFwdParams t{};
    t.src = x;
    t.dst = region(cx, OAA_REGION_X_SPECTRUM);
    t.n_img = p->B;
    t.n_ch = p->C;
    t.H = p->N;
    t.pitch = p->b;
    t.off = 0;
    t.R = p->b;
    t.T = p->T;
    st = timed(cx, OAA_STAGE_X_SPECTRUM, "input block spectra",
               [&] { return oaa::launch_tile_rfft2(p->L, t, s); });
  }
  if (st == OAA_OK && cx.own) p->x_valid = true;
  return st;
}

oaa_status_t run_grad_fft(const Ctx& cx, const float* g) {
  oaa_plan_t p = cx.p;
  hipStream_t s = cx.s;
  if (big_side(p)) {
    // overlap-save: h x h blocks of g; overlap-add: windows of side
    // min(2b, L) of the gradient framed by n - 1 zeros, every b
    const bool oas = p->method == OAA_METHOD_OVERLAP_SAVE;
    oaa_status_t st = big_forward(cx, OAA_STAGE_G_SPECTRUM, oas ? "gradient block spectra" : "gradient window spectra",
                                  g, region(cx, OAA_REGION_G_SPECTRUM), p->B, p->K, p->M, p->b,
                                  oas ? 0 : p->n - 1, oas ? p->b : std::min(2 * p->b, p->L), p->T);
    if (st == OAA_OK && cx.own) p->g_valid = true;
    return st;
  }
  if (p->method == OAA_METHOD_OVERLAP_SAVE) {
    // h x h blocks of g, h = L - n + 1
    oaa_status_t st;
    if (blocks_as_windows(p)) {
      oaa::WindowParams t{};
      t.src = g;
      t.dst = region(cx, OAA_REGION_G_SPECTRUM);
      t.n_img = p->B;
      t.n_ch = p->K;
      t.H = p->M;
      t.n = p->b;
      t.S = p->b;
      t.off = 0;
      t.T = p->T;
      st = timed(cx, OAA_STAGE_G_SPECTRUM, "gradient block spectra",
                 [&] { return oaa::launch_window_rfft2(p->L, t, s); });
    } else {
      oaa::TileFwdParams t{};
      t.src = g;
      t.dst = region(cx, OAA_REGION_G_SPECTRUM);
      t.n_img = p->B;
      t.n_ch = p->K;
      t.H = p->M;
      t.pitch = p->b;
      t.off = 0;
      t.R = p->b;
      t.T = p->T;
      st = timed(cx, OAA_STAGE_G_SPECTRUM, "gradient block spectra",
                 [&] { return oaa::launch_tile_rfft2(p->L, t, s); });
    }
    if (st == OAA_OK && cx.own) p->g_valid = true;
    return st;
  }
  // window (P,Q) of the zero-framed gradient: g[P*n + r - (n-1)][Q*n + s - (n-1)],
  // r, s < 2n
  oaa::WindowParams t{};
  t.src = g;
  t.dst = region(cx, OAA_REGION_G_SPECTRUM);
  t.n_img = p->B;
  t.n_ch = p->K;
  t.H = p->M;
  t.n = p->b;        // window pitch
  t.S = 2 * p->b <= p->L ? 2 * p->b : p->L;  // window side, >= b + n - 1
  t.off = p->n - 1;
  t.T = p->T;
  oaa_status_t st = timed(cx, OAA_STAGE_G_SPECTRUM, "gradient window spectra",
                          [&] { return oaa::launch_window_rfft2(p->L, t, s); });
  if (st == OAA_OK && cx.own) p->g_valid = true;
  return st;
}

oaa_status_t run_gemm(const Ctx& cx, oaa::GemmParams& g, oaa_stage_t stage, const char* what) {
  oaa_plan_t p = cx.p;
  hipStream_t s = cx.s;
  g.F = oaa::unique_bins(p->L);
  g.L = p->L;
  oaa_contraction_t c = p->contraction;
  if (c == OAA_CONTRACTION_AUTO)
    c = oaa::mfma_preferred(g)      ? OAA_CONTRACTION_MFMA
        : oaa::narrow_supported(g) ? OAA_CONTRACTION_NARROW
                                   : OAA_CONTRACTION_VALU;
  if (c == OAA_CONTRACTION_NARROW && !oaa::narrow_supported(g))
    return fail(OAA_ERR_UNSUPPORTED, "%s: the streaming contraction needs C <= %d", what, oaa::kNarrowMaxC);
  return timed(cx, stage, what, [&] {
    switch (c) {
      case OAA_CONTRACTION_MFMA: return oaa::launch_cgemm_mfma(g, s);
      case OAA_CONTRACTION_NARROW: return oaa::launch_cgemm_narrow(g, s);
      default: return oaa::launch_cgemm_valu(g, s);
    }
  });
}

// Estimated time (s) of a training step with T x T tiles of side L per
// plane: the transform stages move every spectrum twice (written by one
// kernel, read by the next) and the planes once each way, at a rate per
// transform side that runs of few tiles per plane lower; the contractions
// run on the matrix cores (C, K >= 32; three products, six flops per complex
// multiply-add) or stream their spectra (few channels). The rates are a fixed
// calibration against the measured training steps of the large layers
// (transform stages at 3.5, 2.5, 2.1 and 1.05 TB/s for L <= 16, 32, 64 and
// 128; 110 TFLOP/s executed on the matrix cores; 4 TB/s streaming), not a
// measured search.
double step_time_estimate(int B, int C, int K, int N, int n, int L, int T) {
  const double M = N - n + 1, BP = double(B) * T * T, Fu = oaa::unique_bins(L);
  const double spec = Fu * BP * 8;  // one spectrum channel, bytes
  const double bytes = 2 * spec * (C + K) + 8.0 * B * (double(C) * N * N + double(K) * M * M);
  const double rate = (L <= 16 ? 3.5 : L == 32 ? 2.5 : L == 64 ? 2.1 : 1.05) * 1e12;
  const double runs = std::pow(std::min(1.0, double(T) * T / 16.0), 0.2);
  double t = bytes / (rate * runs);
  if (std::min(C, K) >= 32)
    t += 18.0 * BP * C * K * Fu / 110e12;
  else
    t += 5.0 * spec * (C + K) / 4e12;  // X and G spectra read and written by the three products
  return t;
}

// Tiling with the least estimated time: transform sides from L0 (the
// smallest power of two >= 2n-1) up to 64 (or L0 itself when it is 128),
// block pitches b in [max(1, n-1), L-n+1]. Ties go to the smaller L, and at
// one L to the larger block (same tile count, fewer zeros).
void choose_tiling(int B, int C, int K, int N, int n, int& L, int& b) {
  const int L0 = pow2_at_least(2 * n - 1);
  double best = 0;
  L = L0;
  b = n;
  for (int Lc = L0; Lc <= std::max(64, L0); Lc *= 2) {
    for (int bc = Lc - n + 1; bc >= (n > 1 ? n - 1 : 1); --bc) {
      const double cost = step_time_estimate(B, C, K, N, n, Lc, (N + bc - 1) / bc);
      if (best == 0 || cost < best) {
        best = cost;
        L = Lc;
        b = bc;
      }
    }
  }
}

// Transform side for the output-tiled method: the side from L0 up to 64 (or
// L0 = 128) with the least estimated time at the hop L - n + 1 over the
// output side M.
int choose_oas_side(int B, int C, int K, int N, int n) {
  const int L0 = pow2_at_least(2 * n - 1);
  const int M = N - n + 1;
  double best = 0;
  int L = L0;
  for (int Lc = L0; Lc <= std::max(64, L0); Lc *= 2) {
    const int h = Lc - n + 1;
    const double cost = step_time_estimate(B, C, K, N, n, Lc, (M + h - 1) / h);
    if (best == 0 || cost < best) {
      best = cost;
      L = Lc;
    }
  }
  return L;
}

// The passes, after validation, on the context's workspace and stream.
oaa_status_t forward_pass(const Ctx& cx, const float* x, const float* w, float* y) {
  oaa_plan_t p = cx.p;
  hipStream_t s = cx.s;
  oaa_status_t st;
  if (w && (st = run_filter_fft(cx, w))) return st;
  if ((st = run_input_fft(cx, x))) return st;
  if (p->fused) {
    oaa::FusedFwdParams f{};
    f.xs = region(cx, OAA_REGION_X_SPECTRUM);
    f.ws = region(cx, OAA_REGION_W_SPECTRUM);
    f.y = y;
    f.B = p->B; f.K = p->K; f.M = p->M; f.T = p->T; f.b = p->b;
    f.KR = p->b + p->n - 1; f.off = p->n - 1;
    return timed(cx, OAA_STAGE_FWD_INVERSE, "fused contraction + inverse transform + overlap-add",
                 [&] { return oaa::launch_fused_forward(f, p->C, s); });
  }
  // Yhat[f] (K x BP) = What[f]^T (K x C) * Xhat[f] (C x BP)
  const long BP = (long)p->B * p->P;
  oaa::GemmParams g{};
  g.A = region(cx, OAA_REGION_W_SPECTRUM);
  g.B = region(cx, OAA_REGION_X_SPECTRUM);
  g.C = region(cx, OAA_REGION_PRODUCT);
  g.M = p->K; g.N = (int)BP; g.Kr = p->C;
  g.lda = p->K; g.ldb = BP; g.ldc = BP;
  g.a_fstride = (size_t)p->C * p->K;
  g.b_fstride = (size_t)p->C * BP;
  g.c_fstride = (size_t)p->K * BP;
  g.nsplit = 1; g.kchunk = p->C; g.c_sstride = 0;
  g.a_trans = true; g.a_conj = false; g.b_trans = false; g.b_conj = false;
  if ((st = run_gemm(cx, g, OAA_STAGE_FWD_PRODUCT, "forward contraction"))) return st;
  if (big_side(p) && p->method == OAA_METHOD_OVERLAP_SAVE)
    return big_inverse(cx, OAA_STAGE_FWD_INVERSE, "inverse transform + overlap-save crop",
                       region(cx, OAA_REGION_PRODUCT), 1, 0, y, p->B, p->K, p->M, p->b, 0, p->T, p->b,
                       (p->L - (p->n - 1)) & (p->L - 1), false);
  if (big_side(p) && (oaa::big_overlap_supported(p->L, p->T) || p->L >= OAA_TWO_STEP_MIN_L))
    return big_inverse(cx, OAA_STAGE_FWD_INVERSE, "inverse transform + overlap-add", region(cx, OAA_REGION_PRODUCT),
                       1, 0, y, p->B, p->K, p->M, p->b, p->n - 1, p->T, p->b + p->n - 1, 0, true);
  if (p->method == OAA_METHOD_OVERLAP_SAVE) {
    // rows and columns [n-1, L) of each window's inverse are its h x h outputs
    oaa::CropParams c{};
    c.src = region(cx, OAA_REGION_PRODUCT);
    c.nsplit = 1; c.split_stride = 0;
    c.dst = y;
    c.n_img = p->B; c.n_ch = p->K;
    c.H = p->M; c.n = p->b; c.T = p->T;
    c.origin = p->n - 1;
    return timed(cx, OAA_STAGE_FWD_INVERSE, "inverse transform + overlap-save crop",
                 [&] { return oaa::launch_irfft2_crop(p->L, c, s); });
  }
  oaa::FoldCropParams o{};
  o.src = region(cx, OAA_REGION_PRODUCT);
  o.dst = y;
  o.n_img = p->B; o.n_ch = p->K;
  o.M = p->M; o.n = p->b; o.off = p->n - 1; o.T = p->T;
  o.To = p->T; o.shift = 0;
  o.S = p->b + p->n - 1;
  // the overlap-add in the frequency domain needs neighbours shifted by b not
  // to wrap into the block (2b <= L); larger blocks add their neighbours in space
  if (2 * p->b <= p->L)
    return timed(cx, OAA_STAGE_FWD_INVERSE, "inverse transform + overlap-add",
                 [&] { return oaa::launch_irfft2_fold_crop(p->L, o, s); });
  return timed(cx, OAA_STAGE_FWD_INVERSE, "inverse transform + overlap-add",
               [&] { return oaa::launch_irfft2_overlap_crop(p->L, o, s); });
}


oaa_status_t backward_data_pass(const Ctx& cx, const float* g, const float* w, float* dx) {
  oaa_plan_t p = cx.p;
  hipStream_t s = cx.s;
  oaa_status_t st;
  if (w && (st = run_filter_fft(cx, w))) return st;
  if (p->fused) {
    oaa::FusedBwdDataParams f{};
    f.g = g;
    f.ws = region(cx, OAA_REGION_W_SPECTRUM);
    f.dx = dx;
    f.B = p->B; f.K = p->K; f.N = p->N; f.M = p->M; f.T = p->T; f.b = p->b;
    f.off = p->n - 1; f.S = std::min(2 * p->b, p->L);
    return timed(cx, OAA_STAGE_BWD_DATA_PRODUCT, "fused gradient windows + contraction + inverse transform",
                 [&] { return oaa::launch_fused_bwd_data(f, p->C, s); });
  }
  if ((st = run_grad_fft(cx, g))) return st;
  // dXhat[f] (C x BP) = conj(What[f]) (C x K) * Ghat[f] (K x BP)
  const long BP = (long)p->B * p->P;
  oaa::GemmParams gm{};
  gm.A = region(cx, OAA_REGION_W_SPECTRUM);
  gm.B = region(cx, OAA_REGION_G_SPECTRUM);
  gm.C = region(cx, OAA_REGION_PRODUCT);
  gm.M = p->C; gm.N = (int)BP; gm.Kr = p->K;
  gm.lda = p->K; gm.ldb = BP; gm.ldc = BP;
  gm.a_fstride = (size_t)p->C * p->K;
  gm.b_fstride = (size_t)p->K * BP;
  gm.c_fstride = (size_t)p->C * BP;
  gm.nsplit = 1; gm.kchunk = p->K; gm.c_sstride = 0;
  gm.a_trans = false; gm.a_conj = true; gm.b_trans = false; gm.b_conj = false;
  if ((st = run_gemm(cx, gm, OAA_STAGE_BWD_DATA_PRODUCT, "backward-data contraction"))) return st;
  if (big_side(p) && p->method != OAA_METHOD_OVERLAP_SAVE)
    return big_inverse(cx, OAA_STAGE_BWD_DATA_INVERSE, "inverse transform + block crop", region(cx, OAA_REGION_PRODUCT),
                       1, 0, dx, p->B, p->C, p->N, p->b, 0, p->T, p->b, 0, false);
  if (big_side(p) && (oaa::big_overlap_supported(p->L, p->T) || p->L >= OAA_TWO_STEP_MIN_L))
    return big_inverse(cx, OAA_STAGE_BWD_DATA_INVERSE, "inverse transform + overlap-add",
                       region(cx, OAA_REGION_PRODUCT), 1, 0, dx, p->B, p->C, p->N, p->b, 0, p->T, p->L, p->n - 1, true);
  if (p->method == OAA_METHOD_OVERLAP_SAVE) {
    // overlap-add of the gradient blocks' results into dx. The contraction
    // used conj(W): each inverse is a circular correlation with support
    // [-(n-1), h), i.e. the block's convolution with the flipped kernel
    // circularly shifted up and left by n-1; the kernel shifts it back.
    oaa::FoldCropParams o{};
    o.src = region(cx, OAA_REGION_PRODUCT);
    o.dst = dx;
    o.n_img = p->B; o.n_ch = p->C;
    o.M = p->N; o.n = p->b; o.off = 0; o.T = p->T;
    o.To = (p->N + p->b - 1) / p->b;
    o.shift = p->n - 1;
    o.S = p->L;
    return timed(cx, OAA_STAGE_BWD_DATA_INVERSE, "inverse transform + overlap-add",
                 [&] { return oaa::launch_irfft2_overlap_crop(p->L, o, s); });
  }
  oaa::CropParams c{};
  c.src = region(cx, OAA_REGION_PRODUCT);
  c.nsplit = 1; c.split_stride = 0;
  c.dst = dx;
  c.n_img = p->B; c.n_ch = p->C;
  c.H = p->N; c.n = p->b; c.T = p->T;
  c.origin = 0;
  return timed(cx, OAA_STAGE_BWD_DATA_INVERSE, "inverse transform + block crop",
               [&] { return oaa::launch_irfft2_crop(p->L, c, s); });
}


oaa_status_t backward_filter_pass(const Ctx& cx, const float* x, const float* g, float* dw) {
  oaa_plan_t p = cx.p;
  hipStream_t s = cx.s;
  oaa_status_t st;
  if (x && (st = run_input_fft(cx, x))) return st;
  if (p->fused) {
    oaa::FusedBwdFilterParams f{};
    f.g = g;
    f.xs = region(cx, OAA_REGION_X_SPECTRUM);
    f.part = region(cx, OAA_REGION_PRODUCT);
    f.B = p->B; f.K = p->K; f.M = p->M; f.T = p->T; f.b = p->b;
    f.off = p->n - 1; f.S = std::min(2 * p->b, p->L);
    f.nsplit = p->fsplit;
    if ((st = timed(cx, OAA_STAGE_BWD_FILTER_PRODUCT, "fused gradient windows + weight-gradient contraction",
                    [&] { return oaa::launch_fused_bwd_filter(f, p->C, s); })))
      return st;
    return big_inverse(cx, OAA_STAGE_BWD_FILTER_INVERSE, "inverse transform of weight gradient",
                       region(cx, OAA_REGION_PRODUCT), p->fsplit, (size_t)p->F * p->C * p->K, dw, p->K, p->C, p->n,
                       p->n, 0, 1, p->n, 0, false);
  }
  if (g && (st = run_grad_fft(cx, g))) return st;
  // dWhat^T[f] (C x K) = conj(Xhat[f]) (C x BP) * Ghat[f]^T (BP x K), split over BP
  const long BP = (long)p->B * p->P;
  oaa::GemmParams gm{};
  gm.A = region(cx, OAA_REGION_X_SPECTRUM);
  gm.B = region(cx, OAA_REGION_G_SPECTRUM);
  gm.C = region(cx, OAA_REGION_PRODUCT);
  gm.M = p->C; gm.N = p->K; gm.Kr = (int)BP;
  gm.lda = BP; gm.ldb = BP; gm.ldc = p->K;
  gm.a_fstride = (size_t)p->C * BP;
  gm.b_fstride = (size_t)p->K * BP;
  gm.c_fstride = (size_t)p->C * p->K;
  gm.nsplit = p->split; gm.kchunk = p->kchunk;
  gm.c_sstride = (size_t)p->F * p->C * p->K;
  gm.a_trans = false; gm.a_conj = true; gm.b_trans = true; gm.b_conj = false;
  if ((st = run_gemm(cx, gm, OAA_STAGE_BWD_FILTER_PRODUCT, "backward-filter contraction"))) return st;
  // overlap-save: the windows carry the conjugate, so dw[u][v] sits at rows
  // and columns (h + u) mod L of the inverse
  const int origin = p->method == OAA_METHOD_OVERLAP_SAVE ? p->b & (p->L - 1) : 0;
  if (big_side(p))
    return big_inverse(cx, OAA_STAGE_BWD_FILTER_INVERSE, "inverse transform of weight gradient",
                       region(cx, OAA_REGION_PRODUCT), p->split, (size_t)p->F * p->C * p->K, dw, p->K, p->C, p->n,
                       p->n, 0, 1, p->n, (p->L - origin) & (p->L - 1), false);
  oaa::CropParams c{};
  c.src = region(cx, OAA_REGION_PRODUCT);
  c.nsplit = p->split;
  c.split_stride = (size_t)p->F * p->C * p->K;
  c.dst = dw;
  c.n_img = p->K; c.n_ch = p->C;   // spectra [F][C][K], output planes dw[k][c]
  c.H = p->n; c.n = p->n; c.T = 1;
  c.origin = origin;
  return timed(cx, OAA_STAGE_BWD_FILTER_INVERSE, "inverse transform of weight gradient",
               [&] { return oaa::launch_irfft2_crop(p->L, c, s); });
}


// Static scratch of oaa_conv_forward_noalloc: spectra of layers whose
// workspace fits, for callers that cannot allocate device memory. Every
// device that runs the library holds its own copy until the process ends.
constexpr size_t kScratchBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch_ptr[kMaxDevices];

// Device address of the current device's copy of `scratch`, looked up once
// per device (with that device current). In host code the array's name
// stands for a host-side symbol, not a device address: only this pointer may
// be handed to kernels.
oaa_status_t scratch_on_current_device(char** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(OAA_ERR_UNSUPPORTED, "device %d is beyond the %d devices the static scratch serves", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e, "hipGetSymbolAddress of the static scratch");
    if (!ptr || reinterpret_cast<uintptr_t>(ptr) % kAlign)
      return fail(OAA_ERR_HIP, "static scratch address %p is not %zu-byte aligned", ptr, kAlign);
    g_scratch_ptr[dev] = static_cast<char*>(ptr);
  }
  *out = g_scratch_ptr[dev];
  return OAA_OK;
}

}  // namespace

extern "C" {

const char* oaa_status_string(oaa_status_t status) {
  switch (status) {
    case OAA_OK: return "OAA_OK";
    case OAA_ERR_INVALID_ARG: return "OAA_ERR_INVALID_ARG";
    case OAA_ERR_UNSUPPORTED: return "OAA_ERR_UNSUPPORTED";
    case OAA_ERR_NO_WORKSPACE: return "OAA_ERR_NO_WORKSPACE";
    case OAA_ERR_NO_CACHE: return "OAA_ERR_NO_CACHE";
    case OAA_ERR_HIP: return "OAA_ERR_HIP";
  }
  return "OAA_ERR_UNKNOWN";
}

const char* oaa_last_error_detail(void) { return g_detail.c_str(); }

oaa_status_t oaa_plan_create(oaa_plan_t* out, int B, int C, int K, int N, int n) {
  if (n >= 1 && n <= kMaxKernel) return oaa_plan_create_tiled(out, B, C, K, N, n, pow2_at_least(2 * n - 1), n);
  return oaa_plan_create_tiled(out, B, C, K, N, n, 0, 0);
}

oaa_status_t oaa_plan_create_tiled(oaa_plan_t* out, int B, int C, int K, int N, int n, int L, int b) {
  return oaa_plan_create_method(out, B, C, K, N, n, L, b, OAA_METHOD_OVERLAP_ADD);
}

oaa_status_t oaa_plan_create_method(oaa_plan_t* out, int B, int C, int K, int N, int n, int L, int b,
                                    oaa_method_t method) {
  if (!out) return fail(OAA_ERR_INVALID_ARG, "plan output pointer is NULL");
  *out = nullptr;
  if (method != OAA_METHOD_OVERLAP_ADD && method != OAA_METHOD_OVERLAP_SAVE)
    return fail(OAA_ERR_INVALID_ARG, "unknown method %d", (int)method);
  if (B < 1 || C < 1 || K < 1 || N < 1 || n < 1)
    return fail(OAA_ERR_INVALID_ARG, "dimensions must be positive (B=%d C=%d K=%d N=%d n=%d)", B, C, K, N, n);
  if (n > N) return fail(OAA_ERR_INVALID_ARG, "kernel side n=%d exceeds input side N=%d", n, N);
  if (n > kMaxKernel)
    return fail(OAA_ERR_UNSUPPORTED, "kernel side n=%d > %d (transform side would exceed %d)", n, kMaxKernel, kMaxSide);
  if (L < 0 || b < 0) return fail(OAA_ERR_INVALID_ARG, "negative tiling (L=%d b=%d)", L, b);
  const int M = N - n + 1;
  int T = 0;
  if (method == OAA_METHOD_OVERLAP_SAVE) {
    if (L == 0) L = choose_oas_side(B, C, K, N, n);
    if (L < 2 || L > kMaxSide || (L & (L - 1)))
      return fail(OAA_ERR_UNSUPPORTED, "transform side L=%d must be a power of two in [2, %d]", L, kMaxSide);
    if (L < 2 * n - 1)
      return fail(OAA_ERR_INVALID_ARG, "overlap-save needs L >= 2n-1 (n=%d, L=%d)", n, L);
    if (b != 0 && b != L - n + 1)
      return fail(OAA_ERR_INVALID_ARG, "overlap-save hop b=%d must be 0 or L-n+1=%d", b, L - n + 1);
    b = L - n + 1;
    T = (M + b - 1) / b;
  } else {
    if (L == 0 && b == 0) {
      choose_tiling(B, C, K, N, n, L, b);
    } else if (L == 0 || b == 0) {
      return fail(OAA_ERR_INVALID_ARG, "give both L and b, or neither (L=%d b=%d)", L, b);
    }
    if (L < 2 || L > kMaxSide || (L & (L - 1)))
      return fail(OAA_ERR_UNSUPPORTED, "transform side L=%d must be a power of two in [2, %d]", L, kMaxSide);
    // block results (support b + n - 1) must fit the transform and may only
    // reach the next block
    if (b < (n > 1 ? n - 1 : 1) || b + n - 1 > L)
      return fail(OAA_ERR_INVALID_ARG, "block pitch b=%d needs max(1, n-1) <= b <= L-n+1 (n=%d, L=%d)", b, n, L);
    T = (N + b - 1) / b;
  }
  const long long P = (long long)T * T;
  const int F = L * (L / 2 + 1);
  const long long BP = (long long)B * P;
  // index ranges the kernels keep in 32-bit integers
  if (BP > kMaxInt || (long long)N * N > kMaxInt || (long long)B * C > kMaxInt || (long long)B * K > kMaxInt ||
      (long long)K * C > kMaxInt)
    return fail(OAA_ERR_UNSUPPORTED, "layer too large for 32-bit tile and plane indices");
  const bool fused_ok = method == OAA_METHOD_OVERLAP_ADD && oaa::fused_supported(L, C, N, n, b, T);
  int fsplit = 1;
  if (fused_ok) fsplit = oaa::fused_filter_split(B, K, T, OAA_FUSED_ITEMS);
  const unsigned long long eW = (unsigned long long)F * C * K;
  const unsigned long long eX = (unsigned long long)F * C * BP;
  const unsigned long long eG = (unsigned long long)F * K * BP;
  if (eX > kMaxElems || eG > kMaxElems || eW > kMaxElems)
    return fail(OAA_ERR_UNSUPPORTED, "spectra exceed the addressable workspace");

  // split of the weight-gradient reduction over B*P, shared by every
  // contraction engine (the inverse adds the partial sums):
  //  * tiled engines: 96- or 128-row by 128-column tiles, two workgroups per
  //    CU, about OAA_SPLIT_TILES tiles; chunks of 16 tiles;
  //  * few input channels (the streaming engine): about 2048 workgroups of 64
  //    kernels, chunks of at least 1024 tiles, a multiple of 128.
  long long split, quantum;
  if (C <= oaa::kNarrowMaxC) {
    const long long groups = (long long)F * ((K + 63) / 64);
    split = groups >= 2048 ? 1 : (2048 + groups - 1) / groups;
    const long long max_split = (BP + 1023) / 1024;
    if (split > max_split) split = max_split;
    quantum = 128;
  } else {
    const long long rows = ((C + 95) / 96) * 96 - C < ((C + 127) / 128) * 128 - C ? (C + 95) / 96 : (C + 127) / 128;
    const long long tiles = rows * ((K + 127) / 128) * F;
    split = tiles >= OAA_SPLIT_TILES ? 1 : (OAA_SPLIT_TILES + tiles - 1) / tiles;
    const long long max_split = (BP + 63) / 64;
    if (split > max_split) split = max_split;
    quantum = 16;
  }
  if (split < 1) split = 1;
  long long kchunk = (BP + split - 1) / split;
  kchunk = (kchunk + quantum - 1) / quantum * quantum;
  split = (BP + kchunk - 1) / kchunk;

  oaa_plan_s* p = new (std::nothrow) oaa_plan_s();
  if (!p) return fail(OAA_ERR_INVALID_ARG, "out of host memory");
  p->B = B; p->C = C; p->K = K; p->N = N; p->n = n; p->b = b;
  p->method = (int)method;
  p->M = M; p->T = T; p->P = (int)P; p->L = L; p->F = F;
  p->split = (int)split;
  p->kchunk = (int)kchunk;
  unsigned long long eProd = eG > eX ? eG : eX;
  if ((unsigned long long)split * eW > eProd) eProd = (unsigned long long)split * eW;
  if ((unsigned long long)fsplit * F * C * K > eProd) eProd = (unsigned long long)fsplit * F * C * K;
  p->size[OAA_REGION_W_SPECTRUM] = size_t(eW) * 8;
  p->size[OAA_REGION_X_SPECTRUM] = size_t(eX) * 8;
  p->size[OAA_REGION_G_SPECTRUM] = size_t(eG) * 8;
  p->size[OAA_REGION_PRODUCT] = size_t(eProd) * 8;
  size_t off = 0;
  for (int r = 0; r < 4; ++r) {
    p->off[r] = off;
    off = align_up(off + p->size[r]);
  }
  // scratch of the overlap-add passes (the forward pass with overlap-add,
  // error propagation with overlap-save) whose planes hold more tiles than
  // one workgroup keeps (from OAA_TWO_STEP_MIN_L; L = 128 has no other kernel)
  p->tiles_off = off;
  p->tiles_size = 0;
  if (L >= OAA_TWO_STEP_MIN_L && L >= OAA_BIG_MIN_L && !oaa::big_overlap_supported(L, T)) {
    p->tiles_size = method == OAA_METHOD_OVERLAP_ADD ? oaa::overlap_tile_bytes((long)B * K, T, b + n - 1)
                                                     : oaa::overlap_tile_bytes((long)B * C, T, L);
    off = align_up(off + p->tiles_size);
  }
  p->ws_bytes = off;
  p->ws = nullptr;
  p->ws_bound = 0;
  p->w_valid = p->x_valid = p->g_valid = false;
  p->contraction = OAA_CONTRACTION_AUTO;
  p->fused_ok = fused_ok;
  p->fused_auto = p->fused = fused_ok && BP >= OAA_FUSED_MIN_TILES;
  p->fsplit = fsplit;
  p->timing = false;
  *out = p;
  return OAA_OK;
}

oaa_status_t oaa_plan_destroy(oaa_plan_t plan) {
  if (!plan) return OAA_OK;
  for (auto& r : plan->records) {
    (void)hipEventSynchronize(r.stop);
    (void)hipEventDestroy(r.start);
    (void)hipEventDestroy(r.stop);
  }
  for (hipEvent_t e : plan->event_pool) (void)hipEventDestroy(e);
  delete plan;
  return OAA_OK;
}

oaa_status_t oaa_plan_set_timing(oaa_plan_t plan, int enable) {
  if (oaa_status_t st = check_plan(plan, false)) return st;
  plan->timing = enable != 0;
  return OAA_OK;
}

oaa_status_t oaa_plan_stage_times(oaa_plan_t plan, double* total_ms, int* launches, int count) {
  if (oaa_status_t st = check_plan(plan, false)) return st;
  if (count < 0) return fail(OAA_ERR_INVALID_ARG, "negative count");
  for (int i = 0; i < count; ++i) {
    if (total_ms) total_ms[i] = 0.0;
    if (launches) launches[i] = 0;
  }
  oaa_status_t result = OAA_OK;
  for (auto& r : plan->records) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(r.stop);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.start, r.stop);
    if (e != hipSuccess && result == OAA_OK) result = hip_status(e, "timing event");
    if (e == hipSuccess && r.stage < count) {
      if (total_ms) total_ms[r.stage] += ms;
      if (launches) launches[r.stage] += 1;
    }
    plan->event_pool.push_back(r.start);
    plan->event_pool.push_back(r.stop);
  }
  plan->records.clear();
  return result;
}

oaa_status_t oaa_plan_geometry(oaa_plan_t plan, oaa_geometry_t* out) {
  if (oaa_status_t st = check_plan(plan, false)) return st;
  if (!out) return fail(OAA_ERR_INVALID_ARG, "geometry output pointer is NULL");
  out->B = plan->B; out->C = plan->C; out->K = plan->K; out->N = plan->N; out->n = plan->n;
  out->M = plan->M; out->T = plan->T; out->P = plan->P; out->L = plan->L; out->F = plan->F;
  out->b = plan->b;
  out->split = plan->fused ? plan->fsplit : plan->split;
  out->method = plan->method;
  out->fused = plan->fused ? 1 : 0;
  return OAA_OK;
}

size_t oaa_plan_workspace_bytes(oaa_plan_t plan) { return plan ? plan->ws_bytes : 0; }

oaa_status_t oaa_plan_region(oaa_plan_t plan, oaa_region_t r, size_t* offset, size_t* bytes) {
  if (oaa_status_t st = check_plan(plan, false)) return st;
  if ((int)r < 0 || (int)r > 3) return fail(OAA_ERR_INVALID_ARG, "unknown region %d", (int)r);
  if (offset) *offset = plan->off[r];
  if (bytes) *bytes = plan->size[r];
  return OAA_OK;
}

oaa_status_t oaa_plan_bind_workspace(oaa_plan_t plan, void* dev_ptr, size_t bytes) {
  if (oaa_status_t st = check_plan(plan, false)) return st;
  plan->w_valid = plan->x_valid = plan->g_valid = false;
  plan->ws = nullptr;
  plan->ws_bound = 0;
  if (!dev_ptr) return fail(OAA_ERR_INVALID_ARG, "workspace pointer is NULL");
  if (reinterpret_cast<uintptr_t>(dev_ptr) % kAlign)
    return fail(OAA_ERR_INVALID_ARG, "workspace pointer is not %zu-byte aligned", kAlign);
  if (bytes < plan->ws_bytes)
    return fail(OAA_ERR_NO_WORKSPACE, "workspace of %zu bytes is smaller than the %zu needed", bytes, plan->ws_bytes);
  plan->ws = static_cast<char*>(dev_ptr);
  plan->ws_bound = bytes;
  return OAA_OK;
}

oaa_status_t oaa_plan_set_contraction(oaa_plan_t plan, oaa_contraction_t which) {
  if (oaa_status_t st = check_plan(plan, false)) return st;
  if (which != OAA_CONTRACTION_AUTO && which != OAA_CONTRACTION_VALU && which != OAA_CONTRACTION_MFMA &&
      which != OAA_CONTRACTION_NARROW && which != OAA_CONTRACTION_FUSED)
    return fail(OAA_ERR_INVALID_ARG, "unknown contraction %d", (int)which);
  if (which == OAA_CONTRACTION_NARROW && plan->C > oaa::kNarrowMaxC)
    return fail(OAA_ERR_UNSUPPORTED, "the streaming contraction needs C <= %d (plan has C=%d)", oaa::kNarrowMaxC,
                plan->C);
  if (which == OAA_CONTRACTION_FUSED && !plan->fused_ok)
    return fail(OAA_ERR_UNSUPPORTED,
                "the fused passes need the overlap-add method, L = 64, C <= %d and at most 8 blocks per side "
                "(plan: method %d, L=%d, C=%d, T=%d)",
                oaa::kFusedMaxC, plan->method, plan->L, plan->C, plan->T);
  const bool fused = which == OAA_CONTRACTION_FUSED || (which == OAA_CONTRACTION_AUTO && plan->fused_auto);
  // the two paths keep their spectra in different layouts
  if (fused != plan->fused) plan->w_valid = plan->x_valid = plan->g_valid = false;
  plan->fused = fused;
  plan->contraction = which;
  return OAA_OK;
}

oaa_status_t oaa_conv_forward(oaa_plan_t p, const float* x, const float* w, float* y, void* stream) {
  if (oaa_status_t st = check_plan(p, true)) return st;
  if (!x || !y) return fail(OAA_ERR_INVALID_ARG, "x and y must be non-NULL");
  if (!w && !p->w_valid) return fail(OAA_ERR_NO_CACHE, "w is NULL and no kernel spectra are cached");
  (void)hipGetLastError();
  return forward_pass(Ctx{p, p->ws, static_cast<hipStream_t>(stream), true}, x, w, y);
}

oaa_status_t oaa_conv_backward_data(oaa_plan_t p, const float* g, const float* w, float* dx, void* stream) {
  if (oaa_status_t st = check_plan(p, true)) return st;
  if (!g || !dx) return fail(OAA_ERR_INVALID_ARG, "g and dx must be non-NULL");
  if (!w && !p->w_valid) return fail(OAA_ERR_NO_CACHE, "w is NULL and no kernel spectra are cached");
  (void)hipGetLastError();
  return backward_data_pass(Ctx{p, p->ws, static_cast<hipStream_t>(stream), true}, g, w, dx);
}

oaa_status_t oaa_conv_backward_filter(oaa_plan_t p, const float* x, const float* g, float* dw, void* stream) {
  if (oaa_status_t st = check_plan(p, true)) return st;
  if (!dw) return fail(OAA_ERR_INVALID_ARG, "dw must be non-NULL");
  if (!x && !p->x_valid) return fail(OAA_ERR_NO_CACHE, "x is NULL and no input block spectra are cached");
  if (!g && p->fused)
    return fail(OAA_ERR_NO_CACHE, "g is NULL: the fused few-channel passes keep no gradient window spectra");
  if (!g && !p->g_valid) return fail(OAA_ERR_NO_CACHE, "g is NULL and no gradient window spectra are cached");
  (void)hipGetLastError();
  return backward_filter_pass(Ctx{p, p->ws, static_cast<hipStream_t>(stream), true}, x, g, dw);
}

size_t oaa_plan_chain_scratch_bytes(oaa_plan_t plan, int J) {
  if (!plan || J < 1) return 0;
  return chain_scratch_bytes(plan, J);
}

oaa_status_t oaa_plan_set_kernel_chain(oaa_plan_t p, const float* w1, int J, int n1, const float* w2, int n2,
                                       void* scratch, size_t scratch_bytes, void* stream) {
  if (oaa_status_t st = check_plan(p, true)) return st;
  if (!w1 || !w2 || !scratch) return fail(OAA_ERR_INVALID_ARG, "w1, w2 and scratch must be non-NULL");
  if (J < 1 || n1 < 1 || n2 < 1) return fail(OAA_ERR_INVALID_ARG, "J=%d, n1=%d, n2=%d must be >= 1", J, n1, n2);
  if (n1 + n2 - 1 != p->n)
    return fail(OAA_ERR_INVALID_ARG, "the stacked kernels make a kernel of side n1 + n2 - 1 = %d; the plan has n=%d",
                n1 + n2 - 1, p->n);
  if (p->fused)
    return fail(OAA_ERR_UNSUPPORTED,
                "the fused passes keep kernel spectra in their own layout: choose another contraction first");
  if ((long long)J * p->C > kMaxInt || (long long)J * p->K > kMaxInt ||
      (unsigned long long)p->F * J * (unsigned long long)std::max(p->C, p->K) > kMaxElems)
    return fail(OAA_ERR_UNSUPPORTED, "J=%d too large", J);
  if (reinterpret_cast<uintptr_t>(scratch) % kAlign)
    return fail(OAA_ERR_INVALID_ARG, "scratch pointer is not %zu-byte aligned", kAlign);
  if (scratch_bytes < chain_scratch_bytes(p, J))
    return fail(OAA_ERR_INVALID_ARG, "scratch of %zu bytes is smaller than the %zu needed", scratch_bytes,
                chain_scratch_bytes(p, J));
  (void)hipGetLastError();
  return kernel_chain(Ctx{p, p->ws, static_cast<hipStream_t>(stream), true}, w1, J, n1, w2, n2,
                      static_cast<char*>(scratch));
}

oaa_status_t oaa_conv_forward_noalloc(oaa_plan_t p, const float* x, const float* w, float* y, void* stream) {
  if (oaa_status_t st = check_plan(p, false)) return st;
  if (!x || !w || !y) return fail(OAA_ERR_INVALID_ARG, "x, w and y must be non-NULL (no cached spectra are used)");
  if (p->ws_bytes > kScratchBytes)
    return fail(OAA_ERR_UNSUPPORTED,
                "the layer needs %zu bytes of spectra, more than the %zu bytes of static scratch "
                "(use oaa_conv_forward with a bound workspace)",
                p->ws_bytes, kScratchBytes);
  char* ws = nullptr;
  if (oaa_status_t st = scratch_on_current_device(&ws)) return st;
  (void)hipGetLastError();
  return forward_pass(Ctx{p, ws, static_cast<hipStream_t>(stream), false}, x, w, y);
}

}  // extern "C"
