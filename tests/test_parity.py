"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Bar: max|gpu - oracle| / max|oracle| <= 2e-5 per output tensor and pass, for
float32 data. Whole arrays are compared wherever the oracle finishes in
seconds; the full-size layers are compared on sampled outputs that the
oracle evaluates one by one, in the same launch configuration bench.py times:
whole images (first and last), every image and channel block on sampled
pixels, and the weight gradient whole for kernel-channel pairs spanning every
output tile.
"""

import numpy as np
import pytest
import torch

import oracle
from oracle import oaa as oaa_oracle
from paper_1601_06815_amd import binding
from paper_1601_06815_amd.workloads import LAYERS, Layer, make_inputs
from tests.conftest import relerr

pytestmark = pytest.mark.gpu
TOL = 2e-5
DEV = "cuda:0"

SMALL = [  # (B, C, K, N, n): every transform size, ragged block rows, n = 1, N = n
    (1, 3, 4, 32, 5),
    (2, 2, 3, 13, 4),
    (1, 1, 1, 9, 3),
    (2, 3, 2, 11, 1),
    (1, 2, 2, 7, 7),
    (1, 1, 2, 10, 6),
    (3, 2, 3, 17, 8),
    (1, 1, 1, 2, 2),
    (2, 2, 3, 40, 16),
    (1, 2, 2, 40, 17),
    (1, 1, 2, 33, 32),
    (2, 70, 66, 12, 2),
    (1, 5, 130, 20, 3),
    (4, 9, 7, 61, 9),
]


def to_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def run_layer(x, w, g, contraction=binding.CONTRACTION_AUTO, tiling="paper", method=binding.METHOD_OVERLAP_ADD):
    B, C, N, _ = x.shape
    K, _, n, _ = w.shape
    plan = binding.Plan(B, C, K, N, n, device=DEV, contraction=contraction, tiling=tiling, method=method)
    xd, wd, gd = to_dev(x), to_dev(w), to_dev(g)
    y = plan.forward(xd, wd)
    dx = plan.backward_data(gd, wd)
    dw = plan.backward_filter(xd, gd)
    torch.cuda.synchronize()
    return plan, y.cpu().numpy(), dx.cpu().numpy(), dw.cpu().numpy()


def check_whole(x, w, g, contraction=binding.CONTRACTION_AUTO, tiling="paper", method=binding.METHOD_OVERLAP_ADD):
    _, y, dx, dw = run_layer(x, w, g, contraction, tiling, method)
    N, n = x.shape[-1], w.shape[-1]
    e = (relerr(y, oracle.conv_forward(x, w)),
         relerr(dx, oracle.conv_backward_data(g, w, N)),
         relerr(dw, oracle.conv_backward_filter(x, g, n)))
    print(f"shape x{x.shape} w{w.shape}: rel err fwd {e[0]:.2e} bwd_data {e[1]:.2e} bwd_filter {e[2]:.2e}",
          flush=True)
    assert max(e) <= TOL, e
    return e


@pytest.mark.parametrize("shape", SMALL, ids=lambda s: "x".join(map(str, s)))
def test_small_layers_all_passes(gpu_lib, shape):
    B, C, K, N, n = shape
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=sum(shape))
    check_whole(x, w, g)


@pytest.mark.parametrize("contraction", [binding.CONTRACTION_VALU, binding.CONTRACTION_MFMA], ids=["valu", "mfma"])
@pytest.mark.parametrize("shape", [(2, 70, 66, 12, 2), (1, 5, 130, 20, 3), (3, 33, 17, 21, 4),
                                   (1, 130, 140, 9, 3), (2, 16, 32, 40, 16), (1, 3, 64, 30, 7)],
                         ids=lambda s: "x".join(map(str, s)))
def test_contraction_variants(gpu_lib, contraction, shape):
    B, C, K, N, n = shape
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=11 + sum(shape))
    check_whole(x, w, g, contraction)


@pytest.mark.parametrize("shape", [
    (4, 40, 128, 60, 9, 32, 24),    # forward rows (K = 128) in 128-row tiles
    (4, 96, 40, 60, 9, 32, 24),     # error-propagation rows (C = 96) in 96-row tiles
    (10, 32, 64, 100, 16, 64, 49),  # B P = 90 columns: 64 x 96 tiles (forward)
], ids=lambda s: "x".join(map(str, s)))
def test_matrix_core_tile_shapes(gpu_lib, shape):
    """The matrix-core contraction's tile shapes (128 x 64, 96 x 64, 64 x 96),
    forced, against the oracle, compared whole."""
    B, C, K, N, n, L, b = shape
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=31 + sum(shape))
    check_whole(x, w, g, binding.CONTRACTION_MFMA, tiling=(L, b))


NARROW = [  # C <= 4: odd and even tile counts, K off multiples of 16, K > 64, K > 256, split reduction
    (1, 1, 1, 9, 3),
    (2, 2, 17, 13, 4),
    (1, 3, 70, 30, 7),
    (2, 4, 300, 12, 2),
    (2, 3, 20, 100, 3),
    (3, 3, 64, 45, 5),
]


@pytest.mark.parametrize("shape", NARROW, ids=lambda s: "x".join(map(str, s)))
def test_narrow_contraction(gpu_lib, shape):
    """The streaming contraction for few input channels, forced, against the
    oracle; and against the tiled vector-ALU contraction on the same inputs."""
    B, C, K, N, n = shape
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=5 + sum(shape))
    check_whole(x, w, g, binding.CONTRACTION_NARROW)
    plan, y, dx, dw = run_layer(x, w, g, binding.CONTRACTION_NARROW)
    _, y2, dx2, dw2 = run_layer(x, w, g, binding.CONTRACTION_VALU)
    for a, b in ((y, y2), (dx, dx2), (dw, dw2)):
        assert relerr(a, b) <= TOL
    if plan.geometry["split"] > 1:
        print(f"split {plan.geometry['split']}", flush=True)


NARROW_FEW = [  # (B, C, K, N, n, L, b): at most 64 tiles per bin, many kernels (kernels over the lanes too)
    (1, 1, 300, 32, 5, 16, 5),     # 49 tiles, K > 256
    (1, 4, 40, 64, 5, 16, 8),      # 64 tiles: the largest few-tile case
    (2, 1, 33, 20, 3, 16, 14),     # two images of 2 x 2 blocks
    (1, 2, 257, 60, 5, 64, 60),    # one tile per bin at L = 64 (the unfused passes)
    (1, 3, 100, 64, 33, 128, 96),  # one tile per bin at L = 128
]


@pytest.mark.parametrize("shape", NARROW_FEW, ids=lambda s: "x".join(map(str, s)))
def test_narrow_contraction_few_tiles(gpu_lib, shape):
    """The streaming contraction with few tiles per bin (forward and error
    propagation spread the kernels over the lanes), forced, against the
    oracle, compared whole."""
    B, C, K, N, n, L, b = shape
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=23 + sum(shape))
    check_whole(x, w, g, binding.CONTRACTION_NARROW, tiling=(L, b))


TILED = [  # (B, C, K, N, n, L, b): b = n - 1, b between n and L/2, b = L/2, L twice the paper's
    (1, 3, 4, 32, 5, 16, 4),
    (2, 2, 3, 13, 4, 8, 4),
    (1, 5, 6, 29, 5, 16, 8),
    (2, 3, 5, 21, 3, 8, 4),
    (1, 4, 7, 40, 7, 32, 16),
    (2, 6, 5, 23, 3, 16, 8),
    (1, 70, 66, 24, 3, 8, 4),
    (2, 1, 2, 17, 1, 4, 2),
    (1, 2, 3, 36, 9, 32, 12),
    (1, 40, 33, 50, 16, 32, 15),
    # blocks over L/2 (overlap-add after the inverse), up to b = L - n + 1
    (1, 3, 4, 32, 5, 16, 12),
    (2, 2, 3, 13, 4, 8, 5),
    (1, 5, 6, 29, 5, 16, 10),
    (2, 3, 5, 21, 3, 8, 6),
    (1, 4, 7, 40, 7, 32, 26),
    (2, 1, 2, 17, 1, 4, 4),
    (1, 2, 3, 9, 1, 2, 2),
    (1, 70, 66, 24, 3, 8, 6),
    (1, 40, 33, 50, 16, 32, 17),
    (2, 3, 64, 60, 7, 16, 10),
    (1, 3, 4, 70, 16, 64, 49),
    (1, 2, 3, 36, 9, 64, 40),
    (1, 2, 2, 9, 9, 32, 24),
]


@pytest.mark.parametrize("shape", TILED, ids=lambda s: "x".join(map(str, s)))
def test_tiled_layers_all_passes(gpu_lib, shape):
    """Blocks of b != n (the library's larger-block tiling) against the oracle."""
    B, C, K, N, n, L, b = shape
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=31 + sum(shape))
    check_whole(x, w, g, tiling=(L, b))


BIG64 = [  # (B, C, K, N, n, L, b, method): transform side 64 through the tile-group kernels
    (2, 16, 24, 128, 16, 64, 49, "oaa"),   # the large-kernel layer's blocks of 49, reduced: T = 3
    (1, 3, 5, 100, 16, 64, 40, "oaa"),     # T = 3, ragged last block row and column
    (2, 2, 3, 70, 16, 64, 49, "oaa"),      # T = 2
    (3, 2, 2, 45, 7, 64, 58, "oaa"),       # one block per plane (FFTconv-like)
    (1, 4, 3, 150, 20, 64, 40, "oaa"),     # T = 4: forward overlap-add through the per-row kernels
    (1, 2, 3, 200, 32, 64, 32, "oaa"),     # the paper's tiling at n = 32: T = 7, frequency-domain fold
    (2, 3, 17, 60, 9, 64, 56, "oaa"),      # odd channel and kernel counts, partial groups
    (2, 5, 6, 100, 20, 64, 0, "oas"),      # overlap-save: h = 45, T = 2
    (1, 3, 4, 120, 10, 64, 0, "oas"),      # overlap-save: h = 55, T = 3
]


@pytest.mark.parametrize("shape", BIG64, ids=lambda s: "x".join(map(str, s)))
def test_transform_side_64(gpu_lib, shape):
    """Every pass at L = 64 against the oracle, compared whole."""
    B, C, K, N, n, L, b, method = shape
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=71 + sum(shape[:7]))
    m = binding.METHOD_OVERLAP_SAVE if method == "oas" else binding.METHOD_OVERLAP_ADD
    check_whole(x, w, g, tiling=(L, b), method=m)


# Shapes for the L = 64 inverses' group walk, with groups of one plane in the
# forward overlap-add (K B groups) and of 8 tiles in the crops (C ceil(B P / 8)
# for the error propagation, C ceil(K / 8) for the weight gradient), on a grid
# of min(256, groups rounded up to 8) workgroups. Teams of 8 (forward) or 2
# (crops) workgroups need a grid that is a multiple of 64 or 16, else each
# workgroup walks alone.
TEAM_WALK = [  # (B, C, K, N, n): at (64, 49)
    (3, 40, 100, 64, 16),   # P = 4: forward 300 groups, teams of 8 with a ragged last range; crops of
                            # 80 (the last group of each channel 4 tiles) and 520 groups in teams of 2
    (1, 9, 65, 64, 16),     # forward 65 groups on 72 workgroups: alone; crops 9 groups in teams of 2
                            # and 81 groups alone
    (2, 24, 64, 64, 16),    # forward 128 groups, teams of 8 over exact ranges; crops 24 (alone), 192
    (4, 16, 48, 128, 16),   # P = 9: forward 192 planes in teams of 8; crops of 80 groups spanning
                            # images and 96 groups, teams of 2
]


@pytest.mark.parametrize("shape", TEAM_WALK, ids=lambda s: "x".join(map(str, s)))
def test_inverse_team_walk_shapes(gpu_lib, shape):
    """Every pass at L = 64 against the oracle, compared whole, on grids that
    take each of the inverses' walks (teams, ragged team ranges, alone)."""
    B, C, K, N, n = shape
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=173 + sum(shape))
    check_whole(x, w, g, tiling=(64, 49))


@pytest.mark.parametrize("shape", [sh for sh in BIG64 if sh[7] == "oaa" and sh[1] <= 4],
                         ids=lambda s: "x".join(map(str, s)))
def test_transform_side_64_unfused(gpu_lib, shape):
    """The few-channel L = 64 layers above through the unfused passes
    (tile-group transforms and the streaming contraction), forced."""
    B, C, K, N, n, L, b, method = shape
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=71 + sum(shape[:7]))
    check_whole(x, w, g, contraction=binding.CONTRACTION_NARROW, tiling=(L, b))


FUSED = [  # (B, C, K, N, n, L, b): the fused few-channel passes (L = 64, C <= 4, T <= 8), forced
    (2, 3, 5, 100, 7, 64, 58),     # the first layer's tiling, reduced: T = 2 (4 planes per item)
    (1, 3, 9, 224, 7, 64, 58),     # the first layer's planes: T = 4, K off a multiple of four
    (2, 1, 3, 60, 5, 64, 60),      # one block per plane, K < 4
    (1, 2, 6, 120, 16, 64, 49),    # T = 3, kernels of 16 (15 carried rows)
    (1, 4, 4, 150, 20, 64, 40),    # C = 4, T = 4, ragged last block
    (1, 2, 3, 200, 32, 64, 32),    # T = 7: one plane per item
    (3, 1, 2, 9, 1, 64, 8),        # n = 1: no overlap, nothing carried
    (1, 3, 4, 80, 33, 64, 32),     # n = 33, b = n - 1: 32 carried rows, KR = 64
    (5, 2, 7, 37, 4, 64, 20),      # odd block count per split, B T not a multiple of the splits
    (2, 2, 64, 100, 7, 64, 58),    # partial sums over block-row ranges, inverted on 16 workgroups in
                                   # teams of two (2 x 64 kernel-channel pairs, groups of 8)
]


@pytest.mark.parametrize("shape", FUSED, ids=lambda s: "x".join(map(str, s)))
def test_fused_few_channel_passes(gpu_lib, shape):
    """The fused passes (taken by default from B T^2 >= 512 tiles; these
    reduced layers choose them explicitly) against the oracle, compared
    whole, in the training-step order (cached kernel and input spectra, g
    given again to the weight gradient) and with explicit inputs."""
    B, C, K, N, n, L, b = shape
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=97 + sum(shape))
    plan = binding.Plan(B, C, K, N, n, device=DEV, tiling=(L, b), contraction=binding.CONTRACTION_FUSED)
    assert plan.geometry["fused"] == 1 and not plan.caches_grad_spectra
    y, dx, dw = run_training_step(plan, x, w, g)
    refs = (oracle.conv_forward(x, w), oracle.conv_backward_data(g, w, N), oracle.conv_backward_filter(x, g, n))
    e = tuple(relerr(a, r) for a, r in zip((y, dx, dw), refs))
    print(f"fused {shape}: rel err fwd {e[0]:.2e} bwd_data {e[1]:.2e} bwd_filter {e[2]:.2e}", flush=True)
    assert max(e) <= TOL, e
    e2 = check_whole(x, w, g, contraction=binding.CONTRACTION_FUSED, tiling=(L, b))
    assert max(e2) <= TOL


def test_fused_spectra_layouts(gpu_lib):
    """The W and X regions of a fused plan against the oracle's kernel and
    block spectra, in the run layouts oaa.h documents, and the weight-gradient
    partial sums in PRODUCT against the oracle's contraction."""
    B, C, K, N, n, L, b = 2, 3, 6, 100, 7, 64, 58
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=13)
    plan = binding.Plan(B, C, K, N, n, device=DEV, tiling=(L, b), contraction=binding.CONTRACTION_FUSED)
    geo = plan.geometry
    T, F, S = geo["T"], geo["F"], geo["split"]
    V = L // 2 + 1
    assert geo["fused"] == 1
    xd, wd, gd = to_dev(x), to_dev(w), to_dev(g)
    plan.forward(xd, wd)
    torch.cuda.synchronize()
    Wh = plan.region(binding.REGION_W_SPECTRUM).cpu().numpy()[:K * C * F].reshape(K, C, L, V)
    Xh = plan.region(binding.REGION_X_SPECTRUM).cpu().numpy()[:B * T * C * F * T].reshape(B, T, C, L, V, T)
    Xh = Xh.transpose(0, 2, 1, 5, 3, 4)                                     # [B,C,T,T,L,V]
    Wo = oaa_oracle.filter_spectra(w, L)
    Xo = oaa_oracle.block_spectra(x, n, L, b)
    keep = np.ones((L, V), bool)
    keep[L // 2 + 1:, 0] = keep[L // 2 + 1:, V - 1] = False
    assert relerr(Wh[..., keep], Wo[..., keep]) < TOL
    assert relerr(Xh[..., keep], Xo[..., keep]) < TOL
    plan.backward_data(gd, None)
    plan.backward_filter(None, gd)
    torch.cuda.synchronize()
    part = plan.region(binding.REGION_PRODUCT).cpu().numpy()[:S * F * C * K].reshape(S, L, V, C, K)
    dWh = part.astype(np.complex128).sum(0)
    Go = oaa_oracle.window_spectra(g, n, N, L, side=min(2 * b, L), b=b)
    assert relerr(dWh.transpose(3, 2, 0, 1)[..., keep], oaa_oracle.backward_filter_product(Go, Xo)[..., keep]) < TOL


def test_forward_transform_alternating_halves(gpu_lib):
    """The L = 64 forward transform in the form that launches of 512 groups
    or more take: the two halves of a workgroup alternate between
    transforming a group and loading the next. The kernel, input-block and
    gradient-window spectra against the oracle's, with 640 groups of
    x (a partial group of four tiles per channel) and some workgroups
    walking an odd number of groups."""
    B, C, K, N, n, L, b = 9, 128, 128, 64, 16, 64, 49
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=29)
    plan = binding.Plan(B, C, K, N, n, device=DEV, tiling=(L, b))
    geo = plan.geometry
    T, F = geo["T"], geo["F"]
    V = L // 2 + 1
    assert geo["fused"] == 0 and T == 2 and C * -(-B * T * T // 8) >= 512
    plan.forward(to_dev(x), to_dev(w))
    plan.backward_data(to_dev(g), None)
    torch.cuda.synchronize()
    keep = np.ones((L, V), bool)
    keep[L // 2 + 1:, 0] = keep[L // 2 + 1:, V - 1] = False
    Wh = plan.region(binding.REGION_W_SPECTRUM).cpu().numpy()[:F * C * K].reshape(L, V, C, K)
    assert relerr(Wh.transpose(3, 2, 0, 1)[..., keep], oaa_oracle.filter_spectra(w, L)[..., keep]) < TOL
    Xh = plan.region(binding.REGION_X_SPECTRUM).cpu().numpy()[:F * C * B * T * T].reshape(L, V, C, B, T, T)
    assert relerr(Xh.transpose(3, 2, 4, 5, 0, 1)[..., keep], oaa_oracle.block_spectra(x, n, L, b)[..., keep]) < TOL
    Gh = plan.region(binding.REGION_G_SPECTRUM).cpu().numpy()[:F * K * B * T * T].reshape(L, V, K, B, T, T)
    Go = oaa_oracle.window_spectra(g, n, N, L, side=min(2 * b, L), b=b)
    assert relerr(Gh.transpose(3, 2, 4, 5, 0, 1)[..., keep], Go[..., keep]) < TOL


BIG128 = [  # (B, C, K, N, n, L, b, method): transform side 128 (kernel sides up to 64)
    (1, 2, 3, 64, 33, 128, 33, "oaa"),     # the paper's tiling at n = 33: T = 2, overlap-add in two steps
    (1, 2, 2, 64, 48, 128, 48, "oaa"),     # T = 2
    (2, 1, 2, 64, 64, 128, 64, "oaa"),     # n = N = 64: one output pixel, one block
    (1, 3, 4, 100, 40, 128, 89, "oaa"),    # b = L - n + 1, T = 2, ragged
    (2, 2, 3, 60, 33, 128, 60, "oaa"),     # one block per plane (FFTconv-like)
    (1, 5, 6, 90, 20, 128, 60, "oaa"),     # a kernel that would also fit L = 64
    (8, 40, 36, 64, 33, 128, 33, "oaa"),   # matrix-core contractions (C, K, B P >= 32)
    (1, 2, 3, 70, 40, 128, 0, "oas"),      # overlap-save, h = 89: one window per plane
    (1, 2, 2, 150, 33, 128, 0, "oas"),     # overlap-save, h = 96, T = 2: error propagation in two steps
]


@pytest.mark.parametrize("shape", BIG128, ids=lambda s: "x".join(map(str, s)))
def test_transform_side_128(gpu_lib, shape):
    """Every pass at L = 128 against the oracle, compared whole."""
    B, C, K, N, n, L, b, method = shape
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=73 + sum(shape[:7]))
    m = binding.METHOD_OVERLAP_SAVE if method == "oas" else binding.METHOD_OVERLAP_ADD
    check_whole(x, w, g, tiling=(L, b), method=m)


FOLD_RUNS = [  # (B, C, K, N, n, L): blocks of L/2, where the forward inverse takes several
    # whole block rows per workgroup (runs of consecutive tiles)
    (2, 3, 512, 64, 5, 32),    # T = 4: four block rows per workgroup
    (1, 2, 1024, 100, 7, 32),  # T = 7: two block rows, the last workgroup with one
    (1, 2, 1024, 128, 5, 16),  # T = 16: one block row
    (4, 2, 256, 50, 3, 8),     # T = 13 at L = 8 (the per-block-row kernel)
    (8, 2, 128, 128, 9, 32),   # T = 8, two block rows (the large-kernel layer's tiling)
    (2, 2, 8, 45, 4, 16),      # T = 6 on few planes, ragged output
]


@pytest.mark.parametrize("shape", FOLD_RUNS, ids=lambda s: "x".join(map(str, s)))
def test_forward_block_row_runs(gpu_lib, shape):
    """Forward pass through the overlap-add inverse on runs of block rows
    against the oracle."""
    B, C, K, N, n, L = shape
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=41 + sum(shape))
    plan = binding.Plan(B, C, K, N, n, device=DEV, tiling=(L, L // 2))
    y = plan.forward(to_dev(x), to_dev(w))
    torch.cuda.synchronize()
    e = relerr(y.cpu().numpy(), oracle.conv_forward(x, w))
    print(f"block-row runs {shape}: rel err fwd {e:.2e}", flush=True)
    assert e <= TOL, e


OVERLAP_WALK = [  # (B, C, K, N, n, L, b), 2b > L, at least 1024 planes: the forward inverse
    # walks down groups of block rows (several per step, or one at L <= 16), each group after
    # the first starting from the tile row above it
    (1, 2, 1200, 60, 5, 16, 12),   # T = 5: four block rows per step, groups of 4 and 1
    (1, 2, 1100, 72, 7, 16, 10),   # T = 8: two per step, four groups of one step each
    (2, 1, 600, 100, 3, 8, 6),     # T = 17 at L = 8: one per step, four groups
    (1, 3, 1100, 44, 9, 32, 20),   # L = 32, T = 3: the whole plane in one step
    (1, 1, 1030, 47, 4, 16, 11),   # T = 5, ragged output
]


@pytest.mark.parametrize("shape", OVERLAP_WALK, ids=lambda s: "x".join(map(str, s)))
def test_forward_overlap_walk(gpu_lib, shape):
    """Forward pass through the walking overlap-add inverse against the oracle."""
    B, C, K, N, n, L, b = shape
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=43 + sum(shape))
    plan = binding.Plan(B, C, K, N, n, device=DEV, tiling=(L, b))
    y = plan.forward(to_dev(x), to_dev(w))
    torch.cuda.synchronize()
    e = relerr(y.cpu().numpy(), oracle.conv_forward(x, w))
    print(f"overlap walk {shape}: rel err fwd {e:.2e}", flush=True)
    assert e <= TOL, e


def test_overlap_save_backward_data_walk(gpu_lib):
    """Overlap-save error propagation on many planes: the overlap-add of the
    gradient blocks walks groups of block rows, with one output block row more
    than tile rows (To = T + 1), the last group holding that row alone."""
    B, C, K, N, n = 1, 1030, 2, 100, 5
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=47)
    plan = binding.Plan(B, C, K, N, n, device=DEV, tiling=(16, 0), method=binding.METHOD_OVERLAP_SAVE)
    dx = plan.backward_data(to_dev(g), to_dev(w))
    torch.cuda.synchronize()
    e = relerr(dx.cpu().numpy(), oracle.conv_backward_data(g, w, N))
    print(f"overlap-save backward data walk: rel err {e:.2e}", flush=True)
    assert e <= TOL, e


WIDE = [  # (B, C, K, N, n, tiling): planes wider than one workgroup's run of tiles, so every
    # transform splits a block row into chunks and the walking kernels take many steps
    (1, 2, 3, 1024, 3, "paper"),     # L = 8, b = 3: T = 342
    (1, 2, 3, 1024, 3, "auto"),
    (1, 3, 2, 700, 16, "auto"),      # L = 32: T = 44
    (1, 2, 2, 900, 9, (32, 24)),     # blocks over L/2 on a wide plane
    (2, 1, 2, 400, 32, "paper"),     # the largest kernel side (L = 64)
]


@pytest.mark.parametrize("shape", WIDE, ids=lambda s: "x".join(map(str, s)))
def test_wide_planes_all_passes(gpu_lib, shape):
    """Maximum plane sizes of the transform kernels' launch shapes: all three
    passes compared whole against the oracle."""
    B, C, K, N, n, tiling = shape
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=61 + B + C + K + N + n)
    check_whole(x, w, g, tiling=tiling)


FFTCONV = [  # (B, C, K, N, n, L): one block per plane, L >= N + n - 1 (the paper's FFTconv)
    (1, 3, 4, 32, 5, 64),
    (2, 2, 3, 13, 4, 16),
    (1, 4, 5, 20, 7, 32),
    (2, 6, 70, 30, 3, 32),
    (1, 2, 2, 1, 1, 2),
    (3, 40, 36, 25, 8, 32),
]


@pytest.mark.parametrize("shape", FFTCONV, ids=lambda s: "x".join(map(str, s)))
def test_single_block_fftconv(gpu_lib, shape):
    """The paper's FFTconv baseline as the library's single-block tiling
    (L, L - n + 1): every pass against the oracle."""
    B, C, K, N, n, L = shape
    b = L - n + 1
    assert -(-N // b) == 1
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=41 + sum(shape))
    check_whole(x, w, g, tiling=(L, b))


@pytest.mark.parametrize("name", ["tiny", "plane224_n3", "plane224_n5", "plane224_n8"])
def test_named_small_layers(gpu_lib, name):
    ly = LAYERS[name]
    x, w, g = make_inputs(ly, seed=0)   # g is drawn for every layer; unused passes still checked
    check_whole(x, w, g)


@pytest.mark.parametrize("tiling", ["paper", "auto"])
@pytest.mark.parametrize("name,batch,C,K", [("first224", 2, None, None), ("mid56", 2, None, None),
                                            ("large128", 1, 16, 32)])
def test_reduced_large_layers_whole(gpu_lib, name, batch, C, K, tiling):
    ly = LAYERS[name]
    ly = Layer(ly.name, batch, C or ly.C, K or ly.K, ly.N, ly.n, ly.x_dist, ly.w_var, ly.g_dist)
    x, w, g = make_inputs(ly, seed=0)
    check_whole(x, w, g, tiling=tiling)


def run_training_step(plan, x, w, g):
    """The three passes as bench.py times them: backward_data reuses the
    forward's kernel spectra, backward_filter the input and gradient spectra
    of the two passes before it (the fused passes keep no gradient spectra
    and take g again)."""
    xd, wd, gd = to_dev(x), to_dev(w), to_dev(g)
    y = plan.forward(xd, wd)
    dx = plan.backward_data(gd, None)
    dw = plan.backward_filter(None, None if plan.caches_grad_spectra else gd)
    torch.cuda.synchronize()
    return y.cpu().numpy(), dx.cpu().numpy(), dw.cpu().numpy()


def _stratified(rng, B, nch, side, per=4, block=32):
    """Index lists (b, ch, i, j): `per` random pixels for every image and
    every block of `block` channels (the row tiles of the contractions span
    whole 32-channel blocks, their column tiles whole images or parts of
    one), plus the last pixel of the last channel of every image."""
    cols = [[], [], [], []]
    for b in range(B):
        for c0 in range(0, nch, block):
            c1 = min(c0 + block, nch)
            cols[0] += [b] * per
            cols[1] += list(rng.integers(c0, c1, per))
            cols[2] += list(rng.integers(0, side, per))
            cols[3] += list(rng.integers(0, side, per))
        cols[0].append(b)
        cols[1].append(nch - 1)
        cols[2].append(side - 1)
        cols[3].append(side - 1)
    return [np.asarray(c) for c in cols]


def _one_per_block(rng, nch, block=32):
    """One random channel from every block of `block`, plus the first and
    last channel."""
    picks = {0, nch - 1}
    for c0 in range(0, nch, block):
        picks.add(int(rng.integers(c0, min(c0 + block, nch))))
    return sorted(picks)


_FULL_INPUTS = {}
_FULL_REFS = {}


def full_size_inputs(name):
    """Seeded inputs of a named layer at full size (drawn once per session)."""
    if name not in _FULL_INPUTS:
        _FULL_INPUTS[name] = make_inputs(LAYERS[name], seed=0)
    return _FULL_INPUTS[name]


def full_size_refs(name):
    """Oracle values for check_full_size, computed once per layer: the first
    and last image whole, stratified pixels, and whole dw planes of kernel-
    channel pairs spanning every 32 x 32 block."""
    if name not in _FULL_REFS:
        ly = LAYERS[name]
        x, w, g = full_size_inputs(name)
        B, C, K, N, n, M = ly.B, ly.C, ly.K, ly.N, ly.n, ly.M
        ends = sorted({0, B - 1})
        rng = np.random.default_rng(1)
        iy = _stratified(rng, B, K, M)
        ix = _stratified(rng, B, C, N)
        cs, ks = _one_per_block(rng, C), _one_per_block(rng, K)
        _FULL_REFS[name] = dict(
            ends=ends, y_ends=oracle.conv_forward(x[ends], w), dx_ends=oracle.conv_backward_data(g[ends], w, N),
            iy=iy, y_at=oracle.conv_forward_at(x, w, *iy), ix=ix, dx_at=oracle.conv_backward_data_at(g, w, N, *ix),
            cs=cs, ks=ks, dw_pairs=oracle.conv_backward_filter(x[:, cs], g[:, ks], n))
    return _FULL_REFS[name]


def check_full_size(name, y, dx, dw, label):
    """Full-size outputs against the oracle:
    * y and dx compared whole for the first and the last image (all output
      and input channels);
    * y and dx on four random pixels of every image and every block of 32
      channels (every column and row tile of the forward and error-propagation
      contractions);
    * dw whole (all n^2 taps) for one input channel from every block of 32
      and one kernel from every block of 32, all pairs of the two sets (every
      output tile of the weight-gradient contraction)."""
    r = full_size_refs(name)
    n = LAYERS[name].n
    e_whole = (relerr(y[r["ends"]], r["y_ends"]), relerr(dx[r["ends"]], r["dx_ends"]))
    e_strat = (relerr(y[tuple(r["iy"])], r["y_at"]), relerr(dx[tuple(r["ix"])], r["dx_at"]))
    e_dw = relerr(dw[np.ix_(r["ks"], r["cs"])], r["dw_pairs"])
    print(f"{label}: whole images {r['ends']}: fwd {e_whole[0]:.2e} bwd_data {e_whole[1]:.2e}; "
          f"{len(r['iy'][0])} y and {len(r['ix'][0])} dx pixels over every image and channel block: "
          f"fwd {e_strat[0]:.2e} bwd_data {e_strat[1]:.2e}; dw {len(r['ks'])}x{len(r['cs'])} kernel-channel "
          f"pairs x {n * n} taps: {e_dw:.2e}", flush=True)
    assert max(e_whole + e_strat + (e_dw,)) <= TOL, (e_whole, e_strat, e_dw)
    assert np.isfinite(y).all() and np.isfinite(dx).all() and np.isfinite(dw).all()


@pytest.mark.parametrize("tiling", ["paper", "auto"])
@pytest.mark.parametrize("name", ["first224", "mid56", "large128"])
def test_full_size_layers(gpu_lib, name, tiling):
    """Full size, in the launch configuration bench.py times (tiling "auto"
    is its default)."""
    ly = LAYERS[name]
    x, w, g = full_size_inputs(name)
    plan = binding.Plan(ly.B, ly.C, ly.K, ly.N, ly.n, device=DEV, tiling=tiling)
    y, dx, dw = run_training_step(plan, x, w, g)
    del plan
    check_full_size(name, y, dx, dw, label=f"{name} {tiling} {y.shape}")


def test_spectra_past_32_bit_offsets(gpu_lib):
    """A layer whose gradient-window and forward-product spectra exceed 4 GB
    (2112 bins x 512 kernels x 576 tiles x 8 bytes = 5.0 GB), so that the
    L = 64 forward transform, the inverse and the matrix-core contraction take
    their 64-bit-offset forms; outputs on stratified samples of every image
    and block of 32 channels, and whole dw planes of kernel-channel pairs
    spanning every block of 32."""
    B, C, K, N, n, L, b = 64, 32, 512, 128, 16, 64, 49
    ly = Layer("wide_spectra", B, C, K, N, n)
    x, w, g = make_inputs(ly, seed=41)
    plan = binding.Plan(B, C, K, N, n, device=DEV, tiling=(L, b))
    geo = plan.geometry
    assert geo["F"] * K * B * geo["T"] ** 2 * 8 > 2 ** 32
    y, dx, dw = run_training_step(plan, x, w, g)
    del plan
    M = ly.M
    rng = np.random.default_rng(5)
    iy, ix = _stratified(rng, B, K, M), _stratified(rng, B, C, N)
    cs, ks = _one_per_block(rng, C), _one_per_block(rng, K)
    e = (relerr(y[tuple(iy)], oracle.conv_forward_at(x, w, *iy)),
         relerr(dx[tuple(ix)], oracle.conv_backward_data_at(g, w, N, *ix)),
         relerr(dw[np.ix_(ks, cs)], oracle.conv_backward_filter(x[:, cs], g[:, ks], n)))
    print(f"spectra past 4 GB: {len(iy[0])} y, {len(ix[0])} dx pixels, dw {len(ks)}x{len(cs)} pairs: "
          f"{e[0]:.2e} {e[1]:.2e} {e[2]:.2e}", flush=True)
    assert max(e) <= TOL, e
    assert np.isfinite(y).all() and np.isfinite(dx).all() and np.isfinite(dw).all()


CHAIN = [  # (B, C, J, K, N, n1, n2, tiling, method): two stacked layers composed in the frequency domain
    (2, 3, 5, 4, 20, 3, 4, "paper", "oaa"),        # L = 16, vector-ALU composition
    (2, 40, 36, 48, 24, 3, 3, "paper", "oaa"),     # matrix-core composition and passes
    (2, 2, 3, 5, 100, 9, 8, (64, 49), "oaa"),      # L = 64 transforms (unfused)
    (1, 3, 4, 2, 70, 20, 14, (128, 0), "oas"),     # L = 128, overlap-save
    (3, 1, 1, 1, 9, 1, 1, "paper", "oaa"),         # 1 x 1 kernels: pure channel mixing
]


@pytest.mark.parametrize("shape", CHAIN, ids=lambda s: "x".join(map(str, s[:7])) + f"-{s[8]}")
def test_kernel_chain_two_stacked_layers(gpu_lib, shape):
    """oaa_plan_set_kernel_chain: the forward pass gives conv(conv(x, w1), w2)
    and the error propagation the gradient through both layers, compared
    whole with the oracle's two layers one after the other."""
    B, C, J, K, N, n1, n2, tiling, method = shape
    rng = np.random.default_rng(sum(shape[:7]))
    x = rng.uniform(-1, 1, (B, C, N, N)).astype(np.float32)
    w1 = (rng.standard_normal((J, C, n1, n1)) / np.sqrt(C * n1 * n1)).astype(np.float32)
    w2 = (rng.standard_normal((K, J, n2, n2)) / np.sqrt(J * n2 * n2)).astype(np.float32)
    n = n1 + n2 - 1
    M = N - n + 1
    g = rng.uniform(-1, 1, (B, K, M, M)).astype(np.float32)
    m = binding.METHOD_OVERLAP_SAVE if method == "oas" else binding.METHOD_OVERLAP_ADD
    plan = binding.Plan(B, C, K, N, n, device=DEV, tiling=tiling, method=m)
    assert plan.geometry["fused"] == 0
    plan.set_kernel_chain(to_dev(w1), to_dev(w2))
    y = plan.forward(to_dev(x), None)
    dx = plan.backward_data(to_dev(g), None)
    torch.cuda.synchronize()
    x64, w164, w264, g64 = (a.astype(np.float64) for a in (x, w1, w2, g))
    y_ref = oracle.conv_forward(oracle.conv_forward(x64, w164), w264)
    dx_ref = oracle.conv_backward_data(oracle.conv_backward_data(g64, w264, N - n1 + 1), w164, N)
    e = (relerr(y.cpu().numpy(), y_ref), relerr(dx.cpu().numpy(), dx_ref))
    print(f"chain {shape}: L={plan.geometry['L']} rel err fwd {e[0]:.2e} bwd_data {e[1]:.2e}", flush=True)
    assert max(e) <= TOL, e


def test_stage_spectra_match_oracle_steps(gpu_lib):
    """Workspace spectra (kernel, input blocks, gradient windows, products)
    against the OaA steps of the oracle, in the layouts oaa.h documents."""
    B, C, K, N, n = 2, 3, 4, 23, 5
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=3)
    plan = binding.Plan(B, C, K, N, n, device=DEV)
    geo = plan.geometry
    L, T, F = geo["L"], geo["T"], geo["F"]
    V = L // 2 + 1
    xd, wd, gd = to_dev(x), to_dev(w), to_dev(g)
    plan.forward(xd, wd)
    torch.cuda.synchronize()
    Wh = plan.region(binding.REGION_W_SPECTRUM).cpu().numpy().reshape(L, V, C, K)
    Xh = plan.region(binding.REGION_X_SPECTRUM).cpu().numpy().reshape(L, V, C, B, T, T)
    Yh = plan.region(binding.REGION_PRODUCT).cpu().numpy()[:F * K * B * T * T].reshape(L, V, K, B, T, T)
    Wo = oaa_oracle.filter_spectra(w, L)                    # [K,C,L,V]
    Xo = oaa_oracle.block_spectra(x, n, L)                  # [B,C,T,T,L,V]
    Yo = oaa_oracle.forward_product(Xo, Wo)                 # [B,K,T,T,L,V]
    # the contractions skip the bins (u > L/2, v in {0, L/2}): there the
    # products are the conjugates of bins (L - u, v)
    keep = np.ones((L, V), bool)
    keep[L // 2 + 1:, 0] = keep[L // 2 + 1:, V - 1] = False
    assert relerr(Wh.transpose(3, 2, 0, 1), Wo) < TOL
    # block and window spectra: bins (u > L/2, v in {0, L/2}) are conjugates that nothing reads
    assert relerr(Xh.transpose(3, 2, 4, 5, 0, 1)[..., keep], Xo[..., keep]) < TOL
    assert relerr(Yh.transpose(3, 2, 4, 5, 0, 1)[..., keep], Yo[..., keep]) < TOL
    plan.backward_data(gd, None)
    torch.cuda.synchronize()
    Gh = plan.region(binding.REGION_G_SPECTRUM).cpu().numpy().reshape(L, V, K, B, T, T)
    dXh = plan.region(binding.REGION_PRODUCT).cpu().numpy()[:F * C * B * T * T].reshape(L, V, C, B, T, T)
    Go = oaa_oracle.window_spectra(g, n, N, L, side=2 * n)   # the library stores 2n x 2n windows
    assert relerr(Gh.transpose(3, 2, 4, 5, 0, 1)[..., keep], Go[..., keep]) < TOL
    assert relerr(dXh.transpose(3, 2, 4, 5, 0, 1)[..., keep], oaa_oracle.backward_data_product(Go, Wo)[..., keep]) < TOL
    plan.backward_filter(None, None)
    torch.cuda.synchronize()
    S = geo["split"]
    part = plan.region(binding.REGION_PRODUCT).cpu().numpy()[:S * F * C * K].reshape(S, L, V, C, K)
    dWh = part.astype(np.complex128).sum(0)
    assert relerr(dWh.transpose(3, 2, 0, 1)[..., keep], oaa_oracle.backward_filter_product(Go, Xo)[..., keep]) < TOL


def test_cached_spectra_reuse_matches_explicit_inputs(gpu_lib):
    B, C, K, N, n = 2, 5, 6, 30, 7
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=5)
    plan = binding.Plan(B, C, K, N, n, device=DEV)
    xd, wd, gd = to_dev(x), to_dev(w), to_dev(g)
    y1 = plan.forward(xd, wd).clone()
    y2 = plan.forward(xd, None).clone()           # cached kernel spectra
    dx1 = plan.backward_data(gd, wd).clone()
    dx2 = plan.backward_data(gd, None).clone()
    dw1 = plan.backward_filter(xd, gd).clone()
    plan.forward(xd, wd)
    plan.backward_data(gd, None)
    dw2 = plan.backward_filter(None, None).clone()  # cached block and window spectra
    torch.cuda.synchronize()
    assert torch.equal(y1, y2) and torch.equal(dx1, dx2) and torch.equal(dw1, dw2)
    assert relerr(dw1.cpu().numpy(), oracle.conv_backward_filter(x, g, n)) <= TOL


def test_bitwise_deterministic(gpu_lib):
    B, C, K, N, n = 2, 66, 70, 24, 3
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=6)
    _, y1, dx1, dw1 = run_layer(x, w, g)
    _, y2, dx2, dw2 = run_layer(x, w, g)
    assert np.array_equal(y1, y2) and np.array_equal(dx1, dx2) and np.array_equal(dw1, dw2)


def test_outputs_overwritten_not_accumulated(gpu_lib):
    B, C, K, N, n = 1, 2, 3, 14, 4
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=7)
    plan = binding.Plan(B, C, K, N, n, device=DEV)
    xd, wd, gd = to_dev(x), to_dev(w), to_dev(g)
    M = N - n + 1
    y = torch.full((B, K, M, M), 1e6, device=DEV)
    dx = torch.full((B, C, N, N), -1e6, device=DEV)
    dw = torch.full((K, C, n, n), 3e5, device=DEV)
    plan.forward(xd, wd, y)
    plan.backward_data(gd, wd, dx)
    plan.backward_filter(xd, gd, dw)
    torch.cuda.synchronize()
    assert relerr(y.cpu().numpy(), oracle.conv_forward(x, w)) <= TOL
    assert relerr(dx.cpu().numpy(), oracle.conv_backward_data(g, w, N)) <= TOL
    assert relerr(dw.cpu().numpy(), oracle.conv_backward_filter(x, g, n)) <= TOL


def test_zero_inputs_give_exact_zeros(gpu_lib):
    B, C, K, N, n = 1, 3, 2, 19, 6
    z = np.zeros((B, C, N, N), np.float32)
    w = np.ones((K, C, n, n), np.float32)
    g = np.zeros((B, K, N - n + 1, N - n + 1), np.float32)
    _, y, dx, dw = run_layer(z, w, g)
    assert not y.any() and not dx.any() and not dw.any()


def test_graph_capture_replays_match_eager(gpu_lib):
    """A training step (forward, backward-data with cached kernel spectra,
    backward-filter with cached input and gradient spectra) captured in a
    HIP graph: several replays, with eager work on the outputs in between,
    each equal bit for bit to the eager step."""
    B, C, K, N, n = 2, 8, 70, 41, 5
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=53)
    plan = binding.Plan(B, C, K, N, n, device=DEV)
    xd, wd, gd = to_dev(x), to_dev(w), to_dev(g)
    M = N - n + 1
    y = torch.empty((B, K, M, M), dtype=torch.float32, device=DEV)
    dx, dw = torch.empty_like(xd), torch.empty_like(wd)

    def step():
        plan.forward(xd, wd, y)
        plan.backward_data(gd, None, dx)
        plan.backward_filter(None, None, dw)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    ref = (y.clone(), dx.clone(), dw.clone())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for i in range(4):
        y.fill_(float(i + 1))
        dx.mul_(0.5)
        dw.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, ref[0]) and torch.equal(dx, ref[1]) and torch.equal(dw, ref[2]), i
    e = relerr(y.cpu().numpy(), oracle.conv_forward(x, w))
    assert e <= TOL, e


def test_named_stream_is_used(gpu_lib):
    B, C, K, N, n = 2, 3, 4, 32, 5
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=8)
    s = torch.cuda.Stream(device=DEV)
    with torch.cuda.stream(s):
        plan = binding.Plan(B, C, K, N, n, device=DEV)
        xd, wd = to_dev(x), to_dev(w)
        y = plan.forward(xd, wd)
    s.synchronize()
    assert relerr(y.cpu().numpy(), oracle.conv_forward(x, w)) <= TOL


def test_autograd_function_matches_oracle(gpu_lib):
    """OaAConv2dFunction: y and both gradients of <y, g> through autograd,
    against the oracle; two forwards before one backward recompute the
    cached spectra."""
    from paper_1601_06815_amd.autograd import OaAConv2d, OaAConv2dFunction
    B, C, K, N, n = 2, 3, 5, 21, 4
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=77)
    plan = binding.Plan(B, C, K, N, n, device=DEV, tiling="auto")
    xd = to_dev(x).requires_grad_(True)
    wd = to_dev(w).requires_grad_(True)
    y = OaAConv2dFunction.apply(xd, wd, plan)
    # a second forward on the same plan with other inputs
    x2, w2, _ = make_inputs(Layer("t", B, C, K, N, n), seed=78)
    OaAConv2dFunction.apply(to_dev(x2), to_dev(w2), plan)
    (y * to_dev(g)).sum().backward()
    torch.cuda.synchronize()
    e = (relerr(y.detach().cpu().numpy(), oracle.conv_forward(x, w)),
         relerr(xd.grad.cpu().numpy(), oracle.conv_backward_data(g, w, N)),
         relerr(wd.grad.cpu().numpy(), oracle.conv_backward_filter(x, g, n)))
    print(f"autograd rel err fwd {e[0]:.2e} dx {e[1]:.2e} dw {e[2]:.2e}", flush=True)
    assert max(e) <= TOL, e
    # the layer module: same three results against torch's float64 autograd on
    # the CPU (cross-correlation with the flipped kernel)
    layer = OaAConv2d(C, K, n, device=DEV)
    with torch.no_grad():
        layer.weight.copy_(to_dev(w))
    xd2 = to_dev(x).requires_grad_(True)
    yl = layer(xd2)
    (yl * to_dev(g)).sum().backward()
    xr = torch.from_numpy(x).double().requires_grad_(True)
    wr = torch.from_numpy(w).double().requires_grad_(True)
    yr = torch.nn.functional.conv2d(xr, wr.flip(-1, -2))
    (yr * torch.from_numpy(g).double()).sum().backward()
    assert relerr(yl.detach().cpu().numpy(), yr.detach().numpy()) <= TOL
    assert relerr(xd2.grad.cpu().numpy(), xr.grad.numpy()) <= TOL
    assert relerr(layer.weight.grad.cpu().numpy(), wr.grad.numpy()) <= TOL


# ---------------------------------------------------------------------------
# output-tiled method: overlap-and-save forward, overlap-add of gradient blocks

OAS = binding.METHOD_OVERLAP_SAVE


@pytest.mark.parametrize("double", [False, True], ids=["L0", "2L0"])
@pytest.mark.parametrize("shape", SMALL, ids=lambda s: "x".join(map(str, s)))
def test_overlap_save_small_layers(gpu_lib, shape, double):
    B, C, K, N, n = shape
    L = 2
    while L < 2 * n - 1:
        L *= 2
    if double:
        L *= 2
    if L > 128:
        pytest.skip("transform side above 128")
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=53 + sum(shape))
    check_whole(x, w, g, tiling=(L, 0), method=OAS)


@pytest.mark.parametrize("contraction", [binding.CONTRACTION_VALU, binding.CONTRACTION_MFMA, binding.CONTRACTION_NARROW],
                         ids=["valu", "mfma", "narrow"])
def test_overlap_save_contraction_engines(gpu_lib, contraction):
    shape = (2, 3, 64, 30, 7) if contraction == binding.CONTRACTION_NARROW else (2, 40, 66, 21, 4)
    B, C, K, N, n = shape
    x, w, g = make_inputs(Layer("t", B, C, K, N, n), seed=61)
    check_whole(x, w, g, contraction=contraction, tiling="auto", method=OAS)


@pytest.mark.parametrize("name,batch,C,K", [("first224", 2, None, None), ("mid56", 2, None, None),
                                            ("large128", 1, 16, 32)])
def test_overlap_save_reduced_large_layers_whole(gpu_lib, name, batch, C, K):
    ly = LAYERS[name]
    ly = Layer(ly.name, batch, C or ly.C, K or ly.K, ly.N, ly.n, ly.x_dist, ly.w_var, ly.g_dist)
    x, w, g = make_inputs(ly, seed=0)
    check_whole(x, w, g, tiling="auto", method=OAS)


@pytest.mark.parametrize("name", ["first224", "mid56", "large128"])
def test_overlap_save_full_size_layers(gpu_lib, name):
    """Full size, in the launch configuration bench.py --method oas times."""
    ly = LAYERS[name]
    x, w, g = full_size_inputs(name)
    plan = binding.Plan(ly.B, ly.C, ly.K, ly.N, ly.n, device=DEV, tiling="auto", method=OAS)
    y, dx, dw = run_training_step(plan, x, w, g)
    del plan
    check_full_size(name, y, dx, dw, label=f"{name} overlap-save")


def test_overlap_save_stage_spectra_match_oracle(gpu_lib):
    """Window spectra of x and block spectra of g, as the kernels store them,
    against the oracle's steps."""
    from oracle import oas
    B, C, K, N, n = 2, 3, 4, 23, 5
    ly = Layer("t", B, C, K, N, n)
    x, w, g = make_inputs(ly, seed=9)
    plan = binding.Plan(B, C, K, N, n, device=DEV, tiling=(16, 0), method=OAS)
    xd, wd, gd = to_dev(x), to_dev(w), to_dev(g)
    plan.forward(xd, wd)
    plan.backward_data(gd, None)
    torch.cuda.synchronize()
    geo = plan.geometry
    L, T, F = geo["L"], geo["T"], geo["F"]
    V = L // 2 + 1
    Xh = plan.region(binding.REGION_X_SPECTRUM).cpu().numpy().reshape(L, V, C, B, T, T)
    Gh = plan.region(binding.REGION_G_SPECTRUM).cpu().numpy().reshape(L, V, K, B, T, T)
    Xo = oas.window_spectra(x, n, L).transpose(4, 5, 1, 0, 2, 3)
    Go = oas.block_spectra(g, n, L).transpose(4, 5, 1, 0, 2, 3)
    # bins (u > L/2, v in {0, L/2}) are conjugates that nothing reads
    keep = np.ones((L, V), bool)
    keep[L // 2 + 1:, 0] = keep[L // 2 + 1:, V - 1] = False
    assert relerr(Xh[keep], Xo[keep]) <= TOL and relerr(Gh[keep], Go[keep]) <= TOL
