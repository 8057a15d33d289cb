"""Pins for the CPU oracle (runs without a GPU).

Each check ties the oracle to something other than itself: library routines
(scipy's 2-D convolution, torch float64 autograd), a hand-derived worked
example, closed forms, invariants of the layer (adjoint identity, linearity,
shift behaviour), exact finite differences of a bilinear form, and the
explicit-DFT route of the convolution theorem. Shapes are asymmetric and
random so that a transposed operand, a missing flip, a wrong offset or a
dropped term fails at least one of them.
"""

import json
import os

import numpy as np
import pytest
import scipy.signal
import torch

import oracle
from oracle import oaa, oas
from tests.conftest import relerr

GOLD = os.path.join(os.path.dirname(__file__), "golden")

SHAPES = [  # (B, C, K, N, n): partial blocks, n = 1, N = n, n even / odd
    (1, 3, 4, 32, 5),
    (2, 2, 3, 13, 4),
    (1, 1, 1, 9, 3),
    (2, 3, 2, 11, 1),
    (1, 2, 2, 7, 7),
    (1, 1, 2, 10, 6),
    (3, 2, 3, 17, 8),
]


def _rand(shape, seed):
    rng = np.random.default_rng(seed)
    B, C, K, N, n = shape
    M = N - n + 1
    return (rng.uniform(-1, 1, (B, C, N, N)), rng.standard_normal((K, C, n, n)),
            rng.uniform(-1, 1, (B, K, M, M)))


@pytest.mark.parametrize("shape", SHAPES)
def test_forward_matches_scipy_convolve2d(shape):
    x, w, _ = _rand(shape, 1)
    B, C, K, N, n = shape
    ref = np.zeros((B, K, N - n + 1, N - n + 1))
    for b in range(B):
        for k in range(K):
            for c in range(C):
                ref[b, k] += scipy.signal.convolve2d(x[b, c], w[k, c], mode="valid")
    assert relerr(oracle.conv_forward(x, w), ref) < 1e-13


@pytest.mark.parametrize("shape", SHAPES)
def test_three_passes_match_torch_float64_autograd(shape):
    x, w, g = _rand(shape, 2)
    xt = torch.tensor(x, requires_grad=True)
    wf = torch.tensor(w[:, :, ::-1, ::-1].copy(), requires_grad=True)  # conv2d correlates
    y = torch.nn.functional.conv2d(xt, wf)
    (y * torch.tensor(g)).sum().backward()
    assert relerr(oracle.conv_forward(x, w), y.detach().numpy()) < 1e-13
    assert relerr(oracle.conv_backward_data(g, w, shape[3]), xt.grad.numpy()) < 1e-13
    assert relerr(oracle.conv_backward_filter(x, g, shape[4]),
                  wf.grad.numpy()[:, :, ::-1, ::-1]) < 1e-13


def test_hand_derived_worked_example():
    d = json.load(open(os.path.join(GOLD, "worked_4x4_2x2.json")))
    x = np.array(d["x"], float)[None, None]
    w = np.array(d["w"], float)[None, None]
    g = np.array(d["g"], float)[None, None]
    np.testing.assert_array_equal(oracle.conv_forward(x, w)[0, 0], np.array(d["y"]))
    np.testing.assert_array_equal(oracle.conv_backward_data(g, w, 4)[0, 0], np.array(d["dx"]))
    np.testing.assert_array_equal(oracle.conv_backward_filter(x, g, 2)[0, 0], np.array(d["dw"]))


@pytest.mark.parametrize("shape", [(1, 2, 3, 8, 3), (2, 1, 2, 12, 5), (1, 3, 1, 6, 1), (1, 1, 1, 5, 5)])
def test_forward_matches_explicit_dft(shape):
    x, w, _ = _rand(shape, 3)
    assert relerr(oracle.conv_forward(x, w), oracle.dft_conv_forward(x, w)) < 1e-12
    # any transform size past N+n-1 gives the same linear convolution
    N, n = shape[3], shape[4]
    assert relerr(oracle.conv_forward(x, w), oracle.dft_conv_forward(x, w, Lc=N + n + 4)) < 1e-12


def test_explicit_dft_detects_aliasing():
    # a transform shorter than N+n-1 must be refused, not silently wrap around
    x, w, _ = _rand((1, 1, 1, 8, 3), 4)
    with pytest.raises(ValueError):
        oracle.dft_conv_forward(x, w, Lc=9)


@pytest.mark.parametrize("n,N", [(3, 9), (4, 10), (1, 5), (5, 5)])
def test_delta_kernels(n, N):
    rng = np.random.default_rng(5)
    x = rng.uniform(-1, 1, (2, 1, N, N))
    M = N - n + 1
    w = np.zeros((1, 1, n, n))
    w[0, 0, 0, 0] = 1.0   # true convolution: y[i,j] = x[i+n-1, j+n-1]
    np.testing.assert_array_equal(oracle.conv_forward(x, w)[:, 0], x[:, 0, n - 1:, n - 1:])
    w[0, 0, 0, 0] = 0.0
    w[0, 0, n - 1, n - 1] = 1.0   # y = x[:M, :M]
    np.testing.assert_array_equal(oracle.conv_forward(x, w)[:, 0], x[:, 0, :M, :M])
    w[0, 0, n - 1, n - 1] = 0.0
    w[0, 0, 0, n - 1] = 1.0       # rows shifted, columns not: y = x[n-1:, :M]
    np.testing.assert_array_equal(oracle.conv_forward(x, w)[:, 0], x[:, 0, n - 1:, :M])


@pytest.mark.parametrize("shape", [(2, 3, 4, 9, 3), (1, 2, 3, 10, 4), (3, 1, 2, 7, 7), (1, 1, 1, 6, 1)])
def test_all_ones_closed_forms(shape):
    B, C, K, N, n = shape
    M = N - n + 1
    x = np.ones((B, C, N, N))
    w = np.ones((K, C, n, n))
    g = np.ones((B, K, M, M))
    np.testing.assert_array_equal(oracle.conv_forward(x, w), np.full((B, K, M, M), C * n * n))
    # dx[p,q] = K * cnt(p) * cnt(q), cnt(p) = #{u < n : 0 <= p-n+1+u < M}
    cnt = np.array([min(p, M - 1) - max(0, p - n + 1) + 1 for p in range(N)], float)
    np.testing.assert_array_equal(oracle.conv_backward_data(g, w, N),
                                  np.broadcast_to(K * np.outer(cnt, cnt), (B, C, N, N)))
    np.testing.assert_array_equal(oracle.conv_backward_filter(x, g, n),
                                  np.full((K, C, n, n), B * M * M))


def test_separable_kernel_is_row_then_column_1d_convolution():
    rng = np.random.default_rng(6)
    N, n = 15, 4
    x = rng.uniform(-1, 1, (1, 1, N, N))
    a, bvec = rng.standard_normal(n), rng.standard_normal(n)
    w = np.outer(a, bvec)[None, None]
    rows = np.stack([np.convolve(r, bvec, mode="valid") for r in x[0, 0]])
    ref = np.stack([np.convolve(col, a, mode="valid") for col in rows.T]).T
    assert relerr(oracle.conv_forward(x, w)[0, 0], ref) < 1e-13


def test_shift_equivariance():
    rng = np.random.default_rng(7)
    x = rng.uniform(-1, 1, (1, 2, 16, 16))
    w = rng.standard_normal((3, 2, 4, 4))
    y = oracle.conv_forward(x, w)
    ys = oracle.conv_forward(x[:, :, 2:14, 3:15], w)      # 12x12 window, shifted by (2, 3)
    np.testing.assert_allclose(ys, y[:, :, 2:11, 3:12], rtol=0, atol=1e-13)


@pytest.mark.parametrize("shape", SHAPES)
def test_adjoint_identity_and_linearity(shape):
    x, w, g = _rand(shape, 8)
    N, n = shape[3], shape[4]
    y = oracle.conv_forward(x, w)
    dx = oracle.conv_backward_data(g, w, N)
    dw = oracle.conv_backward_filter(x, g, n)
    a, b, c = np.vdot(y, g), np.vdot(x, dx), np.vdot(w, dw)
    scale = np.sum(np.abs(y) * np.abs(g))
    assert abs(a - b) < 1e-13 * scale and abs(a - c) < 1e-13 * scale
    x2, w2, _ = _rand(shape, 9)
    assert relerr(oracle.conv_forward(2.5 * x - x2, w),
                  2.5 * y - oracle.conv_forward(x2, w)) < 1e-13
    assert relerr(oracle.conv_forward(x, w + 3 * w2),
                  y + 3 * oracle.conv_forward(x, w2)) < 1e-13


def test_finite_differences_of_bilinear_loss():
    # L(x, w) = <fwd(x, w), g> is linear in each argument, so a central
    # difference with a unit step is exact up to rounding.
    shape = (2, 2, 3, 9, 4)
    x, w, g = _rand(shape, 10)
    N, n = shape[3], shape[4]
    loss = lambda xx, ww: np.vdot(oracle.conv_forward(xx, ww), g)  # noqa: E731
    dx = oracle.conv_backward_data(g, w, N)
    dw = oracle.conv_backward_filter(x, g, n)
    rng = np.random.default_rng(11)
    for _ in range(12):
        idx = tuple(int(rng.integers(0, s)) for s in x.shape)
        e = np.zeros_like(x)
        e[idx] = 1.0
        fd = (loss(x + e, w) - loss(x - e, w)) / 2
        assert abs(fd - dx[idx]) < 1e-12 * max(1.0, abs(dx[idx]))
        idw = tuple(int(rng.integers(0, s)) for s in w.shape)
        e = np.zeros_like(w)
        e[idw] = 1.0
        fd = (loss(x, w + e) - loss(x, w - e)) / 2
        assert abs(fd - dw[idw]) < 1e-12 * max(1.0, abs(dw[idw]))


def test_sampled_elements_match_whole_arrays():
    shape = (2, 3, 4, 12, 5)
    x, w, g = _rand(shape, 12)
    B, C, K, N, n = shape
    M = N - n + 1
    y = oracle.conv_forward(x, w)
    dx = oracle.conv_backward_data(g, w, N)
    dw = oracle.conv_backward_filter(x, g, n)
    rng = np.random.default_rng(13)
    i = [rng.integers(0, s, 20) for s in (B, K, M, M)]
    np.testing.assert_allclose(oracle.conv_forward_at(x, w, *i), y[tuple(i)], rtol=1e-13, atol=1e-13)
    i = [rng.integers(0, s, 20) for s in (B, C, N, N)]
    np.testing.assert_allclose(oracle.conv_backward_data_at(g, w, N, *i), dx[tuple(i)], rtol=1e-13, atol=1e-13)
    i = [rng.integers(0, s, 20) for s in (K, C, n, n)]
    np.testing.assert_allclose(oracle.conv_backward_filter_at(x, g, n, *i), dw[tuple(i)], rtol=1e-13, atol=1e-13)


# ---- the step-by-step OaA oracle (Section 2) against the pinned definition --

@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("Lmode", ["pow2", "2n-1", "big"])
def test_oaa_steps_equal_direct_definition(shape, Lmode):
    x, w, g = _rand(shape, 14)
    N, n = shape[3], shape[4]
    L = {"pow2": oaa.fft_size(n), "2n-1": max(2 * n - 1, 1), "big": oaa.fft_size(n) * 2}[Lmode]
    if L < 2:
        L = 2
    assert relerr(oaa.forward(x, w, L), oracle.conv_forward(x, w)) < 1e-12
    assert relerr(oaa.backward_data(g, w, N, L), oracle.conv_backward_data(g, w, N)) < 1e-12
    assert relerr(oaa.backward_filter(x, g, n, L), oracle.conv_backward_filter(x, g, n)) < 1e-12


@pytest.mark.parametrize("shape", SHAPES)
def test_oaa_backward_independent_of_window_side(shape):
    # windows of side 2n (what the GPU path stores) and L give the results of
    # the 2n-1 windows, which equal the direct definition
    x, w, g = _rand(shape, 16)
    N, n = shape[3], shape[4]
    L = oaa.fft_size(n)
    for side in (2 * n, L):
        if side > L:
            continue
        assert relerr(oaa.backward_data(g, w, N, L, side), oracle.conv_backward_data(g, w, N)) < 1e-12
        assert relerr(oaa.backward_filter(x, g, n, L, side), oracle.conv_backward_filter(x, g, n)) < 1e-12
    with pytest.raises(ValueError):
        oaa.window_spectra(g, n, N, L, side=2 * n - 2)


@pytest.mark.parametrize("shape", SHAPES)
def test_oaa_block_pitch_other_than_n(shape):
    """Blocks of side b != n (the larger-block tiling) reproduce the direct
    definition for every b in [max(1, n-1), L-n+1], in all three passes."""
    x, w, g = _rand(shape, 17)
    N, n = shape[3], shape[4]
    for L in (oaa.fft_size(n), 2 * oaa.fft_size(n)):
        for b in sorted({max(1, n - 1), n, n + 1, L // 2, L - n + 1}):
            if b < max(1, n - 1) or b + n - 1 > L:
                continue
            assert relerr(oaa.forward(x, w, L, b), oracle.conv_forward(x, w)) < 1e-12, (L, b)
            assert relerr(oaa.backward_data(g, w, N, L, b=b), oracle.conv_backward_data(g, w, N)) < 1e-12, (L, b)
            assert relerr(oaa.backward_filter(x, g, n, L, b=b), oracle.conv_backward_filter(x, g, n)) < 1e-12, (L, b)
            # any window side in [b+n-1, L] (the GPU path uses 2b when 2b <= L)
            if 2 * b <= L:
                assert relerr(oaa.backward_data(g, w, N, L, 2 * b, b), oracle.conv_backward_data(g, w, N)) < 1e-12


@pytest.mark.parametrize("shape", [(1, 2, 3, 12, 5), (2, 1, 2, 9, 3), (1, 3, 2, 20, 7)])
def test_oaa_single_block_is_fftconv(shape):
    """With one block per plane (b >= N) the OaA steps are the paper's FFTconv
    (Section 2): the whole plane zero-padded to L >= N + n - 1, one product of
    spectra, one inverse. Pinned against the explicit-DFT convolution at the
    same transform size."""
    B, C, K, N, n = shape
    x, w, _ = _rand(shape, 11 + sum(shape))
    L = 2
    while L < N + n - 1:
        L *= 2
    b = L - n + 1
    assert oaa.block_grid(N, b) == 1
    got = oaa.forward(x, w, L=L, b=b)
    ref = oracle.dft_conv_forward(x, w, Lc=L)
    assert np.max(np.abs(got - ref)) <= 1e-12 * np.max(np.abs(ref))


def test_oaa_tiling_rejects_overlapping_neighbours():
    x = np.zeros((1, 1, 20, 20))
    with pytest.raises(ValueError):
        oaa.block_spectra(x, 7, 16, 5)      # b < n - 1: results reach past the next block
    with pytest.raises(ValueError):
        oaa.block_spectra(x, 7, 16, 11)     # b + n - 1 > L: a block result wraps around


def test_oaa_fft_size_and_block_grid():
    assert [oaa.fft_size(n) for n in (1, 2, 3, 5, 7, 8, 9, 16, 17, 32)] == \
        [2, 4, 8, 16, 16, 16, 32, 32, 64, 64]
    assert [oaa.block_grid(N, n) for N, n in ((32, 5), (224, 3), (224, 7), (56, 3), (128, 16))] == \
        [7, 75, 32, 19, 8]
    # every power-of-two size satisfies L >= 2n, so a block fills at most half a tile
    assert all(oaa.fft_size(n) >= 2 * n for n in range(1, 33))


def test_oaa_spectra_are_explicit_dft_sums():
    rng = np.random.default_rng(15)
    x = rng.uniform(-1, 1, (1, 1, 6, 6))
    n, L = 3, 8
    Xh = oaa.block_spectra(x, n, L)            # [1,1,2,2,L,L/2+1]
    P, Q = 1, 0
    blk = x[0, 0, P * n:P * n + n, Q * n:Q * n + n]
    for u in range(L):
        for v in range(L // 2 + 1):
            ref = sum(blk[r, s] * np.exp(-2j * np.pi * (u * r + v * s) / L)
                      for r in range(n) for s in range(n))
            assert abs(Xh[0, 0, P, Q, u, v] - ref) < 1e-12


def test_half_spectrum_edge_columns_are_hermitian():
    """Why the contractions may skip bins: for real tiles, columns v = 0 and
    v = L/2 of the half spectrum satisfy X[L-u, v] = conj(X[u, v]), and so do
    the bin-wise products of such spectra summed over channels."""
    rng = np.random.default_rng(12)
    x = rng.standard_normal((2, 3, 20, 20))
    w = rng.standard_normal((4, 3, 5, 5))
    L = oaa.fft_size(5)
    Xh = oaa.block_spectra(x, 5, L)
    Yh = oaa.forward_product(Xh, oaa.filter_spectra(w, L))
    for S in (Xh, Yh):
        for v in (0, L // 2):
            col = S[..., v]
            mirrored = np.conj(col[..., (-np.arange(L)) % L])
            assert np.allclose(col, mirrored, rtol=0, atol=1e-12 * np.abs(col).max())
    # the other columns are not symmetric: the skipped set is exactly these two
    col = Xh[..., 1]
    assert not np.allclose(col, np.conj(col[..., (-np.arange(L)) % L]))


# ---------------------------------------------------------------------------
# output-tiled alternative (overlap-and-save forward)

@pytest.mark.parametrize("Lmode", ["min", "double"])
@pytest.mark.parametrize("shape", SHAPES + [(2, 3, 4, 40, 16)])
def test_oas_passes_equal_direct_definition(shape, Lmode):
    """Overlap-and-save forward over windows at hop L - n + 1, the error
    propagation as overlap-and-add over g blocks, and the weight gradient
    from windows and blocks: all equal the plain definitions."""
    x, w, g = _rand(shape, 23 + sum(shape))
    B, C, K, N, n = shape
    L = oaa.fft_size(n) * (2 if Lmode == "double" else 1)
    assert relerr(oas.forward(x, w, L), oracle.conv_forward(x, w)) <= 1e-13
    assert relerr(oas.backward_data(g, w, N, L), oracle.conv_backward_data(g, w, N)) <= 1e-13
    assert relerr(oas.backward_filter(x, g, n, L), oracle.conv_backward_filter(x, g, n)) <= 1e-13


def test_oas_window_count_tiles_the_output():
    """T = ceil(M / h) windows per side with h = L - n + 1: for the 128 x 128
    layer with 16 x 16 kernels at L = 32, 7 windows against 8 blocks."""
    assert oas.hop(16, 32) == 17 and oas.grid(113, 17) == 7 and oaa.block_grid(128, 16) == 8
    x = np.zeros((1, 1, 20, 20))
    assert oas.window_spectra(x, 5, 16).shape[2] == oas.grid(16, 12) == 2


@pytest.mark.parametrize("n,L", [(1, 2), (3, 8), (4, 8), (5, 16), (16, 32)])
def test_flipped_kernel_spectrum_is_phase_times_conjugate(n, L):
    """For a real kernel, the spectrum of w flipped in both axes (padded at
    [0, n)) is exp(-2 pi i (n-1)(u+v)/L) times the conjugate spectrum of w:
    the identity that lets the error propagation reuse the kernel spectra."""
    rng = np.random.default_rng(n + L)
    w = rng.standard_normal((2, 3, n, n))
    u = np.arange(L)[:, None]
    v = np.arange(L // 2 + 1)[None, :]
    phase = np.exp(-2j * np.pi * (n - 1) * (u + v) / L)
    got = oas.kernel_spectra(w, L, flip=True)
    ref = phase * np.conj(oas.kernel_spectra(w, L))
    assert np.max(np.abs(got - ref)) <= 1e-12 * np.max(np.abs(ref))


@pytest.mark.parametrize("shape", [(1, 3, 4, 32, 5), (2, 2, 3, 13, 4), (1, 1, 2, 10, 6), (2, 3, 2, 11, 1)])
def test_oas_weight_gradient_with_conjugated_windows(shape):
    """The same weight gradient with the conjugate on the window spectra:
    the inverse then holds dw[u][v] at rows and columns (h + u) mod L,
    (h + v) mod L (the orientation of the library's contraction)."""
    x, _, g = _rand(shape, 5 + sum(shape))
    B, C, K, N, n = shape
    L = oaa.fft_size(n)
    h = oas.hop(n, L)
    dWh = np.einsum('bkpquv,bcpquv->kcuv', oas.block_spectra(g, n, L), np.conj(oas.window_spectra(x, n, L)))
    c = np.fft.irfft2(dWh, s=(L, L))
    idx = (h + np.arange(n)) % L
    got = c[:, :, idx][:, :, :, idx]
    assert relerr(got, oracle.conv_backward_filter(x, g, n)) <= 1e-13


def test_relerr_sees_imaginary_parts():
    """The comparison used by every parity test: a conjugated or
    sign-flipped spectrum must fail it, and a complex array may not be
    compared with a real one."""
    rng = np.random.default_rng(4)
    z = rng.standard_normal((6, 5)) + 1j * rng.standard_normal((6, 5))
    assert relerr(z, z) == 0.0
    assert relerr(np.conj(z), z) > 0.1
    assert relerr(z.real - 1j * z.imag, z) > 0.1
    assert relerr(1j * z, z) > 0.1
    assert relerr(z.astype(np.complex64), z) < 1e-6
    assert relerr(np.array([1 + 1j, 2]), np.array([1 - 1j, 2])) == 1.0
    with pytest.raises(AssertionError):
        relerr(z.real, z)
    with pytest.raises(AssertionError):
        relerr(z, z.real)


@pytest.mark.parametrize("shape", [(2, 3, 4, 2, 12, 3, 4), (1, 2, 3, 5, 9, 1, 5), (1, 1, 2, 3, 10, 4, 2)])
def test_stacked_layers_are_one_layer_of_the_composed_kernel(shape):
    """Two stacked layers with nothing between them (the reading of the
    Conclusion's frequency-domain layers that the library composes):
    conv(conv(x, w1), w2) equals conv(x, w12) with w12[k][c] the sum over j
    of the full 2-D convolutions of w2[k][j] and w1[j][c] (scipy), and the
    error propagation through both equals that of w12."""
    B, C, J, K, N, n1, n2 = shape
    rng = np.random.default_rng(sum(shape))
    x = rng.uniform(-1, 1, (B, C, N, N))
    w1 = rng.standard_normal((J, C, n1, n1))
    w2 = rng.standard_normal((K, J, n2, n2))
    n = n1 + n2 - 1
    w12 = np.zeros((K, C, n, n))
    for k in range(K):
        for c in range(C):
            for j in range(J):
                w12[k, c] += scipy.signal.convolve2d(w2[k, j], w1[j, c], mode="full")
    y = oracle.conv_forward(oracle.conv_forward(x, w1), w2)
    assert relerr(y, oracle.conv_forward(x, w12)) < 1e-12
    g = rng.uniform(-1, 1, y.shape)
    N1 = N - n1 + 1
    dx = oracle.conv_backward_data(oracle.conv_backward_data(g, w2, N1), w1, N)
    assert relerr(dx, oracle.conv_backward_data(g, w12, N)) < 1e-12
