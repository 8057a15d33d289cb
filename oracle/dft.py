"""Convolution through explicit discrete Fourier matrices, float64 (test
infrastructure).

TEST INFRASTRUCTURE ONLY: the product path never imports this module.

The Introduction of arXiv:1601.06815 recalls that a convolution is a
Hadamard product in the frequency domain. Written as a definition, with no
fast transform and no blocking: every channel plane and every kernel plane is
zero-padded to Lc x Lc with Lc >= N + n - 1 (so the circular convolution of
the padded arrays equals the linear one), multiplied by the DFT matrix
Fm[a, b] = exp(-2 pi i a b / Lc) on both sides, the K x C products are
summed over C, the inverse DFT matrix is applied, and the valid region
[n-1, N) x [n-1, N) of the full linear convolution is kept. This is the
paper's "FFTconv" (Section 2, Table 1) evaluated literally, O(Lc^3) per
plane; it exists only to pin ``direct.conv_forward`` on tiny inputs through a
route that shares nothing with it.
"""

import numpy as np


def _dft_matrix(Lc):
    a = np.arange(Lc)
    return np.exp(-2j * np.pi * np.outer(a, a) / Lc)


def dft_conv_forward(x, w, Lc=None):
    """Valid-mode convolution layer via the convolution theorem with explicit
    DFT matrices. x[B,C,N,N], w[K,C,n,n] -> y[B,K,N-n+1,N-n+1] float64."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    B, C, N, _ = x.shape
    K, _, n, _ = w.shape
    if Lc is None:
        Lc = N + n - 1
    if Lc < N + n - 1:
        raise ValueError("Lc must be at least N + n - 1 for a linear convolution")
    Fm = _dft_matrix(Lc)
    Fi = np.conj(Fm) / Lc
    xp = np.zeros((B, C, Lc, Lc))
    xp[:, :, :N, :N] = x
    wp = np.zeros((K, C, Lc, Lc))
    wp[:, :, :n, :n] = w
    X = Fm @ xp @ Fm.T                     # [B,C,Lc,Lc]
    W = Fm @ wp @ Fm.T                     # [K,C,Lc,Lc]
    Y = np.einsum('bcuv,kcuv->bkuv', X, W)  # Hadamard product, summed over channels
    yfull = (Fi @ Y @ Fi.T).real
    M = N - n + 1
    return np.ascontiguousarray(yfull[:, :, n - 1:n - 1 + M, n - 1:n - 1 + M])
