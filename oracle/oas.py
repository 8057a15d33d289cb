"""Overlap-and-save forward convolution and the output-tiled backward passes,
float64 (test infrastructure).

TEST INFRASTRUCTURE ONLY: the product path never imports this module.

arXiv:1601.06815 names overlap-and-save as the alternative block method
(Introduction; Section 2 uses the name once, for its own method): the input
is read in overlapping windows, each window is convolved circularly with the
zero-padded kernel, and only the part of each circular result that does not
wrap around is kept. Here every pass is tiled by the output side M = N - n + 1
with hop h = L - n + 1, the most outputs one L x L transform can give:

Forward (overlap-and-save). Window (P, Q) of a plane is x[P h + r][Q h + s],
r, s < L (zero beyond N). Its circular convolution with w (zero-padded to L)
equals the linear one on rows and columns [n - 1, L), which are the outputs
y[P h + i][Q h + j], i, j < h. T = ceil(M / h) windows per side.

Error propagation (overlap-and-add over its own input). The error
propagation is the full convolution of g with the flipped kernel
w_f[u][v] = w[n-1-u][n-1-v] (output side M + n - 1 = N). Following
Section 2 on that convolution: g is cut into h x h blocks, each block is
convolved with w_f (support h + n - 1 = L, so the circular convolution at
side L is the linear one), and the block results, h apart, are added.

Weight gradient. dw[u][v] = sum over the batch and the blocks of the
correlation of the g block with the x window at the same origin, at shift
(n-1-u, n-1-v): every index stays inside the window, so the circular
correlation of the padded block with the window is exact there.
"""

import numpy as np

from .oaa import fft_size


def hop(n, L):
    """Outputs per window side: L - n + 1."""
    return L - n + 1


def grid(M, h):
    """Windows (or blocks) per side, ceil(M / h)."""
    return -(-M // h)


def _L(n, L):
    return fft_size(n) if L is None else L


def window_spectra(x, n, L=None):
    """x[B,C,N,N] -> spectra of the L x L windows at hop h:
    [B,C,T,T,L,L//2+1], T = ceil(M/h)."""
    x = np.asarray(x, dtype=np.float64)
    B, C, N, _ = x.shape
    L = _L(n, L)
    h = hop(n, L)
    T = grid(N - n + 1, h)
    S = (T - 1) * h + L
    xz = np.zeros((B, C, max(S, N), max(S, N)))
    xz[:, :, :N, :N] = x
    tiles = np.zeros((B, C, T, T, L, L))
    for P in range(T):
        for Q in range(T):
            tiles[:, :, P, Q] = xz[:, :, P * h:P * h + L, Q * h:Q * h + L]
    return np.fft.rfft2(tiles)


def block_spectra(g, n, L=None):
    """g[B,K,M,M] -> spectra of its h x h blocks zero-padded to L:
    [B,K,T,T,L,L//2+1]."""
    g = np.asarray(g, dtype=np.float64)
    B, K, M, _ = g.shape
    L = _L(n, L)
    h = hop(n, L)
    T = grid(M, h)
    gz = np.zeros((B, K, T * h, T * h))
    gz[:, :, :M, :M] = g
    tiles = np.zeros((B, K, T, T, L, L))
    tiles[..., :h, :h] = gz.reshape(B, K, T, h, T, h).transpose(0, 1, 2, 4, 3, 5)
    return np.fft.rfft2(tiles)


def kernel_spectra(w, L=None, flip=False):
    """w[K,C,n,n] (flipped in both axes if `flip`) zero-padded to L,
    transformed: [K,C,L,L//2+1]."""
    w = np.asarray(w, dtype=np.float64)
    K, C, n, _ = w.shape
    L = _L(n, L)
    tiles = np.zeros((K, C, L, L))
    tiles[:, :, :n, :n] = w[:, :, ::-1, ::-1] if flip else w
    return np.fft.rfft2(tiles)


def forward(x, w, L=None):
    """Overlap-and-save forward: window spectra times kernel spectra summed
    over C, inverse, rows and columns [n-1, L) of each window placed at
    (P h, Q h), valid region [0, M)."""
    w = np.asarray(w, dtype=np.float64)
    K, C, n, _ = w.shape
    N = np.asarray(x).shape[-1]
    L = _L(n, L)
    h = hop(n, L)
    Yh = np.einsum('bcpquv,kcuv->bkpquv', window_spectra(x, n, L), kernel_spectra(w, L))
    t = np.fft.irfft2(Yh, s=(L, L))[..., n - 1:, n - 1:]          # [B,K,T,T,h,h]
    B, _, T, _, _, _ = t.shape
    y = t.transpose(0, 1, 2, 4, 3, 5).reshape(B, K, T * h, T * h)
    M = N - n + 1
    return np.ascontiguousarray(y[:, :, :M, :M])


def backward_data(g, w, N, L=None):
    """Error propagation as overlap-and-add over g: block spectra times the
    flipped kernel's spectra summed over K, inverse (support L), block
    results h apart added, first N rows and columns."""
    w = np.asarray(w, dtype=np.float64)
    K, C, n, _ = w.shape
    L = _L(n, L)
    h = hop(n, L)
    dXh = np.einsum('bkpquv,kcuv->bcpquv', block_spectra(g, n, L), kernel_spectra(w, L, flip=True))
    t = np.fft.irfft2(dXh, s=(L, L))                              # [B,C,T,T,L,L]
    B, _, T, _, _, _ = t.shape
    S = (T - 1) * h + L
    dx = np.zeros((B, C, max(S, N), max(S, N)))
    for P in range(T):
        for Q in range(T):
            dx[:, :, P * h:P * h + L, Q * h:Q * h + L] += t[:, :, P, Q]
    return np.ascontiguousarray(dx[:, :, :N, :N])


def backward_filter(x, g, n, L=None):
    """Weight gradient: conj(block spectra of g) times window spectra of x,
    summed over the batch and the blocks, inverse; dw[u][v] is the result at
    (n-1-u, n-1-v)."""
    L = _L(n, L)
    dWh = np.einsum('bkpquv,bcpquv->kcuv', np.conj(block_spectra(g, n, L)), window_spectra(x, n, L))
    c = np.fft.irfft2(dWh, s=(L, L))[..., :n, :n]
    return np.ascontiguousarray(c[..., ::-1, ::-1])
