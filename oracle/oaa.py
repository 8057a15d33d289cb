"""The overlap-and-add convolution of arXiv:1601.06815, Section 2, in float64
(test infrastructure).

TEST INFRASTRUCTURE ONLY: the product path never imports this module.

Steps, in the paper's order (Section 2 and the zero-padding remarks of
Sections 3.2 and 3.3):

1. Divide each N x N input plane into blocks the size of the kernel, n x n;
   there are ceil(N/n) blocks per side (the paper's N^2/n^2 "rounded up",
   read per side), the last row and column of blocks being zero-filled
   beyond N.
2. Zero-pad every block and every kernel plane to L x L. The paper pads to
   2n-1 per side and suggests rounding up to a power of two for the FFT;
   L = max(2, smallest power of two >= 2n-1) by default. Any L >= 2n-1
   gives the same result.
3. Fourier-transform blocks and kernels (numpy.fft.rfft2: Hermitian
   half-spectrum, L x (L/2+1) bins).
4. Hadamard product of block and kernel spectra, summed over the C channels
   (the layer's K*C convolutions, Introduction).
5. Inverse transform; each block result has support (2n-1) x (2n-1).
6. Overlap the block results by n-1 and add them: block (P, Q) lands at
   (P*n, Q*n) of the full (T*n + n - 1)^2 result.
7. Keep the valid region: rows and columns [n-1, N).

The block pitch b (the block side) is the kernel side n in the paper. Any
b >= n - 1 with b + n - 1 <= L gives the same result: block results then
overlap only their immediate neighbours. The functions below take b as an
option (default n).

The two backward convolutions of Section 3.2 are written as the exact
adjoints of steps 1-7 (the paper gives no formula for them; this is the
reading taken): the upstream gradient g is placed at offset (n-1, n-1) in
zeros (adjoint of step 7), cut into (2n-1) x (2n-1) windows that start at
(P*n, Q*n) and overlap by n-1 (adjoint of step 6), zero-padded to L and
transformed; then

    error propagation:  dX_hat[b,c,P,Q] = sum_k G_hat[b,k,P,Q] * conj(W_hat[k,c])
                        dx block (P,Q) = irfft2(dX_hat)[0:n, 0:n]
    weight gradient:    dW_hat[k,c] = sum_{b,P,Q} G_hat[b,k,P,Q] * conj(X_hat[b,c,P,Q])
                        dw[k,c] = irfft2(dW_hat)[0:n, 0:n]

With L >= 2n-1 the circular correlations involved equal the linear ones on
[0, n), so the results equal the direct definition exactly (up to rounding).

Spectra are returned in this module's own natural layout:
    block spectra   [B, C, T, T, L, L//2+1]   (bin (u, v) = row u, column v)
    kernel spectra  [K, C, L, L//2+1]
    window spectra  [B, K, T, T, L, L//2+1]
"""

import numpy as np


def fft_size(n):
    """Smallest power of two >= 2n-1, at least 2 (Sections 3.2 and 3.3)."""
    L = 2
    while L < 2 * n - 1:
        L *= 2
    return L


def block_grid(N, b):
    """Blocks per side, ceil(N/b) (Section 2, with b = n there)."""
    return -(-N // b)


def check_tiling(n, L, b):
    """Block pitch b and transform side L that reproduce the convolution:
    every block result (support b + n - 1) fits the tile and overlaps only
    its immediate neighbours."""
    if b < max(1, n - 1) or b + n - 1 > L:
        raise ValueError(f"block pitch b={b} needs max(1, n-1) <= b and b + n - 1 <= L (n={n}, L={L})")


def block_spectra(x, n, L=None, b=None):
    """Steps 1-3 on the input: x[B,C,N,N] -> X_hat[B,C,T,T,L,L//2+1], blocks
    of b x b (default n x n)."""
    x = np.asarray(x, dtype=np.float64)
    B, C, N, _ = x.shape
    L = fft_size(n) if L is None else L
    b = n if b is None else b
    check_tiling(n, L, b)
    T = block_grid(N, b)
    xz = np.zeros((B, C, T * b, T * b))
    xz[:, :, :N, :N] = x
    blocks = xz.reshape(B, C, T, b, T, b).transpose(0, 1, 2, 4, 3, 5)   # [B,C,T,T,b,b]
    tiles = np.zeros((B, C, T, T, L, L))
    tiles[..., :b, :b] = blocks
    return np.fft.rfft2(tiles)


def filter_spectra(w, L=None):
    """Steps 2-3 on the kernels: w[K,C,n,n] -> W_hat[K,C,L,L//2+1]."""
    w = np.asarray(w, dtype=np.float64)
    K, C, n, _ = w.shape
    L = fft_size(n) if L is None else L
    tiles = np.zeros((K, C, L, L))
    tiles[:, :, :n, :n] = w
    return np.fft.rfft2(tiles)


def window_spectra(g, n, N, L=None, side=None, b=None):
    """Adjoint of steps 6-7, then 2-3, on the upstream gradient:
    g[B,K,M,M] -> G_hat[B,K,T,T,L,L//2+1]. Windows start every b (default n)
    and are side x side (default b+n-1, for b = n the padded size 2n-1 of
    Section 3.2; any side in [b+n-1, L] gives the same backward results,
    since rows and columns past b+n-2 only meet kernel taps beyond n)."""
    g = np.asarray(g, dtype=np.float64)
    B, K, M, _ = g.shape
    L = fft_size(n) if L is None else L
    b = n if b is None else b
    check_tiling(n, L, b)
    side = b + n - 1 if side is None else side
    if not b + n - 1 <= side <= L:
        raise ValueError("window side must lie in [b+n-1, L]")
    T = block_grid(N, b)
    S = T * b + side
    gfull = np.zeros((B, K, S, S))
    gfull[:, :, n - 1:n - 1 + M, n - 1:n - 1 + M] = g
    tiles = np.zeros((B, K, T, T, L, L))
    for P in range(T):
        for Q in range(T):
            tiles[:, :, P, Q, :side, :side] = gfull[:, :, P * b:P * b + side, Q * b:Q * b + side]
    return np.fft.rfft2(tiles)


def forward_product(Xh, Wh):
    """Step 4: Y_hat[b,k,P,Q] = sum_c X_hat[b,c,P,Q] * W_hat[k,c]."""
    return np.einsum('bcpquv,kcuv->bkpquv', Xh, Wh)


def backward_data_product(Gh, Wh):
    """dX_hat[b,c,P,Q] = sum_k G_hat[b,k,P,Q] * conj(W_hat[k,c])."""
    return np.einsum('bkpquv,kcuv->bcpquv', Gh, np.conj(Wh))


def backward_filter_product(Gh, Xh):
    """dW_hat[k,c] = sum_{b,P,Q} G_hat[b,k,P,Q] * conj(X_hat[b,c,P,Q])."""
    return np.einsum('bkpquv,bcpquv->kcuv', Gh, np.conj(Xh))


def overlap_add(Yh, n, N, L, b=None):
    """Steps 5-7: inverse transform, overlap by n-1 and add, valid crop.
    Y_hat[B,K,T,T,L,L//2+1] -> y[B,K,M,M]; blocks b apart (default n)."""
    b = n if b is None else b
    B, K, T, _, _, _ = Yh.shape
    R = b + n - 1                      # support of a block result
    t = np.fft.irfft2(Yh, s=(L, L))[..., :R, :R]
    S = T * b + n - 1
    yfull = np.zeros((B, K, S, S))
    for P in range(T):
        for Q in range(T):
            yfull[:, :, P * b:P * b + R, Q * b:Q * b + R] += t[:, :, P, Q]
    M = N - n + 1
    return yfull[:, :, n - 1:n - 1 + M, n - 1:n - 1 + M]


def forward(x, w, L=None, b=None):
    """OaA forward convolution layer, steps 1-7."""
    n = np.asarray(w).shape[-1]
    N = np.asarray(x).shape[-1]
    L = fft_size(n) if L is None else L
    return overlap_add(forward_product(block_spectra(x, n, L, b), filter_spectra(w, L)), n, N, L, b)


def backward_data(g, w, N, L=None, side=None, b=None):
    """OaA error propagation: window spectra times conj(kernel spectra), summed
    over K, inverse, top-left b x b of each tile placed at its block."""
    w = np.asarray(w, dtype=np.float64)
    K, C, n, _ = w.shape
    L = fft_size(n) if L is None else L
    b = n if b is None else b
    dXh = backward_data_product(window_spectra(g, n, N, L, side, b), filter_spectra(w, L))
    blk = np.fft.irfft2(dXh, s=(L, L))[..., :b, :b]                     # [B,C,T,T,b,b]
    B, _, T, _, _, _ = blk.shape
    dx = blk.transpose(0, 1, 2, 4, 3, 5).reshape(B, C, T * b, T * b)
    return np.ascontiguousarray(dx[:, :, :N, :N])


def backward_filter(x, g, n, L=None, side=None, b=None):
    """OaA weight gradient: window spectra times conj(block spectra), summed
    over the batch and all blocks, inverse, top-left n x n."""
    N = np.asarray(x).shape[-1]
    L = fft_size(n) if L is None else L
    dWh = backward_filter_product(window_spectra(g, n, N, L, side, b), block_spectra(x, n, L, b))
    return np.ascontiguousarray(np.fft.irfft2(dWh, s=(L, L))[..., :n, :n])
