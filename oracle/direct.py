"""Direct spatial-domain convolution layer in float64 (test infrastructure).

TEST INFRASTRUCTURE ONLY: the product path never imports this module.

Problem statement (arXiv:1601.06815, Introduction and Section 3.2): an input
of C channels, each N x N, and K kernels of C channels, each n x n. Each
channel of each kernel is convolved with the matching input channel and the
C results are summed, giving K output maps; the layer performs K*C 2-D
convolutions. The paper says "convolved" and builds on the convolution
theorem, so the operation is a true convolution (kernel flipped). Only the
positions where the kernel lies fully inside the input are kept ("valid"),
stride 1, giving M = N - n + 1 output pixels per side:

    y[b,k,i,j] = sum_c sum_{u,v<n} w[k,c,u,v] * x[b,c, i+n-1-u, j+n-1-v]

Section 3.2 says the backward pass holds two convolutions per kernel: one
propagates the error through the layer, one forms the change in the weights.
For an upstream gradient g = dL/dy these are the exact derivatives of
<y(x, w), g>:

    dx[b,c,p,q] = sum_k sum_{u,v<n} w[k,c,u,v] * g[b,k, p-n+1+u, q-n+1+v]
                  (g read as 0 outside [0, M)^2: a "full" correlation)
    dw[k,c,u,v] = sum_b sum_{i,j<M} g[b,k,i,j] * x[b,c, i+n-1-u, j+n-1-v]

Evaluation: n^2 shifted slices, each contracted over the channel axis with
numpy.tensordot (a plain matrix product). No transform, no blocking.
Arrays are NCHW; inputs are converted to float64 before any arithmetic.
"""

import numpy as np


def _dims(x, w):
    if x.ndim != 4 or w.ndim != 4:
        raise ValueError("x must be [B,C,N,N] and w [K,C,n,n]")
    B, C, N, N2 = x.shape
    K, C2, n, n2 = w.shape
    if N != N2 or n != n2 or C != C2 or n < 1 or n > N:
        raise ValueError(f"bad shapes x{x.shape} w{w.shape}")
    return B, C, N, K, n, N - n + 1


def conv_forward(x, w):
    """Valid-mode true 2-D convolution layer (Introduction; Section 2 Table 1
    "spaceConv"). x[B,C,N,N], w[K,C,n,n] -> y[B,K,M,M], float64."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    B, C, N, K, n, M = _dims(x, w)
    acc = np.zeros((B, M, M, K))
    for u in range(n):
        for v in range(n):
            xs = x[:, :, n - 1 - u:n - 1 - u + M, n - 1 - v:n - 1 - v + M]  # [B,C,M,M]
            acc += np.tensordot(xs, w[:, :, u, v], axes=([1], [1]))       # [B,M,M,K]
    return np.ascontiguousarray(acc.transpose(0, 3, 1, 2))


def conv_backward_data(g, w, N):
    """Error propagation through the layer (Section 3.2, first of the two
    backward convolutions): dx = d<y, g>/dx. g[B,K,M,M], w[K,C,n,n] ->
    dx[B,C,N,N], float64."""
    g = np.asarray(g, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    K, C, n, _ = w.shape
    B, K2, M, M2 = g.shape
    if K2 != K or M != M2 or M != N - n + 1:
        raise ValueError(f"bad shapes g{g.shape} w{w.shape} N={N}")
    # g placed in a zero frame of width n-1, so gp[b,k,a,c] = g[b,k,a-n+1,c-n+1]
    gp = np.zeros((B, K, M + 2 * (n - 1), M + 2 * (n - 1)))
    gp[:, :, n - 1:n - 1 + M, n - 1:n - 1 + M] = g
    acc = np.zeros((B, N, N, C))
    for u in range(n):
        for v in range(n):
            gs = gp[:, :, u:u + N, v:v + N]                                # g[b,k,p-n+1+u, q-n+1+v]
            acc += np.tensordot(gs, w[:, :, u, v], axes=([1], [0]))       # [B,N,N,C]
    return np.ascontiguousarray(acc.transpose(0, 3, 1, 2))


def conv_backward_filter(x, g, n):
    """Weight gradient (Section 3.2, second backward convolution):
    dw = d<y, g>/dw. x[B,C,N,N], g[B,K,M,M] -> dw[K,C,n,n], float64."""
    x = np.asarray(x, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    B, C, N, _ = x.shape
    B2, K, M, _ = g.shape
    if B2 != B or M != N - n + 1:
        raise ValueError(f"bad shapes x{x.shape} g{g.shape} n={n}")
    dw = np.zeros((K, C, n, n))
    for u in range(n):
        for v in range(n):
            xs = x[:, :, n - 1 - u:n - 1 - u + M, n - 1 - v:n - 1 - v + M]  # [B,C,M,M]
            dw[:, :, u, v] = np.tensordot(g, xs, axes=([0, 2, 3], [0, 2, 3]))
    return dw


# ---------------------------------------------------------------------------
# Single-element evaluation of the same three definitions, for checking
# sampled outputs of layers too large to evaluate whole on the CPU.
# Index arguments are equal-length integer sequences.

def conv_forward_at(x, w, b, k, i, j):
    """y[b,k,i,j] of ``conv_forward`` at the given index lists."""
    n = w.shape[-1]
    out = np.empty(len(b))
    for t, (bb, kk, ii, jj) in enumerate(zip(b, k, i, j)):
        win = np.asarray(x[bb, :, ii:ii + n, jj:jj + n], dtype=np.float64)[:, ::-1, ::-1]
        out[t] = np.sum(win * np.asarray(w[kk], dtype=np.float64))
    return out


def conv_backward_data_at(g, w, N, b, c, p, q):
    """dx[b,c,p,q] of ``conv_backward_data`` at the given index lists."""
    K, C, n, _ = w.shape
    M = g.shape[-1]
    out = np.empty(len(b))
    for t, (bb, cc, pp, qq) in enumerate(zip(b, c, p, q)):
        acc = 0.0
        for u in range(n):
            a = pp - n + 1 + u
            if a < 0 or a >= M:
                continue
            for v in range(n):
                d = qq - n + 1 + v
                if d < 0 or d >= M:
                    continue
                acc += float(np.dot(np.asarray(w[:, cc, u, v], dtype=np.float64),
                                    np.asarray(g[bb, :, a, d], dtype=np.float64)))
        out[t] = acc
    return out


def conv_backward_filter_at(x, g, n, k, c, u, v):
    """dw[k,c,u,v] of ``conv_backward_filter`` at the given index lists."""
    M = g.shape[-1]
    out = np.empty(len(k))
    for t, (kk, cc, uu, vv) in enumerate(zip(k, c, u, v)):
        xs = np.asarray(x[:, cc, n - 1 - uu:n - 1 - uu + M, n - 1 - vv:n - 1 - vv + M], dtype=np.float64)
        out[t] = float(np.sum(xs * np.asarray(g[:, kk], dtype=np.float64)))
    return out
