"""The paper's timing sweeps (arXiv:1601.06815, Section 3) as synthetic
benchmarks of this library on one GPU.

Section 3.2 varies the number of kernels for a 32 x 32 one-channel input and
5 x 5 kernels, forward and backward; Section 3.3 varies the kernel side for a
64 x 64 input and 100 kernels; Section 3.4 varies the input side (4 to 256) for
5 x 5 kernels. The paper plots speed-ups over its own spatial implementation,
which is not part of this library; this module reports the time of each pass
and the direct-convolution-equivalent rate, the shape of those curves.

Kernel sides 33 to 64 run at transform side 128. The number of kernels of
the input-size sweep is not stated and is taken as 100.

--tiling fftconv runs the paper's FFTconv baseline (Section 2): the whole
plane as a single block, zero-padded to L >= N + n - 1, which the library
expresses as the tiling (L, L - n + 1) with one block per plane. Planes that
would need L > 128 are skipped.

    python -m paper_1601_06815_amd.sweeps [--sweep kernels|ksize|input|all] [--tiling paper|auto|fftconv]
                                          [--out FILE]

prints one JSON line per configuration (and with --out also writes them to
FILE, after a line giving the command).
"""

import argparse
import json
import sys

from paper_1601_06815_amd import binding
from paper_1601_06815_amd.workloads import Layer, make_inputs


def sweep_configs(which):
    """(name, B, C, K, N, n) in the order the paper sweeps them."""
    out = []
    if which in ("kernels", "all"):     # Section 3.2: 32 x 32 input, 5 x 5 kernels
        out += [("kernels", 1, 1, K, 32, 5) for K in (25, 50, 100, 200, 300, 400, 500, 600, 750)]
    if which in ("ksize", "all"):       # Section 3.3: 64 x 64 input, 100 kernels
        out += [("ksize", 1, 1, 100, 64, n) for n in range(1, 65)]
    if which in ("input", "all"):       # Section 3.4: 5 x 5 kernels, sides 4 .. 256
        out += [("input", 1, 1, 100, N, 5) for N in range(8, 257, 8)]
    return out


def fftconv_tiling(N, n):
    """(L, b) of a single block covering the N x N plane, or None if the
    linear convolution needs a transform longer than 128."""
    L = 2
    while L < N + n - 1:
        L *= 2
    return (L, L - n + 1) if L <= 128 else None


def time_layer(torch, B, C, K, N, n, tiling, reps):
    """Mean time (ms) of each pass over `reps` repetitions after a warm-up,
    from events on the current stream."""
    ly = Layer("sweep", B, C, K, N, n)
    x, w, g = make_inputs(ly, seed=0)
    dev = torch.device("cuda:0")
    xd, wd, gd = (torch.from_numpy(a).to(dev) for a in (x, w, g))
    plan = binding.Plan(B, C, K, N, n, device=dev, tiling=tiling)
    y = torch.empty((B, K, ly.M, ly.M), device=dev)
    dx, dw = torch.empty_like(xd), torch.empty_like(wd)

    def fwd():
        plan.forward(xd, wd, y)

    def bwd():
        plan.backward_data(gd, None, dx)
        plan.backward_filter(None, None if plan.caches_grad_spectra else gd, dw)

    res = {}
    for name, fn in (("fwd", fwd), ("bwd", bwd)):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        res[name] = e0.elapsed_time(e1) / reps
    return res, plan.geometry, ly


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--sweep", default="all", choices=["kernels", "ksize", "input", "all"])
    ap.add_argument("--tiling", default="paper", choices=["paper", "auto", "fftconv"])
    ap.add_argument("--reps", type=int, default=20)
    ap.add_argument("--out", default=None, help="also write the lines here")
    args = ap.parse_args(argv)
    import torch
    out = None
    if args.out:
        out = open(args.out, "w")
        out.write("command: python -m paper_1601_06815_amd.sweeps " + " ".join(sys.argv[1:] if argv is None else argv)
                  + "\n")
    for name, B, C, K, N, n in sweep_configs(args.sweep):
        tiling = args.tiling
        if tiling == "fftconv":
            tiling = fftconv_tiling(N, n)
            if tiling is None:
                continue
        t, geo, ly = time_layer(torch, B, C, K, N, n, tiling, args.reps)
        direct = ly.direct_flops()
        line = json.dumps({"sweep": name, "B": B, "C": C, "K": K, "N": N, "n": n, "L": geo["L"], "b": geo["b"],
                           "fwd_ms": round(t["fwd"], 4), "bwd_ms": round(t["bwd"], 4),
                           "fwd_direct_tflops": round(direct / t["fwd"] * 1e-9, 4),
                           "bwd_direct_tflops": round(2 * direct / t["bwd"] * 1e-9, 4)})
        print(line, flush=True)
        if out:
            out.write(line + "\n")
            out.flush()
    if out:
        out.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
