"""Host-side checks of the C ABI (no GPU needed).

The library is loaded (it is built first if absent), every function that
include/oaa.h declares must be exported, and plan creation, geometry,
workspace layout and argument validation are exercised. Only calls that fail
validation before any launch are made here, so no device is touched.
"""

import ctypes
import os
import re

import numpy as np

import pytest

from paper_1601_06815_amd import binding, build
from paper_1601_06815_amd.workloads import LAYERS

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "oaa.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(build.LIB_PATH):
        build.build()
    return binding.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(oaa_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert len(names) >= 12
    for name in names:
        assert hasattr(lib, name), f"{name} declared in oaa.h but not exported"
    assert set(names) == set(binding.SIGNATURES), "binding and header disagree"


def test_status_strings(lib):
    for code, name in binding.STATUS.items():
        assert binding.oaa_status_string(code) == name
    assert binding.oaa_status_string(99) == "OAA_ERR_UNKNOWN"


@pytest.mark.parametrize("name,expect", [
    ("tiny", dict(M=28, T=7, P=49, L=16, F=144)),
    ("plane224_n3", dict(M=222, T=75, P=5625, L=8, F=40)),
    ("plane224_n5", dict(M=220, T=45, P=2025, L=16, F=144)),
    ("plane224_n8", dict(M=217, T=28, P=784, L=16, F=144)),
    ("first224", dict(M=218, T=32, P=1024, L=16, F=144)),
    ("mid56", dict(M=54, T=19, P=361, L=8, F=40)),
    ("large128", dict(M=113, T=8, P=64, L=32, F=544)),
])
def test_geometry_of_named_layers(lib, name, expect):
    ly = LAYERS[name]
    h = binding.oaa_plan_create(ly.B, ly.C, ly.K, ly.N, ly.n)
    try:
        g = binding.oaa_plan_geometry(h)
        for k, v in expect.items():
            assert g[k] == v, (k, g[k], v)
        BP = ly.B * g["P"]
        F = g["F"]
        sizes = {}
        offs = []
        for r, elems in [(binding.REGION_W_SPECTRUM, F * ly.C * ly.K),
                         (binding.REGION_X_SPECTRUM, F * ly.C * BP),
                         (binding.REGION_G_SPECTRUM, F * ly.K * BP)]:
            off, size = binding.oaa_plan_region(h, r)
            assert size == 8 * elems and off % 256 == 0
            sizes[r] = size
            offs.append((off, size))
        off, size = binding.oaa_plan_region(h, binding.REGION_PRODUCT)
        assert size == 8 * max(F * ly.K * BP, F * ly.C * BP, g["split"] * F * ly.C * ly.K)
        offs.append((off, size))
        offs.sort()
        for (o1, s1), (o2, _) in zip(offs, offs[1:]):
            assert o1 + s1 <= o2, "regions overlap"
        assert offs[-1][0] + offs[-1][1] <= binding.oaa_plan_workspace_bytes(h)
        assert g["split"] >= 1
        assert g["b"] == ly.n          # the paper's tiling: blocks of the kernel's size
    finally:
        binding.oaa_plan_destroy(h)


@pytest.mark.parametrize("name,L,b", [("tiny", 16, 12), ("mid56", 16, 14), ("first224", 64, 58), ("large128", 64, 49)])
def test_library_tiling_choice(lib, name, L, b):
    """L = b = 0: fewer, larger blocks where that cuts the estimated work."""
    ly = LAYERS[name]
    h = binding.oaa_plan_create_tiled(ly.B, ly.C, ly.K, ly.N, ly.n, 0, 0)
    try:
        g = binding.oaa_plan_geometry(h)
        assert (g["L"], g["b"]) == (L, b)
        assert g["T"] == -(-ly.N // b) and g["P"] == g["T"] ** 2 and g["F"] == L * (L // 2 + 1)
    finally:
        binding.oaa_plan_destroy(h)


@pytest.mark.parametrize("dims,status", [
    ((1, 1, 1, 20, 5, 16, 8), 0), ((1, 1, 1, 20, 5, 16, 4), 0), ((1, 1, 1, 20, 5, 16, 3), 1),   # b < n-1
    ((1, 1, 1, 20, 5, 16, 12), 0), ((1, 1, 1, 20, 5, 16, 13), 1),                                # b > L-n+1
    ((1, 1, 1, 20, 5, 12, 6), 2), ((1, 1, 1, 20, 5, 256, 8), 2), ((1, 1, 1, 20, 5, 128, 8), 0),
    ((1, 1, 1, 20, 1, 4, 4), 0),
    ((1, 1, 1, 20, 5, 16, 0), 1), ((1, 1, 1, 20, 5, 0, 8), 1), ((1, 1, 1, 20, 1, 2, 1), 0),
    ((1, 1, 1, 20, 5, 0, 0), 0), ((1, 1, 1, 20, 5, -2, 4), 1),
])
def test_tiled_plan_validation(lib, dims, status):
    h = ctypes.c_void_p(12345)
    st = lib.oaa_plan_create_tiled(ctypes.byref(h), *dims)
    assert st == status, (dims, st, binding.oaa_last_error_detail())
    if status == 0:
        g = binding.oaa_plan_geometry(h.value)
        if dims[5]:
            assert (g["L"], g["b"]) == dims[5:]
        lib.oaa_plan_destroy(h)
    else:
        assert h.value is None


@pytest.mark.parametrize("dims,status", [
    ((0, 1, 1, 8, 3), 1), ((1, 0, 1, 8, 3), 1), ((1, 1, 0, 8, 3), 1), ((1, 1, 1, 0, 1), 1),
    ((1, 1, 1, 8, 0), 1), ((1, 1, 1, 4, 5), 1), ((1, 1, 1, 64, 33), 0), ((1, 1, 1, 64, 64), 0),
    ((1, 1, 1, 80, 65), 2), ((1, 1, 1, 64, 32), 0),
    ((1, 1, 1, 1, 1), 0), ((1 << 20, 1, 1, 4096, 2), 2),
])
def test_plan_create_validation(lib, dims, status):
    h = ctypes.c_void_p(12345)
    st = lib.oaa_plan_create(ctypes.byref(h), *dims)
    assert st == status, (dims, st, binding.oaa_last_error_detail())
    if status == 0:
        assert h.value
        lib.oaa_plan_destroy(h)
    else:
        assert h.value is None
        assert binding.oaa_last_error_detail()


def test_null_and_workspace_validation(lib):
    assert lib.oaa_plan_create(None, 1, 1, 1, 8, 3) == 1
    assert lib.oaa_plan_destroy(None) == 0
    assert lib.oaa_plan_workspace_bytes(None) == 0
    assert lib.oaa_conv_forward(None, 256, 256, 256, None) == 1
    h = binding.oaa_plan_create(2, 3, 4, 16, 5)
    try:
        fake = 1 << 40   # never dereferenced: every call below fails validation first
        assert lib.oaa_conv_forward(h, fake, fake, fake, None) == 3        # no workspace
        assert lib.oaa_conv_backward_data(h, fake, fake, fake, None) == 3
        assert lib.oaa_conv_backward_filter(h, fake, fake, fake, None) == 3
        need = binding.oaa_plan_workspace_bytes(h)
        assert lib.oaa_plan_bind_workspace(h, fake, need - 1) == 3        # too small
        assert lib.oaa_plan_bind_workspace(h, fake + 8, need) == 1        # misaligned
        assert lib.oaa_plan_bind_workspace(h, None, need) == 1
        assert lib.oaa_plan_bind_workspace(h, fake, need) == 0
        assert lib.oaa_conv_forward(h, None, fake, fake, None) == 1       # x NULL
        assert lib.oaa_conv_forward(h, fake, fake, None, None) == 1       # y NULL
        assert lib.oaa_conv_forward(h, fake, None, fake, None) == 4       # no cached kernel spectra
        assert lib.oaa_conv_backward_data(h, fake, None, fake, None) == 4
        assert lib.oaa_conv_backward_data(h, None, fake, fake, None) == 1
        assert lib.oaa_conv_backward_filter(h, None, fake, fake, None) == 4   # no cached block spectra
        assert lib.oaa_conv_backward_filter(h, fake, None, fake, None) == 4   # no cached window spectra
        assert lib.oaa_conv_backward_filter(h, fake, fake, None, None) == 1
        assert lib.oaa_plan_set_contraction(h, 7) == 1
        assert lib.oaa_plan_set_contraction(h, 4) == 2                    # fused: needs L = 64
        assert lib.oaa_plan_set_contraction(h, 3) == 0                    # streaming: C = 3 <= 4
        assert lib.oaa_plan_set_contraction(h, 1) == 0
        assert lib.oaa_plan_region(h, 4, None, None) == 1
        g = binding.Geometry()
        assert lib.oaa_plan_geometry(h, None) == 1
        assert lib.oaa_plan_geometry(h, ctypes.byref(g)) == 0 and g.L == 16 and g.T == 4
    finally:
        binding.oaa_plan_destroy(h)


def test_fused_passes_selection_and_caches(lib):
    """Overlap-add plans at L = 64 with C <= 4 and at most 8 blocks per side
    take the fused passes by default: kernel spectra bin-contiguous per kernel,
    one weight-gradient partial sum per range of block rows, and no gradient
    spectra to reuse. Switching the contraction discards cached spectra."""
    h = binding.oaa_plan_create_tiled(64, 3, 64, 224, 7, 64, 58)   # the first layer's tiling: T = 4
    try:
        g = binding.oaa_plan_geometry(h)
        assert g["fused"] == 1 and g["T"] == 4 and g["split"] == 8   # 32 kernel pairs x 8 ranges of rows
        _, wbytes = binding.oaa_plan_region(h, binding.REGION_W_SPECTRUM)
        assert wbytes == 8 * g["F"] * 3 * 64
        fake = 1 << 40   # never dereferenced: the calls below fail validation first
        assert lib.oaa_plan_bind_workspace(h, fake, binding.oaa_plan_workspace_bytes(h)) == 0
        assert lib.oaa_conv_backward_filter(h, fake, None, fake, None) == 4
        assert "fused" in binding.oaa_last_error_detail()
        assert lib.oaa_plan_set_contraction(h, binding.CONTRACTION_NARROW) == 0
        g = binding.oaa_plan_geometry(h)
        assert g["fused"] == 0 and g["split"] != 8
        assert lib.oaa_plan_set_contraction(h, binding.CONTRACTION_FUSED) == 0
        assert binding.oaa_plan_geometry(h)["fused"] == 1
        assert lib.oaa_plan_set_contraction(h, binding.CONTRACTION_AUTO) == 0
        assert binding.oaa_plan_geometry(h)["fused"] == 1
    finally:
        binding.oaa_plan_destroy(h)
    for dims, tiling, method in [((1, 5, 4, 100, 7), (64, 58), 0),    # C = 5
                                 ((1, 3, 4, 100, 7), (32, 26), 0),    # L = 32
                                 ((1, 3, 4, 600, 7), (64, 58), 0),    # T = 11
                                 ((1, 3, 4, 100, 7), (64, 0), 1)]:    # overlap-save
        h = binding.oaa_plan_create_method(*dims, *tiling, method)
        try:
            assert binding.oaa_plan_geometry(h)["fused"] == 0
            assert lib.oaa_plan_set_contraction(h, binding.CONTRACTION_FUSED) == 2
        finally:
            binding.oaa_plan_destroy(h)


def test_streaming_contraction_needs_few_channels(lib):
    h = binding.oaa_plan_create(1, 5, 4, 16, 3)
    try:
        assert lib.oaa_plan_set_contraction(h, binding.CONTRACTION_NARROW) == 2
        assert "C <= 4" in binding.oaa_last_error_detail()
        assert lib.oaa_plan_set_contraction(h, binding.CONTRACTION_MFMA) == 0
    finally:
        binding.oaa_plan_destroy(h)


@pytest.mark.parametrize("dims,split", [((64, 3, 64, 224, 7), 15), ((2, 3, 64, 224, 7), 2), ((1, 3, 4, 32, 5), 1),
                                        ((2, 3, 20, 100, 3), 3)])
def test_split_for_few_channels(lib, dims, split):
    """Few input channels: chunks of at least 1024 tiles in multiples of 128."""
    h = binding.oaa_plan_create(*dims)
    try:
        assert binding.oaa_plan_geometry(h)["split"] == split
    finally:
        binding.oaa_plan_destroy(h)


def test_binding_raises_with_detail(lib):
    with pytest.raises(binding.OaaError) as e:
        binding.oaa_plan_create(1, 1, 1, 8, 9)
    assert "exceeds" in str(e.value)


def test_twiddle_table_matches_libm(tmp_path):
    """The compile-time twiddles (csrc/twiddle.hpp, plain C++) against the C
    library's cos/sin in double, rounded to float."""
    import shutil
    import subprocess
    import numpy as np
    cxx = shutil.which("g++")
    if cxx is None:
        pytest.skip("no host C++ compiler")
    src = tmp_path / "tw.cpp"
    src.write_text('#include "twiddle.hpp"\n#include <cstdio>\n'
                   'template <int L> void dump() { for (int k = 0; k < L; ++k) '
                   'std::printf("%d %d %.9e %.9e\\n", L, k, (double)oaa::tw::kTable<L>.c[k], '
                   '(double)oaa::tw::kTable<L>.s[k]); }\n'
                   'int main() { dump<2>(); dump<4>(); dump<8>(); dump<16>(); dump<32>(); dump<64>(); }\n')
    exe = tmp_path / "tw"
    csrc = os.path.join(os.path.dirname(build.LIB_PATH), "csrc")
    subprocess.run([cxx, "-std=c++17", "-O1", "-I", csrc, str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split("\n")
    worst = 0
    for line in filter(None, out):
        L, k, c, s = line.split()
        L, k = int(L), int(k)
        ang = 2 * np.pi * k / L
        rc, rs = np.float32(np.cos(ang)), np.float32(np.sin(ang))
        for got, ref in ((np.float32(float(c)), rc), (np.float32(float(s)), rs)):
            ulp = np.spacing(np.float32(max(abs(ref), 1e-30)))
            worst = max(worst, abs(float(got) - float(ref)) / float(ulp) if abs(ref) > 1e-7 else abs(float(got)) * 1e7)
    assert worst <= 1.0


def test_paper_sweep_configurations():
    """The three sweeps of Section 3 as configured for the benchmark module."""
    from paper_1601_06815_amd.sweeps import sweep_configs
    k = sweep_configs("kernels")
    assert all(c[1:] == (1, 1, c[3], 32, 5) for c in k) and [c[3] for c in k][0] == 25 and k[-1][3] == 750
    s = sweep_configs("ksize")
    assert [c[5] for c in s] == list(range(1, 65)) and all(c[3:5] == (100, 64) for c in s)
    i = sweep_configs("input")
    assert [c[4] for c in i] == list(range(8, 257, 8)) and all(c[5] == 5 for c in i)
    assert len(sweep_configs("all")) == len(k) + len(s) + len(i)


@pytest.mark.parametrize("name,L,h,T", [("large128", 32, 17, 7), ("mid56", 16, 14, 4), ("first224", 16, 10, 22),
                                       ("tiny", 16, 12, 3)])
def test_overlap_save_geometry(lib, name, L, h, T):
    """The output-tiled method: hop h = L - n + 1 reported as b, and
    T = ceil(M / h) windows per side (the large layer: 7, against 8 blocks
    of the overlap-add tiling)."""
    ly = LAYERS[name]
    handle = binding.oaa_plan_create_method(ly.B, ly.C, ly.K, ly.N, ly.n, L, 0, binding.METHOD_OVERLAP_SAVE)
    try:
        geo = binding.oaa_plan_geometry(handle)
        assert (geo["L"], geo["b"], geo["T"], geo["P"], geo["method"]) == (L, h, T, T * T, 1)
        assert geo["M"] == ly.M and T == -(-ly.M // h)
    finally:
        binding.oaa_plan_destroy(handle)
    auto = binding.oaa_plan_create_method(ly.B, ly.C, ly.K, ly.N, ly.n, 0, 0, binding.METHOD_OVERLAP_SAVE)
    try:
        g2 = binding.oaa_plan_geometry(auto)
        assert g2["b"] == g2["L"] - ly.n + 1 and g2["T"] == -(-ly.M // g2["b"])
    finally:
        binding.oaa_plan_destroy(auto)


@pytest.mark.parametrize("dims,status", [
    ((1, 1, 1, 16, 5, 8, 0, 1), 1),   # L < 2n - 1
    ((1, 1, 1, 16, 5, 16, 11, 1), 1),  # b not the hop
    ((1, 1, 1, 16, 5, 24, 0, 1), 2),   # L not a power of two
    ((1, 1, 1, 16, 5, 16, 0, 7), 1),   # unknown method
])
def test_method_plan_validation(lib, dims, status):
    h = ctypes.c_void_p()
    st = lib.oaa_plan_create_method(ctypes.byref(h), *dims)
    assert st == status and not h.value
    assert lib.oaa_last_error_detail()


def test_small_division_by_reciprocal_is_exact():
    """The inverse kernels divide small lane indices x < 2^16 by a divisor
    d < 2^16 as floor(x m / 2^32) with m = floor((2^32 - 1) / d) + 1 (d >= 2;
    d = 1 is taken apart, m would be 2^32): exact for every such x."""
    x = np.arange(1 << 16, dtype=np.uint64)
    for d in list(range(2, 1025)) + [4095, 4096, 4097, 65535]:
        m = np.uint64(0xFFFFFFFF // d + 1)
        assert m < (1 << 32)
        assert np.array_equal((x * m) >> np.uint64(32), x // np.uint64(d)), d
    assert (0xFFFFFFFF // 1 + 1) & 0xFFFFFFFF == 0  # why d = 1 needs its own path


def test_forward_noalloc_validation(lib):
    """oaa_conv_forward_noalloc refuses NULL tensors and layers whose spectra
    exceed its 64 MiB static scratch before touching any device."""
    h = binding.oaa_plan_create(32, 96, 256, 128, 16)
    try:
        assert binding.oaa_plan_workspace_bytes(h) > 64 << 20
        st = lib.oaa_conv_forward_noalloc(h, 256, 256, 256, None)
        assert binding.STATUS[st] == "OAA_ERR_UNSUPPORTED"
        assert "static scratch" in binding.oaa_last_error_detail()
    finally:
        binding.oaa_plan_destroy(h)
    h = binding.oaa_plan_create(1, 3, 4, 32, 5)
    try:
        for args in ((None, 256, 256), (256, None, 256), (256, 256, None)):
            st = lib.oaa_conv_forward_noalloc(h, *args, None)
            assert binding.STATUS[st] == "OAA_ERR_INVALID_ARG"
        assert binding.STATUS[lib.oaa_conv_forward_noalloc(None, 256, 256, 256, None)] == "OAA_ERR_INVALID_ARG"
    finally:
        binding.oaa_plan_destroy(h)


def test_register_fft_matches_numpy(tmp_path):
    """The in-register transform of csrc/fft_core.hpp (radix-2^2 stages, a
    last radix-2 stage for odd log2 L), run on the host: every size L = 2 to
    64, both signs, with and without the zero upper half, against numpy's
    FFT in double, coefficient k read at position bitrev(k)."""
    import shutil
    import subprocess
    import numpy as np
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("no hipcc")
    src = tmp_path / "fft.cpp"
    src.write_text(r'''#include "fft_core.hpp"
#include <cstdio>
template <int L, int SIGN, bool ZH> void run(unsigned seed) {
  float re[L], im[L];
  unsigned s = seed;
  for (int i = 0; i < L; ++i) {
    s = s * 1664525u + 1013904223u; float a = float(s >> 8) / 16777216.0f - 0.5f;
    s = s * 1664525u + 1013904223u; float b = float(s >> 8) / 16777216.0f - 0.5f;
    re[i] = (ZH && i >= L / 2) ? 0.f : a; im[i] = (ZH && i >= L / 2) ? 0.f : b;
    std::printf("i %d %d %d %d %.9e %.9e\n", L, SIGN, int(ZH), i, re[i], im[i]);
  }
  oaa::fft_dif<L, SIGN, ZH>(re, im);
  for (int i = 0; i < L; ++i) std::printf("o %d %d %d %d %.9e %.9e\n", L, SIGN, int(ZH), i, re[i], im[i]);
}
template <int L> void all() { run<L, -1, false>(L); run<L, 1, false>(L + 7); run<L, -1, true>(L + 3); run<L, 1, true>(L + 5); }
int main() { all<2>(); all<4>(); all<8>(); all<16>(); all<32>(); all<64>(); }
''')
    exe = tmp_path / "fft"
    csrc = os.path.join(os.path.dirname(build.LIB_PATH), "csrc")
    subprocess.run([hipcc, "-std=c++17", "-O1", "--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang",
                    "-packed-fp32-ops", "-I", csrc, "-x", "hip", str(src), "-o", str(exe)], check=True,
                   capture_output=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split("\n")
    data = {}
    for line in filter(None, out):
        kind, L, sign, zh, i, a, b = line.split()
        data.setdefault((int(L), int(sign), int(zh)), {}).setdefault(kind, {})[int(i)] = complex(float(a), float(b))

    def bitrev(k, L):
        r, b = 0, 1
        while b < L:
            r, k, b = (r << 1) | (k & 1), k >> 1, b << 1
        return r

    assert len(data) == 24
    for (L, sign, zh), d in data.items():
        x = np.array([d["i"][i] for i in range(L)])
        X = np.fft.fft(x) if sign < 0 else L * np.fft.ifft(x)
        got = np.array([d["o"][bitrev(k, L)] for k in range(L)])
        err = np.max(np.abs(got - X)) / np.max(np.abs(X))
        assert err < 2e-6, (L, sign, zh, err)


def test_kernel_chain_validation(lib):
    """oaa_plan_set_kernel_chain: scratch size, and every argument error
    before any launch (a fake device pointer is never dereferenced)."""
    h = binding.oaa_plan_create(2, 3, 4, 20, 6)          # n = 6: n1 + n2 - 1
    try:
        g = binding.oaa_plan_geometry(h)
        F, J = g["F"], 5
        align = lambda v: (v + 255) // 256 * 256
        need = align(F * 3 * J * 8) + align(F * J * 4 * 8)
        assert binding.oaa_plan_chain_scratch_bytes(h, J) == need
        assert binding.oaa_plan_chain_scratch_bytes(h, 0) == 0
        fake = 1 << 40
        assert lib.oaa_plan_set_kernel_chain(h, fake, J, 3, fake, 4, fake, need, None) == 3   # no workspace
        assert lib.oaa_plan_bind_workspace(h, fake, binding.oaa_plan_workspace_bytes(h)) == 0
        assert lib.oaa_plan_set_kernel_chain(h, fake, J, 3, fake, 3, fake, need, None) == 1   # 3 + 3 - 1 != 6
        assert "n1 + n2 - 1" in binding.oaa_last_error_detail()
        assert lib.oaa_plan_set_kernel_chain(h, None, J, 3, fake, 4, fake, need, None) == 1
        assert lib.oaa_plan_set_kernel_chain(h, fake, 0, 3, fake, 4, fake, need, None) == 1
        assert lib.oaa_plan_set_kernel_chain(h, fake, J, 3, fake, 4, fake, need - 1, None) == 1
        assert lib.oaa_plan_set_kernel_chain(h, fake, J, 3, fake, 4, fake + 8, need, None) == 1  # alignment
    finally:
        binding.oaa_plan_destroy(h)
    h = binding.oaa_plan_create_tiled(64, 3, 64, 224, 7, 64, 58)   # fused passes by default
    try:
        fake = 1 << 40
        assert lib.oaa_plan_bind_workspace(h, fake, binding.oaa_plan_workspace_bytes(h)) == 0
        need = binding.oaa_plan_chain_scratch_bytes(h, 8)
        assert lib.oaa_plan_set_kernel_chain(h, fake, 8, 4, fake, 4, fake, need, None) == 2
        assert "fused" in binding.oaa_last_error_detail()
    finally:
        binding.oaa_plan_destroy(h)
