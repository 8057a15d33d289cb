"""CPU oracle for the overlap-and-add (OaA) FFT convolution layer.

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or
execute this package: only the test suite, the smoke check in
``__graft_entry__`` and the ``cpu_baseline`` leg of ``bench.py`` use it.

Source: T. Highlander and A. Rodriguez, "Very Efficient Training of
Convolutional Neural Networks using Fast Fourier Transform and
Overlap-and-Add", arXiv:1601.06815 (BMVC 2015).

Modules
-------
direct
    The plain definition of one convolutional layer (forward, error
    propagation, weight gradient) evaluated in the spatial domain in float64
    (the paper's "spaceConv", Table 1). This is what every GPU result is
    compared with.
dft
    Convolution through an explicitly built discrete Fourier matrix (the
    convolution theorem the paper's Introduction relies on; the paper's
    "FFTconv" written as a definition, no fast transform). Used only to pin
    ``direct`` on tiny inputs.
oaa
    The paper's OaA algorithm (Section 2) in float64 with numpy's FFT, step by
    step in the paper's order: divide into n x n blocks, zero-pad, transform,
    Hadamard product with channel sum, inverse transform, overlap by n-1 and
    add. Its intermediate spectra are what the GPU stages are compared with.
oas
    The output-tiled alternative: overlap-and-save forward over L x L windows
    of x at hop L - n + 1, the error propagation as overlap-and-add over
    blocks of g, and the weight gradient from the same windows and blocks.

Every function states the passage it follows. Pins (tests/test_oracle.py)
tie each function to library routines, closed forms and invariants that are
independent of this code.
"""

from .direct import (conv_forward, conv_backward_data, conv_backward_filter,  # noqa: F401
                     conv_forward_at, conv_backward_data_at, conv_backward_filter_at)
from .dft import dft_conv_forward  # noqa: F401
from . import oaa  # noqa: F401
from . import oas  # noqa: F401
