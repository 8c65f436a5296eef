"""Float64 CPU oracle for the DONN physics kernel of LightRidge (arXiv 2306.11268).

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute anything in this package: only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code,
tables or constants with the HIP library in ``paper_2306_11268_amd/`` and it
imports nothing from there.

Everything here is plain numpy in float64 / complex128.  Discrete Fourier
transforms are the naive O(M^3) matrix products of their definition (the DFT
matrix is built from integer-reduced exponents); numpy's BLAS only executes
those products.  No FFT library is used by the oracle.
"""

from .donn import (  # noqa: F401
    FRESNEL,
    ANGULAR_SPECTRUM,
    Detector,
    dft_matrix,
    dft2,
    idft2,
    frequencies,
    transfer_function,
    propagate,
    encode_amplitude,
    modulate,
    intensity,
    detector_readout,
    donn_forward,
    softmax_cross_entropy,
    mse_softmax_loss,
    region_scatter,
    donn_backward,
)
