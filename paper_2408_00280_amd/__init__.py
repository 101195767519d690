"""Temporally fused LIF spiking-neuron layer for MI355X (gfx950).

The compute path is the HIP library ``libsnnlif.so`` behind the C ABI of
``include/snn_lif.h``; :mod:`paper_2408_00280_amd.native` is its thin binding
(import it to use the GPU path; it raises if the library is not built) and
:mod:`paper_2408_00280_amd.layer` wraps it as a torch autograd function and
module.  ``build()`` compiles the library.
"""
from .build import build  # noqa: F401
