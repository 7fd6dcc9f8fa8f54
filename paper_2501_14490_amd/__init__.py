"""MI355X-native mul-free channel-wise Parallel Spiking Neuron (arXiv 2501.14490).

The training step of the neuron (forward charge + fire, surrogate-gradient
backward, power-of-two weight quantizer) runs in hand-written HIP kernels for
gfx950 behind the C ABI declared in ``include/mfpsn.h`` (``libmfpsn.so``).
``paper_2501_14490_amd.mfpsn`` is the thin Python binding with the same names.

Importing the package does not load the native library; ``mfpsn`` does, and
raises if it has not been built.
"""
__all__ = ["mfpsn", "workloads"]
