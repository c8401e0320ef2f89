"""MI355X-native Adaptive Gradient Scaling (AGS) step with gradient statistics.

The hot path of the Tula method (arXiv 2603.18112) for one data-parallel
training step: K replica gradients averaged on the GPU, per-layer segmented
statistics (||w||^2, ||g||^2, cross-replica variance, small-batch norm),
the gradient-variability decision of Eq. (5) and the layerwise-scaled
momentum-SGD update of Algorithm 1, in hand-written HIP kernels for gfx950
behind the C-ABI library ``libags.so`` (see ``include/ags.h``).

``paper_2603_18112_amd.ags`` is the Python binding (ctypes marshalling
only); ``layouts`` and ``synth`` describe flat layouts and draw seeded
synthetic inputs.
"""

__all__ = ["layouts", "synth", "ags"]
