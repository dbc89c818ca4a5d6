"""Seeded synthetic inputs for the per-hit classifier.

This package only draws random numbers and lays them out in arrays: ADC
planes, hit lists, pre-cut patch batches and He-normal weights.  It holds none
of the classifier's arithmetic, so the CPU oracle and the GPU path can both take
their inputs from it without sharing any of the method.
"""

from .gen import (  # noqa: F401
    PATCH, KSIZE, NCH, FMAP, FC1_IN, FC1_OUT, FC2_OUT, NCLS,
    WEIGHT_SHAPES, WEIGHT_ORDER, he_normal_weights, n_parameters,
    Plane, gen_plane, config1, config2, config3, config4_patches,
    config5_requests, coord_image,
)
