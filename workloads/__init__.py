"""Seeded synthetic workloads for the StructADMM hot path.

This package holds layer shapes, kept-count rounding and seeded tensor
generators only.  It contains none of the method's arithmetic, so both the
CPU oracle (``oracle/``) and the GPU library can be fed from it without
sharing any computation.
"""
from .configs import (  # noqa: F401
    ConvLayer, Workload, WORKLOADS, get_workload, kept_count,
    alexnet_layers, resnet50_layers, FILTER, CHANNEL, SHAPE, ELEMENT, KIND_NAMES,
    PAPER_TABLE_SPARSITY, PAPER_ELEMENT_SPARSITY, kept_from_sparsity,
)
from .gen import layer_tensors, input_nchw, normal_f32  # noqa: F401
