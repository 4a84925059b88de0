"""Seeded synthetic workloads shared by the oracle and the HIP path.

This package holds only *inputs*: CNN architectures written as fused-layer
lists, and seeded generators for weights, batch-norm statistics and input
images, plus seeded request traces and cluster plans for the request
scheduler (serving.py).  It contains none of the forward-pass arithmetic (no convolution,
pooling, normalisation folding or shape inference); both the CPU oracle and
the GPU library consume what it produces, and neither imports the other.
"""
from .zoo import Layer, Model, MODELS, model, param_count
from .gen import (Workload, WORKLOADS, workload, layer_params, model_params,
                  partition_input, to_dtype_values, DTYPES)

__all__ = ["Layer", "Model", "MODELS", "model", "param_count", "Workload",
           "WORKLOADS", "workload", "layer_params", "model_params",
           "partition_input", "to_dtype_values", "DTYPES"]
