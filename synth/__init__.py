"""Seeded synthetic workloads for the decoder-layer shard.

This package only describes workloads (shapes, partitions, positions) and
draws their random inputs. It holds none of the layer's arithmetic: both the
fp64 oracle and the HIP path receive the same fp16 arrays from it.
"""
from .configs import WORKLOADS, Workload, LayerDims, get
from .gen import LayerInputs, layer_inputs

__all__ = ["WORKLOADS", "Workload", "LayerDims", "get", "LayerInputs", "layer_inputs"]
