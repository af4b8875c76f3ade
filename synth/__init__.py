"""Seeded synthetic workloads shared by the GPU path's tests and the oracle's.

This module only describes workload shapes and draws random numbers; it holds
none of the optimizer's arithmetic.  Host arrays come from numpy's Philox
generator keyed by (seed, step, worker); device arrays come from a
torch.Generator seeded the same way.  Both the GPU path and the oracle receive
the same arrays (the oracle gets host copies).

The workloads stand in for BERT pre-training (Section 7.1 of the paper):
only the model shapes (BERT-Base L=12 H=768, BERT-Large L=24 H=1024, FFN 4H,
vocabulary 30522, 512 positions) are used; the data and gradients are
synthetic.
"""
from .workloads import (  # noqa: F401
    Workload, WORKLOADS, bert_tensor_shapes, stress_sizes, get,
    host_normal, host_params, host_grads, grad_scale_per_element,
    device_params, device_grads, device_bits_and_scales, host_bits_and_scales,
)
