"""Seeded synthetic inputs shaped like the paper's workloads.

Data only: this module draws activations, weights and output derivatives and
rounds them to the storage dtype. It holds none of the method's arithmetic
(no patterns, no sampling, no layer math) and is shared by the tests, the
benchmark and the oracle comparisons, which all receive the same tensors.

Distributions (all fp32 draws from a torch.Generator seeded per workload):
  normal(std)      - N(0, std^2)
  uniform(a)       - U(-a, a)
  xavier(n, k)     - N(0, 2 / (fan_in + fan_out))
  he(n, k)         - N(0, 2 / fan_in)
bf16 workloads round the fp32 draws to bf16 (round to nearest even); the
oracle receives exactly those rounded values, widened to fp64.
"""

import math

import torch


def generator(seed):
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    return g


def normal(g, shape, std=1.0):
    return torch.randn(*shape, generator=g, dtype=torch.float32) * std


def uniform(g, shape, a):
    return (torch.rand(*shape, generator=g, dtype=torch.float32) * 2.0 - 1.0) * a


def xavier(g, n_out, n_in):
    return normal(g, (n_out, n_in), math.sqrt(2.0 / (n_in + n_out)))


def he(g, n_out, n_in):
    return normal(g, (n_out, n_in), math.sqrt(2.0 / n_in))


def storage_dtype(name):
    return {"f32": torch.float32, "bf16": torch.bfloat16}[name]


def to_storage(t, dtype_name):
    """Round an fp32 tensor to the storage dtype (bf16: nearest even)."""
    return t.to(storage_dtype(dtype_name)).contiguous()


def as_f64(t):
    """The exact values of a storage tensor as an fp64 CPU tensor."""
    return t.detach().to("cpu").to(torch.float64)
