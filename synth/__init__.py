"""Seeded synthetic inputs shared by the tests, the benchmark and smoke().

This module only draws random numbers: it holds none of the method's
arithmetic. Both the HIP path and the CPU oracle receive the very same
tensors from it.

Recipe: every tensor is drawn as float32 N(0, 1) from a ``torch.Generator``
on the tensor's device, seeded from a tuple (workload id, layer, chunk,
tensor id), then rounded once to bfloat16 (round-to-nearest-even, torch's
conversion). The oracle reads the bf16 values back as float64, so both sides
see identical inputs. CPU and GPU generators give different streams; tests
always hand the same materialised tensor to both sides.
"""

import hashlib

import torch

# tensor ids inside a seed tuple
Q, K, V, X, Y_FULL, Y_LOCAL = range(6)


def seed_of(*parts):
    """A 63-bit seed from a tuple of ints (stable across runs and hosts)."""
    h = hashlib.sha256(repr(tuple(int(p) for p in parts)).encode()).digest()
    return int.from_bytes(h[:8], "little") & ((1 << 63) - 1)


def normal(shape, seed, device="cpu", dtype=torch.bfloat16, scale=1.0):
    """N(0, scale^2) draws of ``shape``; float32 first, then cast to ``dtype``."""
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    t = torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32)
    if scale != 1.0:
        t.mul_(scale)
    return t.to(dtype)


def chunk_qkv(workload, layer, chunk, n_q, cache_len, hidden, device="cpu",
              q_scale=1.0, capacity=None):
    """Q [n_q, hidden] and a K/V cache [capacity, hidden] (bf16).

    ``capacity`` >= cache_len rows are allocated; only the first cache_len
    rows are meaningful, the rest are filled with large values so that a
    kernel reading beyond cache_len would be caught by parity.
    """
    cap = cache_len if capacity is None else capacity
    q = normal((n_q, hidden), seed_of(workload, layer, chunk, Q), device, scale=q_scale)
    k = normal((cap, hidden), seed_of(workload, layer, chunk, K), device)
    v = normal((cap, hidden), seed_of(workload, layer, chunk, V), device)
    if cap > cache_len:
        k[cache_len:] = 30.0
        v[cache_len:] = 1.0e4
    return q, k, v


def rollout_chunk(layer, chunk, n_q, hidden, device="cpu", workload=5):
    """One chunk of a streaming rollout for one layer: the chunk's queries and
    the keys and values it appends to the layer's cache, each [n_q, hidden]
    bf16, drawn fresh per (layer, chunk)."""
    return tuple(normal((n_q, hidden), seed_of(workload, layer, chunk, t), device) for t in (Q, K, V))
