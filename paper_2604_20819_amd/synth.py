"""Seeded synthetic inputs shared by the tests, the bench and the oracle checks.

This module holds no attention arithmetic.  It only draws the workloads the
paper evaluates on: zero-mean, unit-variance Gaussian Q, K, V and dO with
fixed seeds (Section 4.1), generated with numpy's PCG64 in float32, drawn in
the order Q, K, V, dO with layout [B, L, H, d], then cast with
round-to-nearest-even to the input dtype (bf16, fp16) or kept as fp32.
"""
import numpy as np
import torch

_TORCH_DTYPES = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def torch_dtype(name):
    return _TORCH_DTYPES[name]


def _draw(gen, shape, out, chunk_elems=1 << 26):
    """Fill `out` (a CPU torch tensor of `shape`) with standard normals drawn
    sequentially from `gen` in float32, converting chunk by chunk so a 1M-token
    tensor never needs a full float32 copy."""
    flat = out.view(-1)
    n = flat.numel()
    for s in range(0, n, chunk_elems):
        e = min(n, s + chunk_elems)
        x = gen.standard_normal(e - s, dtype=np.float32)
        flat[s:e].copy_(torch.from_numpy(x))


def make_inputs(seed, B, L, H, d, dtype="bf16", with_dO=False, pin_memory=False):
    """Return (Q, K, V) or (Q, K, V, dO) as CPU torch tensors [B, L, H, d]."""
    gen = np.random.Generator(np.random.PCG64(seed))
    names = ["Q", "K", "V"] + (["dO"] if with_dO else [])
    out = []
    for _ in names:
        t = torch.empty((B, L, H, d), dtype=torch_dtype(dtype), pin_memory=pin_memory)
        _draw(gen, (B, L, H, d), t)
        out.append(t)
    return tuple(out)


def sample_rows(seed, L, n, H):
    """Per-head sorted query-row samples of size min(n, L), always holding rows
    0 and L-1 (seeded choice without replacement)."""
    gen = np.random.Generator(np.random.PCG64(seed))
    rows = []
    for _ in range(H):
        if n >= L:
            rows.append(np.arange(L, dtype=np.int64))
            continue
        r = gen.choice(L - 2, size=n - 2, replace=False) + 1
        rows.append(np.sort(np.concatenate([[0, L - 1], r]).astype(np.int64)))
    return rows


def as_f64(t):
    """Exact float64 copy (numpy) of a CPU torch tensor of any input dtype."""
    return t.to(torch.float64).numpy()
