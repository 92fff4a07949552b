"""Seeded synthetic inputs shaped like the paper's workloads.

These stand in for the weights and KV activations the paper measures on
(Llama-3.1-8B-Instruct weights, WikiText-2 KV activations), which are not
available here: same shapes, dtypes and value structure (heavy tails, outlier
columns or channels, per-output-channel scales), drawn from seeded generators.
This module holds no codec arithmetic; it is the only code that both the
oracle-side tests and the HIP path consume.
"""
import math

import numpy as np
import torch

# Llama-3.1-8B linear shapes [out, in]: tiles run along the input dimension.
LLAMA_LINEARS = (
    ("q", 4096, 4096),
    ("k", 1024, 4096),
    ("v", 1024, 4096),
    ("o", 4096, 4096),
    ("gate", 14336, 4096),
    ("up", 14336, 4096),
    ("down", 4096, 14336),
)
LLAMA_LAYERS = 32


def _gen(device, seed):
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def single_matrix_fp32(seed=0, shape=(512, 512), std=0.02):
    """Single fp32 matrix, entries iid N(0, std^2) (numpy PCG64, seed 0)."""
    rng = np.random.default_rng(seed)
    return (rng.standard_normal(shape) * std).astype(np.float32)


def heavy_tailed_weight(device="cpu", seed=2, shape=(4096, 4096), std=0.02, n_outlier_cols=16,
                        outlier_scale=20.0):
    """bf16 weight, Student-t (nu = 4) scaled to std 0.02, plus random columns x20."""
    g = _gen(device, seed)
    rows, cols = shape
    nrm = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    # chi-square with 4 degrees of freedom = sum of 4 squared normals
    chi = torch.zeros(shape, device=device, dtype=torch.float32)
    for _ in range(4):
        e = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
        chi += e * e
    t = nrm / torch.sqrt(chi / 4.0)
    w = t * (std / math.sqrt(2.0))  # Var(t_4) = 2
    cols_idx = torch.randperm(cols, generator=g, device=device)[:n_outlier_cols]
    w[:, cols_idx] *= outlier_scale
    return w.to(torch.bfloat16)


def llama_linear_seed(layer, idx, base=3000):
    return base + layer * 8 + idx


def llama_linear(layer, idx, device="cpu", std=0.02, rows=None):
    """One Llama-shaped linear: bf16 N(0, std^2) with per-output-channel scales
    drawn log-uniform in [0.5, 2].  `rows` limits the output rows (for sampling)."""
    name, out_f, in_f = LLAMA_LINEARS[idx]
    g = _gen(device, llama_linear_seed(layer, idx))
    w = torch.randn((out_f, in_f), generator=g, device=device, dtype=torch.float32) * std
    u = torch.rand((out_f, 1), generator=g, device=device, dtype=torch.float32)
    scale = torch.exp(math.log(0.5) + u * (math.log(2.0) - math.log(0.5)))
    w = (w * scale).to(torch.bfloat16)
    if rows is not None:
        w = w[:rows].contiguous()
    return w


def kv_cache(device="cpu", seed=4, batch=16, seq=8192, heads=8, head_dim=128,
             n_outlier_channels=4, outlier_scale=10.0, role="k"):
    """KV cache tensor [batch, seq, heads, head_dim] bf16: N(0, 1); keys carry
    4 fixed channels per head scaled x10 (the same channels for every token)."""
    g = _gen(device, seed + (0 if role == "k" else 1))
    x = torch.randn((batch, seq, heads, head_dim), generator=g, device=device, dtype=torch.float32)
    if role == "k":
        gc = _gen("cpu", seed + 100)
        for h in range(heads):
            ch = torch.randperm(head_dim, generator=gc)[:n_outlier_channels].to(device)
            x[:, :, h, ch] *= outlier_scale
    return x.to(torch.bfloat16)


def activations(device="cpu", seed=5, tokens=4096, features=4096, outlier_frac=0.01,
                outlier_scale=30.0):
    """Activations [tokens, features] bf16 N(0, 1) with 1% of the feature
    channels (fixed across tokens) scaled x30."""
    g = _gen(device, seed)
    a = torch.randn((tokens, features), generator=g, device=device, dtype=torch.float32)
    gc = _gen("cpu", seed + 100)
    n_out = max(1, int(round(outlier_frac * features)))
    ch = torch.randperm(features, generator=gc)[:n_out].to(device)
    a[:, ch] *= outlier_scale
    return a.to(torch.bfloat16)


def gaussian_tiles(n_tiles, tile=128, seed=42, device="cpu", dtype=torch.float32):
    """iid N(0, 1) tiles, the calibration source of the paper's App. B."""
    g = _gen(device, seed)
    return torch.randn((n_tiles, tile), generator=g, device=device, dtype=torch.float32).to(dtype)


def queries(n=1024, dim=128, seed=7, device="cpu"):
    g = _gen(device, seed)
    return torch.randn((n, dim), generator=g, device=device, dtype=torch.float32)
