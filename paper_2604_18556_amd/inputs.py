"""Seeded synthetic inputs for the GSQ layer step (weights W and calibration Gram H = X^T X).

This module holds no part of the method: it only draws layers and calibration
activations shaped like the paper's workloads (§4.1: Llama-3.1-8B/70B linear
layers, Kimi-K2.5 routed experts; calibration of 4096 sequences), so the HIP
path, the oracle, the tests and the benchmark can all consume the same
numbers.  The paper's datasets and checkpoints are not used; the recipe is:

* W ~ N(0, 0.02^2); for the bf16 workloads 0.1 % of the entries (chosen
  uniformly without replacement) are multiplied by 10 (outlier weights), then
  rounded to bfloat16;
* X has i.i.d. Normal (tiny workload) or Student-t(4) (heavy-tailed) entries,
  and every input channel j is multiplied by lambda_j ~ LogNormal(0, 0.5);
* H = X^T X (no normalisation);
* MoE token counts per expert follow a Zipf(1.2) profile over a seeded
  permutation of 64 expert ranks, 16384 routed token slots in total.

Random streams: numpy PCG64 seeded with 1000 + workload index.
"""
from dataclasses import dataclass

import numpy as np

L4 = (-1.5, -0.5, 0.5, 1.5)
L3 = (-1.0, 0.0, 1.0)
L8 = (-3.5, -2.5, -1.5, -0.5, 0.5, 1.5, 2.5, 3.5)


@dataclass(frozen=True)
class Workload:
    name: str
    index: int                 # seeds PCG64(1000 + index)
    batch: int
    out_features: int
    in_features: int
    levels: tuple
    group_size: int
    layout: str                # "group" | "superblock"
    precision: str             # "fp32" | "bf16"
    tokens: int                # calibration tokens (per expert: see moe_token_counts)
    steps: int
    x_dist: str                # "normal" | "student_t4"
    outliers: bool
    lr_scales: float
    relaxation: str = "grid"   # "grid" | "shift" | "ternary"


WORKLOADS = {
    w.name: w for w in (
        Workload("tiny-256x256-k4", 0, 1, 256, 256, L4, 128, "group", "fp32",
                 512, 100, "normal", False, 5e-5),
        Workload("attn-4096x4096-k3", 1, 1, 4096, 4096, L3, 128, "group", "bf16",
                 4096, 500, "student_t4", True, 5e-5),
        Workload("mlp-up-14336x4096-k8", 2, 1, 14336, 4096, L8, 128, "group", "bf16",
                 8192, 500, "student_t4", True, 5e-5),
        Workload("mlp-down-4096x14336-k8", 3, 1, 4096, 14336, L8, 128, "group", "bf16",
                 8192, 500, "student_t4", True, 5e-5),
        Workload("down-8192x28672-k4", 4, 1, 8192, 28672, L4, 64, "group", "bf16",
                 8192, 300, "student_t4", True, 5e-5),
        Workload("moe-64x2048x7168-superblock", 5, 64, 2048, 7168, L8, 16, "superblock", "bf16",
                 2048, 200, "student_t4", True, 0.0),
        # the same layers under the paper's other relaxations (same seeds, same data)
        Workload("mlp-down-4096x14336-shift8", 3, 1, 4096, 14336, L8, 128, "group", "bf16",
                 8192, 500, "student_t4", True, 5e-5, "shift"),
        Workload("attn-4096x4096-ternary", 1, 1, 4096, 4096, L3, 128, "base3", "bf16",
                 4096, 500, "student_t4", True, 5e-5, "ternary"),
        # the K-quant experts with the local shift, App. E's relaxation for sets of more than
        # four values
        Workload("moe-64x2048x7168-superblock-shift8", 5, 64, 2048, 7168, L8, 16, "superblock",
                 "bf16", 2048, 200, "student_t4", True, 0.0, "shift"),
    )
}


def rng_for(index, salt=0):
    return np.random.Generator(np.random.PCG64(1000 + index + 7919 * salt))


def to_bf16_values(x):
    """Round float32 values to the nearest bfloat16 (ties to even); float32 array out."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = (b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))) & np.uint64(0xFFFF0000)
    return b.astype(np.uint32).view(np.float32)


def make_weights(rng, batch, O, I, outliers, bf16):
    W = rng.normal(0.0, 0.02, size=(batch, O, I)).astype(np.float32)
    if outliers:
        flat = W.reshape(batch, -1)
        n_out = max(1, int(round(0.001 * O * I)))
        for b in range(batch):
            idx = rng.choice(O * I, size=n_out, replace=False)
            flat[b, idx] *= np.float32(10.0)
    return to_bf16_values(W) if bf16 else W


def make_activations(rng, tokens, I, dist):
    if dist == "normal":
        X = rng.standard_normal((tokens, I))
    else:
        X = rng.standard_t(4.0, size=(tokens, I))
    lam = rng.lognormal(0.0, 0.5, size=I)
    return (X * lam[None, :]).astype(np.float32)


def moe_token_counts(rng, n_experts=64, routed=16384, s=1.2):
    ranks = rng.permutation(n_experts) + 1
    z = np.arange(1, n_experts + 1, dtype=np.float64) ** -s
    return np.maximum(1, np.rint(routed * ranks.astype(np.float64) ** -s / z.sum())).astype(int)


def gram(X, device=None):
    """H = X^T X in float32 (float64 accumulation on the CPU path)."""
    if device is not None:
        import torch
        Xt = torch.as_tensor(X, device=device)
        return (Xt.t() @ Xt).float()
    X64 = np.asarray(X, dtype=np.float64)
    return (X64.T @ X64).astype(np.float32)


def make_layer(w, out_rows=None, in_features=None, batch=None, device=None, tokens=None):
    """Draw (W, H) for workload ``w``, optionally shrunk (rows / inputs / experts / tokens).

    Returns W as float32 values (bfloat16-representable for bf16 workloads),
    shape (batch, O, I), and H float32 (batch, I, I) as numpy arrays, or H as a
    torch tensor on ``device`` when one is given.
    """
    O = out_rows or w.out_features
    I = in_features or w.in_features
    B = batch or w.batch
    rng = rng_for(w.index)
    W = make_weights(rng, B, O, I, w.outliers, w.precision == "bf16")
    if w.layout == "superblock":
        counts = moe_token_counts(rng_for(w.index, 1), n_experts=max(B, 64))[:B]
    else:
        counts = [tokens or w.tokens] * B
    Hs = []
    for b in range(B):
        X = make_activations(rng_for(w.index, 2 + b), int(tokens or counts[b]), I, w.x_dist)
        Hs.append(gram(X, device))
    if device is not None:
        import torch
        return W, torch.stack(Hs)
    return W, np.stack(Hs)
