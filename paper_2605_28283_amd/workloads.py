"""Seeded synthetic inputs for the sparse-FFN forward.

This module only draws random numbers and rounds them to bf16; it holds none
of the method's arithmetic.  Both the oracle-based tests and the HIP path
consume exactly the arrays produced here (bf16 values are carried as their
uint16 bit patterns).

Recipe (the paper's datasets and trained checkpoints are not available, so
these synthetic layers stand in for them):
  * one ``numpy.random.default_rng(seed)`` (PCG64) stream per layer, drawn in
    the fixed order W_r, W_gate, W_up, W_down, then the layer extras (skewed
    router bias);
  * expert/gate/up/down weights ~ N(0, 0.02^2);  router weights
    ~ N(0, (3/sqrt(d))^2) so that logits of a unit-variance token have std ~3
    (sharp routing distributions, which the paper's entropy loss aims for);
  * tokens come from a separate stream: x ~ N(0, 1), optionally each row scaled
    by LogNormal(0, 0.5) (prefill workload), and for the skewed workload a
    per-token temperature ~ U(0.5, 2) passed as its inverse;
  * the skewed workload adds a per-expert router bias ~ Gumbel(0, 1.5);
  * every value is drawn in fp32 and rounded to bf16 with round-to-nearest-even;
  * router-loss batches: logits [B, E] fp32 ~ N(0, 3^2) (the synthetic
    routers' logit scale), each row scaled by LogNormal(0, 0.5) so that sharp
    and flat routing distributions mix, plus a per-expert Gumbel(0, 1) offset
    so that the batch-mean probabilities are uneven (a non-trivial L_bal);
    the training-step workload is B = 16384 rows (8 sequences of 2048 tokens)
    over the LLaMA-3-8B split, E = 112;
  * the 32-layer stack (11.3 GB of weights) draws its layers on the GPU with
    torch's Philox generator, seeded 0x5EED0000 + 64 * seed + layer, in the
    same order and distributions (host PCG64 would take minutes per layer);
    its first residual x_0 comes from the host stream as above.
"""
from dataclasses import dataclass, field
from typing import Dict, Optional, Tuple

import numpy as np

EXPERT_WIDTH = 128


def bf16_bits(a) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); return uint16 bits.
    (torch's CPU conversion is the same rounding, multithreaded.)"""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def bf16_to_f32(bits) -> np.ndarray:
    """Exact fp32 value of bf16 bit patterns."""
    b = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32)


@dataclass
class Layer:
    d: int
    d_ff: int
    E: int
    W_r: np.ndarray      # [E, d]    bf16 bits
    W_gate: np.ndarray   # [d_ff, d] bf16 bits
    W_up: np.ndarray     # [d_ff, d] bf16 bits
    W_down: np.ndarray   # [d, d_ff] bf16 bits
    bias: Optional[np.ndarray] = None   # [E] fp32 (skewed router only)
    perm: Optional[np.ndarray] = None   # [d_ff] int32 neuron permutation


def make_layer(d: int, d_ff: int, E: int, seed, *, weight_std: float = 0.02,
               router_std: Optional[float] = None, skewed: bool = False,
               perm: bool = False) -> Layer:
    """One bias-free SwiGLU FFN layer with its linear router."""
    rng = np.random.default_rng(seed)
    if router_std is None:
        router_std = 3.0 / np.sqrt(d)
    W_r = bf16_bits(rng.standard_normal((E, d), dtype=np.float32) * np.float32(router_std))
    W_gate = bf16_bits(rng.standard_normal((d_ff, d), dtype=np.float32) * np.float32(weight_std))
    W_up = bf16_bits(rng.standard_normal((d_ff, d), dtype=np.float32) * np.float32(weight_std))
    W_down = bf16_bits(rng.standard_normal((d, d_ff), dtype=np.float32) * np.float32(weight_std))
    bias = None
    if skewed:
        bias = rng.gumbel(0.0, 1.5, size=E).astype(np.float32)
    p = None
    if perm:
        p = rng.permutation(d_ff).astype(np.int32)
    return Layer(d, d_ff, E, W_r, W_gate, W_up, W_down, bias, p)


def make_tokens(T: int, d: int, seed, *, row_lognormal_sigma: float = 0.0,
                temperature: bool = False) -> Tuple[np.ndarray, Optional[np.ndarray]]:
    """x [T, d] bf16 bits and, for the skewed workload, inv_temp [T] fp32."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((T, d), dtype=np.float32)
    if row_lognormal_sigma > 0.0:
        s = rng.lognormal(0.0, row_lognormal_sigma, size=(T, 1)).astype(np.float32)
        x = x * s
    inv_temp = None
    if temperature:
        inv_temp = (1.0 / rng.uniform(0.5, 2.0, size=T)).astype(np.float32)
    return bf16_bits(x), inv_temp


ROUTER_LOSS_B, ROUTER_LOSS_E = 16384, 112


def make_clustered_features(n: int, D: int, k: int, seed, *, centre_std: float = 0.02,
                            noise_std: float = 0.02):
    """Neuron feature rows for the clustering step: n rows of D bf16 values
    around k planted centres (n / k rows each), centre ~ N(0, centre_std^2),
    row = centre + N(0, noise_std^2), rows shuffled; plus k distinct row
    indices for the initial centroids.  Returns (F bits [n, D], planted group
    [n], init rows [k])."""
    rng = np.random.default_rng(seed)
    centres = rng.standard_normal((k, D), dtype=np.float32) * np.float32(centre_std)
    group = np.repeat(np.arange(k), n // k)
    rng.shuffle(group)
    F = centres[group] + rng.standard_normal((n, D), dtype=np.float32) * np.float32(noise_std)
    init = rng.choice(n, size=k, replace=False).astype(np.int32)
    return bf16_bits(F), group.astype(np.int32), init


def make_router_logits(B: int, E: int, seed, *, std: float = 3.0,
                       row_lognormal_sigma: float = 0.5, expert_gumbel: float = 1.0) -> np.ndarray:
    """Router logits [B, E] fp32 for the routing-regulariser kernels."""
    rng = np.random.default_rng(seed)
    g = rng.standard_normal((B, E), dtype=np.float32) * np.float32(std)
    if row_lognormal_sigma > 0.0:
        g *= rng.lognormal(0.0, row_lognormal_sigma, size=(B, 1)).astype(np.float32)
    if expert_gumbel > 0.0:
        g += rng.gumbel(0.0, expert_gumbel, size=(1, E)).astype(np.float32)
    return np.ascontiguousarray(g, dtype=np.float32)


# --------------------------------------------------------------------------
# The workloads.  Token streams use seed + 1000 so that changing T never
# changes the weights.

@dataclass(frozen=True)
class Workload:
    name: str
    d: int
    d_ff: int
    E: int
    T: Tuple[int, ...]
    taus: Tuple[float, ...]
    layers: int = 1
    skewed: bool = False
    row_lognormal_sigma: float = 0.0
    mlp: bool = False      # non-gated GELU MLP with biases (GPT-2) instead of SwiGLU
    notes: str = ""


WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload("tiny", 512, 2048, 16, (4,), (0.9,),
                     notes="single FFN layer, E=16 experts of 128 neurons, T=4 decode"),
    "llama8b_decode": Workload("llama8b_decode", 4096, 14336, 112, (1, 8, 32, 64),
                               (0.5, 0.7, 0.9, 1.0),
                               notes="LLaMA-3-8B-shaped FFN layer, decode batches"),
    "llama8b_stack32": Workload("llama8b_stack32", 4096, 14336, 112, (16,), (0.8,), layers=32,
                                notes="32 layers chained by residual add + RMSNorm(eps 1e-5)"),
    "llama8b_prefill": Workload("llama8b_prefill", 4096, 14336, 112, (2048,), (0.7, 0.9),
                                row_lognormal_sigma=0.5,
                                notes="prefill, rows scaled by LogNormal(0, 0.5)"),
    "gpt2m_decode": Workload("gpt2m_decode", 1024, 4096, 32, (1, 8, 32, 64), (0.5, 0.7, 0.9, 1.0),
                             mlp=True, notes="GPT-2 Medium MLP layer (GELU, biases), decode batches"),
    "qwen7b_skewed": Workload("qwen7b_skewed", 3584, 18944, 148, (64,), (0.5, 0.9),
                              skewed=True,
                              notes="Gumbel(0,1.5) router bias, per-token temperature U(0.5,2)"),
}


@dataclass
class MlpLayer:
    """Non-gated GELU MLP (GPT-2 style) with its linear router."""
    d: int
    d_ff: int
    E: int
    W_r: np.ndarray      # [E, d]    bf16 bits
    W_fc: np.ndarray     # [d_ff, d] bf16 bits
    b_fc: np.ndarray     # [d_ff]    fp32
    W_proj: np.ndarray   # [d, d_ff] bf16 bits
    b_proj: np.ndarray   # [d]       fp32
    perm: Optional[np.ndarray] = None
    bias: Optional[np.ndarray] = None   # [E] fp32 router bias (none in these workloads)


def make_mlp_layer(d: int, d_ff: int, E: int, seed, *, weight_std: float = 0.02,
                   bias_std: float = 0.02, perm: bool = False) -> MlpLayer:
    """GPT-2-style MLP layer: weights N(0, 0.02^2) (GPT-2's initialisation
    scale) rounded to bf16, biases N(0, 0.02^2) in fp32, router as in
    make_layer; drawn in the order W_r, W_fc, b_fc, W_proj, b_proj[, perm]."""
    rng = np.random.default_rng(seed)
    W_r = bf16_bits(rng.standard_normal((E, d), dtype=np.float32) * np.float32(3.0 / np.sqrt(d)))
    W_fc = bf16_bits(rng.standard_normal((d_ff, d), dtype=np.float32) * np.float32(weight_std))
    b_fc = (rng.standard_normal(d_ff, dtype=np.float32) * np.float32(bias_std)).astype(np.float32)
    W_proj = bf16_bits(rng.standard_normal((d, d_ff), dtype=np.float32) * np.float32(weight_std))
    b_proj = (rng.standard_normal(d, dtype=np.float32) * np.float32(bias_std)).astype(np.float32)
    p = rng.permutation(d_ff).astype(np.int32) if perm else None
    return MlpLayer(d, d_ff, E, W_r, W_fc, b_fc, W_proj, b_proj, p)


def make_layer_device(d: int, d_ff: int, E: int, seed: int, device="cuda", *,
                      weight_std: float = 0.02, router_std: Optional[float] = None):
    """One layer drawn on the GPU: dict of torch int16 tensors (bf16 bits)
    W_r [E,d], W_gate/W_up [d_ff,d], W_down [d,d_ff]."""
    import torch
    if router_std is None:
        router_std = 3.0 / np.sqrt(d)
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    out = {}
    for name, shape, std in (("W_r", (E, d), router_std), ("W_gate", (d_ff, d), weight_std),
                             ("W_up", (d_ff, d), weight_std), ("W_down", (d, d_ff), weight_std)):
        a = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
        a.mul_(float(np.float32(std)))
        out[name] = a.to(torch.bfloat16).view(torch.int16)
        del a
    return out


def stack_layer_seed(layer: int, seed: int = 0) -> int:
    return 0x5EED0000 + 64 * seed + layer


def workload_layer(w: Workload, seed: int = 0, layer: int = 0):
    if w.layers > 1:
        s = np.random.SeedSequence(seed).spawn(w.layers + 1)[layer]
    else:
        s = seed
    if w.mlp:
        return make_mlp_layer(w.d, w.d_ff, w.E, s)
    return make_layer(w.d, w.d_ff, w.E, s, skewed=w.skewed)


def workload_tokens(w: Workload, T: int, seed: int = 0):
    if w.layers > 1:
        s = np.random.SeedSequence(seed).spawn(w.layers + 1)[w.layers]
    else:
        s = seed + 1000
    return make_tokens(T, w.d, s, row_lognormal_sigma=w.row_lognormal_sigma,
                       temperature=w.skewed)
