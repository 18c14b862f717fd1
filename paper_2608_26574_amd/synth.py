"""Seeded synthetic inputs shaped like the paper's decoding workloads.

This module only draws random numbers and names workload shapes: random-init
model weights, prompt ids, per-position token states with their confidences.
It holds none of the decoding method's arithmetic and is the only code that the
HIP path's tests and the CPU oracle both use.

Recipes (seeds: weights 1, inputs 2, per-step state draw 1000 + t):
  * weights ~ N(0, 0.02) rounded to the storage type; RMSNorm gains
    1 + N(0, 0.02) so that the gain multiply is exercised;
  * prompt / candidate ids uniform on [0, V-1); id V-1 is [Mask];
  * tiny block states i.i.d. M/C/U with p = 0.5/0.25/0.25;
  * workload states: n_C = round(f*B) candidates, the rest split evenly into
    M (rounded up) and U, positions from a random permutation, candidate
    confidences distinct and uniform in (tau_c, tau_u], U confidences in
    (tau_u, 1), M confidences in [0, tau_c].
"""
from __future__ import annotations

import math
from dataclasses import dataclass, asdict

import numpy as np
import torch

STATE_M, STATE_C, STATE_U = 0, 1, 2


@dataclass(frozen=True)
class Dims:
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    max_pos: int
    dtype: str          # 'bf16' or 'f32'
    norm_eps: float = 1e-5
    rope_theta: float = 10000.0
    kv_dtype: str = ""  # KV-cache storage: "" = dtype, "fp8" = OCP FP8 E4M3 (bf16 models)

    def as_dict(self):
        return asdict(self)

    @property
    def mask_id(self):
        return self.vocab - 1


# Model shapes of the workloads (random-init; no trained weights exist here).
TINY = Dims(2, 256, 4, 4, 64, 1024, 2048, 4096, "f32")
LLADA8B = Dims(32, 4096, 32, 32, 128, 12288, 126464, 4096, "bf16")
DREAM7B = Dims(28, 3584, 28, 4, 128, 18944, 152064, 4096, "bf16")


def truncated(dims: Dims, n_layers: int) -> Dims:
    d = dims.as_dict()
    d["n_layers"] = n_layers
    return Dims(**d)


def with_fp8_kv(dims: Dims) -> Dims:
    d = dims.as_dict()
    d["kv_dtype"] = "fp8"
    return Dims(**d)


def torch_dtype(dims: Dims):
    return torch.bfloat16 if dims.dtype == "bf16" else torch.float32


def weight_shapes(dims: Dims):
    """Logical weight list: name -> shape ([out, in] for projections)."""
    d, F, V = dims.d_model, dims.ffn_dim, dims.vocab
    qd = dims.n_heads * dims.head_dim
    kd = dims.n_kv_heads * dims.head_dim
    shapes = [("embed", (V, d))]
    for layer in range(dims.n_layers):
        p = f"layers.{layer}."
        shapes += [(p + "attn_norm", (d,)), (p + "wq", (qd, d)), (p + "wk", (kd, d)),
                   (p + "wv", (kd, d)), (p + "wo", (d, qd)), (p + "ffn_norm", (d,)),
                   (p + "w_gate", (F, d)), (p + "w_up", (F, d)), (p + "w_down", (d, F))]
    shapes += [("final_norm", (d,)), ("lm_head", (V, d))]
    return shapes


def make_weights(dims: Dims, seed: int = 1, device="cpu", std: float = 0.02):
    """Random-init weights in the logical layout, as torch tensors of the
    storage dtype on ``device``.  Returns an ordered dict name -> tensor."""
    g = torch.Generator(device=device).manual_seed(seed)
    out = {}
    for name, shape in weight_shapes(dims):
        x = torch.randn(shape, generator=g, device=device, dtype=torch.float32) * std
        if name.endswith("norm"):
            x = x + 1.0
        out[name] = x.to(torch_dtype(dims))
    return out


class OracleWeights:
    """float64 numpy view of the weights in the nesting the oracle reads
    (``w['embed']``, ``w['layers'][l]['wq']``, ...).  Layers are converted on
    access so that a 32-layer model never sits in host memory as float64.
    With ``host_copy`` every tensor is first copied once into host memory as
    float32 (exact for bf16 and fp32 values), so that repeated passes over a
    deep model convert from there instead of fetching it again."""

    def __init__(self, dims: Dims, tensors, host_copy: bool = False):
        self.dims = dims
        self.t = tensors
        if host_copy:
            self.t = {k: v.detach().to("cpu", torch.float32).numpy() for k, v in tensors.items()}
        self.layers = _LayerView(self)

    @staticmethod
    def _np(t):
        if isinstance(t, np.ndarray):
            return t.astype(np.float64)
        return t.detach().to("cpu", torch.float32).numpy().astype(np.float64)

    def __getitem__(self, key):
        if key == "layers":
            return self.layers
        return self._np(self.t[key])


class _LayerView:
    def __init__(self, parent):
        self.p = parent

    def __len__(self):
        return self.p.dims.n_layers

    def __getitem__(self, layer):
        pre = f"layers.{layer}."
        names = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")
        return {n: self.p._np(self.p.t[pre + n]) for n in names}


def prompt_ids(b: int, P: int, vocab: int, seed: int = 2):
    rng = np.random.default_rng(seed)
    return rng.integers(0, vocab - 1, size=(b, P), dtype=np.int64).astype(np.int32)


def tiny_block(b: int, B: int, vocab: int, seed: int = 2, tau_c=0.4, tau_u=0.9):
    """Block of the tiny workload: states i.i.d. M/C/U with p = .5/.25/.25."""
    rng = np.random.default_rng(seed)
    state = rng.choice(3, size=(b, B), p=[0.5, 0.25, 0.25]).astype(np.uint8)
    tok = rng.integers(0, vocab - 1, size=(b, B)).astype(np.int32)
    tok[state == STATE_M] = vocab - 1
    conf = _confs(rng, state, tau_c, tau_u)
    return tok, state, conf


def _confs(rng, state, tau_c, tau_u):
    """Confidences consistent with the thresholds; C confidences distinct."""
    conf = np.zeros(state.shape, dtype=np.float32)
    nM = int((state == STATE_M).sum())
    nU = int((state == STATE_U).sum())
    conf[state == STATE_M] = rng.uniform(0.0, tau_c, size=nM)
    conf[state == STATE_U] = rng.uniform(tau_u, 1.0, size=nU) + 1e-6
    for row in range(state.shape[0]):
        idx = np.nonzero(state[row] == STATE_C)[0]
        if len(idx):
            # distinct values in (tau_c, tau_u]: a shuffled even grid plus jitter
            grid = tau_c + (tau_u - tau_c) * (np.arange(len(idx)) + 0.5 +
                                              0.25 * rng.uniform(-1, 1, len(idx))) / len(idx)
            conf[row, idx] = rng.permutation(grid)
    return np.minimum(conf, np.float32(1.0))


def workload_block(b: int, B: int, cand_frac: float, vocab: int, seed: int,
                   tau_c=0.4, tau_u=0.9):
    """Block states of the attention / full-step workloads: n_C = round(f*B),
    n_M = ceil((B - n_C) / 2), n_U = the rest; positions permuted per sequence."""
    rng = np.random.default_rng(seed)
    nC = int(round(cand_frac * B))
    nM = int(math.ceil((B - nC) / 2))
    base = np.array([STATE_C] * nC + [STATE_M] * nM + [STATE_U] * (B - nC - nM), dtype=np.uint8)
    state = np.stack([rng.permutation(base) for _ in range(b)]).astype(np.uint8)
    tok = rng.integers(0, vocab - 1, size=(b, B)).astype(np.int32)
    tok[state == STATE_M] = vocab - 1
    conf = _confs(rng, state, tau_c, tau_u)
    return tok, state, conf


def qkv(b: int, rows: int, n_heads: int, n_kv: int, dh: int, keys: int, seed: int = 2,
        dtype=torch.bfloat16, device="cpu"):
    """Q [b, rows, Hq, dh] and K/V caches [b, Hkv, keys, dh], N(0, 1)."""
    g = torch.Generator(device=device).manual_seed(seed)
    q = torch.randn((b, rows, n_heads, dh), generator=g, device=device).to(dtype)
    k = torch.randn((b, n_kv, keys, dh), generator=g, device=device).to(dtype)
    v = torch.randn((b, n_kv, keys, dh), generator=g, device=device).to(dtype)
    return q, k, v
