"""Seeded synthetic workloads shaped like the paper's models and data.

The paper fine-tunes GPT2 (12 blocks) and DistilGPT2 (6 blocks), width 768,
vocabulary 50257, tied or untied embeddings (Sec. "Models"), on GLUE prompts of
at most 128 tokens with batch 24 (Sec. "Tasks and Dataset", "Training
Configurations"). No dataset or checkpoint is available here, so every array
below is drawn from a seeded numpy generator with the shapes and value
distributions of those workloads.

Recipe (all draws fp32, then rounded to bf16 by round-to-nearest-even when the
workload is bf16):
  * one independent stream per tensor and example: the [B, T, w] draws of
    example b come from ``np.random.default_rng([seed, tag, b])`` with a fixed
    integer tag per tensor (other shapes: one stream ``default_rng([seed,
    tag])``), so any subset of tensors or examples can be regenerated alone
    and always gets the same values, and examples are drawn in parallel;
  * linear layer l: activations A ~ N(0, a_std) [B,T,d_in] (tag 2l),
    output grads G ~ N(0, g_std) [B,T,d_out] (tag 2l+1); "N(0,s)" means
    standard deviation s;
  * token ids: uniform over V (tiny config) or truncated Zipf, p(k) ~ k^-1.1
    for k = 1..V, id = k-1 (tag 1000);
  * head hidden states H ~ N(0,1) [B,T,d] (tag 1001);
  * logit grads of a causal LM: for t < T-1,
    Gz[t] = (softmax(z_t) - onehot(ids[t+1])) / T with z_t ~ N(0,1) over V
    (tag 1002); the last row has no next token and is zero;
  * input-embedding output grads dE ~ N(0, e_std) [B,T,d] (tag 1003);
  * with ``full_params``: every linear layer's bias shares that layer's G; each
    LayerNorm k (two per block, then the final one) gets normalised inputs
    xhat ~ N(0,1) [B,T,d] (tag 3000+2k) and output grads gy ~ N(0, g_std)
    (tag 3001+2k) for its gain and bias; the position table (1024 rows, or
    2T in the tiny configs) shares the embedding-output grads dE.

bf16 tensors are held as their uint16 bit patterns; fp32 tensors as float32.
Nothing here computes any part of the DP-SGD method.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

__all__ = [
    "GPT2_VOCAB", "GPT2_WIDTH", "GPT2_POSITIONS",
    "f32_to_bf16_bits", "bf16_bits_to_f32",
    "block_linears", "model_linears", "gpt2_param_count",
    "LinearInputs", "HeadInputs", "VectorInputs", "Workload", "CONFIG_NAMES", "make_workload",
    "zipf_ids", "logit_grads", "draw", "draw_ids",
]

GPT2_VOCAB = 50257
GPT2_WIDTH = 768
GPT2_POSITIONS = 1024

TAG_IDS, TAG_H, TAG_Z, TAG_DE = 1000, 1001, 1002, 1003
TAG_LN = 3000


# --------------------------------------------------------------------------
# bf16 encoding
# --------------------------------------------------------------------------
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round to nearest, ties to even); uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


# --------------------------------------------------------------------------
# Model shapes
# --------------------------------------------------------------------------
def block_linears(d: int = GPT2_WIDTH):
    """The four weight matrices of one GPT-2 block as (name, d_in, d_out)."""
    return [("attn.c_attn", d, 3 * d), ("attn.c_proj", d, d),
            ("mlp.c_fc", d, 4 * d), ("mlp.c_proj", 4 * d, d)]


def model_linears(n_blocks: int, d: int = GPT2_WIDTH):
    out = []
    for b in range(n_blocks):
        for name, di, do in block_linears(d):
            out.append((f"h.{b}.{name}", di, do))
    return out


def gpt2_param_count(n_blocks: int, tied: bool, V: int = GPT2_VOCAB,
                     d: int = GPT2_WIDTH, n_pos: int = GPT2_POSITIONS) -> int:
    """Trainable parameters of a GPT-2-style model with these shapes.

    Per block: the four weight matrices and their biases plus two LayerNorms
    (gain and bias); then the final LayerNorm, position embeddings, the token
    embedding and, when untied, a separate output projection of the same size.
    """
    per_block = sum(di * do + do for _, di, do in block_linears(d)) + 2 * (2 * d)
    return n_blocks * per_block + 2 * d + n_pos * d + V * d * (1 if tied else 2)


# --------------------------------------------------------------------------
# Draws
# --------------------------------------------------------------------------
def _rng(seed: int, tag: int, example: Optional[int] = None) -> np.random.Generator:
    key = [int(seed), int(tag)] if example is None else [int(seed), int(tag), int(example)]
    return np.random.default_rng(key)


_POOL: Optional[ThreadPoolExecutor] = None


def _per_example(fn, B: int) -> None:
    """fn(b) for every example b, on a thread pool (numpy's generators and
    ufuncs release the GIL on large arrays)."""
    global _POOL
    if B == 1:
        fn(0)
        return
    if _POOL is None:
        _POOL = ThreadPoolExecutor(max_workers=max(1, min(16, os.cpu_count() or 1)))
    for f in [_POOL.submit(fn, b) for b in range(B)]:
        f.result()


def _normal(seed, tag, shape, std, enc=None) -> np.ndarray:
    """N(0, std) draws of one tensor; a [B, T, w] tensor takes one stream per
    example. enc (optional) encodes each example's draws (fp32 -> bf16 bits)."""
    shape = tuple(int(x) for x in shape)
    if len(shape) != 3:
        x = _rng(seed, tag).standard_normal(size=shape, dtype=np.float32)
        if std != 1.0:
            x *= np.float32(std)
        return x if enc is None else enc(x)
    out = None

    def one(b):
        nonlocal out
        x = _rng(seed, tag, b).standard_normal(size=shape[1:], dtype=np.float32)
        if std != 1.0:
            x *= np.float32(std)
        out[b] = x if enc is None else enc(x)
    probe = np.zeros((1, 1), np.float32) if enc is None else enc(np.zeros((1, 1), np.float32))
    out = np.empty(shape, dtype=probe.dtype)
    _per_example(one, shape[0])
    return out


def zipf_ids(rng: np.random.Generator, shape, V: int, s: float = 1.1) -> np.ndarray:
    """Truncated Zipf over V ids: P(id = k-1) proportional to k^-s, k = 1..V."""
    k = np.arange(1, V + 1, dtype=np.float64)
    p = k ** (-s)
    cdf = np.cumsum(p)
    cdf /= cdf[-1]
    u = rng.random(size=shape)
    ids = np.searchsorted(cdf, u, side="right")
    return np.minimum(ids, V - 1).astype(np.int32)


def logit_grads(z: np.ndarray, ids: np.ndarray) -> np.ndarray:
    """Cross-entropy logit gradients of a causal LM, fp32 [B,T,V].

    Row t is (softmax(z_t) - onehot(ids[t+1])) / T; row T-1 is zero.
    ``z`` is overwritten.
    """
    B, T, V = z.shape
    z -= z.max(axis=-1, keepdims=True)
    np.exp(z, out=z)
    z /= z.sum(axis=-1, keepdims=True)
    bi, ti = np.meshgrid(np.arange(B), np.arange(T - 1), indexing="ij")
    z[bi, ti, ids[:, 1:]] -= np.float32(1.0)
    z[:, T - 1, :] = 0.0
    z /= np.float32(T)
    return z


def draw(seed: int, tag: int, shape, std: float = 1.0, dtype: str = "bf16") -> np.ndarray:
    """One seeded N(0, std) tensor, encoded as bf16 bits or fp32."""
    return _normal(seed, tag, shape, std, f32_to_bf16_bits if dtype == "bf16" else None)


def draw_ids(seed: int, tag: int, shape, V: int, kind: str = "zipf") -> np.ndarray:
    """Seeded token ids: "zipf" (s = 1.1), "uniform", "same" (all one id) or
    "distinct" (a random injection into [0, V); needs the last axis <= V)."""
    rng = _rng(seed, tag)
    if kind == "zipf":
        return zipf_ids(rng, shape, V, 1.1)
    if kind == "uniform":
        return rng.integers(0, V, size=shape, dtype=np.int64).astype(np.int32)
    if kind == "same":
        return np.full(shape, int(rng.integers(0, V)), dtype=np.int32)
    if kind == "distinct":
        flat = np.stack([rng.permutation(V)[: shape[-1]] for _ in range(int(np.prod(shape[:-1])))])
        return flat.reshape(shape).astype(np.int32)
    raise ValueError(kind)


# --------------------------------------------------------------------------
# Workloads
# --------------------------------------------------------------------------
@dataclass
class LinearInputs:
    name: str
    d_in: int
    d_out: int
    A: np.ndarray  # [B,T,d_in]  uint16 bf16 bits or float32
    G: np.ndarray  # [B,T,d_out]


@dataclass
class HeadInputs:
    V: int
    d: int
    ids: np.ndarray            # int32 [B,T]
    dE: np.ndarray             # [B,T,d] grads w.r.t. the input-embedding output
    H: Optional[np.ndarray]    # [B,T,d] hidden states entering the output head
    Gz: Optional[np.ndarray]   # [B,T,ldz] logit grads; columns >= V are zero
    ldz: int
    tied: bool


@dataclass
class VectorInputs:
    """A vector parameter applied to every token: its per-example gradient is
    the sum over tokens of G (a bias; X is None) or of X * G (a LayerNorm gain,
    X the normalised input)."""
    name: str
    d: int
    X: Optional[np.ndarray]    # [B,T,d] or None
    G: np.ndarray              # [B,T,d] (a slice of a linear layer's G for a bias)


@dataclass
class Workload:
    name: str
    dtype: str                 # "bf16" or "f32"
    B: int
    T: int
    C: float
    sigma: float
    linears: List[LinearInputs] = field(default_factory=list)
    head: Optional[HeadInputs] = None
    description: str = ""
    vectors: List[VectorInputs] = field(default_factory=list)
    n_pos: int = 0             # rows of the position table (0: no position embedding)

    def n_coordinates(self) -> int:
        n = sum(l.d_in * l.d_out for l in self.linears)
        if self.head is not None:
            h = self.head
            n += h.V * h.d * (1 if (h.tied or h.H is None) else 2)
        n += sum(v.d for v in self.vectors)
        if self.n_pos:
            n += self.n_pos * self.head.d
        return n


CONFIG_NAMES = ("c1", "c1-tied", "c2", "c3", "c4", "c5", "gpt2-step", "gpt2-full")

_DEFAULTS = {
    # name: (dtype, B, T, n_blocks, head kind, description)
    "c1": ("f32", 4, 16, None, "embed",
           "tiny untied toy: one 64->64 linear, embedding V=512 x d=64, fp32"),
    "c1-tied": ("f32", 4, 16, None, "tied",
                "tiny tied toy: one 64->64 linear, tied V=512 x d=64 head, fp32"),
    "c2": ("bf16", 32, 128, 12, None,
           "GPT-2-small body, untied: 12 blocks x 4 linears, B=32 T=128, bf16"),
    "c3": ("bf16", 32, 128, 0, "tied",
           "GPT-2-small tied head: V=50257 d=768, Zipf ids, B=32 T=128, bf16"),
    "c4": ("bf16", 64, 256, 6, "tied",
           "DistilGPT2-shaped tied step: 6 blocks + tied head, B=64 T=256, bf16"),
    "c5": ("bf16", 16, 1024, 12, "untied",
           "long-sequence GPT-2-small untied step: 12 blocks + head + E_in, B=16 T=1024, bf16"),
    "gpt2-step": ("bf16", 32, 128, 12, "tied",
                  "GPT-2-small tied step: 12 blocks + tied V=50257 head, B=32 T=128, bf16"),
    "gpt2-full": ("bf16", 32, 128, 12, "tied",
                  "GPT-2-small tied step, every parameter (weights, biases, LayerNorms, "
                  "position table, tied embedding): 124,439,808 coordinates, B=32 T=128, bf16"),
}


def make_workload(name: str, seed: int = 0, *, B: Optional[int] = None,
                  T: Optional[int] = None, n_blocks: Optional[int] = None,
                  layers: Optional[List[int]] = None, ldz: Optional[int] = None,
                  V: Optional[int] = None, d: Optional[int] = None,
                  with_head: bool = True, C: float = 1.0,
                  sigma: float = 1.0, full_params: bool = False) -> Workload:
    """Draw the inputs of one named workload (optionally at reduced size).

    ``layers`` selects a subset of the linear layers by index (each keeps the
    values it has in the full workload). ``ldz`` pads logit-grad rows to a
    row stride >= V with zeros. ``full_params`` adds the remaining GPT-2
    parameters: linear biases, LayerNorm gains and biases (two per block and a
    final one) and the position table (needs the head's embedding inputs).
    """
    if name not in _DEFAULTS:
        raise KeyError(f"unknown workload {name!r}; choose from {CONFIG_NAMES}")
    dtype, B0, T0, nb0, head_kind, desc = _DEFAULTS[name]
    full_params = full_params or name == "gpt2-full"
    B = B0 if B is None else int(B)
    T = T0 if T is None else int(T)
    if B <= 0 or T <= 0:
        raise ValueError("B and T must be positive")
    enc = f32_to_bf16_bits if dtype == "bf16" else (lambda x: np.ascontiguousarray(x, np.float32))

    if name.startswith("c1"):
        dd = 64 if d is None else int(d)
        shapes = [("linear", dd, dd)]
        a_std, g_std, e_std = 1.0, 0.01, 0.01
        Vh = 512 if V is None else int(V)
    else:
        dd = GPT2_WIDTH if d is None else int(d)
        nb = nb0 if n_blocks is None else int(n_blocks)
        shapes = model_linears(nb, dd)
        a_std, g_std, e_std = 1.0, 1e-3, 1e-3
        Vh = GPT2_VOCAB if V is None else int(V)

    wl = Workload(name=name, dtype=dtype, B=B, T=T, C=C, sigma=sigma, description=desc)
    idx = range(len(shapes)) if layers is None else layers
    for l in idx:
        lname, di, do = shapes[l]
        A = _normal(seed, 2 * l, (B, T, di), a_std, enc)
        G = _normal(seed, 2 * l + 1, (B, T, do), g_std, enc)
        wl.linears.append(LinearInputs(lname, di, do, A, G))

    if head_kind is None or not with_head:
        return wl

    rng_ids = _rng(seed, TAG_IDS)
    if name.startswith("c1"):
        ids = rng_ids.integers(0, Vh, size=(B, T), dtype=np.int64).astype(np.int32)
    else:
        ids = zipf_ids(rng_ids, (B, T), Vh, 1.1)
    dE = _normal(seed, TAG_DE, (B, T, dd), e_std, enc)
    H = Gz = None
    ldz_eff = Vh if ldz is None else int(ldz)
    if ldz_eff < Vh:
        raise ValueError("ldz must be >= V")
    if head_kind in ("tied", "untied"):
        H = _normal(seed, TAG_H, (B, T, dd), 1.0, enc)
        Gz = None

        def one(b):
            # example b's logits, its logit gradients, padded to ldz, encoded
            z = _rng(seed, TAG_Z, b).standard_normal(size=(1, T, Vh), dtype=np.float32)
            gz = logit_grads(z, ids[b:b + 1])[0]
            if ldz_eff > Vh:
                pad = np.zeros((T, ldz_eff), dtype=np.float32)
                pad[:, :Vh] = gz
                gz = pad
            Gz[b] = enc(gz)
        probe = enc(np.zeros((1, 1), np.float32))
        Gz = np.empty((B, T, ldz_eff), dtype=probe.dtype)
        _per_example(one, B)
    wl.head = HeadInputs(V=Vh, d=dd, ids=ids, dE=dE, H=H, Gz=Gz, ldz=ldz_eff,
                         tied=(head_kind == "tied"))
    if full_params:
        _add_full_params(wl, seed, enc, g_std, n_blocks=(1 if name.startswith("c1") else nb),
                         n_pos=(2 * T if name.startswith("c1") else GPT2_POSITIONS))
    return wl


def _add_full_params(wl: Workload, seed: int, enc, g_std: float, n_blocks: int,
                     n_pos: int) -> None:
    """Biases of the linear layers, LayerNorm gains and biases, position table."""
    B, T, d = wl.B, wl.T, wl.head.d
    if T > n_pos:
        raise ValueError(f"T = {T} exceeds the position table ({n_pos} rows)")
    for lin in wl.linears:
        wl.vectors.append(VectorInputs(lin.name + ".bias", lin.d_out, None, lin.G))
    names = [f"h.{b}.{ln}" for b in range(n_blocks) for ln in ("ln_1", "ln_2")] + ["ln_f"]
    for k, name in enumerate(names):
        xhat = _normal(seed, TAG_LN + 2 * k, (B, T, d), 1.0, enc)
        gy = _normal(seed, TAG_LN + 2 * k + 1, (B, T, d), g_std, enc)
        wl.vectors.append(VectorInputs(name + ".weight", d, xhat, gy))
        wl.vectors.append(VectorInputs(name + ".bias", d, None, gy))
    wl.n_pos = n_pos
