"""fp64 CPU oracle for the DP-SGD ghost-clipping hot path.

TEST INFRASTRUCTURE. Only the test suite, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run this module. The GPU
library never calls it, and it shares no code with the GPU library.

It follows the definitions, not the fast identities: every per-example
gradient is materialised in fp64 and its norm taken directly.

  * DP-SGD (Sec. "Differentially Private Stochastic Gradient Descent"):
    per-example gradient g_i; clipped gradient g_i * min(1, C/||g_i||)
    (eq. 2); privatised gradient (sum of clipped gradients + N(0, s^2 C^2 I))
    divided by the batch size (eq. 3).
  * Ghost clipping (Sec. "Ghost Clipping Mechanism"): a linear layer's
    per-example weight gradient is built from activations a and
    back-propagated errors delta (eq. 4, one outer product per token, summed
    over the tokens of the example); the squared norm of the whole gradient is
    the sum of the per-layer squared norms (eq. 6, eq. 10); clip factor
    R_i = min(1, C/||g_i||) (eq. 7).
  * Weight tying (Sec. "Weight Tying in Decoder-Only LLMs", eq. 8): the output
    projection is the embedding matrix E in R^{V x d}; the tied gradient is the
    sum of the input-embedding and output-projection contributions, whose
    squared norm carries the cross term 2<g_in, g_out> (eq. 11, eq. 13).

Readings taken where the paper is silent:
  * ||g_i|| = 0 gives R_i = 1 (the limit of min(1, C/x) as x -> 0).
  * A squared norm that is not finite gives R_i = 0 (min(1, C/inf) = 0; NaN
    is read the same way), and such an example is left out of every clipped
    sum rather than multiplied by 0, so the bound of eq. 2 holds for it.
  * The batch divisor of eq. 3 is the actual batch size B.
  * "N(0, s^2 C^2 I)" is drawn with standard deviation s*C per coordinate; a
    tied matrix is one tensor and is noised once.
  * Gaussians come from the Philox4x32-10 counter-based generator (Salmon et
    al., SC'11) and the Box-Muller transform (Box & Muller, 1958), keyed by
    (seed, tensor_id, step); see ``gaussian``.
  * Gradient layout is [d_in, d_out] (activations on the rows); norms do not
    depend on it.
  * The parameters the paper counts besides the weight matrices (its table of
    trainable-parameter counts: biases, LayerNorm gains and biases, position
    embeddings) enter the flat norm of eq. 6 like every other parameter; their
    per-example gradients follow from the chain rule (``vector_grad``,
    ``positional_grad``).
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import numpy as np

__all__ = [
    "decode", "linear_grad", "embedding_grad", "head_grad", "sqnorm",
    "linear_norm2", "embedding_norm2", "head_norm2", "tied_cross", "tied_norm2",
    "buckets", "clip_factors", "clipped_sum_linear", "clipped_sum_embedding",
    "clipped_sum_head", "vector_grad", "positional_grad", "vector_norm2", "positional_norm2",
    "clipped_sum_vector", "clipped_sum_positional", "philox4x32_10", "gaussian", "add_noise",
    "per_example_norms", "step",
]


# --------------------------------------------------------------------------
# Input decoding (exact)
# --------------------------------------------------------------------------
def decode(x: np.ndarray, dtype: str) -> np.ndarray:
    """Widen stored inputs exactly to fp64: bf16 bit patterns or fp32 values."""
    if dtype == "bf16":
        u = np.asarray(x, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return u.view(np.float32).astype(np.float64)
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


# --------------------------------------------------------------------------
# Per-example gradients (materialised)
# --------------------------------------------------------------------------
def linear_grad(A_i: np.ndarray, G_i: np.ndarray) -> np.ndarray:
    """Per-example weight gradient of one linear layer, [d_in, d_out].

    eq. 4 gives the gradient of one token as the outer product of its error
    signal and its activation; over the T tokens of an example the layer's
    gradient is the sum of those outer products, i.e. A_i^T G_i.
    """
    return A_i.T @ G_i


def embedding_grad(ids_i: np.ndarray, dE_i: np.ndarray, V: int) -> np.ndarray:
    """Per-example gradient of the input-embedding lookup, [V, d].

    The lookup reads row ids[t] of E (eq. 8 context) for each token, so the
    gradient of that row is the sum of the output-gradients of the tokens that
    carry that id; all other rows are zero.
    """
    g = np.zeros((V, dE_i.shape[1]), dtype=np.float64)
    np.add.at(g, ids_i, dE_i)
    return g


def head_grad(H_i: np.ndarray, Gz_i: np.ndarray, V: int) -> np.ndarray:
    """Per-example gradient of the output projection W_out, [V, d].

    logits = H W_out^T, so dL/dW_out = Gz^T H over the example's tokens.
    ``Gz_i`` may carry padding columns beyond V; they are ignored.
    """
    return Gz_i[:, :V].T @ H_i


def vector_grad(X_i: Optional[np.ndarray], G_i: np.ndarray) -> np.ndarray:
    """Per-example gradient of a vector parameter applied to every token, [d].

    A bias b enters every token's output as y_t = ... + b, so its gradient is
    the sum over tokens of the output grads G_t (X_i is None). A LayerNorm gain
    enters as y_t = gamma * xhat_t + beta, so its gradient is the sum over tokens
    of xhat_t * G_t (X_i = xhat), and the LayerNorm bias is again the plain sum.
    """
    return G_i.sum(axis=0) if X_i is None else (X_i * G_i).sum(axis=0)


def positional_grad(dE_i: np.ndarray, n_pos: int) -> np.ndarray:
    """Per-example gradient of a learned position table, [n_pos, d].

    Token t adds row t of the table to its input embedding, so row t receives
    that token's embedding-output grad dE_t; rows at or past T receive nothing.
    """
    g = np.zeros((n_pos, dE_i.shape[1]), dtype=np.float64)
    g[: dE_i.shape[0]] = dE_i
    return g


def sqnorm(g: np.ndarray) -> float:
    return float(np.sum(g * g))


# --------------------------------------------------------------------------
# Per-example squared norms
# --------------------------------------------------------------------------
def linear_norm2(A: np.ndarray, G: np.ndarray) -> np.ndarray:
    """||A_i^T G_i||_F^2 per example, by materialising the gradient."""
    return np.array([sqnorm(linear_grad(A[i], G[i])) for i in range(A.shape[0])])


def embedding_norm2(ids: np.ndarray, dE: np.ndarray, V: int) -> np.ndarray:
    return np.array([sqnorm(embedding_grad(ids[i], dE[i], V)) for i in range(ids.shape[0])])


def head_norm2(H: np.ndarray, Gz: np.ndarray, V: int) -> np.ndarray:
    return np.array([sqnorm(head_grad(H[i], Gz[i], V)) for i in range(H.shape[0])])


def vector_norm2(X: Optional[np.ndarray], G: np.ndarray) -> np.ndarray:
    return np.array([sqnorm(vector_grad(None if X is None else X[i], G[i]))
                     for i in range(G.shape[0])])


def positional_norm2(dE: np.ndarray, n_pos: int) -> np.ndarray:
    return np.array([sqnorm(positional_grad(dE[i], n_pos)) for i in range(dE.shape[0])])


def tied_cross(ids, dE, H, Gz, V) -> np.ndarray:
    """<g_in,i, g_out,i>: the interaction term of eq. 11, by materialising both."""
    out = np.empty(ids.shape[0])
    for i in range(ids.shape[0]):
        out[i] = float(np.sum(embedding_grad(ids[i], dE[i], V) * head_grad(H[i], Gz[i], V)))
    return out


def tied_norm2(ids, dE, H, Gz, V) -> np.ndarray:
    """||g_in + g_out||^2 of the shared matrix, taken directly (eq. 13 left side)."""
    out = np.empty(ids.shape[0])
    for i in range(ids.shape[0]):
        g = embedding_grad(ids[i], dE[i], V) + head_grad(H[i], Gz[i], V)
        out[i] = sqnorm(g)
    return out


def buckets(ids: np.ndarray):
    """Token buckets of each example: dense rank of every id, and #unique ids.

    seg_id[i, t] is the position of ids[i, t] among the sorted distinct ids of
    example i; n_unique[i] is the number of distinct ids.
    """
    B, T = ids.shape
    seg = np.empty((B, T), dtype=np.int32)
    nu = np.empty(B, dtype=np.int32)
    for i in range(B):
        uniq, inv = np.unique(ids[i], return_inverse=True)
        seg[i] = inv.reshape(-1)
        nu[i] = len(uniq)
    return seg, nu


# --------------------------------------------------------------------------
# Clipping and the clipped sum
# --------------------------------------------------------------------------
def clip_factors(norm2: np.ndarray, C: float) -> np.ndarray:
    """R_i = min(1, C / ||g_i||) (eq. 2, eq. 7), with R_i = 1 when ||g_i|| = 0
    and R_i = 0 when ||g_i||^2 is not finite (inf, where min(1, C/inf) = 0,
    and NaN, read the same way so that such an example can never enter the
    sum unclipped)."""
    n2 = np.asarray(norm2, dtype=np.float64)
    c = np.zeros(n2.shape)
    fin = np.isfinite(n2)
    n = np.sqrt(np.where(fin & (n2 > 0), n2, 1.0))
    c[fin] = np.where(n2[fin] > 0, np.minimum(1.0, C / n[fin]), 1.0)
    return c


def _kept(c, i) -> bool:
    """An example with R_i = 0 contributes nothing to a clipped sum: it is
    left out rather than multiplied by 0 (0 * inf would be NaN)."""
    return c[i] != 0.0


def clipped_sum_linear(A, G, c) -> np.ndarray:
    """sum_i c_i g_i for one linear layer (the bracket of eq. 3 without noise)."""
    S = np.zeros((A.shape[2], G.shape[2]))
    for i in range(A.shape[0]):
        if _kept(c, i):
            S += c[i] * linear_grad(A[i], G[i])
    return S


def clipped_sum_embedding(ids, dE, c, V) -> np.ndarray:
    S = np.zeros((V, dE.shape[2]))
    for i in range(ids.shape[0]):
        if _kept(c, i):
            S += c[i] * embedding_grad(ids[i], dE[i], V)
    return S


def clipped_sum_head(H, Gz, c, V) -> np.ndarray:
    S = np.zeros((V, H.shape[2]))
    for i in range(H.shape[0]):
        if _kept(c, i):
            S += c[i] * head_grad(H[i], Gz[i], V)
    return S


def clipped_sum_vector(X: Optional[np.ndarray], G: np.ndarray, c) -> np.ndarray:
    S = np.zeros(G.shape[2])
    for i in range(G.shape[0]):
        if _kept(c, i):
            S += c[i] * vector_grad(None if X is None else X[i], G[i])
    return S


def clipped_sum_positional(dE: np.ndarray, c, n_pos: int) -> np.ndarray:
    S = np.zeros((n_pos, dE.shape[2]))
    for i in range(dE.shape[0]):
        if _kept(c, i):
            S += c[i] * positional_grad(dE[i], n_pos)
    return S


# --------------------------------------------------------------------------
# Noise: Philox4x32-10 + Box-Muller
# --------------------------------------------------------------------------
_MASK32 = np.uint64(0xFFFFFFFF)
# Philox4x32 round multipliers and key increments (Salmon et al., SC'11).
_PHILOX_M = (np.uint64(0xD2511F53), np.uint64(0xCD9E8D57))
_PHILOX_W = (np.uint64(0x9E3779B9), np.uint64(0xBB67AE85))


def philox4x32_10(ctr: Sequence[np.ndarray], key: Sequence[int]):
    """Philox4x32 with 10 rounds on arrays of 32-bit counters.

    Each round multiplies counter words 0 and 2 by the two round constants,
    keeps both 32-bit halves of the 64-bit products, and mixes them with words
    1 and 3 and the key; the key is advanced by the Weyl increments between
    rounds. Returns four uint32 arrays.
    """
    c = [np.asarray(x, dtype=np.uint64) & _MASK32 for x in ctr]
    k0 = np.uint64(int(key[0]) & 0xFFFFFFFF)
    k1 = np.uint64(int(key[1]) & 0xFFFFFFFF)
    for r in range(10):
        if r:
            k0 = (k0 + _PHILOX_W[0]) & _MASK32
            k1 = (k1 + _PHILOX_W[1]) & _MASK32
        p0 = _PHILOX_M[0] * c[0]
        p1 = _PHILOX_M[1] * c[2]
        hi0, lo0 = p0 >> np.uint64(32), p0 & _MASK32
        hi1, lo1 = p1 >> np.uint64(32), p1 & _MASK32
        c = [hi1 ^ c[1] ^ k0, lo1, hi0 ^ c[3] ^ k1, lo0]
    return [x.astype(np.uint32) for x in c]


def gaussian(n: int, seed: int, tensor_id: int, step: int, start: int = 0) -> np.ndarray:
    """Standard normal draws z[start : start+n] of one tensor, fp64.

    Element j uses Philox block j // 4 with key (seed low word, seed high word)
    and counter (block low word, block high word, tensor_id, step); the four
    32-bit outputs x_0..x_3 become uniforms u_a = (x_a + 1/2) 2^-32 in (0, 1),
    and Box-Muller turns (u_0, u_1) into (r cos t, r sin t) and (u_2, u_3)
    likewise, with r = sqrt(-2 ln u_even) and t = 2 pi u_odd. Element j takes
    output number j % 4.
    """
    if n == 0:
        return np.zeros(0)
    j = np.arange(start, start + n, dtype=np.uint64)
    blk = j >> np.uint64(2)
    blocks = np.unique(blk)
    x = philox4x32_10([blocks & _MASK32, blocks >> np.uint64(32),
                       np.full(blocks.shape, tensor_id & 0xFFFFFFFF, np.uint64),
                       np.full(blocks.shape, step & 0xFFFFFFFF, np.uint64)],
                      (seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF))
    u = [(xa.astype(np.float64) + 0.5) * 2.0 ** -32 for xa in x]
    r01 = np.sqrt(-2.0 * np.log(u[0]))
    r23 = np.sqrt(-2.0 * np.log(u[2]))
    z = np.stack([r01 * np.cos(2 * np.pi * u[1]), r01 * np.sin(2 * np.pi * u[1]),
                  r23 * np.cos(2 * np.pi * u[3]), r23 * np.sin(2 * np.pi * u[3])], axis=1)
    rows = np.searchsorted(blocks, blk)
    return z[rows, (j & np.uint64(3)).astype(np.int64)]


def add_noise(S: np.ndarray, sigma: float, C: float, B: int, seed: int,
              tensor_id: int, step: int) -> np.ndarray:
    """(S + N(0, sigma^2 C^2 I)) / B, eq. 3; B = 0 means no division."""
    z = gaussian(S.size, seed, tensor_id, step).reshape(S.shape)
    out = S + sigma * C * z
    return out / B if B else out


# --------------------------------------------------------------------------
# The whole step on a workload (duck-typed: see workloads.gen.Workload)
# --------------------------------------------------------------------------
def per_example_norms(wl, examples: Optional[List[int]] = None) -> Dict[str, np.ndarray]:
    """Every squared-norm term of the examples listed (default: all)."""
    ex = list(range(wl.B)) if examples is None else list(examples)
    dt = wl.dtype
    out: Dict[str, np.ndarray] = {}
    lin = np.zeros((len(wl.linears), len(ex)))
    for l, L in enumerate(wl.linears):
        for k, i in enumerate(ex):
            lin[l, k] = sqnorm(linear_grad(decode(L.A[i], dt), decode(L.G[i], dt)))
    out["linear"] = lin
    total = lin.sum(axis=0)
    h = wl.head
    if h is not None:
        V = h.V
        n_in = np.zeros(len(ex)); n_out = np.zeros(len(ex))
        cross = np.zeros(len(ex)); tied = np.zeros(len(ex))
        for k, i in enumerate(ex):
            gE = embedding_grad(h.ids[i], decode(h.dE[i], dt), V)
            n_in[k] = sqnorm(gE)
            if h.H is not None:
                gW = head_grad(decode(h.H[i], dt), decode(h.Gz[i], dt), V)
                n_out[k] = sqnorm(gW)
                cross[k] = float(np.sum(gE * gW))
                if h.tied:
                    tied[k] = sqnorm(gE + gW)
                del gW
            del gE
        out["in"], out["out"], out["cross"] = n_in, n_out, cross
        if h.H is not None and h.tied:
            out["tied"] = tied
            total = total + tied
        else:
            total = total + n_in + n_out
    vecs = getattr(wl, "vectors", [])
    if vecs:
        vn = np.zeros((len(vecs), len(ex)))
        for v, vec in enumerate(vecs):
            for k, i in enumerate(ex):
                X = None if vec.X is None else decode(vec.X[i], dt)
                vn[v, k] = sqnorm(vector_grad(X, decode(vec.G[i], dt)))
        out["vector"] = vn
        total = total + vn.sum(axis=0)
    if getattr(wl, "n_pos", 0):
        pos = np.array([sqnorm(positional_grad(decode(h.dE[i], dt), wl.n_pos)) for i in ex])
        out["pos"] = pos
        total = total + pos
    out["total"] = total
    return out


def step(wl, seed: int = 0, step_id: int = 0, examples: Optional[List[int]] = None,
         noise: bool = True) -> Dict[str, object]:
    """One DP-SGD aggregation on the listed examples: norms, clip, sums, noise.

    Tensor ids for the noise: linear layer l uses l; then the input embedding
    (or the tied matrix) uses L, and an untied output head uses L+1; the vector
    parameters follow in their order, then the position table.
    """
    ex = list(range(wl.B)) if examples is None else list(examples)
    dt = wl.dtype
    norms = per_example_norms(wl, ex)
    c = clip_factors(norms["total"], wl.C)
    sums: Dict[str, np.ndarray] = {}
    L = len(wl.linears)
    for l, lay in enumerate(wl.linears):
        S = np.zeros((lay.d_in, lay.d_out))
        for k, i in enumerate(ex):
            if not _kept(c, k):
                continue
            S += c[k] * linear_grad(decode(lay.A[i], dt), decode(lay.G[i], dt))
        sums[lay.name] = S
    h = wl.head
    if h is not None:
        SE = np.zeros((h.V, h.d))
        for k, i in enumerate(ex):
            if not _kept(c, k):
                continue
            SE += c[k] * embedding_grad(h.ids[i], decode(h.dE[i], dt), h.V)
        if h.H is not None:
            SW = np.zeros((h.V, h.d))
            for k, i in enumerate(ex):
                if not _kept(c, k):
                    continue
                SW += c[k] * head_grad(decode(h.H[i], dt), decode(h.Gz[i], dt), h.V)
            if h.tied:
                sums["wte"] = SE + SW
            else:
                sums["wte"], sums["lm_head"] = SE, SW
        else:
            sums["wte"] = SE
    for vec in getattr(wl, "vectors", []):
        S = np.zeros(vec.d)
        for k, i in enumerate(ex):
            if not _kept(c, k):
                continue
            X = None if vec.X is None else decode(vec.X[i], dt)
            S += c[k] * vector_grad(X, decode(vec.G[i], dt))
        sums[vec.name] = S
    if getattr(wl, "n_pos", 0):
        SP = np.zeros((wl.n_pos, h.d))
        for k, i in enumerate(ex):
            if not _kept(c, k):
                continue
            SP += c[k] * positional_grad(decode(h.dE[i], dt), wl.n_pos)
        sums["wpe"] = SP
    noisy: Dict[str, np.ndarray] = {}
    if noise:
        names = [lay.name for lay in wl.linears] + [n for n in ("wte", "lm_head") if n in sums]
        names += [vec.name for vec in getattr(wl, "vectors", [])]
        names += ["wpe"] if "wpe" in sums else []
        for tid, name in enumerate(names):
            noisy[name] = add_noise(sums[name], wl.sigma, wl.C, len(ex), seed, tid, step_id)
    return {"norms": norms, "c": c, "sums": sums, "noisy": noisy}
