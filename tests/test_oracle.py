"""Pins of the fp64 oracle against facts fixed outside the oracle itself.

Each pin checks the oracle against something it does not compute the same way:
torch autograd on a small model, a closed form the paper prints (eq. 5), the
decomposition the paper writes for tied weights (eq. 11/13), an independent
algebraic identity (the Gram form of the Frobenius norm), the Philox published
known-answer vectors, distribution statistics, or plain integer brute force.
The mutation tests at the end plant plausible mistakes in a copy of the oracle
and check that some pin catches each one.
"""
import os
import types

import numpy as np
import pytest
import torch

import oracle as O
from workloads import gen

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
RNG = np.random.default_rng(12345)


def _rand(*shape, scale=1.0):
    return RNG.standard_normal(shape) * scale


# ---------------------------------------------------------------------------
# Pin 1: per-example linear gradient and its norm
# ---------------------------------------------------------------------------
def check_linear_grad_autograd(o, B=3, T=5, d_in=4, d_out=6):
    """Per-example dL/dW of y = x W (W [d_in, d_out]) from autograd."""
    A = _rand(B, T, d_in)
    R = _rand(B, T, d_out)
    W = torch.tensor(_rand(d_in, d_out), dtype=torch.float64, requires_grad=True)
    for i in range(B):
        W.grad = None
        y = torch.tensor(A[i]) @ W
        (y * torch.tensor(R[i])).sum().backward()   # dL/dy = R
        g_ref = W.grad.numpy()
        g = o.linear_grad(A[i], R[i])
        assert g.shape == g_ref.shape
        np.testing.assert_allclose(g, g_ref, rtol=1e-12, atol=1e-12)
        assert abs(o.sqnorm(g) - float((W.grad ** 2).sum())) <= 1e-12 * max(1.0, o.sqnorm(g))


def test_linear_grad_matches_autograd():
    check_linear_grad_autograd(O)


@pytest.mark.parametrize("T", [1, 2, 3, 16, 17])
@pytest.mark.parametrize("d_in,d_out", [(1, 1), (5, 3), (64, 64), (1, 5)])
def test_linear_norm_equals_gram_identity(T, d_in, d_out):
    """||A^T G||_F^2 = sum_{t,s} (A A^T)_{ts} (G G^T)_{ts}: an independent formula."""
    B = 3
    A = _rand(B, T, d_in)
    G = _rand(B, T, d_out, scale=1e-2)
    got = O.linear_norm2(A, G)
    for i in range(B):
        gram = float(np.sum((A[i] @ A[i].T) * (G[i] @ G[i].T)))
        assert abs(got[i] - gram) <= 1e-11 * abs(gram)


def test_linear_norm_T1_closed_form():
    """eq. 5: with one token the norm is ||delta||^2 ||a||^2."""
    A = _rand(4, 1, 7)
    G = _rand(4, 1, 9)
    got = O.linear_norm2(A, G)
    ref = (A[:, 0] ** 2).sum(-1) * (G[:, 0] ** 2).sum(-1)
    np.testing.assert_allclose(got, ref, rtol=1e-13)


def test_linear_norm_scaling_and_permutation():
    A = _rand(5, 6, 4)
    G = _rand(5, 6, 3)
    n = O.linear_norm2(A, G)
    np.testing.assert_allclose(O.linear_norm2(A, 3.0 * G), 9.0 * n, rtol=1e-13)
    perm = RNG.permutation(5)
    np.testing.assert_allclose(O.linear_norm2(A[perm], G[perm]), n[perm], rtol=1e-14)
    # permuting tokens inside an example leaves its gradient unchanged
    tp = RNG.permutation(6)
    np.testing.assert_allclose(O.linear_norm2(A[:, tp], G[:, tp]), n, rtol=1e-12)


# ---------------------------------------------------------------------------
# Pin 2: embedding gradient, head gradient, tied composition
# ---------------------------------------------------------------------------
def _tiny_tied_lm(B, T, V, d, seed=0):
    """A small causal LM with E tied to the output head, all fp64 autograd.

    emb = E[ids]; h = tanh(emb W1) + emb; logits = h E^T;
    loss_i = sum_t CE(logits[t], ids[t+1]) / T.
    Returns per-example tied gradients and the captured (dE, H, Gz).
    """
    g = torch.Generator().manual_seed(seed)
    E = torch.randn(V, d, generator=g, dtype=torch.float64, requires_grad=True)
    W1 = torch.randn(d, d, generator=g, dtype=torch.float64) * 0.3
    ids = torch.randint(0, V, (B, T), generator=g)
    ids[0, : T // 2] = ids[0, 0]          # forces repeated ids in example 0
    grads, dEs, Hs, Gzs = [], [], [], []
    for i in range(B):
        E.grad = None
        emb = E[ids[i]]
        emb.retain_grad()
        h = torch.tanh(emb @ W1) + emb
        h.retain_grad()
        logits = h @ E.T
        logits.retain_grad()
        loss = torch.nn.functional.cross_entropy(logits[:-1], ids[i, 1:], reduction="sum") / T
        loss.backward()
        grads.append(E.grad.numpy().copy())
        dEs.append(emb.grad.numpy().copy())
        Hs.append(h.detach().numpy().copy())
        Gzs.append(logits.grad.numpy().copy())
    return ids.numpy().astype(np.int32), np.stack(grads), np.stack(dEs), np.stack(Hs), np.stack(Gzs)


def check_tied_against_autograd(o, B=3, T=9, V=11, d=5):
    ids, g_true, dE, H, Gz = _tiny_tied_lm(B, T, V, d)
    for i in range(B):
        gE = o.embedding_grad(ids[i], dE[i], V)
        gW = o.head_grad(H[i], Gz[i], V)
        np.testing.assert_allclose(gE + gW, g_true[i], rtol=1e-10, atol=1e-12)
    tn = o.tied_norm2(ids, dE, H, Gz, V)
    np.testing.assert_allclose(tn, (g_true ** 2).sum(axis=(1, 2)), rtol=1e-10)
    # eq. 11 / eq. 13: ||gin + gout||^2 = ||gin||^2 + ||gout||^2 + 2 <gin, gout>
    n_in = o.embedding_norm2(ids, dE, V)
    n_out = o.head_norm2(H, Gz, V)
    cross = o.tied_cross(ids, dE, H, Gz, V)
    np.testing.assert_allclose(n_in + n_out + 2 * cross, tn, rtol=1e-10)
    # the naive sum of eq. 12 differs from the true norm by exactly 2*cross
    assert np.all(np.abs(cross) > 0)
    np.testing.assert_allclose(tn - (n_in + n_out), 2 * cross, rtol=1e-9)


def test_tied_gradient_matches_autograd():
    check_tied_against_autograd(O)


def test_cross_cauchy_schwarz_and_sign():
    ids, _, dE, H, Gz = _tiny_tied_lm(4, 12, 7, 6, seed=3)
    n_in = O.embedding_norm2(ids, dE, 7)
    n_out = O.head_norm2(H, Gz, 7)
    cross = O.tied_cross(ids, dE, H, Gz, 7)
    assert np.all(np.abs(cross) <= np.sqrt(n_in * n_out) * (1 + 1e-12))
    # flipping the sign of the embedding pathway flips the cross term only
    np.testing.assert_allclose(O.tied_cross(ids, -dE, H, Gz, 7), -cross, rtol=1e-14)


def test_cross_special_cases():
    """One bucket: when every token of an example has id x, the input-embedding
    gradient is a single row sum_t dE_t at x, so the cross term is that row
    dotted with row x of the head gradient, sum_s Gz[s, x] h_s. Distinct ids:
    each token's row meets only its own column of Gz, so the cross term is
    sum_t <dE_t, sum_s Gz[s, x_t] h_s>, one dot product per token."""
    T, d, V = 9, 6, 11
    dE, H, Gz = _rand(1, T, d), _rand(1, T, d), _rand(1, T, V)
    same = np.full((1, T), 4, np.int32)
    want = dE[0].sum(0) @ (Gz[0][:, 4] @ H[0])
    np.testing.assert_allclose(O.tied_cross(same, dE, H, Gz, V)[0], want, rtol=1e-12)
    distinct = RNG.permutation(V)[:T].astype(np.int32)[None]
    want = sum(dE[0, t] @ (Gz[0][:, distinct[0, t]] @ H[0]) for t in range(T))
    np.testing.assert_allclose(O.tied_cross(distinct, dE, H, Gz, V)[0], want, rtol=1e-12)


def test_embedding_special_cases():
    T, d, V = 8, 5, 32
    dE = _rand(1, T, d)
    distinct = RNG.permutation(V)[:T].astype(np.int32)[None]
    np.testing.assert_allclose(O.embedding_norm2(distinct, dE, V)[0], (dE[0] ** 2).sum(), rtol=1e-13)
    same = np.full((1, T), 3, np.int32)
    np.testing.assert_allclose(O.embedding_norm2(same, dE, V)[0], (dE[0].sum(0) ** 2).sum(), rtol=1e-13)
    # the embedding is a linear layer whose input is onehot(ids)
    ids = RNG.integers(0, 4, size=(3, T)).astype(np.int32)
    dE3 = _rand(3, T, d)
    onehot = np.eye(V)[ids]
    np.testing.assert_allclose(O.embedding_norm2(ids, dE3, V), O.linear_norm2(onehot, dE3), rtol=1e-12)
    # ... so, written out pairwise (the form the short-example kernel sums):
    # sum_{t,s} [x_t = x_s] <e_t, e_s>
    pair = np.array([sum(float(dE3[i, t] @ dE3[i, u]) for t in range(T) for u in range(T)
                         if ids[i, t] == ids[i, u]) for i in range(3)])
    np.testing.assert_allclose(O.embedding_norm2(ids, dE3, V), pair, rtol=1e-12)


def test_head_is_linear_layer_d_to_V():
    H = _rand(2, 6, 4)
    Gz = _rand(2, 6, 9)
    np.testing.assert_allclose(O.head_norm2(H, Gz, 9), O.linear_norm2(H, Gz), rtol=1e-13)
    # padding columns beyond V are ignored
    Gzp = np.concatenate([Gz, _rand(2, 6, 3)], axis=2)
    np.testing.assert_allclose(O.head_norm2(H, Gzp, 9), O.linear_norm2(H, Gz), rtol=1e-13)


# ---------------------------------------------------------------------------
# Pin 3: buckets (integer brute force)
# ---------------------------------------------------------------------------
def test_buckets_brute_force():
    ids = RNG.integers(0, 20, size=(5, 33)).astype(np.int32)
    ids[1] = 7
    ids[2] = np.arange(33)
    seg, nu = O.buckets(ids)
    for i in range(5):
        distinct = sorted(set(int(x) for x in ids[i]))
        rank = {v: r for r, v in enumerate(distinct)}
        assert nu[i] == len(distinct)
        assert [rank[int(x)] for x in ids[i]] == seg[i].tolist()


# ---------------------------------------------------------------------------
# Pin 4: clipping (eq. 2, eq. 7)
# ---------------------------------------------------------------------------
def check_clip(o):
    A = _rand(6, 5, 4)
    G = _rand(6, 5, 3)
    G[2] = 0.0                       # zero gradient
    G[3] *= 1e-3                     # well under C
    C = 0.7
    n2 = o.linear_norm2(A, G)
    c = o.clip_factors(n2, C)
    assert c[2] == 1.0
    for i in range(6):
        N = np.sqrt(n2[i])
        clipped = c[i] * o.linear_grad(A[i], G[i])
        Nc = np.sqrt((clipped ** 2).sum())
        assert Nc <= C * (1 + 1e-12)
        if N > C:
            assert abs(Nc - C) <= 1e-12 * C
        else:
            assert c[i] == 1.0


def test_clip_bounds():
    check_clip(O)


def check_nonfinite_norms(o):
    """A squared norm that is not finite (inf from an overflow, NaN) gives a
    clip factor of 0 (min(1, C/inf) = 0; NaN read the same way), and the
    example is left out of the clipped sum, which stays finite: the bound
    ||c_i g_i|| <= C of eq. 2 holds for every example."""
    c = o.clip_factors(np.array([np.inf, np.nan, -np.inf, 4.0, 0.0, -1e-20]), 1.0)
    np.testing.assert_array_equal(c, [0.0, 0.0, 0.0, 0.5, 1.0, 1.0])
    A = _rand(5, 4, 3)
    G = _rand(5, 4, 2)
    A[1, 2, 0] = np.nan
    G[3, 0, 1] = np.inf
    C = 0.8
    n2 = o.linear_norm2(A, G)
    assert not np.isfinite(n2[1]) and not np.isfinite(n2[3])
    c = o.clip_factors(n2, C)
    assert c[1] == 0.0 and c[3] == 0.0 and np.all(c[[0, 2, 4]] > 0)
    S = o.clipped_sum_linear(A, G, c)
    assert np.isfinite(S).all()
    keep = [0, 2, 4]
    ref = np.einsum("i,itm,itn->mn", c[keep], A[keep], G[keep])
    np.testing.assert_allclose(S, ref, rtol=1e-12, atol=1e-12)
    for i in keep:
        assert np.sqrt(o.sqnorm(c[i] * o.linear_grad(A[i], G[i]))) <= C * (1 + 1e-12)


def test_nonfinite_norms_are_clipped_to_zero():
    check_nonfinite_norms(O)


def test_nonfinite_example_left_out_of_every_sum():
    """The whole step on a tied full-parameter workload with one NaN
    activation in example 1 and one inf embedding gradient in example 2:
    both get c = 0, every clipped sum is finite, and equals the step over the
    other examples with the same factors."""
    wl = gen.make_workload("c1-tied", full_params=True)
    wl.linears[0].A = wl.linears[0].A.copy()
    wl.linears[0].A[1, 3, 5] = np.nan
    wl.head.dE = wl.head.dE.copy()
    wl.head.dE[2, 0, 7] = np.inf
    r = O.step(wl, noise=False)
    assert r["c"][1] == 0.0 and r["c"][2] == 0.0 and np.all(r["c"][[0, 3]] > 0)
    r_ok = O.step(wl, examples=[0, 3], noise=False)
    np.testing.assert_array_equal(r_ok["c"], r["c"][[0, 3]])
    for k, S in r["sums"].items():
        assert np.isfinite(S).all(), k
        np.testing.assert_allclose(S, r_ok["sums"][k], rtol=1e-12, atol=1e-15, err_msg=k)


def check_huge_C_is_plain_gradient(o):
    """C -> infinity: the clipped sum is the non-private gradient, one GEMM over B*T rows."""
    A = _rand(4, 6, 5)
    G = _rand(4, 6, 3)
    c = o.clip_factors(o.linear_norm2(A, G), 1e30)
    assert np.all(c == 1.0)
    S = o.clipped_sum_linear(A, G, c)
    ref = A.reshape(-1, 5).T @ G.reshape(-1, 3)
    np.testing.assert_allclose(S, ref, rtol=1e-12, atol=1e-12)


def test_huge_C_is_plain_gradient():
    check_huge_C_is_plain_gradient(O)


def test_small_C_linearity_and_permutation_invariance():
    A = _rand(5, 4, 3)
    G = _rand(5, 4, 2)
    n2 = O.linear_norm2(A, G)
    S1 = O.clipped_sum_linear(A, G, O.clip_factors(n2, 1e-6))
    S2 = O.clipped_sum_linear(A, G, O.clip_factors(n2, 2e-6))
    np.testing.assert_allclose(S2, 2 * S1, rtol=1e-12)
    perm = RNG.permutation(5)
    S1p = O.clipped_sum_linear(A[perm], G[perm], O.clip_factors(n2[perm], 1e-6))
    np.testing.assert_allclose(S1p, S1, rtol=1e-12)


def test_embedding_and_head_sums_match_linear_forms():
    V, T, d = 10, 7, 3
    ids = RNG.integers(0, V, size=(3, T)).astype(np.int32)
    dE = _rand(3, T, d)
    H = _rand(3, T, d)
    Gz = _rand(3, T, V)
    c = np.array([0.5, 1.0, 0.25])
    onehot = np.eye(V)[ids]
    np.testing.assert_allclose(O.clipped_sum_embedding(ids, dE, c, V),
                               O.clipped_sum_linear(onehot, dE, c), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(O.clipped_sum_head(H, Gz, c, V),
                               O.clipped_sum_linear(Gz, H, c), rtol=1e-12, atol=1e-14)


# ---------------------------------------------------------------------------
# Pin 5: noise (eq. 3), Philox known answers, Gaussian statistics
# ---------------------------------------------------------------------------
def _kat_rows():
    rows = []
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            v = [int(x, 16) for x in line.split()]
            rows.append((v[0:4], v[4:6], v[6:10]))
    return rows


def check_philox_kat(o):
    for ctr, key, out in _kat_rows():
        got = o.philox4x32_10([np.array([c], np.uint64) for c in ctr], key)
        assert [int(g[0]) for g in got] == out


def test_philox_known_answers():
    assert len(_kat_rows()) == 3
    check_philox_kat(O)


def test_gaussian_statistics():
    n = 1 << 20
    z = O.gaussian(n, seed=7, tensor_id=3, step=11)
    se = 1.0 / np.sqrt(n)
    assert abs(z.mean()) < 5 * se
    assert abs(z.std() - 1.0) < 5 * np.sqrt(0.5) * se
    # fourth moment of a standard normal is 3
    assert abs((z ** 4).mean() - 3.0) < 5 * np.sqrt(96.0) * se
    from scipy import stats
    assert stats.kstest(z[: 1 << 16], "norm").pvalue > 1e-4
    # the four outputs of one Philox block are not copies of each other
    zz = z.reshape(-1, 4)
    assert abs(np.corrcoef(zz[:, 0], zz[:, 1])[0, 1]) < 5 * np.sqrt(4.0 / n)


def test_gaussian_streams_are_keyed_and_sliceable():
    a = O.gaussian(1000, 1, 2, 3)
    np.testing.assert_array_equal(O.gaussian(10, 1, 2, 3, start=995)[:5], a[995:])
    assert not np.allclose(a, O.gaussian(1000, 1, 2, 4))
    assert not np.allclose(a, O.gaussian(1000, 1, 5, 3))
    assert not np.allclose(a, O.gaussian(1000, 2, 2, 3))
    # the 64-bit seed uses both halves
    assert not np.allclose(a, O.gaussian(1000, 1 + (1 << 32), 2, 3))


def test_noise_sigma_zero_and_scale():
    S = _rand(7, 9)
    np.testing.assert_array_equal(O.add_noise(S, 0.0, 1.0, 4, 0, 0, 0), S / 4)
    np.testing.assert_array_equal(O.add_noise(S, 0.0, 1.0, 0, 0, 0, 0), S)
    z = O.gaussian(S.size, 5, 1, 2).reshape(S.shape)
    np.testing.assert_allclose(O.add_noise(S, 2.0, 0.5, 3, 5, 1, 2), (S + 1.0 * z) / 3, rtol=1e-14)


# ---------------------------------------------------------------------------
# Pin 6: generator facts the workloads rely on
# ---------------------------------------------------------------------------
def test_param_counts_match_paper_table():
    with open(os.path.join(GOLDEN, "gpt2_param_counts.txt")) as f:
        rows = [l.split() for l in f if l.strip() and not l.startswith("#")]
    assert len(rows) == 4
    for _, nb, tied, n in rows:
        assert gen.gpt2_param_count(int(nb), bool(int(tied))) == int(n)
    # untying adds exactly one V x d matrix
    assert gen.gpt2_param_count(12, False) - gen.gpt2_param_count(12, True) == 50257 * 768


def test_logit_grads_match_cross_entropy_autograd():
    B, T, V = 2, 6, 13
    z = RNG.standard_normal((B, T, V)).astype(np.float32)
    ids = RNG.integers(0, V, size=(B, T)).astype(np.int32)
    zt = torch.tensor(z.astype(np.float64), requires_grad=True)
    loss = 0
    for i in range(B):
        loss = loss + torch.nn.functional.cross_entropy(
            zt[i, :-1], torch.tensor(ids[i, 1:]).long(), reduction="sum") / T
    loss.backward()
    got = gen.logit_grads(z.copy(), ids)
    np.testing.assert_allclose(got, zt.grad.numpy(), rtol=1e-5, atol=1e-7)
    np.testing.assert_allclose(got[:, :-1].sum(-1), 0.0, atol=1e-6)
    assert np.all(got[:, -1] == 0)


def test_zipf_frequencies():
    rng = np.random.default_rng(0)
    ids = gen.zipf_ids(rng, (200000,), 50257, 1.1)
    k = np.arange(1, 50258, dtype=np.float64)
    p = k ** -1.1
    p /= p.sum()
    for r in range(5):
        f = np.mean(ids == r)
        assert abs(f - p[r]) < 5 * np.sqrt(p[r] * (1 - p[r]) / ids.size)
    assert ids.min() >= 0 and ids.max() < 50257


def test_bf16_rounding():
    x = np.array([1.0, 1.00390625, 1.01171875, -2.5, 3.0e-3, 1e30], np.float32)
    b = gen.f32_to_bf16_bits(x)
    back = gen.bf16_bits_to_f32(b)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: goes to even (1.0)
    assert back[0] == 1.0 and back[1] == 1.0
    assert back[2] == np.float32(1.015625)       # 1 + 3*2^-8 ties up to even
    np.testing.assert_allclose(back, x, rtol=2 ** -8)
    np.testing.assert_array_equal(O.decode(b, "bf16"), back.astype(np.float64))


def test_workload_streams_are_per_tensor():
    full = gen.make_workload("c1", B=4, T=16)
    again = gen.make_workload("c1", B=4, T=16)
    np.testing.assert_array_equal(full.linears[0].A, again.linears[0].A)
    np.testing.assert_array_equal(full.head.ids, again.head.ids)
    sub = gen.make_workload("c2", B=2, T=8, n_blocks=2, layers=[5], with_head=False)
    full2 = gen.make_workload("c2", B=2, T=8, n_blocks=2, with_head=False)
    np.testing.assert_array_equal(sub.linears[0].A, full2.linears[5].A)


# ---------------------------------------------------------------------------
# Whole-step consistency on the tiny workloads
# ---------------------------------------------------------------------------
def test_step_tiny_tied_consistency():
    wl = gen.make_workload("c1-tied", B=4, T=16)
    r = O.step(wl, seed=3, step_id=1)
    n = r["norms"]
    np.testing.assert_allclose(n["in"] + n["out"] + 2 * n["cross"], n["tied"], rtol=1e-10)
    np.testing.assert_allclose(n["total"], n["linear"].sum(0) + n["tied"], rtol=1e-13)
    assert set(r["noisy"]) == {"linear", "wte"}
    # sigma = 0 reproduces the clipped mean exactly
    wl.sigma = 0.0
    r0 = O.step(wl, seed=3, step_id=1)
    for k in r0["sums"]:
        np.testing.assert_array_equal(r0["noisy"][k], r0["sums"][k] / wl.B)


# ---------------------------------------------------------------------------
# Pin: biases, LayerNorm gain/bias and the position table (the parameters the
# paper's parameter-count table includes besides the weight matrices)
# ---------------------------------------------------------------------------
def check_vector_and_position_grads_autograd(o, B=3, T=5, d=6, d_out=4, n_pos=8):
    """Per-example grads of a block h0 = tok + wpe[t], h1 = LayerNorm(h0) with
    gain and bias, y = h1 W + b, loss_i = sum(y * R_i), from fp64 autograd;
    the upstream grads the oracle takes (dL/dy, dL/dh1, dL/dh0) come from
    autograd too."""
    g = torch.Generator().manual_seed(7)
    f64 = dict(dtype=torch.float64)
    wpe = torch.randn(n_pos, d, generator=g, **f64).requires_grad_()
    gamma = (1 + 0.3 * torch.randn(d, generator=g, **f64)).requires_grad_()
    beta = (0.3 * torch.randn(d, generator=g, **f64)).requires_grad_()
    W = torch.randn(d, d_out, generator=g, **f64).requires_grad_()
    b = torch.randn(d_out, generator=g, **f64).requires_grad_()
    for i in range(B):
        for p in (wpe, gamma, beta, W, b):
            p.grad = None
        tok = torch.randn(T, d, generator=g, **f64).requires_grad_()
        R = torch.randn(T, d_out, generator=g, **f64)
        h0 = tok + wpe[torch.arange(T)]
        h1 = torch.nn.functional.layer_norm(h0, (d,), gamma, beta)
        y = h1 @ W + b
        h1.retain_grad(); y.retain_grad()
        (y * R).sum().backward()
        xhat = torch.nn.functional.layer_norm(h0.detach(), (d,))
        dE, G1, Gy = tok.grad.numpy(), h1.grad.numpy(), y.grad.numpy()
        np.testing.assert_allclose(o.vector_grad(None, Gy), b.grad.numpy(), rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(o.vector_grad(xhat.numpy(), G1), gamma.grad.numpy(),
                                   rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(o.vector_grad(None, G1), beta.grad.numpy(), rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(o.positional_grad(dE, n_pos), wpe.grad.numpy(),
                                   rtol=1e-12, atol=1e-12)
        # the flat norm of eq. 6 over every parameter of the block
        flat = torch.cat([p.grad.reshape(-1) for p in (wpe, gamma, beta, W, b)])
        ours = (o.sqnorm(o.positional_grad(dE, n_pos)) + o.sqnorm(o.vector_grad(xhat.numpy(), G1))
                + o.sqnorm(o.vector_grad(None, G1)) + o.sqnorm(o.linear_grad(h1.detach().numpy(), Gy))
                + o.sqnorm(o.vector_grad(None, Gy)))
        np.testing.assert_allclose(ours, float(flat @ flat), rtol=1e-12)


def test_vector_and_position_grads_match_autograd():
    check_vector_and_position_grads_autograd(O)


def test_position_grad_is_embedding_grad_of_distinct_positions():
    T, d, n_pos = 7, 5, 12
    dE = _rand(T, d)
    np.testing.assert_array_equal(O.positional_grad(dE, n_pos),
                                  O.embedding_grad(np.arange(T), dE, n_pos))
    # distinct rows: the squared norm is the sum of the rows' squared norms
    np.testing.assert_allclose(O.positional_norm2(dE[None], n_pos), [np.sum(dE * dE)], rtol=1e-13)


def test_vector_norm_special_cases():
    G = _rand(2, 1, 6)
    X = _rand(2, 1, 6)
    # one token: the gain's gradient is x * g, the bias's g
    np.testing.assert_allclose(O.vector_norm2(X, G), np.sum((X * G) ** 2, axis=(1, 2)), rtol=1e-13)
    np.testing.assert_allclose(O.vector_norm2(None, G), np.sum(G * G, axis=(1, 2)), rtol=1e-13)
    # the bias gradient is the Gram form with A a column of ones: 1^T (G G^T) 1
    G = _rand(3, 9, 5)
    gram = np.array([np.sum(G[i] @ G[i].T) for i in range(3)])
    np.testing.assert_allclose(O.vector_norm2(None, G), gram, rtol=1e-12)
    np.testing.assert_allclose(O.vector_norm2(None, G),
                               O.linear_norm2(np.ones((3, 9, 1)), G), rtol=1e-12)


def test_full_param_workloads_cover_the_paper_counts():
    with open(os.path.join(GOLDEN, "gpt2_param_counts.txt")) as f:
        rows = {(int(r[1]), int(r[2])): int(r[3]) for r in
                (l.split() for l in f if l.strip() and not l.startswith("#"))}
    for name, nb, tied in (("gpt2-step", 12, 1), ("c4", 6, 1), ("c5", 12, 0)):
        wl = gen.make_workload(name, B=1, T=4, full_params=True)
        assert wl.n_coordinates() == rows[(nb, tied)], name


def check_full_step_composition(o):
    """Flat per-example norm over every parameter tensor of a tiny full-parameter
    tied workload, from the materialised gradients, against the step's total;
    huge C gives the plain sums."""
    wl = gen.make_workload("c1-tied", B=3, T=6, full_params=True)
    dec = lambda x: O.decode(x, wl.dtype)
    h = wl.head
    for i in range(wl.B):
        parts = [O.linear_grad(dec(l.A[i]), dec(l.G[i])) for l in wl.linears]
        parts.append(O.embedding_grad(h.ids[i], dec(h.dE[i]), h.V)
                     + O.head_grad(dec(h.H[i]), dec(h.Gz[i]), h.V))
        parts += [O.vector_grad(None if v.X is None else dec(v.X[i]), dec(v.G[i]))
                  for v in wl.vectors]
        parts.append(O.positional_grad(dec(h.dE[i]), wl.n_pos))
        flat = np.concatenate([p.reshape(-1) for p in parts])
        assert flat.size == wl.n_coordinates()
        n = o.per_example_norms(wl, [i])["total"][0]
        np.testing.assert_allclose(n, flat @ flat, rtol=1e-12)
    wl.C = 1e30
    r = o.step(wl, noise=False)
    for v in wl.vectors:
        X = 1.0 if v.X is None else dec(v.X)
        np.testing.assert_allclose(r["sums"][v.name], (X * dec(v.G)).sum(axis=(0, 1)), rtol=1e-12)
    np.testing.assert_allclose(r["sums"]["wpe"][: wl.T], dec(h.dE).sum(axis=0), rtol=1e-12)
    assert not r["sums"]["wpe"][wl.T:].any()


def test_full_step_composition():
    check_full_step_composition(O)


def test_full_step_noise_ids_follow_the_tensors():
    wl = gen.make_workload("c1-tied", B=2, T=4, full_params=True)
    r = O.step(wl, seed=5, step_id=3)
    names = list(r["noisy"])
    assert names[:2] == ["linear", "wte"] and names[-1] == "wpe"
    assert names[2:-1] == [v.name for v in wl.vectors]
    for tid, name in enumerate(names):
        S = r["sums"][name]
        z = O.gaussian(S.size, 5, tid, 3).reshape(S.shape)
        np.testing.assert_allclose(r["noisy"][name], (S + wl.sigma * wl.C * z) / wl.B, rtol=1e-13)


# ---------------------------------------------------------------------------
# Mutation tests: plausible mistakes planted in a copy of the oracle
# ---------------------------------------------------------------------------
def _mutant(**overrides):
    m = types.SimpleNamespace(**{k: getattr(O, k) for k in O.__all__})
    for k, v in overrides.items():
        setattr(m, k, v)
    return m


def _fails(check, o):
    try:
        check(o)
    except AssertionError:
        return True
    return False


def test_pins_catch_transposed_linear_grad():
    m = _mutant(linear_grad=lambda A, G: G.T @ A)
    assert _fails(check_linear_grad_autograd, m)


def test_pins_catch_dropped_cross_term():
    def tied_norm2_naive(ids, dE, H, Gz, V):
        return O.embedding_norm2(ids, dE, V) + O.head_norm2(H, Gz, V)
    assert _fails(check_tied_against_autograd, _mutant(tied_norm2=tied_norm2_naive))


def test_pins_catch_wrong_head_orientation():
    def head_grad_bad(H_i, Gz_i, V):
        return Gz_i[:, :V].T @ H_i[::-1]     # tokens of H misaligned with Gz
    assert _fails(check_tied_against_autograd, _mutant(head_grad=head_grad_bad))


def test_pins_catch_clip_max_instead_of_min():
    def clip_bad(norm2, C):
        n = np.sqrt(norm2)
        c = np.ones_like(n)
        nz = n > 0
        c[nz] = np.maximum(1.0, C / n[nz])
        return c
    assert _fails(check_clip, _mutant(clip_factors=clip_bad))


def test_pins_catch_nan_norm_summed_unclipped():
    def clip_nan_is_one(norm2, C):     # NaN fails n > 0, so it keeps c = 1
        n = np.sqrt(np.asarray(norm2, np.float64))
        c = np.ones_like(n)
        nz = n > 0
        c[nz] = np.minimum(1.0, C / n[nz])
        return c
    assert _fails(check_nonfinite_norms, _mutant(clip_factors=clip_nan_is_one))


def test_pins_catch_zero_factor_multiplied_not_skipped():
    def sum_multiplies(A, G, c):       # 0 * inf = NaN
        return np.einsum("i,itm,itn->mn", c, A, G)
    assert _fails(check_nonfinite_norms, _mutant(clipped_sum_linear=sum_multiplies))


def test_pins_catch_philox_wrong_rounds():
    def philox9(ctr, key):
        c = [np.asarray(x, np.uint64) for x in ctr]
        out = O.philox4x32_10(c, key)
        return [o ^ np.uint32(1) for o in out]
    assert _fails(check_philox_kat, _mutant(philox4x32_10=philox9))


def test_pins_catch_gain_treated_as_bias():
    m = _mutant(vector_grad=lambda X, G: G.sum(axis=0))
    assert _fails(check_vector_and_position_grads_autograd, m)


def test_pins_catch_shifted_positions():
    def pos_bad(dE_i, n_pos):
        g = np.zeros((n_pos, dE_i.shape[1]))
        g[1: dE_i.shape[0] + 1] = dE_i
        return g
    assert _fails(check_vector_and_position_grads_autograd, _mutant(positional_grad=pos_bad))


def test_pins_catch_dropped_vector_norms():
    def norms_without_vectors(wl, examples=None):
        saved = wl.vectors
        wl.vectors = []
        try:
            return O.per_example_norms(wl, examples)
        finally:
            wl.vectors = saved
    assert _fails(check_full_step_composition, _mutant(per_example_norms=norms_without_vectors))
