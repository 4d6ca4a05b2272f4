"""GPU parity of the remaining GPT-2 parameters against the fp64 oracle:
vector parameters (linear biases, LayerNorm gains and biases) and the
learned position table, their per-example norms, clipped sums and noise.

Inputs are seeded draws (workloads.gen); expected values come only from the
oracle. Per-example gradients of these parameters are small, so full GPT-2
sizes are checked in full.
"""
import sys

import numpy as np
import pytest

import oracle as O
from workloads import gen
from tests.helpers import TOL, assert_close, dev, host, rel

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def dp():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_40335_amd.dpghost as d
    d.lib()
    return d


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _nan_pad(x, d):
    """Fill the row-stride padding past column d with NaN (bf16 or fp32)."""
    if x.shape[2] > d:
        x[:, :, d:] = 0x7FC0 if x.dtype == np.uint16 else np.nan
    return x


VEC_CASES = [
    # dtype, B, T, d, with X, row stride (None: d)
    ("bf16", 3, 37, 520, True, None),      # ragged T (not a multiple of 16 rows), 2 chunks
    ("bf16", 2, 130, 77, False, 80),       # width not a multiple of 8, aligned padded stride
    ("bf16", 2, 5, 3000, True, None),      # 6 feature chunks, fewer rows than waves x unroll
    ("bf16", 4, 1, 64, True, None),        # T = 1: x * g
    ("bf16", 2, 16, 101, True, 103),       # unaligned stride: element-wise loads
    ("f32", 4, 16, 64, True, None),
    ("f32", 2, 33, 300, False, 303),       # unaligned fp32 stride
    ("f32", 3, 70, 260, True, 264),        # 2 fp32 chunks, aligned padded stride
]


@pytest.mark.parametrize("case", VEC_CASES, ids=lambda c: "-".join(str(x) for x in c))
def test_vector_grads_and_norms(dp, case):
    dtype, B, T, d, with_x, ld = case
    _say(f"vector grads {case}")
    ld = ld or d
    G = _nan_pad(gen.draw(71, 1, (B, T, ld), 1e-2, dtype), d)
    X = _nan_pad(gen.draw(71, 2, (B, T, ld), 1.0, dtype), d) if with_x else None
    Gd = O.decode(G[:, :, :d], dtype)
    Xd = None if X is None else O.decode(X[:, :, :d], dtype)
    ref_g = np.stack([O.vector_grad(None if Xd is None else Xd[i], Gd[i]) for i in range(B)])
    ref_n = O.vector_norm2(Xd, Gd)
    grads = [torch.full((B, d), 7.0, device="cuda")]
    Xt = None if X is None else dev(X, dtype)[:, :, :d]
    n2 = torch.full((B,), 2.0, device="cuda")
    dp.dp_vector_grads_grouped([(Xt, dev(G, dtype)[:, :, :d])], grads, n2, accumulate=True)
    got = host(grads[0])
    assert np.isfinite(got).all()
    for i in range(B):
        assert_close(got[i], ref_g[i], TOL[dtype], i)
    assert rel(host(n2) - 2.0, ref_n).max() <= TOL[dtype]
    # overwrite mode, no norm output
    n3 = torch.full((B,), 5.0, device="cuda")
    dp.dp_vector_grads_grouped([(Xt, dev(G, dtype)[:, :, :d])], grads, n3, accumulate=False)
    assert rel(host(n3), ref_n).max() <= TOL[dtype]
    dp.dp_vector_grads_grouped([(Xt, dev(G, dtype)[:, :, :d])], grads, None)


def test_vector_grads_grouped_mixed(dp):
    """Biases and gains of several widths, aligned and unaligned, one call."""
    B, T = 3, 40
    specs = [(96, False, None), (520, True, None), (77, True, 80), (33, False, 35), (1024, True, None)]
    params, refs, norm_ref = [], [], np.zeros(B)
    for k, (d, with_x, ld) in enumerate(specs):
        ld = ld or d
        G = gen.draw(80 + k, 1, (B, T, ld), 1e-2, "bf16")
        X = gen.draw(80 + k, 2, (B, T, ld), 1.0, "bf16") if with_x else None
        Gd = O.decode(G[:, :, :d], "bf16")
        Xd = None if X is None else O.decode(X[:, :, :d], "bf16")
        refs.append(np.stack([O.vector_grad(None if Xd is None else Xd[i], Gd[i])
                              for i in range(B)]))
        norm_ref += O.vector_norm2(Xd, Gd)
        params.append((None if X is None else dev(X, "bf16")[:, :, :d], dev(G, "bf16")[:, :, :d]))
    grads = [torch.empty(B, d, device="cuda") for d, _, _ in specs]
    n2 = torch.zeros(B, device="cuda")
    dp.dp_vector_grads_grouped(params, grads, n2)
    for g, r in zip(grads, refs):
        assert_close(host(g), r, TOL["bf16"])
    assert rel(host(n2), norm_ref).max() <= TOL["bf16"]


def test_vector_grads_layernorm_pairs(dp):
    """A gain and a bias on one G buffer take one fused pass; listed in either
    order, next to a bias on another buffer and a gain whose bias differs in
    width (not fused)."""
    B, T = 3, 45
    G1 = gen.draw(120, 1, (B, T, 768), 1e-2, "bf16")
    X1 = gen.draw(120, 2, (B, T, 768), 1.0, "bf16")
    G2 = gen.draw(121, 1, (B, T, 136), 1e-2, "bf16")
    X2 = gen.draw(121, 2, (B, T, 136), 1.0, "bf16")
    g1, x1, g2, x2 = dev(G1, "bf16"), dev(X1, "bf16"), dev(G2, "bf16"), dev(X2, "bf16")
    params = [(None, g1), (x2, g2), (x1, g1), (None, g2[:, :, :100])]
    grads = [torch.empty(B, p[1].shape[2], device="cuda") for p in params]
    n2 = torch.zeros(B, device="cuda")
    dp.dp_vector_grads_grouped(params, grads, n2)
    norm = np.zeros(B)
    for (X, G), g, Xh, Gh in zip(params, grads, [None, X2, X1, None],
                                 [G1, G2, G1, G2[:, :, :100]]):
        Gd = O.decode(Gh, "bf16")
        Xd = None if Xh is None else O.decode(Xh, "bf16")
        ref = np.stack([O.vector_grad(None if Xd is None else Xd[i], Gd[i]) for i in range(B)])
        assert_close(host(g), ref, TOL["bf16"])
        norm += (ref * ref).sum(axis=1)
    assert rel(host(n2), norm).max() <= TOL["bf16"]


def test_vector_clipped_sum_noised(dp):
    """outs = (prior + sum_i c_i g_i + sigma C z) / B against the oracle's
    add_noise with the same stream; widths not multiples of 4."""
    B = 5
    sigma, C, seed, step = 0.8, 1.3, 0xBEEF, 7
    ds = [3, 64, 517, 2304]
    tids = [4, 11, 12, 40]
    acc = [False, True, False, True]
    c = np.linspace(0.2, 1.0, B).astype(np.float32)
    grads, outs, refs = [], [], []
    for k, d in enumerate(ds):
        g = gen.draw(90 + k, 1, (B, d), 1.0, "f32")
        prior = gen.draw(90 + k, 2, (d,), 1e-1, "f32") if acc[k] else np.zeros(d, np.float32)
        S = (c.astype(np.float64)[:, None] * g.astype(np.float64)).sum(axis=0)
        refs.append(O.add_noise(prior.astype(np.float64) + S, sigma, C, B, seed, tids[k], step))
        grads.append(dev(g))
        outs.append(dev(prior.copy()))
    dp.dp_vector_clipped_sum_noised_grouped(grads, outs, dev(c), tids, sigma, C, B, seed, step,
                                            accumulate=acc)
    for k in range(len(ds)):
        err = assert_close(host(outs[k]), refs[k], TOL["f32"])
        _say(f"  d={ds[k]} fro / element rel err {err[0]:.2e} / {err[1]:.2e}")
    # sigma = 0, B_norm = 0: the plain clipped sum
    plain = [torch.zeros(d, device="cuda") for d in ds]
    dp.dp_vector_clipped_sum_noised_grouped(grads, plain, dev(c), tids, 0.0, C, 0, seed, step)
    for k, d in enumerate(ds):
        S = (c.astype(np.float64)[:, None] * host(grads[k]).astype(np.float64)).sum(axis=0)
        assert_close(host(plain[k]), S, 1e-6)


@pytest.mark.parametrize("dtype,B,T,d,ld", [("bf16", 3, 37, 768, None), ("bf16", 2, 20, 77, 80),
                                            ("f32", 4, 16, 64, None), ("f32", 2, 9, 101, 103)])
def test_positional_norm(dp, dtype, B, T, d, ld):
    ld = ld or d
    dE = _nan_pad(gen.draw(101, 1, (B, T, ld), 1e-2, dtype), d)
    ref = O.positional_norm2(O.decode(dE[:, :, :d], dtype), 2 * T)
    n2 = torch.full((B,), 1.5, device="cuda")
    dp.dp_ghost_norm_positional(dev(dE, dtype)[:, :, :d], n2, accumulate=True)
    assert rel(host(n2) - 1.5, ref).max() <= TOL[dtype]


@pytest.mark.parametrize("dtype,B,T,d,n_pos,acc", [("bf16", 3, 37, 768, 64, False),
                                                   ("bf16", 2, 16, 77, 16, True),
                                                   ("f32", 4, 10, 101, 23, True)])
def test_positional_clipped_sum_noised(dp, dtype, B, T, d, n_pos, acc):
    """Rows t < T get the clipped sum, every row the noise of element t*d + f;
    a width not a multiple of 4 draws per element."""
    sigma, C, seed, step, tid = 0.6, 0.9, 12345, 3, 17
    dE = gen.draw(111, 1, (B, T, d), 1e-2, dtype)
    c = np.linspace(0.3, 1.0, B).astype(np.float32)
    S = O.clipped_sum_positional(O.decode(dE, dtype), c.astype(np.float64), n_pos)
    prior = gen.draw(111, 2, (n_pos, d), 1e-2, "f32") if acc else np.zeros((n_pos, d), np.float32)
    ref = O.add_noise(prior.astype(np.float64) + S, sigma, C, B, seed, tid, step)
    out = dev(prior.copy())
    dp.dp_clipped_grad_sum_positional_noised(dev(dE, dtype), dev(c), out, tid, sigma, C, B, seed,
                                             step, accumulate=acc)
    got = host(out)
    assert_close(got[:T], ref[:T], TOL[dtype])
    if n_pos > T:
        assert_close(got[T:], ref[T:], TOL["f32"])   # noise (and prior) only


def test_full_param_tiny_step(dp):
    """Every parameter of a tiny tied model (weights, biases, LayerNorms,
    position table, tied embedding/head): norms, clip factors and noised sums
    through the C ABI against the oracle's step."""
    wl = gen.make_workload("c1-tied", full_params=True)
    ref = O.step(wl, seed=9, step_id=4)
    B, h = wl.B, wl.head
    lin = wl.linears[0]
    A, G = dev(lin.A), dev(lin.G)
    ids, dE, H = dev(h.ids), dev(h.dE), dev(h.H)
    Gz = dev(h.Gz)[:, :, :h.V]
    n2 = torch.zeros(B, device="cuda")
    dp.dp_ghost_norm_linear_grouped([(A, G), (H, Gz)], n2)
    dp.dp_ghost_norm_embedding(ids, dE, h.V, n2, accumulate=True)
    dp.dp_tied_cross_term(ids, dE, H, Gz, h.V, n2, scale=2.0, accumulate=True)
    vg = dp.VectorGroup([(None if v.X is None else dev(v.X), dev(v.G)) for v in wl.vectors])
    vg.grads_and_norm(n2, accumulate=True)
    dp.dp_ghost_norm_positional(dE, n2, accumulate=True)
    assert rel(host(n2), ref["norms"]["total"]).max() <= TOL["f32"]
    c = torch.empty(B, device="cuda")
    c_b = torch.empty(B, device="cuda")
    dp.dp_clip_factors_scaled(n2, wl.C, 1.0 / B, c_b, c=c)
    assert rel(host(c), ref["c"]).max() <= TOL["f32"]
    names = list(ref["noisy"])
    tid = {n: k for k, n in enumerate(names)}
    S = torch.empty(lin.d_in, lin.d_out, device="cuda")
    E = torch.empty(h.V, h.d, device="cuda")
    dp.dp_clipped_grad_sum_noised_grouped([(A, G), (Gz, H)], [S, E], c,
                                          [tid["linear"], tid["wte"]], wl.sigma, wl.C, B, 9, 4)
    dp.dp_clipped_grad_sum(None, dE, c_b, E, ids=ids, V=h.V, accumulate=True)
    outs = [torch.empty(v.d, device="cuda") for v in wl.vectors]
    vg.clipped_sum_noised(c, outs, [tid[v.name] for v in wl.vectors], wl.sigma, wl.C, B, 9, 4)
    P = torch.empty(wl.n_pos, h.d, device="cuda")
    dp.dp_clipped_grad_sum_positional_noised(dE, c, P, tid["wpe"], wl.sigma, wl.C, B, 9, 4)
    assert_close(host(S), ref["noisy"]["linear"], TOL["f32"])
    assert_close(host(E), ref["noisy"]["wte"], TOL["f32"])
    for v, o in zip(wl.vectors, outs):
        assert_close(host(o), ref["noisy"][v.name], TOL["f32"], v.name)
    assert_close(host(P), ref["noisy"]["wpe"], TOL["f32"])


def test_full_size_gpt2_vectors(dp):
    """All 98 vector parameters and the position table of GPT-2-small at the
    benchmark's B = 32, T = 128, checked in full against the oracle."""
    wl = gen.make_workload("gpt2-step", full_params=True)
    B, h = wl.B, wl.head
    _say(f"full-size vectors: {len(wl.vectors)} parameters, B={B}, T={wl.T}")
    bufs = {}

    def once(a):  # one device buffer per host array: LayerNorm gain/bias pairs fuse
        if id(a) not in bufs:
            bufs[id(a)] = dev(a)
        return bufs[id(a)]
    vg = dp.VectorGroup([(None if v.X is None else dev(v.X), once(v.G)) for v in wl.vectors])
    n2 = torch.zeros(B, device="cuda")
    vg.grads_and_norm(n2)
    dE = dev(h.dE)
    npos = torch.zeros(B, device="cuda")
    dp.dp_ghost_norm_positional(dE, npos)
    ref_n = np.zeros(B)
    worst = 0.0
    for v, g in zip(wl.vectors, vg.grads):
        Xd = None if v.X is None else O.decode(v.X, "bf16")
        Gd = O.decode(v.G, "bf16")
        ref_g = np.stack([O.vector_grad(None if Xd is None else Xd[i], Gd[i]) for i in range(B)])
        worst = max(worst, assert_close(host(g), ref_g, TOL["bf16"])[1])
        ref_n += (ref_g * ref_g).sum(axis=1)
    _say(f"  worst per-parameter gradient rel err {worst:.2e}")
    assert worst <= TOL["bf16"]
    assert rel(host(n2), ref_n).max() <= TOL["bf16"]
    assert rel(host(npos), O.positional_norm2(O.decode(h.dE, "bf16"), wl.n_pos)).max() <= TOL["bf16"]
    c = (0.25 + 0.75 * np.arange(B) / B).astype(np.float32)
    P = torch.empty(wl.n_pos, h.d, device="cuda")
    dp.dp_clipped_grad_sum_positional_noised(dE, dev(c), P, 7, 0.0, 1.0, 0, 1, 0)
    ref_p = O.clipped_sum_positional(O.decode(h.dE, "bf16"), c.astype(np.float64), wl.n_pos)
    assert_close(host(P), ref_p, TOL["bf16"])


# ---------------------------------------------------------------------------
# Linear-layer biases fused into the grouped norm
# ---------------------------------------------------------------------------
BIAS_CASES = [
    # dtype, B, T, layers: (d_in, d_out, bias?, G row stride or None, algo)
    ("bf16", 4, 64, [(96, 200, True, None, "gram"), (64, 72, False, None, "gram"),
                     (128, 520, True, None, "gram")]),            # single-tile Gram: fused
    ("bf16", 3, 200, [(96, 136, True, None, "gram"), (72, 64, True, None, "gram")]),  # whole
    ("bf16", 2, 300, [(64, 96, True, None, "gram")]),             # tile pairs: vector pass
    ("bf16", 2, 64, [(64, 4200, True, None, "gram")]),            # G in 2 chunks: fused
    ("bf16", 3, 40, [(80, 101, True, 103, "gram"),                # unaligned rows: vector pass
                     (64, 64, True, None, "direct")]),            # direct norm: vector pass
    ("f32", 3, 50, [(48, 70, True, None, "gram"), (32, 40, False, None, "gram")]),
    ("bf16", 1, 1, [(64, 72, True, None, "gram")]),               # one example, one token
    ("bf16", 2, 129, [(64, 200, True, None, "gram")]),            # whole kernel, ragged T
    ("bf16", 2, 256, [(128, 64, True, None, "gram")]),            # whole kernel, full T
]


@pytest.mark.parametrize("case", BIAS_CASES, ids=lambda c: f"{c[0]}-B{c[1]}-T{c[2]}-{len(c[3])}")
def test_linear_norm_with_biases(dp, case):
    dtype, B, T, spec = case
    _say(f"linear norm with biases {dtype} B={B} T={T} {spec}")
    algos = {"gram": dp.DP_NORM_GRAM, "direct": dp.DP_NORM_DIRECT}
    layers, biases, ref_n2, refs = [], [], np.zeros(B), []
    for k, (di, do, has_b, ldg, algo) in enumerate(spec):
        ldg = ldg or do
        A = gen.draw(81 + k, 1, (B, T, di), 1.0, dtype)
        G = _nan_pad(gen.draw(81 + k, 2, (B, T, ldg), 1e-2, dtype), do)
        Ad, Gd = O.decode(A, dtype), O.decode(G[:, :, :do], dtype)
        ref_n2 = ref_n2 + O.linear_norm2(Ad, Gd)
        layers.append((dev(A, dtype), dev(G, dtype)[:, :, :do], algos[algo]))
        if has_b:
            refs.append(np.stack([O.vector_grad(None, Gd[i]) for i in range(B)]))
            ref_n2 = ref_n2 + O.vector_norm2(None, Gd)
            biases.append(torch.full((B, do), 7.0, device="cuda"))
        else:
            refs.append(None)
            biases.append(None)
    n2 = torch.full((B,), 3.0, device="cuda")
    grp = dp.LinearGroup(layers, bias_grads=biases)
    grp.ghost_norm(n2, accumulate=True)
    got_n2 = host(n2) - 3.0
    _say(f"  norm rel err {rel(got_n2, ref_n2).max():.2e}")
    assert rel(got_n2, ref_n2).max() <= TOL[dtype]
    for k, (g, r) in enumerate(zip(biases, refs)):
        if g is None:
            continue
        got = host(g)
        assert np.isfinite(got).all(), k
        for i in range(B):
            assert_close(got[i], r[i], TOL[dtype], (k, i))
    # overwrite mode gives the same norms; a group without biases gives the
    # weight-only part
    n3 = torch.full((B,), 9.0, device="cuda")
    grp.ghost_norm(n3, accumulate=False)
    assert rel(host(n3), ref_n2).max() <= TOL[dtype]
    n4 = torch.zeros(B, device="cuda")
    dp.LinearGroup(layers).ghost_norm(n4)
    bias_n2 = sum(O.vector_norm2(None, O.decode(
        gen.draw(81 + k, 2, (B, T, s[3] or s[1]), 1e-2, dtype)[:, :, :s[1]], dtype))
        for k, s in enumerate(spec) if s[2])
    assert rel(host(n4), ref_n2 - bias_n2).max() <= TOL[dtype]
