"""GPU parity: every entry point of libdpghost against the fp64 oracle.

Inputs are seeded draws (workloads.gen) shared by both sides; expected values
come only from the oracle. Sizes span several tiles with ragged tails, plus
sampled outputs at the full GPT-2 shapes.
"""
import sys

import numpy as np
import pytest

import oracle as O
from workloads import gen
from tests.helpers import TOL, assert_close, dev, fro_rel, host, rel

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


def _layer_inputs(dtype, B, T, d_in, d_out, seed, ldg=None, lda=None, g_std=1e-2):
    A = gen.draw(seed, 1, (B, T, lda or d_in), 1.0, dtype)
    G = gen.draw(seed, 2, (B, T, ldg or d_out), g_std, dtype)
    return A, G


def _oracle_linear_norm2(A, G, d_in, d_out, dtype):
    return O.linear_norm2(O.decode(A[:, :, :d_in], dtype), O.decode(G[:, :, :d_out], dtype))


# ---------------------------------------------------------------------------
# a1 / a10: linear ghost norm (Gram and direct)
# ---------------------------------------------------------------------------
NORM_CASES = [
    # dtype, B, T, d_in, d_out, lda, ldg
    ("f32", 4, 16, 64, 64, None, None),        # the tiny fp32 config
    ("f32", 3, 130, 40, 72, None, None),       # two T-tiles, ragged T
    ("f32", 2, 37, 33, 50, 36, 53),            # odd widths, padded strides
    ("bf16", 3, 128, 768, 2304, None, None),   # GPT-2 qkv shape, one T-tile
    ("bf16", 2, 300, 96, 200, None, None),     # three T-tiles, ragged T
    ("bf16", 2, 64, 100, 77, None, None),      # widths not multiples of 8
    ("bf16", 2, 50, 64, 40, 72, 48),           # padded aligned strides
    ("bf16", 2, 17, 24, 5000, None, 5008),     # G chunked (> 4096 features) + ragged tail
    ("bf16", 1, 1, 8, 8, None, None),          # T = 1
    ("bf16", 3, 96, 100, 77, 104, 80),         # last chunk straddles d, aligned strides
    ("bf16", 2, 200, 64, 4500, None, 4504),    # two T-tiles (off-diagonal pair) + G chunks
    ("bf16", 3, 64, 300, 520, None, None),     # 2 x 3 ragged output tiles for the direct norm
]


@pytest.mark.parametrize("algo", ["gram", "direct"])
@pytest.mark.parametrize("case", NORM_CASES, ids=lambda c: "-".join(str(x) for x in c))
def test_linear_norm(dp, case, algo):
    dtype, B, T, d_in, d_out, lda, ldg = case
    _say(f"linear norm {algo} {case}")
    A, G = _layer_inputs(dtype, B, T, d_in, d_out, seed=11, lda=lda, ldg=ldg)
    # Stride padding holds NaN: no kernel may let features past d reach a sum.
    nan = np.uint16(0x7FC0) if dtype == "bf16" else np.float32("nan")
    A[:, :, d_in:] = nan
    G[:, :, d_out:] = nan
    ref = _oracle_linear_norm2(A, G, d_in, d_out, dtype)
    At = dev(A, dtype)[:, :, :d_in]
    Gt = dev(G, dtype)[:, :, :d_out]
    n2 = torch.full((B,), 7.0, device="cuda")
    a = dp.DP_NORM_GRAM if algo == "gram" else dp.DP_NORM_DIRECT
    dp.dp_ghost_norm_linear(At, Gt, n2, accumulate=False, algo=a)
    got = host(n2)
    err = rel(got, ref).max()
    _say(f"  max rel err {err:.3e}")
    assert err <= TOL[dtype]
    # accumulate adds onto what is there
    dp.dp_ghost_norm_linear(At, Gt, n2, accumulate=True, algo=a)
    assert rel(host(n2), 2 * ref).max() <= TOL[dtype]


def test_linear_norm_grouped_mixed_algos(dp):
    """Several layers in one call, Gram and direct mixed, summed per example (eq. 6)."""
    B, T = 3, 140
    shapes = [(64, 192), (96, 96), (128, 40), (40, 128)]
    layers, ref = [], np.zeros(B)
    for l, (di, do) in enumerate(shapes):
        A, G = _layer_inputs("bf16", B, T, di, do, seed=100 + l)
        ref += _oracle_linear_norm2(A, G, di, do, "bf16")
        algo = dp.DP_NORM_DIRECT if l % 2 else dp.DP_NORM_GRAM
        layers.append((dev(A, "bf16"), dev(G, "bf16"), algo))
    n2 = torch.zeros(B, device="cuda")
    dp.dp_ghost_norm_linear_grouped(layers, n2)
    assert rel(host(n2), ref).max() <= TOL["bf16"]


def test_linear_norm_deterministic(dp):
    A, G = _layer_inputs("bf16", 4, 256, 256, 512, seed=5)
    At, Gt = dev(A), dev(G)
    outs = []
    for _ in range(3):
        n2 = torch.zeros(4, device="cuda")
        dp.dp_ghost_norm_linear(At, Gt, n2)
        outs.append(host(n2).tobytes())
    assert outs[0] == outs[1] == outs[2]


# ---------------------------------------------------------------------------
# a2: output head (linear d -> V) ghost norm
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("dtype,V,ldz", [("bf16", 5003, 5003), ("bf16", 5003, 5008),
                                         ("f32", 512, 512)])
def test_head_norm(dp, dtype, V, ldz):
    B, T, d = 3, 130, 96
    _say(f"head norm {dtype} V={V} ldz={ldz}")
    ids = gen.draw_ids(3, 1, (B, T), V, "zipf")
    H = gen.draw(3, 2, (B, T, d), 1.0, dtype)
    z = gen._normal(3, 3, (B, T, V), 1.0)
    gz = gen.logit_grads(z, ids)
    Gz = np.zeros((B, T, ldz), np.float32)
    Gz[:, :, :V] = gz
    Gz = gen.f32_to_bf16_bits(Gz) if dtype == "bf16" else Gz
    ref = O.head_norm2(O.decode(H, dtype), O.decode(Gz, dtype), V)
    n2 = torch.zeros(B, device="cuda")
    dp.dp_ghost_norm_linear(dev(H, dtype), dev(Gz, dtype)[:, :, :V], n2)
    err = rel(host(n2), ref).max()
    _say(f"  max rel err {err:.3e}")
    assert err <= TOL[dtype]


# ---------------------------------------------------------------------------
# a3 / a4: bucketing and the input-embedding norm
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("kind,T,V", [("zipf", 130, 50257), ("uniform", 16, 512),
                                      ("same", 64, 1000), ("distinct", 100, 300),
                                      ("zipf", 1, 50257), ("zipf", 1024, 50257),
                                      ("zipf", 256, 50257), ("zipf", 257, 50257),
                                      ("same", 300, 1000),
                                      ("zipf", 4096, 50257),   # the most tokens bucketed in LDS
                                      ("zipf", 4097, 50257),   # past it: the workspace sort
                                      ("zipf", 12000, 50257),  # three sort blocks per example
                                      ("same", 9000, 1000)])   # one run across sort blocks
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("d,lde", [(200, 200), (201, 201), (200, 204)],
                         ids=["d200", "d201-scalar-rows", "d200-lde204"])
def test_embedding_norm_and_buckets(dp, kind, T, V, dtype, d, lde):
    """d = 200: rows read 8 bytes per lane, each example's runs split over
    workgroups (counting rank up to T = 256, the LDS radix sort to 4096, the
    workspace radix sort beyond); d = 201 (rows not a multiple of 8 bytes in
    bf16): the per-feature kernel, which sorts in LDS and is refused past
    T = 4096; lde = 204: padded rows (NaN in the padding, never read)."""
    B = 3
    _say(f"embedding {kind} T={T} V={V} {dtype} d={d} lde={lde}")
    ids = gen.draw_ids(4, 1, (B, T), V, kind)
    dE = gen.draw(4, 2, (B, T, d), 1e-2, dtype)
    ref = O.embedding_norm2(ids, O.decode(dE, dtype), V)
    seg_ref, nu_ref = O.buckets(ids)
    n2 = torch.zeros(B, device="cuda")
    seg = torch.full((B, T), -1, dtype=torch.int32, device="cuda")
    nu = torch.zeros(B, dtype=torch.int32, device="cuda")
    dEd = dev(dE, dtype)
    if lde != d:
        pad = torch.full((B, T, lde), float("nan"), device="cuda", dtype=dEd.dtype)
        pad[:, :, :d] = dEd
        dEd = pad[:, :, :d]
    if T > 4096 and (d * (2 if dtype == "bf16" else 4)) % 8:
        with pytest.raises(dp.DPError, match="8-byte"):
            dp.dp_ghost_norm_embedding(dev(ids), dEd, V, n2, seg_id=seg, n_unique=nu)
        return
    dp.dp_ghost_norm_embedding(dev(ids), dEd, V, n2, seg_id=seg, n_unique=nu)
    np.testing.assert_array_equal(host(seg), seg_ref)
    np.testing.assert_array_equal(host(nu), nu_ref)
    err = rel(host(n2), ref).max()
    _say(f"  max rel err {err:.3e}")
    assert err <= TOL[dtype]


@pytest.mark.parametrize("kind,B,T,V,d,lde", [
    ("zipf", 4, 128, 50257, 768, 768),     # GPT-2 shape: eight 96-feature chunks, four row blocks
    ("zipf", 3, 100, 50257, 200, 208),     # ragged row block, last chunk past d, NaN padding
    ("same", 3, 33, 1000, 64, 64),         # one bucket; a second row block of one row
    ("distinct", 2, 32, 300, 136, 136),    # every id once; one row block, 8-feature tail piece
    ("uniform", 3, 128, 512, 768, 768),    # many repeats per id
    ("zipf", 2, 1, 50257, 8, 8),           # T = 1, one 8-feature piece
])
def test_embedding_norm_pairwise_form(dp, kind, B, T, V, d, lde):
    """bf16 examples up to T = 128 with 16-byte rows take the pairwise form,
    sum_{t,s} [x_t = x_s] <dE_t, dE_s> on MFMA (the ghost-norm identity with
    one-hot inputs), next to a workgroup that ranks the ids for the buckets."""
    _say(f"embedding pairwise {kind} B={B} T={T} V={V} d={d} lde={lde}")
    ids = gen.draw_ids(5, 1, (B, T), V, kind)
    dE = gen.draw(5, 2, (B, T, d), 1e-2, "bf16")
    ref = O.embedding_norm2(ids, O.decode(dE, "bf16"), V)
    seg_ref, nu_ref = O.buckets(ids)
    dEd = dev(dE, "bf16")
    if lde != d:
        pad = torch.full((B, T, lde), float("nan"), device="cuda", dtype=dEd.dtype)
        pad[:, :, :d] = dEd
        dEd = pad[:, :, :d]
    n2 = torch.full((B,), 9.0, device="cuda")
    seg = torch.full((B, T), -1, dtype=torch.int32, device="cuda")
    nu = torch.zeros(B, dtype=torch.int32, device="cuda")
    dp.dp_ghost_norm_embedding(dev(ids), dEd, V, n2, seg_id=seg, n_unique=nu)
    np.testing.assert_array_equal(host(seg), seg_ref)
    np.testing.assert_array_equal(host(nu), nu_ref)
    got = host(n2)
    _say(f"  max rel err {rel(got, ref).max():.3e}")
    assert rel(got, ref).max() <= TOL["bf16"]
    # without buckets (no ranking workgroup), accumulating onto what is there
    dp.dp_ghost_norm_embedding(dev(ids), dEd, V, n2, accumulate=True)
    assert rel(host(n2), 2 * ref).max() <= TOL["bf16"]
    # one of the two bucket outputs alone
    seg2 = torch.full((B, T), -1, dtype=torch.int32, device="cuda")
    dp.dp_ghost_norm_embedding(dev(ids), dEd, V, n2, seg_id=seg2)
    np.testing.assert_array_equal(host(seg2), seg_ref)
    nu2 = torch.zeros(B, dtype=torch.int32, device="cuda")
    dp.dp_ghost_norm_embedding(dev(ids), dEd, V, n2, n_unique=nu2)
    np.testing.assert_array_equal(host(nu2), nu_ref)
    assert rel(host(n2), ref).max() <= TOL["bf16"]


# ---------------------------------------------------------------------------
# a5: tied cross term
# ---------------------------------------------------------------------------
def _tied_inputs(dtype, B, T, V, d, ldz, seed, kind="zipf"):
    ids = gen.draw_ids(seed, 1, (B, T), V, kind)
    dE = gen.draw(seed, 2, (B, T, d), 1e-2, dtype)
    H = gen.draw(seed, 3, (B, T, d), 1.0, dtype)
    z = gen._normal(seed, 4, (B, T, V), 1.0)
    Gz = np.zeros((B, T, ldz), np.float32)
    Gz[:, :, :V] = gen.logit_grads(z, ids)
    if dtype == "bf16":
        Gz = gen.f32_to_bf16_bits(Gz)
    return ids, dE, H, Gz


@pytest.mark.parametrize("dtype,B,T,V,d,ldz", [("f32", 4, 16, 512, 64, 512),
                                               ("bf16", 4, 128, 50257, 768, 50304),
                                               ("bf16", 3, 100, 3000, 200, 3000),
                                               ("bf16", 3, 32, 2000, 40, 2000),
                                               ("bf16", 1, 1, 300, 16, 304),
                                               ("bf16", 3, 130, 5003, 96, 5003),
                                               ("bf16", 2, 256, 50257, 768, 50304),
                                               ("bf16", 2, 260, 777, 100, 784)])
def test_tied_cross_term(dp, dtype, B, T, V, d, ldz):
    """fp32: the register-staged kernel; bf16 up to T = 128: 32 x 32 blocks
    with the tokens in sorted-id order (GPT-2 shape, ragged T, a partial
    16-feature step, T = 1); longer: the direct-load 64-row kernel."""
    _say(f"cross {dtype} B={B} T={T} V={V} d={d}")
    ids, dE, H, Gz = _tied_inputs(dtype, B, T, V, d, ldz, seed=21)
    dEd, Hd, Gzd = O.decode(dE, dtype), O.decode(H, dtype), O.decode(Gz, dtype)
    cross = O.tied_cross(ids, dEd, Hd, Gzd, V)
    n_in = O.embedding_norm2(ids, dEd, V)
    n_out = O.head_norm2(Hd, Gzd, V)
    out = torch.zeros(B, device="cuda")
    dp.dp_tied_cross_term(dev(ids), dev(dE, dtype), dev(H, dtype), dev(Gz, dtype)[:, :, :V], V,
                          out)
    got = host(out)
    bound = TOL[dtype] * np.sqrt(n_in * n_out)
    _say(f"  max |err| / (||gin|| ||gout||) {np.max(np.abs(got - cross) / np.sqrt(n_in * n_out)):.3e}")
    assert np.all(np.abs(got - cross) <= bound)
    # folding 2*cross into a norm: the corrected tied norm of eq. 13
    tied_ref = O.tied_norm2(ids, dEd, Hd, Gzd, V)
    n2 = torch.tensor(n_in + n_out, dtype=torch.float32, device="cuda")
    dp.dp_tied_cross_term(dev(ids), dev(dE, dtype), dev(H, dtype), dev(Gz, dtype)[:, :, :V], V,
                          n2, scale=2.0, accumulate=True)
    assert rel(host(n2), tied_ref).max() <= TOL[dtype]


@pytest.mark.parametrize("kind", ["same", "distinct"])
@pytest.mark.parametrize("T", [64, 128, 200])
def test_tied_cross_term_degenerate_ids(dp, kind, T):
    """Every token of an example with one id (one bucket: every pair (t, s)
    meets at the same logit column, so cross = <sum_t dE_t, sum_s Gz[s, x] h_s>)
    and every id distinct, in the register-direct kernel (T <= 128) and the
    direct-load one (T = 200)."""
    B, V, d = 3, 1000, 128
    _say(f"cross degenerate ids {kind} T={T}")
    ids, dE, H, Gz = _tied_inputs("bf16", B, T, V, d, V, seed=25, kind=kind)
    dEd, Hd, Gzd = O.decode(dE, "bf16"), O.decode(H, "bf16"), O.decode(Gz, "bf16")
    cross = O.tied_cross(ids, dEd, Hd, Gzd, V)
    if kind == "same":
        assert all(len(np.unique(ids[b])) == 1 for b in range(B))
        closed = np.array([dEd[b].sum(0) @ (Gzd[b][:, ids[b, 0]] @ Hd[b]) for b in range(B)])
        np.testing.assert_allclose(cross, closed, rtol=1e-10, atol=1e-12)
    else:
        assert all(len(np.unique(ids[b])) == T for b in range(B))
    n_in = O.embedding_norm2(ids, dEd, V)
    n_out = O.head_norm2(Hd, Gzd, V)
    out = torch.zeros(B, device="cuda")
    dp.dp_tied_cross_term(dev(ids), dev(dE, "bf16"), dev(H, "bf16"), dev(Gz, "bf16"), V, out)
    got = host(out)
    _say(f"  max |err| / (||gin|| ||gout||) {np.max(np.abs(got - cross) / np.sqrt(n_in * n_out)):.3e}")
    assert np.all(np.abs(got - cross) <= TOL["bf16"] * np.sqrt(n_in * n_out))


@pytest.mark.parametrize("T", [100, 200])
def test_tied_cross_term_padded_rows(dp, T):
    """dE and H on 16-byte aligned strides wider than d (NaN in the padding):
    the last feature chunk straddles d, in the register-direct kernel
    (T = 100) and the direct-load one (T = 200)."""
    B, V, d, ld = 2, 900, 100, 104
    ids, dE, H, Gz = _tied_inputs("bf16", B, T, V, d, V, seed=23)
    dEp = np.full((B, T, ld), 0x7FC0, np.uint16)
    Hp = np.full((B, T, ld), 0x7FC0, np.uint16)
    dEp[:, :, :d], Hp[:, :, :d] = dE, H
    dEd, Hd, Gzd = O.decode(dE, "bf16"), O.decode(H, "bf16"), O.decode(Gz, "bf16")
    cross = O.tied_cross(ids, dEd, Hd, Gzd, V)
    n_in = O.embedding_norm2(ids, dEd, V)
    n_out = O.head_norm2(Hd, Gzd, V)
    out = torch.zeros(B, device="cuda")
    dp.dp_tied_cross_term(dev(ids), dev(dEp, "bf16")[:, :, :d], dev(Hp, "bf16")[:, :, :d],
                          dev(Gz, "bf16"), V, out)
    got = host(out)
    assert np.all(np.abs(got - cross) <= TOL["bf16"] * np.sqrt(n_in * n_out))


# ---------------------------------------------------------------------------
# a6: clip factors
# ---------------------------------------------------------------------------
def test_clip_factors(dp):
    n2 = np.array([0.0, 1e-12, 0.25, 1.0, 1.0000001, 4.0, 1e6, 3.3e-3], np.float32)
    for C in (1.0, 0.05, 0.5):
        ref = O.clip_factors(n2.astype(np.float64), C)
        c = torch.empty(len(n2), device="cuda")
        dp.dp_clip_factors(dev(n2), C, c)
        got = host(c)
        assert rel(got, ref).max() <= 1e-6
        assert got[0] == 1.0
        assert np.all(got * np.sqrt(n2.astype(np.float64)) <= C * (1 + 1e-5))


def test_clip_factors_scaled(dp):
    n2 = np.array([0.0, 1e-12, 0.25, 1.0, 1.0000001, 4.0, 1e6, 3.3e-3, 17.0], np.float32)
    for C, scale in ((1.0, 1 / 32), (0.05, 1 / 24), (0.5, 3.0)):
        ref = O.clip_factors(n2.astype(np.float64), C)
        c = torch.full((len(n2),), -1.0, device="cuda")
        cs = torch.empty(len(n2), device="cuda")
        dp.dp_clip_factors_scaled(dev(n2), C, scale, cs, c=c)
        assert rel(host(cs), np.float32(scale) * ref).max() <= 1e-6
        plain = torch.empty(len(n2), device="cuda")
        dp.dp_clip_factors(dev(n2), C, plain)
        assert torch.equal(c, plain)
        cs2 = torch.empty(len(n2), device="cuda")
        dp.dp_clip_factors_scaled(dev(n2), C, scale, cs2)   # without c
        assert torch.equal(cs, cs2)


def test_clip_factors_of_two_norm_parts(dp):
    """The squared norm given as two arrays whose sum is the total (eq. 6 is
    a sum over parameter tensors): the factors are those of the sum."""
    rng = np.random.default_rng(11)
    a = np.array([0.0, 0.0, 0.2, 1.0, 0.5, 3e5, 1e-3, 9.0, 0.7], np.float32)
    b = np.array([0.0, 1e-12, 0.05, 0.0, 0.5000001, 7e5, 2.3e-3, 8.0, 0.3], np.float32)
    a = np.concatenate([a, rng.gamma(2.0, 1.0, 300).astype(np.float32)])
    b = np.concatenate([b, rng.gamma(2.0, 1.0, 300).astype(np.float32)])
    total = a.astype(np.float64) + b.astype(np.float64)
    for C, scale in ((1.0, 1 / 32), (0.5, 1 / 7)):
        ref = O.clip_factors(total, C)
        c = torch.full((len(a),), -1.0, device="cuda")
        cs = torch.empty(len(a), device="cuda")
        dp.dp_clip_factors_scaled2(dev(a), dev(b), C, scale, cs, c=c)
        assert rel(host(c), ref).max() <= 1e-6
        assert rel(host(cs), np.float32(scale) * ref).max() <= 1e-6
        assert host(c)[0] == 1.0


# ---------------------------------------------------------------------------
# a7 / a8: clipped sums
# ---------------------------------------------------------------------------
SUM_CASES = [
    ("f32", 4, 16, 64, 64, None, None),
    ("bf16", 3, 130, 768, 300, None, None),    # ragged K = 390 and N
    ("bf16", 2, 70, 100, 77, None, None),      # unaligned widths
    ("bf16", 2, 64, 520, 264, 528, 272),       # padded strides, two M tiles
    ("f32", 2, 33, 50, 300, 52, None),
]


@pytest.mark.parametrize("transpose", [False, True])
@pytest.mark.parametrize("case", SUM_CASES, ids=lambda c: "-".join(str(x) for x in c))
def test_clipped_sum_linear(dp, case, transpose):
    dtype, B, T, d_in, d_out, lda, ldg = case
    _say(f"clipped sum {case} transpose={transpose}")
    A, G = _layer_inputs(dtype, B, T, d_in, d_out, seed=31, lda=lda, ldg=ldg)
    c = np.linspace(0.2, 1.0, B).astype(np.float32)
    ref = O.clipped_sum_linear(O.decode(A[:, :, :d_in], dtype), O.decode(G[:, :, :d_out], dtype),
                               c.astype(np.float64))
    shape = (d_out, d_in) if transpose else (d_in, d_out)
    out = torch.full(shape, 3.0, device="cuda")
    dp.dp_clipped_grad_sum(dev(A, dtype)[:, :, :d_in], dev(G, dtype)[:, :, :d_out], dev(c), out,
                           transpose_out=transpose)
    got = host(out)
    got = got.T if transpose else got
    err = assert_close(got, ref, TOL[dtype])
    _say(f"  fro / element rel err {err[0]:.3e} / {err[1]:.3e}")
    dp.dp_clipped_grad_sum(dev(A, dtype)[:, :, :d_in], dev(G, dtype)[:, :, :d_out], dev(c), out,
                           transpose_out=transpose, accumulate=True)
    got2 = host(out)
    got2 = got2.T if transpose else got2
    assert_close(got2, 2 * ref, TOL[dtype])


@pytest.mark.parametrize("dtype,T", [("bf16", 64), ("f32", 64), ("bf16", 48)],
                         ids=["bf16-direct-load", "f32-register-staged", "bf16-staged-rows"])
def test_clipped_sum_wide_factor_range(dp, dtype, T):
    """Examples with finite but huge gradients (G scaled by 2^60) next to
    ordinary ones, with clip factors ~2^-60 against 1, as min(1, C/N) gives
    them: every clipped contribution is O(1). The kernels that scale their
    fp32 accumulators by c_prev / c_next at each example boundary then
    multiply by factors up to ~2^61 and back; the sum must keep fp32's
    relative precision across that range (T = 48 takes the kernel that scales
    the rows as it stages them)."""
    B, d_in, d_out = 6, 300, 520
    _say(f"clipped sum wide factor range {dtype} T={T}")
    A, G = _layer_inputs(dtype, B, T, d_in, d_out, seed=37)
    Ad, Gd = O.decode(A, dtype), O.decode(G, dtype)
    big = [1, 3, 5]
    Gd[big] *= 2.0 ** 60                     # exact: a power of two
    G = gen.f32_to_bf16_bits(Gd.astype(np.float32)) if dtype == "bf16" else Gd.astype(np.float32)
    assert np.array_equal(O.decode(G, dtype), Gd)
    c = np.array([1.0, 0.5 * 2.0 ** -60, 0.7, 0.3 * 2.0 ** -60, 1.0, 2.0 ** -61], np.float32)
    ref = O.clipped_sum_linear(Ad, Gd, c.astype(np.float64))
    # every example contributes at the same scale
    parts = [np.abs(c[i] * O.linear_grad(Ad[i], Gd[i])).max() for i in range(B)]
    assert max(parts) / min(parts) < 1e3
    out = torch.zeros((d_in, d_out), device="cuda")
    dp.dp_clipped_grad_sum(dev(A, dtype), dev(G, dtype), dev(c), out)
    got = host(out)
    assert np.isfinite(got).all()
    err = assert_close(got, ref, TOL[dtype])
    _say(f"  fro / element rel err {err[0]:.3e} / {err[1]:.3e}")


# bf16 sums on 16-byte aligned rows with T % 32 == 0 take the direct-load
# kernel (rows loaded straight into LDS, 4-stage ring, per-example factors on
# the accumulators); these cases pin its edges.
DL_CASES = [
    # B, T, d_in, d_out, lda, ldg, c
    (5, 32, 300, 520, 304, 528, [0.0, 1.0, 0.5, 0.0, 0.25]),   # c = 0 first/middle, ragged tiles
    (1, 32, 64, 64, None, None, [0.7]),                       # one stage (less than the ring)
    (3, 96, 256, 256, None, None, [1.0, 1.0, 1.0]),            # all c = 1, exact tiles
    (4, 64, 520, 264, 528, 272, [0.9, 0.1, 0.6, 0.0]),         # last example skipped
]


@pytest.mark.parametrize("transpose", [False, True])
@pytest.mark.parametrize("case", DL_CASES, ids=lambda c: "-".join(str(x) for x in c[:6]))
def test_clipped_sum_direct_load(dp, case, transpose):
    B, T, d_in, d_out, lda, ldg, cl = case
    _say(f"direct-load sum {case[:6]} transpose={transpose}")
    A, G = _layer_inputs("bf16", B, T, d_in, d_out, seed=37, lda=lda, ldg=ldg)
    # Stride padding holds NaN: the kernel loads whole 256-column tile rows,
    # and what lies past the valid columns may only reach unstored outputs.
    if lda:
        A[:, :, d_in:] = 0x7FC0
    if ldg:
        G[:, :, d_out:] = 0x7FC0
    c = np.asarray(cl, np.float32)
    ref = O.clipped_sum_linear(O.decode(A[:, :, :d_in], "bf16"),
                               O.decode(G[:, :, :d_out], "bf16"), c.astype(np.float64))
    shape = (d_out, d_in) if transpose else (d_in, d_out)
    out = torch.full(shape, 3.0, device="cuda")
    dp.dp_clipped_grad_sum(dev(A, "bf16")[:, :, :d_in], dev(G, "bf16")[:, :, :d_out], dev(c), out,
                           transpose_out=transpose)
    got = host(out)
    got = got.T if transpose else got
    assert np.isfinite(got).all()
    err = assert_close(got, ref, TOL["bf16"])
    _say(f"  fro / element rel err {err[0]:.3e} / {err[1]:.3e}")


NOISED_CASES = [
    # dtype, B, T, [(d_in, d_out), ...]
    ("bf16", 3, 64, [(300, 520), (256, 256)]),   # direct-load kernel, ragged tiles
    ("bf16", 2, 70, [(100, 77), (64, 40)]),      # general kernel, row lengths not 4-aligned
    ("f32", 2, 33, [(50, 300), (72, 64)]),       # fp32 general kernel
]


@pytest.mark.parametrize("transpose", [False, True])
@pytest.mark.parametrize("case", NOISED_CASES, ids=lambda c: f"{c[0]}-B{c[1]}-T{c[2]}")
def test_clipped_sum_noised(dp, case, transpose):
    """Clipped sum with the Gaussian mechanism fused into its store equals the
    oracle's add_noise(prior + sum) with the same (seed, tensor id, step), and
    the unfused GPU path (grouped sum, then dp_add_noise)."""
    dtype, B, T, shapes = case
    sigma, C, seed, step = 0.7, 0.9, 0xC0FFEE, 11
    tids = [5, 9]
    acc = [False, True]
    c = np.linspace(0.3, 1.0, B).astype(np.float32)
    layers, outs, refs, priors = [], [], [], []
    for l, (di, do) in enumerate(shapes):
        A, G = _layer_inputs(dtype, B, T, di, do, seed=60 + l)
        layers.append((dev(A, dtype), dev(G, dtype)))
        S = O.clipped_sum_linear(O.decode(A, dtype), O.decode(G, dtype), c.astype(np.float64))
        S = S.T if transpose else S
        prior = gen.draw(61 + l, 3, S.shape, 1e-2, "f32") if acc[l] else np.zeros(S.shape, np.float32)
        priors.append(prior)
        outs.append(dev(prior.copy()))
        refs.append(O.add_noise(prior.astype(np.float64) + S, sigma, C, B, seed, tids[l], step))
    dp.dp_clipped_grad_sum_noised_grouped(layers, outs, dev(c), tids, sigma, C, B, seed, step,
                                          accumulate=acc, transpose_out=transpose)
    plain = [dev(p.copy()) for p in priors]
    dp.dp_clipped_grad_sum_grouped(layers, plain, dev(c), transpose_out=transpose)
    for l in range(len(shapes)):
        got = host(outs[l])
        assert_close(got, refs[l], TOL[dtype])
        if acc[l]:
            plain[l] += dev(priors[l])
        dp.dp_add_noise(plain[l], sigma, C, B, seed, tids[l], step)
        _say(f"  layer {l}: fused vs oracle {fro_rel(got, refs[l]):.2e}, "
             f"fused vs unfused {fro_rel(got, host(plain[l])):.2e}")
        # The fused launch may swap the GEMM operands (its rows must be the
        # output's rows). Where bf16 rows are scaled while staged (T not a
        # multiple of the stage depth) the rounding then falls on the other
        # operand; elsewhere the two paths agree to fp32 accumulation.
        exact = dtype == "f32" or T % 64 == 0
        assert_close(got, host(plain[l]), 1e-5 if exact else 2e-3)


SPLIT_CASES = [
    # B, T, [(d_in, d_out), ...], c (None: linspace); widths multiples of 8 (16-byte rows)
    (4, 64, [(520, 304)], None),                           # 6 ragged tiles, all split
    (4, 64, [(2304, 3072)] * 3, None),                     # 324 tiles: 256 whole + 68 split
    (5, 96, [(768, 768), (296, 1000)], [0.5, 0.0, 1.0, 0.25, 0.7]),  # ranges start mid-example
]


@pytest.mark.parametrize("case", SPLIT_CASES, ids=lambda c: f"B{c[0]}-T{c[1]}-{len(c[2])}")
def test_clipped_sum_split_tail(dp, case):
    """The workspace form splits the last round's tiles along K; its result
    equals the unsplit call's up to fp32 rounding, and the oracle's."""
    B, T, shapes, cl = case
    sigma, C, seed, step = 0.5, 1.1, 77, 4
    c = np.asarray(cl if cl is not None else np.linspace(0.3, 1.0, B), np.float32)
    layers, refs, priors = [], [], []
    for l, (di, do) in enumerate(shapes):
        A, G = _layer_inputs("bf16", B, T, di, do, seed=130 + l)
        layers.append((dev(A, "bf16"), dev(G, "bf16")))
        S = O.clipped_sum_linear(O.decode(A, "bf16"), O.decode(G, "bf16"), c.astype(np.float64))
        prior = gen.draw(131 + l, 3, S.shape, 1e-2, "f32") if l % 2 else np.zeros(S.shape, np.float32)
        priors.append(prior)
        refs.append(O.add_noise(prior.astype(np.float64) + S, sigma, C, B, seed, 10 + l, step))
    tids = [10 + l for l in range(len(shapes))]
    acc = [bool(l % 2) for l in range(len(shapes))]
    split = [dev(p.copy()) for p in priors]
    grp = dp.LinearGroup(layers, split)
    assert grp  # the group passes its workspace
    grp.clipped_sum_noised(dev(c), tids, sigma, C, B, seed, step, accumulate=acc)
    plain = [dev(p.copy()) for p in priors]
    dp.dp_clipped_grad_sum_noised_grouped(layers, plain, dev(c), tids, sigma, C, B, seed, step,
                                          accumulate=acc)
    assert grp._split_ws is not None   # these launches do split their tail
    for l in range(len(shapes)):
        got, ref = host(split[l]), refs[l]
        assert np.isfinite(got).all()
        assert_close(got, host(plain[l]), 1e-5)
        err = assert_close(got, ref, TOL["bf16"])
        _say(f"  split tail layer {l}: vs oracle {err[0]:.2e} / {err[1]:.2e}")


def test_clipped_sum_many_examples(dp):
    """B above the direct-load kernel's factor table (4096): general kernel."""
    B, T, d_in, d_out = 4100, 32, 64, 72
    A, G = _layer_inputs("bf16", B, T, d_in, d_out, seed=38)
    c = gen.draw(38, 3, (B,), 1.0, "f32")
    c = np.abs(c).astype(np.float32)
    ref = O.clipped_sum_linear(O.decode(A, "bf16"), O.decode(G, "bf16"), c.astype(np.float64))
    out = torch.zeros((d_in, d_out), device="cuda")
    dp.dp_clipped_grad_sum(dev(A, "bf16"), dev(G, "bf16"), dev(c), out)
    assert_close(host(out), ref, TOL["bf16"])


def test_clipped_sum_grouped(dp):
    B, T = 2, 96
    shapes = [(64, 192), (200, 96), (768, 768)]
    c = np.array([0.5, 0.9], np.float32)
    layers, outs, refs = [], [], []
    for l, (di, do) in enumerate(shapes):
        A, G = _layer_inputs("bf16", B, T, di, do, seed=40 + l)
        layers.append((dev(A), dev(G)))
        outs.append(torch.zeros(di, do, device="cuda"))
        refs.append(O.clipped_sum_linear(O.decode(A, "bf16"), O.decode(G, "bf16"),
                                         c.astype(np.float64)))
    dp.dp_clipped_grad_sum_grouped(layers, outs, dev(c))
    for o, r in zip(outs, refs):
        assert_close(host(o), r, TOL["bf16"])


@pytest.mark.parametrize("dtype,B,T,V,d,kind", [("f32", 4, 16, 512, 64, "uniform"),
                                                ("bf16", 3, 130, 5003, 96, "zipf"),
                                                ("bf16", 2, 64, 300, 40, "same"),
                                                ("bf16", 16, 1024, 50257, 64, "zipf")])
def test_clipped_sum_embedding(dp, dtype, B, T, V, d, kind):
    _say(f"embedding sum {dtype} B={B} T={T} V={V} {kind}")
    ids = gen.draw_ids(6, 1, (B, T), V, kind)
    dE = gen.draw(6, 2, (B, T, d), 1e-2, dtype)
    c = np.linspace(0.3, 1.0, B).astype(np.float32)
    ref = O.clipped_sum_embedding(ids, O.decode(dE, dtype), c.astype(np.float64), V)
    out = torch.full((V, d), 5.0, device="cuda")
    dp.dp_clipped_grad_sum(None, dev(dE, dtype), dev(c), out, ids=dev(ids), V=V)
    err = assert_close(host(out), ref, TOL[dtype])
    _say(f"  fro / element rel err {err[0]:.3e} / {err[1]:.3e}")
    outT = torch.zeros((d, V), device="cuda")
    dp.dp_clipped_grad_sum(None, dev(dE, dtype), dev(c), outT, ids=dev(ids), V=V,
                           transpose_out=True)
    assert_close(host(outT).T, ref, TOL[dtype])


def test_clipped_sum_embedding_invalid_ids(dp):
    """Ids outside [0, V) contribute nothing (header contract); they sort after
    every valid id, so each valid id still forms one run."""
    B, T, V, d = 4, 96, 300, 72
    ids = gen.draw_ids(12, 1, (B, T), V, "zipf")
    bad = np.zeros((B, T), bool)
    bad[:, ::7] = True
    ids = ids.copy()
    ids[bad] = np.where(np.arange(bad.sum()) % 2 == 0, -1, V + 7)
    dE = gen.draw(12, 2, (B, T, d), 1e-2, "bf16")
    c = np.linspace(0.4, 1.0, B).astype(np.float32)
    ids_ref = np.where(bad, 0, ids)
    dE_ref = O.decode(dE, "bf16").copy()
    dE_ref[bad] = 0.0
    ref = O.clipped_sum_embedding(ids_ref, dE_ref, c.astype(np.float64), V)
    out = torch.full((V, d), 2.0, device="cuda")
    dp.dp_clipped_grad_sum(None, dev(dE, "bf16"), dev(c), out, ids=dev(ids), V=V)
    assert_close(host(out), ref, TOL["bf16"])


@pytest.mark.parametrize("T,ldz", [(100, 1001), (64, 1008)])   # general / direct-load head
def test_tied_clipped_sum_one_buffer(dp, T, ldz):
    """Tied E: the head sum and the embedding sum land in one [V, d] buffer."""
    dtype, B, V, d = "bf16", 3, 1001, 64
    ids, dE, H, Gz = _tied_inputs(dtype, B, T, V, d, ldz, seed=8)
    c = np.array([0.3, 1.0, 0.7], np.float32)
    dEd, Hd, Gzd = O.decode(dE, dtype), O.decode(H, dtype), O.decode(Gz, dtype)
    ref = (O.clipped_sum_head(Hd, Gzd, c.astype(np.float64), V)
           + O.clipped_sum_embedding(ids, dEd, c.astype(np.float64), V))
    out = torch.empty((V, d), device="cuda")
    dp.dp_clipped_grad_sum(dev(Gz, dtype)[:, :, :V], dev(H, dtype), dev(c), out)   # Gz^T H -> [V, d]
    dp.dp_clipped_grad_sum(None, dev(dE, dtype), dev(c), out, ids=dev(ids), V=V, accumulate=True)
    assert_close(host(out), ref, TOL[dtype])


# ---------------------------------------------------------------------------
# a9: noise
# ---------------------------------------------------------------------------
def test_noise_matches_oracle_stream(dp):
    n = 1_000_003
    S = gen.draw(9, 1, (n,), 1e-3, "f32")
    sigma, C, B = 1.3, 0.5, 24
    ref = O.add_noise(S.astype(np.float64), sigma, C, B, seed=0x1234_5678_9ABC, tensor_id=7,
                      step=42)
    g = dev(S)
    dp.dp_add_noise(g, sigma, C, B, seed=0x1234_5678_9ABC, tensor_id=7, step=42)
    got = host(g)
    err = assert_close(got, ref, TOL["f32"])
    _say(f"  noise fro / element rel err {err[0]:.3e} / {err[1]:.3e}")
    z = (got.astype(np.float64) * B - S) / (sigma * C)
    zref = O.gaussian(n, seed=0x1234_5678_9ABC, tensor_id=7, step=42)
    zerr = np.abs(z - zref)
    _say(f"  z max abs err {zerr.max():.3e}, rms {np.sqrt((zerr ** 2).mean()):.3e}")
    # fp32 Box-Muller on the hardware log/sqrt/sin/cos: absolute error well
    # below 1e-4 even in the tails (|z| up to ~5.5 here).
    assert zerr.max() < 1e-4
    assert abs(z.mean()) < 5 / np.sqrt(n)
    assert abs(z.std() - 1) < 5 * np.sqrt(0.5 / n)


def test_noise_sigma_zero_and_unaligned(dp):
    S = gen.draw(9, 2, (1001,), 1.0, "f32")
    g = dev(S)
    dp.dp_add_noise(g, 0.0, 1.0, 4, 1, 2, 3)
    assert_close(host(g), S / 4, 1e-7)
    g2 = dev(S)
    sub = g2[1:]  # 4-byte but not 16-byte aligned
    dp.dp_add_noise(sub, 1.0, 1.0, 0, 1, 2, 3)
    ref = O.add_noise(S[1:].astype(np.float64), 1.0, 1.0, 0, 1, 2, 3)
    assert_close(host(sub), ref, TOL["f32"])


@pytest.mark.parametrize("n,offset", [(1_000_003, 0), (1001, 1), (4, 0), (3, 2)])
def test_noise_fill(dp, n, offset):
    """Noise alone equals dp_add_noise on zeros bit for bit, without reading
    the output (it starts as NaN), aligned or not, with a ragged tail."""
    sigma, C, B = 1.3, 0.5, 24
    buf = torch.full((n + offset,), float("nan"), device="cuda")
    out = buf[offset:]
    dp.dp_noise_fill(out, sigma, C, B, seed=99, tensor_id=4, step=11)
    zeros = torch.zeros(n, device="cuda")
    dp.dp_add_noise(zeros, sigma, C, B, seed=99, tensor_id=4, step=11)
    assert torch.equal(out, zeros)
    ref = O.add_noise(np.zeros(n), sigma, C, B, seed=99, tensor_id=4, step=11)
    assert_close(host(out), ref, TOL["f32"])


# ---------------------------------------------------------------------------
# The whole step on the tiny configs, against oracle.step
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("name", ["c1", "c1-tied"])
def test_tiny_step(dp, name):
    wl = gen.make_workload(name)
    ref = O.step(wl, seed=3, step_id=5)
    B, T, dt = wl.B, wl.T, wl.dtype
    lin = wl.linears[0]
    A, G = dev(lin.A), dev(lin.G)
    h = wl.head
    ids, dE = dev(h.ids), dev(h.dE)
    n2 = torch.zeros(B, device="cuda")
    dp.dp_ghost_norm_linear(A, G, n2)
    dp.dp_ghost_norm_embedding(ids, dE, h.V, n2, accumulate=True)
    if h.H is not None:
        Hd, Gzd = dev(h.H), dev(h.Gz)[:, :, :h.V]
        dp.dp_ghost_norm_linear(Hd, Gzd, n2, accumulate=True)
        dp.dp_tied_cross_term(ids, dE, Hd, Gzd, h.V, n2, scale=2.0, accumulate=True)
    assert rel(host(n2), ref["norms"]["total"]).max() <= TOL[dt]
    c = torch.empty(B, device="cuda")
    dp.dp_clip_factors(n2, wl.C, c)
    assert rel(host(c), ref["c"]).max() <= TOL[dt]
    S = torch.empty(lin.d_in, lin.d_out, device="cuda")
    dp.dp_clipped_grad_sum(A, G, c, S)
    E = torch.empty(h.V, h.d, device="cuda")
    if h.H is not None:
        dp.dp_clipped_grad_sum(Gzd, Hd, c, E)
        dp.dp_clipped_grad_sum(None, dE, c, E, ids=ids, V=h.V, accumulate=True)
    else:
        dp.dp_clipped_grad_sum(None, dE, c, E, ids=ids, V=h.V)
    assert_close(host(S), ref["sums"]["linear"], TOL[dt])
    assert_close(host(E), ref["sums"]["wte"], TOL[dt])
    dp.dp_add_noise(S, wl.sigma, wl.C, B, 3, 0, 5)
    dp.dp_add_noise(E, wl.sigma, wl.C, B, 3, 1, 5)
    assert_close(host(S), ref["noisy"]["linear"], TOL[dt])
    assert_close(host(E), ref["noisy"]["wte"], TOL[dt])
    # The same step in the benchmark's order: the noise fused into the GEMM
    # store (the tied head written first), then the embedding part added with
    # the factors c/B; an embedding without a tied head starts from noise alone.
    S2 = torch.empty(lin.d_in, lin.d_out, device="cuda")
    E2 = torch.full((h.V, h.d), float("nan"), device="cuda")
    c2, c_b = torch.empty(B, device="cuda"), torch.empty(B, device="cuda")
    dp.dp_clip_factors_scaled(n2, wl.C, 1.0 / B, c_b, c=c2)
    assert torch.equal(c2, c)
    if h.H is not None:
        dp.dp_clipped_grad_sum_noised_grouped([(A, G), (Gzd, Hd)], [S2, E2], c, [0, 1],
                                              wl.sigma, wl.C, B, 3, 5)
    else:
        dp.dp_clipped_grad_sum_noised_grouped([(A, G)], [S2], c, [0], wl.sigma, wl.C, B, 3, 5)
        dp.dp_noise_fill(E2, wl.sigma, wl.C, B, 3, 1, 5)
    dp.dp_clipped_grad_sum(None, dE, c_b, E2, ids=ids, V=h.V, accumulate=True)
    assert_close(host(S2), ref["noisy"]["linear"], TOL[dt])
    assert_close(host(E2), ref["noisy"]["wte"], TOL[dt])


# ---------------------------------------------------------------------------
# Full GPT-2-small sizes, in the grouped launches the benchmark times,
# checked on sampled examples / rows the oracle can compute one at a time.
# ---------------------------------------------------------------------------
def test_full_size_gpt2_body_sampled(dp):
    wl = gen.make_workload("c2", layers=[0, 1, 2, 3, 44, 45, 46, 47])
    B = wl.B
    _say(f"full-size body: {len(wl.linears)} layers, B={B}, T={wl.T}")
    layers = [(dev(l.A), dev(l.G)) for l in wl.linears]
    n2 = torch.zeros(B, device="cuda")
    dp.dp_ghost_norm_linear_grouped(layers, n2)
    got = host(n2)
    for i in (0, B - 1):
        ref = sum(O.sqnorm(O.linear_grad(O.decode(l.A[i], "bf16"), O.decode(l.G[i], "bf16")))
                  for l in wl.linears)
        assert rel(got[i], ref) <= TOL["bf16"], i
    # clipped sum with a known c: sampled rows of S against the oracle
    c = (0.25 + 0.75 * np.arange(B) / B).astype(np.float32)
    outs = [torch.empty(l.d_in, l.d_out, device="cuda") for l in wl.linears]
    dp.dp_clipped_grad_sum_grouped(layers, outs, dev(c))
    for l, o in zip(wl.linears[:4], outs[:4]):
        rows = [0, l.d_in // 2 + 3, l.d_in - 1]
        Ad = O.decode(l.A[:, :, rows], "bf16")         # [B, T, 3]
        Gd = O.decode(l.G, "bf16")
        ref = sum(c[i] * Ad[i].T @ Gd[i] for i in range(B))
        assert_close(host(o)[rows], ref, TOL["bf16"])


@pytest.mark.parametrize("algo", ["gram", "direct"])
def test_full_size_long_sequence(dp, algo):
    """T = 1024 at GPT-2 widths (the long-sequence config's shapes): the
    multi-tile Gram and the direct norm, for a body layer and the head."""
    a = dp.DP_NORM_GRAM if algo == "gram" else dp.DP_NORM_DIRECT
    B, T = 2, 1024
    A, G = _layer_inputs("bf16", B, T, 768, 2304, seed=51, g_std=1e-3)
    n2 = torch.zeros(B, device="cuda")
    dp.dp_ghost_norm_linear(dev(A, "bf16"), dev(G, "bf16"), n2, algo=a)
    ref = _oracle_linear_norm2(A, G, 768, 2304, "bf16")
    _say(f"  long-T {algo} body max rel err {rel(host(n2), ref).max():.3e}")
    assert rel(host(n2), ref).max() <= TOL["bf16"]
    V, d = 50257, 768
    ids, dE, H, Gz = _tied_inputs("bf16", 1, T, V, d, 50304, seed=52)
    n_out = torch.zeros(1, device="cuda")
    dp.dp_ghost_norm_linear(dev(H, "bf16"), dev(Gz, "bf16")[:, :, :V], n_out, algo=a)
    ref_out = O.sqnorm(O.head_grad(O.decode(H[0], "bf16"), O.decode(Gz[0], "bf16"), V))
    assert rel(host(n_out)[0], ref_out) <= TOL["bf16"]


def _norm_group(n_tiles, B, spe, cus):
    """Examples per work item of the direct-load direct norm, as the library
    chooses them: the fewest rounds times the item length (stages of its
    examples plus ~6 of fill and drain). Only names the case below."""
    best, best_cost = 1, None
    for eg in range(1, min(B, 512) + 1):
        rounds = -(-n_tiles * -(-B // eg) // cus)
        cost = rounds * (eg * spe + 6)
        if best_cost is None or cost < best_cost:
            best, best_cost = eg, cost
    return best


@pytest.mark.parametrize("B,T,d_in,d_out,lda,ldg", [
    (45, 1024, 300, 520, 304, 520),     # 2 x 3 ragged tiles, 32 stages per example
    (13, 64, 2500, 1500, 2504, 1504),   # 10 x 6 ragged tiles, 2 stages per example
])
def test_direct_norm_example_groups(dp, B, T, d_in, d_out, lda, ldg):
    """The direct-load direct norm gives a work item a run of consecutive
    examples when that shortens the launch (eq. 6 per example, reduced at each
    example boundary): a ragged last group, ragged output tiles, NaN in the
    stride padding."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    tiles = -(-d_in // 256) * -(-d_out // 256)
    eg = _norm_group(tiles, B, T // 32, cus)
    _say(f"direct norm groups B={B} T={T} {d_in}x{d_out}: {eg} examples per item on {cus} CUs")
    assert eg > 1 and B % eg != 0
    A, G = _layer_inputs("bf16", B, T, d_in, d_out, seed=61, lda=lda, ldg=ldg)
    nan = np.uint16(0x7FC0)
    A[:, :, d_in:] = nan
    G[:, :, d_out:] = nan
    ref = _oracle_linear_norm2(A, G, d_in, d_out, "bf16")
    n2 = torch.full((B,), 3.0, device="cuda")
    At, Gt = dev(A, "bf16")[:, :, :d_in], dev(G, "bf16")[:, :, :d_out]
    dp.dp_ghost_norm_linear(At, Gt, n2, accumulate=False, algo=dp.DP_NORM_DIRECT)
    got = host(n2)
    _say(f"  max rel err {rel(got, ref).max():.3e}")
    assert rel(got, ref).max() <= TOL["bf16"]
    dp.dp_ghost_norm_linear(At, Gt, n2, accumulate=True, algo=dp.DP_NORM_DIRECT)
    assert rel(host(n2), 2 * ref).max() <= TOL["bf16"]
    # The partials are reduced in a fixed order: the same bits every call.
    n2b = torch.zeros(B, device="cuda")
    dp.dp_ghost_norm_linear(At, Gt, n2b, accumulate=False, algo=dp.DP_NORM_DIRECT)
    assert host(n2b).tobytes() == got.tobytes()


def test_full_size_gpt2_head_sampled(dp):
    wl = gen.make_workload("c3")
    h = wl.head
    B = wl.B
    _say(f"full-size tied head V={h.V} B={B} T={wl.T}")
    ids, dE, H = dev(h.ids), dev(h.dE), dev(h.H)
    Gz = dev(h.Gz)[:, :, :h.V]
    n_out = torch.zeros(B, device="cuda")
    dp.dp_ghost_norm_linear(H, Gz, n_out)
    n_in = torch.zeros(B, device="cuda")
    seg = torch.empty((B, wl.T), dtype=torch.int32, device="cuda")
    nu = torch.empty(B, dtype=torch.int32, device="cuda")
    dp.dp_ghost_norm_embedding(ids, dE, h.V, n_in, seg_id=seg, n_unique=nu)
    cross = torch.zeros(B, device="cuda")
    dp.dp_tied_cross_term(ids, dE, H, Gz, h.V, cross)
    seg_ref, nu_ref = O.buckets(h.ids)
    np.testing.assert_array_equal(host(seg), seg_ref)
    np.testing.assert_array_equal(host(nu), nu_ref)
    ref_in = O.embedding_norm2(h.ids, O.decode(h.dE, "bf16"), h.V)
    assert rel(host(n_in), ref_in).max() <= TOL["bf16"]
    for i in (0, B - 1):
        gE = O.embedding_grad(h.ids[i], O.decode(h.dE[i], "bf16"), h.V)
        gW = O.head_grad(O.decode(h.H[i], "bf16"), O.decode(h.Gz[i], "bf16"), h.V)
        assert rel(host(n_out)[i], O.sqnorm(gW)) <= TOL["bf16"]
        cr = float(np.sum(gE * gW))
        assert abs(host(cross)[i] - cr) <= TOL["bf16"] * np.sqrt(O.sqnorm(gE) * O.sqnorm(gW))


@pytest.mark.parametrize("n_layers", [52, 53])
def test_layer_table_extremes(dp, n_layers):
    """As many layers as one launch's table holds (52: every lane of the
    work-item decode used) and one more (two launches): grouped Gram norms
    with fused biases, direct norms and the grouped clipped sum against the
    oracle, all layers of distinct widths."""
    B, T = 3, 64
    _say(f"layer table: {n_layers} layers")
    layers, biases, sums, ref_n2, refs = [], [], [], np.zeros(B), []
    c = np.array([0.3, 1.0, 0.55], np.float32)
    for l in range(n_layers):
        di, do = 32 + 8 * (l % 7), 40 + 16 * (l % 11)
        A, G = _layer_inputs("bf16", B, T, di, do, seed=300 + l)
        Ad, Gd = O.decode(A, "bf16"), O.decode(G, "bf16")
        ref_n2 = ref_n2 + O.linear_norm2(Ad, Gd)
        algo = dp.DP_NORM_DIRECT if l % 5 == 4 else dp.DP_NORM_GRAM
        layers.append((dev(A, "bf16"), dev(G, "bf16"), algo))
        if l % 3 == 0:
            ref_n2 = ref_n2 + O.vector_norm2(None, Gd)
            biases.append(torch.zeros(B, do, device="cuda"))
        else:
            biases.append(None)
        refs.append(O.clipped_sum_linear(Ad, Gd, c.astype(np.float64)))
        sums.append(torch.empty(di, do, device="cuda"))
    n2 = torch.zeros(B, device="cuda")
    dp.LinearGroup(layers, bias_grads=biases).ghost_norm(n2)
    assert rel(host(n2), ref_n2).max() <= TOL["bf16"]
    dp.dp_clipped_grad_sum_grouped([(a, g) for a, g, _ in layers], sums, dev(c))
    worst = max(assert_close(host(o), r, TOL["bf16"])[1] for o, r in zip(sums, refs))
    _say(f"  norm rel err {rel(host(n2), ref_n2).max():.2e}, worst clipped sum {worst:.2e}")
    assert worst <= TOL["bf16"]
