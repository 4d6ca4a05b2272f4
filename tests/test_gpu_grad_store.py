"""GPU: the per-example gradient store, the materialising form of the clipped
sum (eq. 2-3) for long sequences. dp_ghost_norm_linear_store takes every
layer's direct norm and keeps each example's fp32 gradient tiles;
dp_clipped_grad_sum_noised_store then adds them with the clip factors and the
fused Gaussian mechanism. Checked element by element against the fp64 oracle
(with the noise, and without it so that the noise cannot hide the sums), and
against the GEMM form of the same call.
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


NAN = np.uint16(0x7FC0)

CASES = [
    # B, T, [(d_in, d_out, lda, ldg), ...], c (None: linspace 0.3 .. 1)
    # ragged 256-wide tiles, NaN in the stride padding, one example left out (c = 0)
    (5, 64, [(300, 520, 304, 520), (256, 256, 256, 256)], [0.5, 0.0, 1.0, 0.25, 0.7]),
    # 32 stages per example, two examples per work item (boundaries inside the K loop)
    (45, 1024, [(300, 520, 304, 520)], None),
    # three layers of mixed shapes, 136-feature rows
    (3, 96, [(64, 768, 64, 768), (768, 64, 768, 64), (128, 136, 136, 136)], None),
    # 53 layers: two launches of the layer table, store slots numbered across them
    (2, 64, [(64, 72, 64, 72)] * 53, None),
]


def _case_inputs(B, T, shapes, seed):
    layers_np, layers = [], []
    for l, (di, do, lda, ldg) in enumerate(shapes):
        A = gen.draw(seed + l, 1, (B, T, lda), 1.0, "bf16")
        G = gen.draw(seed + l, 2, (B, T, ldg), 1e-2, "bf16")
        A[:, :, di:] = NAN
        G[:, :, do:] = NAN
        layers_np.append((O.decode(A[:, :, :di], "bf16"), O.decode(G[:, :, :do], "bf16")))
        layers.append((dev(A, "bf16")[:, :, :di], dev(G, "bf16")[:, :, :do]))
    return layers_np, layers


@pytest.mark.parametrize("transpose", [False, True, "mixed"])
@pytest.mark.parametrize("case", CASES, ids=lambda c: f"B{c[0]}-T{c[1]}-{len(c[2])}layers")
def test_store_norms_and_noised_sums(dp, case, transpose):
    """transpose: every output [d_in, d_out], every one [d_out, d_in], or the
    layers alternating (the layout is chosen per layer)."""
    B, T, shapes, c = case
    c = np.linspace(0.3, 1.0, B) if c is None else np.asarray(c)
    c = c.astype(np.float32)
    _say(f"gradient store B={B} T={T} shapes={shapes} transpose={transpose}")
    layers_np, layers = _case_inputs(B, T, shapes, seed=80)
    tiles = sum(-(-di // 256) * -(-do // 256) for di, do, _, _ in shapes)
    nbytes = dp.dp_grad_store_bytes(layers)
    assert nbytes == B * tiles * 256 * 256 * 4 + -(-(B * tiles * 4) // 256) * 256
    store = torch.empty(nbytes, dtype=torch.uint8, device="cuda")

    # norms: the direct form's bits, and the oracle's values
    n2 = torch.full((B,), 4.0, device="cuda")
    dp.dp_ghost_norm_linear_store(layers, n2, store)
    n2d = torch.zeros(B, device="cuda")
    dp.dp_ghost_norm_linear_grouped([(A, G, dp.DP_NORM_DIRECT) for A, G in layers], n2d)
    assert host(n2).tobytes() == host(n2d).tobytes()
    ref_n2 = sum(O.linear_norm2(A, G) for A, G in layers_np)
    _say(f"  norms max rel err {rel(host(n2), ref_n2).max():.3e}")
    assert rel(host(n2), ref_n2).max() <= TOL["bf16"]
    # accumulate adds onto what is there (and rewrites the same tiles)
    n2a = n2.clone()
    dp.dp_ghost_norm_linear_store(layers, n2a, store, accumulate=True)
    assert rel(host(n2a), 2 * ref_n2).max() <= TOL["bf16"]

    sigma, C, seed, step = 0.7, 0.9, 0xBEEF, 5
    tids = [3 + l for l in range(len(shapes))]
    acc = [l % 2 == 1 for l in range(len(shapes))]
    tr = [l % 2 == 1 for l in range(len(shapes))] if transpose == "mixed" \
        else [transpose] * len(shapes)
    sums, priors = [], []
    for l, (A, G) in enumerate(layers_np):
        S = O.clipped_sum_linear(A, G, c.astype(np.float64))
        sums.append(S.T if tr[l] else S)
        priors.append(gen.draw(90 + l, 3, sums[-1].shape, 1e-2, "f32") if acc[l]
                      else np.zeros(sums[-1].shape, np.float32))

    # without noise (sigma = 0, B_norm = 0): the sums themselves
    outs0 = [dev(p.copy()) for p in priors]
    dp.dp_clipped_grad_sum_noised_store(layers, outs0, dev(c), tids, 0.0, C, 0, seed, step,
                                        store, accumulate=acc, transpose_out=tr)
    for l in range(len(shapes)):
        err = assert_close(host(outs0[l]), priors[l].astype(np.float64) + sums[l], TOL["bf16"],
                           f"layer {l} sum")
        _say(f"  layer {l}: noise-free fro / element rel err {err[0]:.2e} / {err[1]:.2e}")

    # with noise: the oracle's add_noise(prior + sum), and the GEMM form's output
    outs = [dev(p.copy()) for p in priors]
    dp.dp_clipped_grad_sum_noised_store(layers, outs, dev(c), tids, sigma, C, B, seed, step,
                                        store, accumulate=acc, transpose_out=tr)
    gemm = [dev(p.copy()) for p in priors]
    for l in range(len(shapes)):   # the GEMM form takes one layout per call
        dp.dp_clipped_grad_sum_noised_grouped([layers[l]], [gemm[l]], dev(c), [tids[l]], sigma,
                                              C, B, seed, step, accumulate=acc[l],
                                              transpose_out=tr[l])
    for l in range(len(shapes)):
        ref = O.add_noise(priors[l].astype(np.float64) + sums[l], sigma, C, B, seed, tids[l], step)
        got = host(outs[l])
        assert np.isfinite(got).all()
        assert_close(got, ref, TOL["bf16"], f"layer {l} noised")
        # the same noise draws; the sums differ by fp32 rounding order only
        assert_close(got, host(gemm[l]), 1e-4, f"layer {l} store vs GEMM")


def test_store_reused_across_steps(dp):
    """A second step with other inputs and a smaller batch through the same
    store buffer: no tile of the first step leaks into the second."""
    shapes = [(300, 520, 304, 520)]
    store = None
    for step, (B, seed) in enumerate([(6, 100), (4, 200)]):
        layers_np, layers = _case_inputs(B, 64, shapes, seed)
        nbytes = dp.dp_grad_store_bytes(layers)
        if store is None:
            store = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        assert store.numel() >= nbytes
        c = np.linspace(1.0, 0.4, B).astype(np.float32)
        n2 = torch.zeros(B, device="cuda")
        dp.dp_ghost_norm_linear_store(layers, n2, store)
        out = torch.zeros((300, 520), device="cuda")
        dp.dp_clipped_grad_sum_noised_store(layers, [out], dev(c), [1], 0.0, 1.0, 0, 1, step,
                                            store)
        A, G = layers_np[0]
        assert rel(host(n2), O.linear_norm2(A, G)).max() <= TOL["bf16"]
        assert_close(host(out), O.clipped_sum_linear(A, G, c.astype(np.float64)), TOL["bf16"])
