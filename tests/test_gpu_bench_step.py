"""The benchmark's step (bench.Step: every entry point, two clipped-sum
launches and the sums on a second stream) against the oracle's step, on
reduced workloads: the order of its launches across streams is part of what
is checked."""
import os
import sys

import numpy as np
import pytest

import oracle as O
from workloads import gen
from tests.helpers import TOL, fro_rel, rel

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def parts():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    sys.path.insert(0, ROOT)
    import bench
    import paper_2609_40335_amd.dpghost as dp
    dp.lib()
    return bench, dp


CASES = [
    ("c1-tied", dict(full_params=True)),                              # fp32, every parameter
    ("gpt2-full", dict(B=4, T=32, n_blocks=1, V=4000, ldz=4032)),     # bf16, tied, every parameter
    ("c5", dict(B=2, T=64, n_blocks=1, V=3000, ldz=3008)),            # bf16, untied head + E_in
]


@pytest.mark.parametrize("name,kw", CASES, ids=[c[0] for c in CASES])
def test_bench_step_matches_oracle(parts, name, kw):
    bench, dp = parts
    wl = gen.make_workload(name, **kw)
    st = bench.Step(wl, dp, torch)
    st.run()
    torch.cuda.synchronize()
    ref = O.step(wl, seed=1234, step_id=0)
    tol = TOL[wl.dtype]
    assert rel(st.total_norm2().cpu().numpy(), ref["norms"]["total"]).max() <= tol
    assert rel(st.c.cpu().numpy(), ref["c"]).max() <= tol
    got = {l.name: o for l, o in zip(wl.linears, st.outs)}
    got["wte"] = st.E
    if wl.head.H is not None and not wl.head.tied:
        got["lm_head"] = st.W
    for v, o in zip(wl.vectors, st.vec_outs):
        got[v.name] = o
    if wl.n_pos:
        got["wpe"] = st.P
    assert set(got) == set(ref["noisy"])
    for k, t in got.items():
        err = fro_rel(t.cpu().numpy(), ref["noisy"][k])
        assert err <= tol, (k, err)


def _say(*a):
    print(*a, flush=True)


def test_full_size_step_sampled(parts):
    """The benchmark's step at its full size (GPT-2-small, tied head V = 50257,
    B = 32, T = 128: every GEMM-shaped tensor in one noised launch with its
    split tail, the embedding rows on the second stream) against the oracle
    on what it can compute one piece at a time: every example's norm (for
    the clip factors), and sampled rows of the noisy sums of five linear
    layers and of the tied matrix, noise included."""
    bench, dp = parts
    wl = gen.make_workload("gpt2-step", ldz=50304)
    B, T, L, h = wl.B, wl.T, len(wl.linears), wl.head
    _say(f"full-size step: {L} linears + tied head V={h.V}, B={B}, T={T}")
    st = bench.Step(wl, dp, torch)
    st.run()
    torch.cuda.synchronize()
    seed, step_id = 1234, 0                     # the step's noise key (first step)
    norms = O.per_example_norms(wl)
    _say("  oracle norms done")
    c = O.clip_factors(norms["total"], wl.C)
    tol = TOL["bf16"]
    assert rel(st.total_norm2().cpu().numpy(), norms["total"]).max() <= tol
    assert rel(st.c.cpu().numpy(), c).max() <= tol
    sc = wl.sigma * wl.C
    for l in (0, 1, 2, 3, L - 1):
        lay = wl.linears[l]
        rows = [0, lay.d_in // 2 + 3, lay.d_in - 1]
        S = sum(c[i] * O.linear_grad(O.decode(lay.A[i][:, rows], "bf16"),
                                     O.decode(lay.G[i], "bf16")) for i in range(B))
        z = np.stack([O.gaussian(lay.d_out, seed, l, step_id, start=r * lay.d_out) for r in rows])
        got = st.outs[l].cpu().numpy()[rows]
        err = fro_rel(got, (S + sc * z) / B)
        # the noise (~sigma C) dwarfs the clipped sum (~1e-3 here): the sum
        # is also checked alone, with the oracle's noise taken out
        err_s = fro_rel(got * B - sc * z, S)
        _say(f"  linear {l} ({lay.d_in}x{lay.d_out}) rows {rows}: fro rel err {err:.2e}, "
             f"clipped sum alone {err_s:.2e}")
        assert err <= tol and err_s <= tol, (l, err, err_s)
    # tied matrix rows: the most frequent id, an id no token carries, the last
    # rows (the head's last output tiles)
    ids = h.ids
    counts = np.bincount(ids.ravel(), minlength=h.V)
    absent = int(np.flatnonzero(counts == 0)[0])
    rows = [int(counts.argmax()), absent, h.V - 300, h.V - 1]
    n = len(rows)
    where = {v: k for k, v in enumerate(rows)}
    S = np.zeros((n, h.d))
    for i in range(B):
        ids_map = np.array([where.get(int(v), n) for v in ids[i]])
        gE = O.embedding_grad(ids_map, O.decode(h.dE[i], "bf16"), n + 1)[:n]
        gW = O.head_grad(O.decode(h.H[i], "bf16"), O.decode(h.Gz[i][:, rows], "bf16"), n)
        S += c[i] * (gE + gW)
    z = np.stack([O.gaussian(h.d, seed, L, step_id, start=r * h.d) for r in rows])
    got = st.E.cpu().numpy()[rows]
    err = fro_rel(got, (S + sc * z) / B)
    err_s = fro_rel(got * B - sc * z, S)
    _say(f"  tied matrix rows {rows}: fro rel err {err:.2e}, clipped sum alone {err_s:.2e}")
    assert err <= tol and err_s <= tol


def _snapshot(st):
    outs = [st.total_norm2(), st.c, st.c_b, *st.outs, st.E]
    for name in ("W", "P"):
        t = getattr(st, name, None)
        if t is not None:
            outs.append(t)
    outs += list(getattr(st, "vec_outs", None) or [])
    return [t.detach().clone() for t in outs]


@pytest.mark.parametrize("name,kw", [
    ("gpt2-full", dict(B=4, T=32, n_blocks=1, V=4000, ldz=4032)),
    ("gpt2-step", dict(ldz=50304)),
], ids=["gpt2-full-small", "gpt2-step"])
def test_bench_step_is_deterministic(parts, name, kw):
    """Two runs of the benchmark's step with the same noise key give the same
    bits in every output: its reductions have a fixed order (no float
    atomics), across both streams and the split tail."""
    bench, dp = parts
    wl = gen.make_workload(name, **kw)
    st = bench.Step(wl, dp, torch)
    runs = []
    for _ in range(2):
        st.step_id = 0
        st.run()
        torch.cuda.synchronize()
        runs.append(_snapshot(st))
    for k, (a, b) in enumerate(zip(*runs)):
        assert torch.equal(a, b), k
