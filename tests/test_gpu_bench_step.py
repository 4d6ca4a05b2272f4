"""The benchmark's step (bench.Step: every entry point, the grouped
clipped-sum launch and the sums on a second stream) against the oracle's
step: the order of its launches across streams is part of what is checked.

Each step runs twice: with the workload's noise (sigma = 1, which at these
sizes is ~1e3 times the clipped sum, so that comparison sees the noise and
little else), and with sigma = 0, whose outputs are the clipped sums of eq. 3
divided by B and are compared with the oracle's sums element by element."""
import dataclasses
import os
import sys

import numpy as np
import pytest

import oracle as O
from workloads import gen
from tests.helpers import TOL, assert_close, rel

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SEED = 1234          # the step's noise key (bench.Step)


@pytest.fixture(scope="module")
def parts():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    sys.path.insert(0, ROOT)
    import bench
    import paper_2609_40335_amd.dpghost as dp
    dp.lib()
    return bench, dp


def _say(*a):
    print(*a, flush=True)


def _outputs(st, wl):
    got = {l.name: o for l, o in zip(wl.linears, st.outs)}
    got["wte"] = st.E
    if wl.head.H is not None and not wl.head.tied:
        got["lm_head"] = st.W
    for v, o in zip(wl.vectors, st.vec_outs):
        got[v.name] = o
    if wl.n_pos:
        got["wpe"] = st.P
    return got


def _run(st, sigma, step_id=0):
    st.wl = dataclasses.replace(st.wl, sigma=sigma)
    st.step_id = step_id
    st.run()
    torch.cuda.synchronize()


CASES = [
    ("c1-tied", dict(full_params=True)),                              # fp32, every parameter
    ("gpt2-full", dict(B=4, T=32, n_blocks=1, V=4000, ldz=4032)),     # bf16, tied, every parameter
    ("c5", dict(B=2, T=64, n_blocks=1, V=3000, ldz=3008)),            # bf16, untied head + E_in
    ("c4", dict(B=3, T=256, n_blocks=1, V=3000, ldz=3008)),           # bf16, T = 256 whole-example Gram
    # d = 64: every layer takes the direct norm at T = 64, so the step keeps the
    # examples' gradient tiles and forms the clipped sums from them
    ("c5", dict(B=3, T=64, n_blocks=1, V=3000, ldz=3008, d=64)),
]


def _case_id(c):
    return c[0] + ("-store" if c[1].get("d") == 64 else "")


@pytest.mark.parametrize("name,kw", CASES, ids=[_case_id(c) for c in CASES])
def test_bench_step_matches_oracle(parts, name, kw):
    bench, dp = parts
    _say(f"bench step {name} {kw}")
    wl = gen.make_workload(name, **kw)
    st = bench.Step(wl, dp, torch)
    _run(st, wl.sigma)
    ref = O.step(wl, seed=SEED, step_id=0)
    tol = TOL[wl.dtype]
    assert rel(st.total_norm2().cpu().numpy(), ref["norms"]["total"]).max() <= tol
    assert rel(st.c.cpu().numpy(), ref["c"]).max() <= tol
    got = _outputs(st, wl)
    assert set(got) == set(ref["noisy"])
    for k, t in got.items():
        assert_close(t.cpu().numpy(), ref["noisy"][k], tol, f"noisy {k}")
    # sigma = 0: the same launches on both streams, outputs = sums / B
    _run(st, 0.0)
    for k, t in got.items():
        f, e = assert_close(t.cpu().numpy(), ref["sums"][k] / wl.B, tol, f"sum {k}")
        _say(f"  {k}: clipped sum fro / element rel err {f:.2e} / {e:.2e}")


NONFINITE_CASES = [
    ("gpt2-full", dict(B=4, T=32, n_blocks=1, V=4000, ldz=4032)),   # direct-load GEMM, split tail
    ("gpt2-full", dict(B=4, T=40, n_blocks=1, V=4000, ldz=4032)),   # rows scaled while staged
    ("c1-tied", dict(full_params=True)),                              # fp32
    ("c5", dict(B=4, T=64, n_blocks=1, V=3000, ldz=3008, d=64)),      # per-example gradient store
]


@pytest.mark.parametrize("name,kw", NONFINITE_CASES,
                         ids=["T32", "T40", "c1-tied-f32", "c5-store"])
def test_nonfinite_example_left_out(parts, name, kw):
    """One NaN activation in example 1 and one inf embedding-output gradient
    in example 2: their squared norms are not finite, their clip factors are
    0 (eq. 2 read for non-finite norms), and every output of the step is
    finite and equals the oracle's, which leaves both examples out."""
    bench, dp = parts
    _say(f"non-finite examples {name} {kw}")
    wl = gen.make_workload(name, **kw)
    bf = wl.dtype == "bf16"
    wl.linears[0].A = wl.linears[0].A.copy()
    wl.linears[0].A[1, 3, 5] = 0x7FC0 if bf else np.nan
    wl.head.dE = wl.head.dE.copy()
    wl.head.dE[2, 0, 7] = 0x7F80 if bf else np.inf
    ref = O.step(wl, seed=SEED, step_id=0)
    assert np.all(ref["c"][[1, 2]] == 0.0) and np.all(ref["c"][[0, 3]] > 0)
    st = bench.Step(wl, dp, torch)
    tol = TOL[wl.dtype]
    for sigma in (wl.sigma, 0.0):
        _run(st, sigma)
        n2 = st.total_norm2().cpu().numpy()
        assert not np.isfinite(n2[[1, 2]]).any()
        assert rel(n2[[0, 3]], ref["norms"]["total"][[0, 3]]).max() <= tol
        c = st.c.cpu().numpy()
        assert np.all(c[[1, 2]] == 0.0)
        assert rel(c[[0, 3]], ref["c"][[0, 3]]).max() <= tol
        for k, t in _outputs(st, wl).items():
            got = t.cpu().numpy()
            assert np.isfinite(got).all(), k
            want = ref["noisy"][k] if sigma else ref["sums"][k] / wl.B
            assert_close(got, want, tol, f"{k} sigma={sigma}")


def _tied_rows(h, c, rows, B):
    """Rows of sum_i c_i (g_in,i + g_out,i) for the listed ids (eq. 8, 11)."""
    n = len(rows)
    where = {v: k for k, v in enumerate(rows)}
    SE, SW = np.zeros((n, h.d)), np.zeros((n, h.d))
    for i in range(B):
        if c[i] == 0.0:
            continue
        ids_map = np.array([where.get(int(v), n) for v in h.ids[i]])
        SE += c[i] * O.embedding_grad(ids_map, O.decode(h.dE[i], "bf16"), n + 1)[:n]
        if h.H is not None:
            SW += c[i] * O.head_grad(O.decode(h.H[i], "bf16"), O.decode(h.Gz[i][:, rows], "bf16"), n)
    return SE, SW


@pytest.mark.parametrize("name", ["gpt2-step", "c4", "c5"])
def test_full_size_step_sampled(parts, name):
    """The benchmark's step at full size, with the algorithm choice left to
    the library (DP_NORM_AUTO):
      gpt2-step  GPT-2-small, tied head V = 50257, B = 32, T = 128
      c4         DistilGPT2 (6 blocks), tied head, B = 64, T = 256: the
                 whole-example Gram, the head's logit features in chunks,
                 B*T = 16384 tokens sorted for the embedding sum
      c5         GPT-2-small, untied head + input embedding, B = 16, T = 1024:
                 the direct norm, the noise-filled embedding then its sum
    against the oracle on what it computes one piece at a time: every
    example's norm (for the clip factors), and sampled rows of five linear
    layers and of the embedding / head matrices, with noise and at sigma = 0."""
    bench, dp = parts
    wl = gen.make_workload(name, ldz=50304)
    B, T, L, h = wl.B, wl.T, len(wl.linears), wl.head
    _say(f"full-size step {name}: {L} linears + {'tied' if h.tied else 'untied'} head "
         f"V={h.V}, B={B}, T={T}")
    st = bench.Step(wl, dp, torch)
    _run(st, wl.sigma)
    n2_gpu, c_gpu = st.total_norm2().cpu().numpy(), st.c.cpu().numpy()
    lin_rows = {l: [0, wl.linears[l].d_in // 2 + 3, wl.linears[l].d_in - 1]
                for l in (0, 1, 2, 3, L - 1)}
    counts = np.bincount(h.ids.ravel(), minlength=h.V)
    v_rows = [int(counts.argmax()), int(np.flatnonzero(counts == 0)[0]), h.V - 300, h.V - 1]
    noisy = {l: st.outs[l].cpu().numpy()[r] for l, r in lin_rows.items()}
    noisy["E"] = st.E.cpu().numpy()[v_rows]
    if not h.tied:
        noisy["W"] = st.W.cpu().numpy()[v_rows]
    _run(st, 0.0)
    plain = {l: st.outs[l].cpu().numpy()[r] for l, r in lin_rows.items()}
    plain["E"] = st.E.cpu().numpy()[v_rows]
    if not h.tied:
        plain["W"] = st.W.cpu().numpy()[v_rows]
    _say("  GPU steps done")

    norms = O.per_example_norms(wl)
    _say("  oracle norms done")
    c = O.clip_factors(norms["total"], wl.C)
    tol = TOL["bf16"]
    assert rel(n2_gpu, norms["total"]).max() <= tol
    assert rel(c_gpu, c).max() <= tol
    sc = wl.sigma * wl.C

    def check(what, got_noisy, got_plain, S, tid, row_starts, width):
        z = np.stack([O.gaussian(width, SEED, tid, 0, start=r0) for r0 in row_starts])
        fn, en = assert_close(got_noisy, (S + sc * z) / B, tol, f"{what} noisy")
        fp, ep = assert_close(got_plain, S / B, tol, f"{what} sum")
        _say(f"  {what}: noisy {fn:.1e}/{en:.1e}, clipped sum {fp:.1e}/{ep:.1e} (fro/element)")

    for l, rows in lin_rows.items():
        lay = wl.linears[l]
        S = sum(c[i] * O.linear_grad(O.decode(lay.A[i][:, rows], "bf16"),
                                     O.decode(lay.G[i], "bf16"))
                for i in range(B) if c[i] != 0.0)
        check(f"linear {l} ({lay.d_in}x{lay.d_out}) rows {rows}", noisy[l], plain[l], S, l,
              [r * lay.d_out for r in rows], lay.d_out)
    SE, SW = _tied_rows(h, c, v_rows, B)
    starts = [r * h.d for r in v_rows]
    if h.tied:
        check(f"tied matrix rows {v_rows}", noisy["E"], plain["E"], SE + SW, L, starts, h.d)
    else:
        check(f"input embedding rows {v_rows}", noisy["E"], plain["E"], SE, L, starts, h.d)
        check(f"output head rows {v_rows}", noisy["W"], plain["W"], SW, L + 1, starts, h.d)


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
    _say(f"determinism {name}")
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
