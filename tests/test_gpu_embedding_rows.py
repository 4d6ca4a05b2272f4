"""GPU: the embedding form of the clipped sum in two calls (dp_embedding_rows,
then dp_embedding_rows_add) against the one-call form and the fp64 oracle.
Batches of up to 16384 tokens are sorted in one workgroup, larger ones by the
radix sort through the workspace (to B*T = 65536 at V = 50257).

The two-call form adds each run's finished row with one fp32 addition, as the
one-call form does, so the two agree bit for bit; the oracle bounds both.
"""
import sys

import numpy as np
import pytest

import oracle as O
from workloads import gen
from tests.helpers import TOL, assert_close, dev, host

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


def _case(seed, dtype, B, T, V, d, kind, bad_every=0):
    ids = gen.draw_ids(seed, 1, (B, T), V, kind).copy()
    bad = np.zeros((B, T), bool)
    if bad_every:
        bad[:, ::bad_every] = True
        ids[bad] = np.where(np.arange(bad.sum()) % 2 == 0, -1, V + 3)
    dE = gen.draw(seed, 2, (B, T, d), 1e-2, dtype)
    c = np.linspace(0.3, 1.0, B).astype(np.float32)
    if B > 2:
        c[1] = 0.0                      # an example with factor 0 adds zeros
    return ids, dE, c, bad


def _oracle(ids, dE, c, bad, V, dtype):
    ids_ref = np.where(bad, 0, ids)
    dE_ref = O.decode(dE, dtype).copy()
    dE_ref[bad] = 0.0                   # ids outside [0, V) contribute nothing
    return O.clipped_sum_embedding(ids_ref, dE_ref, c.astype(np.float64), V)


CASES = [
    # dtype, B, T, V, d, ids, invalid-id stride, transposed output
    ("f32", 4, 16, 512, 64, "uniform", 0, False),
    ("bf16", 3, 50, 97, 70, "zipf", 7, False),      # K = 150 (ragged block), d % 4 != 0
    ("bf16", 2, 100, 1000, 128, "zipf", 0, True),   # transposed [d, V] output
    ("bf16", 4, 64, 50, 64, "same", 0, False),      # one run through every block
    ("f32", 1, 1, 10, 8, "uniform", 0, False),      # a single token
    ("bf16", 32, 128, 50257, 768, "zipf", 0, False),  # GPT-2 step
    ("bf16", 64, 256, 50257, 768, "zipf", 0, False),  # B*T = 16384, the most one workgroup sorts
    # past it, the radix sort through the workspace:
    ("bf16", 65, 256, 50257, 768, "zipf", 0, False),  # B*T = 16640, a ragged last sort block
    ("bf16", 128, 256, 50257, 768, "zipf", 0, False),  # B*T = 32768
    ("bf16", 256, 256, 50257, 256, "zipf", 0, False),  # B*T = 65536, the most a 32-bit key holds
    ("f32", 40, 500, 3000, 40, "zipf", 9, True),      # B*T = 20000, invalid ids, transposed
    ("bf16", 20, 1000, 64, 32, "same", 0, False),     # one run across every sort block
]


@pytest.mark.parametrize("dtype,B,T,V,d,kind,bad_every,tr", CASES)
def test_rows_then_add_equals_one_call(dp, dtype, B, T, V, d, kind, bad_every, tr):
    _say(f"embedding rows {dtype} B={B} T={T} V={V} d={d} {kind} bad={bad_every} tr={tr}")
    ids, dE, c, bad = _case(5, dtype, B, T, V, d, kind, bad_every)
    shape = (d, V) if tr else (V, d)
    prior = torch.randn(shape, device="cuda", generator=torch.Generator("cuda").manual_seed(1))
    one = prior.clone()
    dp.dp_clipped_grad_sum(None, dev(dE, dtype), dev(c), one, ids=dev(ids), V=V,
                           transpose_out=tr, accumulate=True)
    rows = dp.EmbeddingRows(B, T, V, d)
    two = prior.clone()
    rows.compute(dev(dE, dtype), dev(ids), dev(c))
    rows.add_to(two, transpose_out=tr)
    torch.cuda.synchronize()
    assert torch.equal(one, two)
    ref = _oracle(ids, dE, c, bad, V, dtype)
    got = host(two - prior)
    err = assert_close(got.T if tr else got, ref, TOL[dtype])
    _say(f"  fro / element rel err vs oracle {err[0]:.3e} / {err[1]:.3e}")


def test_workspace_reused_with_new_ids(dp):
    """A second compute on the same workspace replaces the run list (a
    different number of runs) before its add."""
    B, T, V, d = 4, 96, 300, 72
    rows = dp.EmbeddingRows(B, T, V, d)
    for seed, kind in ((3, "zipf"), (4, "same"), (5, "uniform")):
        ids, dE, c, bad = _case(seed, "bf16", B, T, V, d, kind)
        out = torch.zeros((V, d), device="cuda")
        rows.compute(dev(dE, "bf16"), dev(ids), dev(c))
        rows.add_to(out)
        ref = _oracle(ids, dE, c, bad, V, "bf16")
        assert_close(host(out), ref, TOL["bf16"], kind)


def test_rows_beside_a_writer_of_out(dp):
    """The intended use: rows on a second stream while the main stream
    writes `out`; the add follows both. Same result as the one-call form
    after the writer."""
    B, T, V, d = 8, 64, 4000, 256
    ids, dE, c, _ = _case(9, "bf16", B, T, V, d, "zipf")
    dEd, idsd, cd = dev(dE, "bf16"), dev(ids), dev(c)
    base = torch.randn((V, d), device="cuda", generator=torch.Generator("cuda").manual_seed(2))
    rows = dp.EmbeddingRows(B, T, V, d)
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    out = torch.empty((V, d), device="cuda")
    ev = torch.cuda.Event()
    start = torch.cuda.Event()
    start.record(main)
    side.wait_event(start)
    with torch.cuda.stream(side):
        rows.compute(dEd, idsd, cd)
        ev.record(side)
    out.copy_(base)                     # the writer, on the main stream
    main.wait_event(ev)
    rows.add_to(out)
    ref = base.clone()
    dp.dp_clipped_grad_sum(None, dEd, cd, ref, ids=idsd, V=V, accumulate=True)
    torch.cuda.synchronize()
    assert torch.equal(out, ref)
