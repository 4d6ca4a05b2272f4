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
