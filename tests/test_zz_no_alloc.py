"""The no-allocation grouped norm (dp_ghost_norm_linear_bias_grouped_noalloc,
partials in the library's static device scratch) against the workspace form
of the same entry point, and the oracle: two calls in a row on one device,
the second smaller, so the second reads nothing the first left behind."""
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


def _case(dp, seed, B, T, shapes, with_bias):
    """(layers, bias tensors or None, oracle squared norms incl. biases, bias refs)."""
    layers, bias, ref, bias_ref = [], [], np.zeros(B), []
    for l, (di, do, algo) in enumerate(shapes):
        A = gen.draw(seed, 2 * l, (B, T, di), 1.0, "bf16")
        G = gen.draw(seed, 2 * l + 1, (B, T, do), 1e-2, "bf16")
        Ad, Gd = O.decode(A, "bf16"), O.decode(G, "bf16")
        ref += O.linear_norm2(Ad, Gd)
        layers.append((dev(A, "bf16"), dev(G, "bf16"), algo))
        if with_bias and l % 2 == 0:
            bias.append(torch.full((B, do), float("nan"), device="cuda"))
            g = np.stack([O.vector_grad(None, Gd[i]) for i in range(B)])
            bias_ref.append(g)
            ref += (g * g).sum(axis=1)
        else:
            bias.append(None)
            bias_ref.append(None)
    return layers, (bias if with_bias else None), ref, bias_ref


CALLS = [
    # B, T, [(d_in, d_out, algo)], biases: GPT-2 widths with a chunked
    # 5000-feature output, one layer forced to the direct norm
    (8, 128, [(768, 2304, 0), (768, 768, 0), (3072, 768, 2), (768, 5000, 0)], True),
    (2, 32, [(256, 512, 0), (64, 72, 2)], False),                       # smaller, after it
]


def test_noalloc_norm_matches_workspace_form(dp):
    for k, (B, T, shapes, with_bias) in enumerate(CALLS):
        _say(f"no-alloc grouped norm call {k}: B={B} T={T} layers={shapes} biases={with_bias}")
        layers, bias, ref, bias_ref = _case(dp, 70 + k, B, T, shapes, with_bias)
        n2_static = torch.full((B,), float("nan"), device="cuda")
        dp.dp_ghost_norm_linear_bias_grouped_noalloc(layers, bias, n2_static)
        got_bias = [None if b is None else b.clone() for b in (bias or [])]
        n2_ws = torch.full((B,), float("nan"), device="cuda")
        if bias is not None:
            for b in bias:
                if b is not None:
                    b.fill_(float("nan"))
        dp.LinearGroup(layers, bias_grads=bias).ghost_norm(n2_ws)
        torch.cuda.synchronize()
        # the same kernels in the same order: the same bits
        assert torch.equal(n2_static, n2_ws)
        for a, b in zip(got_bias, bias or []):
            if b is not None:
                assert torch.equal(a, b)
        err = rel(host(n2_static), ref).max()
        _say(f"  vs oracle: max rel err {err:.2e}")
        assert err <= TOL["bf16"]
        for a, r in zip(got_bias, bias_ref):
            if r is not None:
                assert_close(host(a), r, TOL["bf16"], "bias gradient")
        # accumulate = 1 adds onto the prior
        dp.dp_ghost_norm_linear_bias_grouped_noalloc(layers, bias, n2_static, accumulate=True)
        torch.cuda.synchronize()
        assert rel(host(n2_static), 2 * ref).max() <= TOL["bf16"]


def test_noalloc_norm_rejects_a_call_beyond_its_scratch(dp):
    # 17 x 17 direct-norm tiles per example at B = 8192: 9.5 MB of partials
    B, d = 8192, 4352
    A = torch.zeros((B, 1, d), dtype=torch.bfloat16, device="cuda")
    n2 = torch.zeros(B, device="cuda")
    with pytest.raises(dp.DPError, match="static scratch"):
        dp.dp_ghost_norm_linear_bias_grouped_noalloc([(A, A, dp.DP_NORM_DIRECT)], None, n2)
    torch.cuda.synchronize()
