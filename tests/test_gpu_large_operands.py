"""GPU: an operand spanning more than 4 GiB, past the reach of 32-bit buffer
offsets. The direct-load GEMM (clipped sum, direct norm) moves its
descriptors' base to each stage's first row; the Gram kernels address each
example from its own base. Checked element by element against the fp64
oracle on the same inputs.

G is a [B, T, 200] bf16 view of rows 65536 elements long (128 KiB), so its
33 * 1024 rows span 4.43 GB: every example after the 32nd starts past 4 GiB.
Columns 200..255 of each row hold NaN: the last 256-wide tile loads them and
they only reach outputs that are never stored.
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


B, T, D_IN, D_OUT, LDG = 33, 1024, 64, 200, 65536


@pytest.fixture(scope="module")
def inputs():
    A = gen.draw(7, 1, (B, T, D_IN), 1.0, "bf16")
    Gv = gen.draw(7, 2, (B, T, D_OUT), 1e-2, "bf16")
    c = np.linspace(0.2, 1.0, B).astype(np.float32)
    c[3] = 0.0                       # left out of the sum
    Gfull = torch.empty((B, T, LDG), dtype=torch.bfloat16, device="cuda")
    Gfull[:, :, :D_OUT] = dev(Gv, "bf16")
    Gfull[:, :, D_OUT:256] = float("nan")
    assert Gfull.numel() * 2 > (4 << 30)
    Ad, Gd = dev(A, "bf16"), Gfull[:, :, :D_OUT]
    Ao, Go = O.decode(A, "bf16"), O.decode(Gv, "bf16")
    yield Ad, Gd, c, Ao, Go
    del Gfull
    torch.cuda.empty_cache()


@pytest.mark.parametrize("transpose", [False, True])
def test_clipped_sum_past_4gib(dp, inputs, transpose):
    Ad, Gd, c, Ao, Go = inputs
    _say(f"clipped sum with G spanning 4.43 GB, transpose={transpose}")
    ref = O.clipped_sum_linear(Ao, Go, c.astype(np.float64))
    out = torch.full((D_OUT, D_IN) if transpose else (D_IN, D_OUT), 3.0, device="cuda")
    dp.dp_clipped_grad_sum(Ad, Gd, dev(c), out, transpose_out=transpose)
    got = host(out)
    err = assert_close(got.T if transpose else got, ref, TOL["bf16"])
    _say(f"  fro / element rel err {err[0]:.3e} / {err[1]:.3e}")


def test_noised_sum_past_4gib_split_tail(dp, inputs):
    """The one tile of this launch is split into K ranges (the split tail):
    each range starts past 4 GiB from its own stage. sigma = 0, so the
    result is the clipped sum over B."""
    Ad, Gd, c, Ao, Go = inputs
    ref = O.clipped_sum_linear(Ao, Go, c.astype(np.float64)) / B
    out = torch.full((D_IN, D_OUT), 3.0, device="cuda")
    grp = dp.LinearGroup([(Ad, Gd)], [out])
    grp.clipped_sum_noised(dev(c), [0], 0.0, 1.0, B, seed=1, step=0)
    err = assert_close(host(out), ref, TOL["bf16"])
    _say(f"  noised (sigma = 0) fro / element rel err {err[0]:.3e} / {err[1]:.3e}")


@pytest.mark.parametrize("algo", ["gram", "direct"])
def test_norms_past_4gib(dp, inputs, algo):
    Ad, Gd, c, Ao, Go = inputs
    ref = O.linear_norm2(Ao, Go)
    n2 = torch.zeros(B, device="cuda")
    dp.dp_ghost_norm_linear(Ad, Gd, n2, algo=dp.DP_NORM_GRAM if algo == "gram"
                            else dp.DP_NORM_DIRECT)
    err = rel(host(n2), ref).max()
    _say(f"  {algo} norm max rel err {err:.3e}")
    assert err <= TOL["bf16"]
