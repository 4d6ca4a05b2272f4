"""The parity bars themselves (CPU): the element-wise bound rejects the
mistakes a whole-tensor Frobenius ratio lets through at the bf16 bar, and
accepts what fp32 accumulation order leaves behind."""
import numpy as np

from tests.helpers import TOL, assert_close, elem_rel, fro_rel
from workloads import gen


def test_zeroed_tile_of_a_head_sized_output_is_rejected():
    # the tied head's clipped sum is [V, d] = [50257, 768]; one 32 x 32 MFMA
    # block left at zero moves the Frobenius ratio by ~5e-3 only
    rng = np.random.default_rng(0)
    y = rng.standard_normal((50257, 768), dtype=np.float32)
    x = y.copy()
    x[20000:20032, 256:288] = 0.0
    assert fro_rel(x, y) < TOL["bf16"]
    assert elem_rel(x, y) > 0.5


def test_dropped_token_of_an_embedding_sum_is_rejected():
    # B = 16, T = 1024 embedding clipped sum with Zipf ids over V = 50257:
    # one token's row missing moves the Frobenius ratio by well under 1 %
    B, T, V, d = 16, 1024, 50257, 64
    ids = gen.draw_ids(6, 1, (B, T), V, "zipf").reshape(-1)
    rng = np.random.default_rng(1)
    e = rng.standard_normal((B * T, d)) * 1e-2
    y = np.zeros((V, d))
    np.add.at(y, ids, e)
    counts = np.bincount(ids, minlength=V)
    k = int(np.flatnonzero(counts[ids] == 3)[0])   # a token whose id occurs 3 times
    x = y.copy()
    x[ids[k]] -= e[k]
    assert fro_rel(x, y) < TOL["bf16"]
    assert elem_rel(x, y) > 0.1


def test_zero_rows_must_stay_zero():
    y = np.zeros((4, 8))
    y[1] = np.arange(8) + 1.0
    x = y.copy()
    x[3, 2] = 1e-3 * np.sqrt(np.mean(y * y))      # a row that should be empty is not
    assert abs(elem_rel(x, y) - 1e-3) < 1e-12
    x[3, 2] = np.nan
    assert elem_rel(x, y) == np.inf


def test_fp32_rounding_is_accepted():
    rng = np.random.default_rng(2)
    y = rng.standard_normal((300, 517)) * 1e-3
    y[:, :5] *= 1e-6                                 # near-cancelled elements
    x = (y * (1 + 1e-6 * rng.standard_normal(y.shape))).astype(np.float32)
    f, e = assert_close(x, y, TOL["f32"])
    assert e < 1e-5 and f < 1e-5
