"""The C ABI on a host without a GPU: exports, workspace sizes, validation.

Only invalid arguments are passed to entry points that launch kernels: they
must be rejected on the host before any HIP call, so these run anywhere.
"""
import ctypes
import os
import re

import pytest

from paper_2609_40335_amd import build as B
from paper_2609_40335_amd import dpghost as D

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dpghost.h")
EINVAL, EUNSUP = 1, 2


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(D.library_path()):
        B.build()
    return D.lib()


def _declared():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(dp_[a-z0-9_]+)\s*\(", txt)))


def test_every_declared_symbol_is_exported(L):
    names = _declared()
    assert len(names) >= 15
    for n in names:
        assert hasattr(L, n), n
    assert set(n for n in names) >= {
        "dp_ghost_norm_linear", "dp_ghost_norm_embedding", "dp_tied_cross_term",
        "dp_clip_factors", "dp_clipped_grad_sum", "dp_add_noise"}


def test_binding_covers_every_entry_point():
    for n in _declared():
        assert n in D._SIGS, n


def test_version_and_strings(L):
    assert L.dp_abi_version() == 3
    assert L.dp_status_string(0) == b"ok"
    assert L.dp_status_string(1) == b"invalid argument"


def _lin(A=1 << 20, lda=64, d_in=64, G=1 << 21, ldg=64, d_out=64, algo=0):
    return D.dp_linear_t(A, lda, d_in, G, ldg, d_out, algo)


def _head_chunks(width, ks, per_chunk, other, slots):
    """The planner's chunk count for a long G range: chunks of at most 4096 and at
    least 1024 features (whole stages of ks) whose launch, with `other` items,
    leaves the smallest idle fraction of `slots` in its last round."""
    cdiv = lambda a, b: -(-a // b)
    lo = cdiv(width, 4096)
    hi = max(lo, cdiv(width, 1024))
    best, best_idle = lo, 2.0
    for nc in range(lo, hi + 1):
        kg = cdiv(cdiv(width, nc), ks) * ks
        eff = cdiv(width, kg)
        total = other + per_chunk * eff
        idle = (cdiv(total, slots) * slots - total) / total
        if idle < best_idle - 1e-9:
            best, best_idle = eff, idle
    return best


def test_norm_workspace_sizes(L):
    one = (D.dp_linear_t * 1)(_lin(algo=D.DP_NORM_GRAM))
    # T = 16: one T-tile pair per example, one G chunk -> 4 bytes per example
    assert L.dp_ghost_norm_linear_workspace(one, 1, 4, 16, D.DP_F32) == 256
    # T = 300 -> 3 T-tiles -> 6 pairs
    assert L.dp_ghost_norm_linear_workspace(one, 1, 100, 300, D.DP_F32) == 2560
    head = (D.dp_linear_t * 1)(_lin(d_in=768, lda=768, d_out=50257, ldg=50304))
    # bf16 head: V = 50257 features in chunks; the chunk count is the one whose
    # items best fill the last round of 512 workgroups (256 CUs, two per CU)
    assert L.dp_ghost_norm_linear_workspace(head, 1, 1, 128, D.DP_BF16) == 256
    for B in (32, 100):
        nc = _head_chunks(50257, 64, B, 0, 512)
        assert 50257 / nc <= 4096 and 50257 / nc >= 1024 - 64
        ws = L.dp_ghost_norm_linear_workspace(head, 1, B, 128, D.DP_BF16)
        assert ws == ((B * nc * 4 + 255) // 256) * 256
    assert _head_chunks(50257, 64, 32, 0, 512) == 16          # 512 items: one full round
    assert _head_chunks(50257, 64, 32, 48 * 32, 512) == 16    # with 48 body layers: 2048 items
    # an operand spanning 4 GiB or more (G: 1000 * 128 rows of 50304 bf16) is
    # taken only where the direct-load kernels rebase per example or per stage
    # (bf16, 16-byte rows, T a multiple of 32), refused otherwise (32-bit
    # buffer offsets across the batch)
    assert L.dp_ghost_norm_linear_workspace(head, 1, 1000, 128, D.DP_BF16) > 0
    assert L.dp_ghost_norm_linear_workspace(head, 1, 1000, 100, D.DP_BF16) == 0
    assert L.dp_ghost_norm_linear_grouped(head, 1, 1000, 100, D.DP_BF16, 1 << 22, 0, 1 << 23,
                                          1 << 30, None) == EUNSUP
    assert b"4 GiB" in L.dp_last_error()
    odd = (D.dp_linear_t * 1)(_lin(d_in=768, lda=768, d_out=50257, ldg=50257))  # rows not 16 B
    assert L.dp_ghost_norm_linear_workspace(odd, 1, 1000, 128, D.DP_BF16) == 0
    # AUTO picks the direct form once T + 1 > R * 2 d_in d_out / (d_in + d_out)
    # (R * 64 here): one 256x256 output tile per example
    auto = (D.dp_linear_t * 1)(_lin())
    assert L.dp_ghost_norm_linear_workspace(auto, 1, 100, 300, D.DP_F32) == 512
    # R = 0.49 when G is read whole: at d_in = d_out = 512 the switch sits at
    # T + 1 > 250.88, so T = 249 keeps the Gram (2 T-tiles, 3 pairs per
    # example) and T = 250 goes direct (2 x 2 tiles)
    sq = (D.dp_linear_t * 1)(_lin(d_in=512, lda=512, d_out=512, ldg=512))
    assert L.dp_ghost_norm_linear_workspace(sq, 1, 100, 249, D.DP_F32) == 1280
    assert L.dp_ghost_norm_linear_workspace(sq, 1, 100, 250, D.DP_F32) == 1792
    # R = 0.38 when G is read in feature chunks (d_out > 4096): at d_in = 768,
    # d_out = 50304 the switch sits at T + 1 > 574.93 (with 0.49: 741.4)
    def ws(d_out, T, algo):
        h = (D.dp_linear_t * 1)(_lin(d_in=768, lda=768, d_out=d_out, ldg=d_out, algo=algo))
        return L.dp_ghost_norm_linear_workspace(h, 1, 2, T, D.DP_BF16)
    for T in (573, 574):
        want = D.DP_NORM_GRAM if T == 573 else D.DP_NORM_DIRECT
        assert ws(50304, T, D.DP_NORM_AUTO) == ws(50304, T, want)
    assert ws(50304, 573, D.DP_NORM_GRAM) != ws(50304, 573, D.DP_NORM_DIRECT)
    assert L.dp_ghost_norm_linear_workspace(None, 1, 4, 16, D.DP_F32) == 0


def test_grad_store_size_and_argument_checks(L):
    """The per-example gradient store: B * tiles * 256 KB of fp32 tiles plus
    B * tiles norm partials; only bf16, T % 32 == 0 and 16-byte rows; every
    failure is found on the host before any launch."""
    two = (D.dp_linear_t * 2)(_lin(d_in=300, lda=304, d_out=520, ldg=520),   # 2 x 3 tiles
                              _lin(d_in=256, lda=256, d_out=256, ldg=256))   # 1 tile
    tiles, B, T = 7, 5, 64
    need = B * tiles * 256 * 256 * 4 + 256                    # partials: 140 B, one 256-B unit
    assert L.dp_grad_store_bytes(two, 2, B, T, D.DP_BF16) == need
    assert L.dp_grad_store_bytes(two, 2, B, T, D.DP_F32) == 0
    assert L.dp_grad_store_bytes(two, 2, B, 48, D.DP_BF16) == 0     # T not a multiple of 32
    odd = (D.dp_linear_t * 1)(_lin(d_in=300, lda=300, d_out=520, ldg=520))  # 600-byte rows
    assert L.dp_grad_store_bytes(odd, 1, B, T, D.DP_BF16) == 0
    n2, st = ctypes.c_void_p(1 << 22), ctypes.c_void_p(1 << 24)
    f = L.dp_ghost_norm_linear_store
    assert f(two, 2, B, T, D.DP_BF16, n2, 0, st, need - 1, None) == EINVAL
    assert b"gradient store of" in L.dp_last_error()
    assert f(two, 2, B, T, D.DP_BF16, None, 0, st, need, None) == EINVAL
    assert f(two, 2, B, T, D.DP_BF16, n2, 0, ctypes.c_void_p((1 << 24) + 8), need, None) == EINVAL
    assert b"16-byte" in L.dp_last_error()
    assert f(two, 2, B, T, D.DP_F32, n2, 0, st, need, None) == EUNSUP
    assert f(odd, 1, B, T, D.DP_BF16, n2, 0, st, need, None) == EUNSUP
    assert b"16-byte aligned rows" in L.dp_last_error()
    g = L.dp_clipped_grad_sum_noised_store
    outs = (ctypes.c_void_p * 2)(1 << 26, 1 << 27)
    tids = (ctypes.c_uint64 * 2)(1, 2)
    c = ctypes.c_void_p(1 << 23)
    tiles_bytes = B * tiles * 256 * 256 * 4                  # the sum reads the tiles only
    assert g(two, outs, tids, None, None, 2, c, B, T, D.DP_BF16, 1.0, 1.0, B, 7, 0, st,
             tiles_bytes - 1, None) == EINVAL
    assert g(two, None, tids, None, None, 2, c, B, T, D.DP_BF16, 1.0, 1.0, B, 7, 0, st,
             tiles_bytes, None) == EINVAL
    assert g(two, outs, tids, None, None, 2, c, B, T, D.DP_BF16, -1.0, 1.0, B, 7, 0, st,
             tiles_bytes, None) == EINVAL                     # sigma < 0
    assert g(two, outs, tids, None, None, 2, c, B, T, D.DP_F32, 1.0, 1.0, B, 7, 0, st,
             tiles_bytes, None) == EUNSUP
    big = (ctypes.c_uint64 * 2)(1, 1 << 32)
    assert g(two, outs, big, None, None, 2, c, B, T, D.DP_BF16, 1.0, 1.0, B, 7, 0, st,
             tiles_bytes, None) == EINVAL


def test_linear_norm_rejects_bad_arguments(L):
    n2 = ctypes.c_void_p(1 << 22)
    ws = ctypes.c_void_p(1 << 23)
    f = L.dp_ghost_norm_linear
    assert f(None, 64, 1 << 21, 64, 4, 16, 64, 64, 0, 0, n2, 0, ws, 1 << 20, None) == EINVAL
    assert b"NULL" in L.dp_last_error()
    assert f(1 << 20, 32, 1 << 21, 64, 4, 16, 64, 64, 0, 0, n2, 0, ws, 1 << 20, None) == EINVAL
    assert f(1 << 20, 64, 1 << 21, 64, 0, 16, 64, 64, 0, 0, n2, 0, ws, 1 << 20, None) == EINVAL
    assert f(1 << 20, 64, 1 << 21, 64, 4, 16, 64, 64, 7, 0, n2, 0, ws, 1 << 20, None) == EINVAL
    assert f(1 << 20, 64, 1 << 21, 64, 4, 16, 64, 64, 0, 9, n2, 0, ws, 1 << 20, None) == EINVAL
    assert f(1 << 20, 64, 1 << 21, 64, 4, 16, 64, 64, 0, 0, None, 0, ws, 1 << 20, None) == EINVAL
    # workspace too small / missing
    assert f(1 << 20, 64, 1 << 21, 64, 4, 16, 64, 64, 0, 0, n2, 0, ws, 8, None) == EINVAL
    assert b"workspace" in L.dp_last_error()
    assert f(1 << 20, 64, 1 << 21, 64, 4, 16, 64, 64, 0, 0, n2, 0, None, 0, None) == EINVAL
    assert f(1 << 20, 64, 1 << 21, 64, 4, 70000, 64, 64, 0, 0, n2, 0, ws, 1 << 30,
             None) == EUNSUP


def test_grouped_rejects_bad_layers(L):
    arr = (D.dp_linear_t * 2)(_lin(), _lin(G=0))
    assert L.dp_ghost_norm_linear_grouped(arr, 2, 4, 16, 0, 1 << 22, 0, 1 << 23, 1 << 20,
                                          None) == EINVAL
    assert b"layer 1" in L.dp_last_error()
    assert L.dp_ghost_norm_linear_grouped(arr, 0, 4, 16, 0, 1 << 22, 0, 1 << 23, 1 << 20,
                                          None) == EINVAL


def test_noalloc_norm_rejects_bad_and_oversized_calls(L):
    """The no-allocation grouped norm validates like the workspace form, and
    rejects a call whose partials exceed its static scratch before any HIP
    call (so this runs without a GPU)."""
    f = L.dp_ghost_norm_linear_bias_grouped_noalloc
    arr = (D.dp_linear_t * 2)(_lin(), _lin(G=0))
    assert f(arr, None, 2, 4, 16, 0, 1 << 22, 0, None) == EINVAL
    assert b"layer 1" in L.dp_last_error()
    one = (D.dp_linear_t * 1)(_lin())
    assert f(one, None, 1, 4, 16, 0, None, 0, None) == EINVAL           # no norm2
    assert f(None, None, 1, 4, 16, 0, 1 << 22, 0, None) == EINVAL
    # direct norm of a 4352 x 4352 layer: 17 x 17 tiles per example, so at
    # B = 8192 the partials take 8192 * 289 * 4 bytes > 8 MiB
    big = (D.dp_linear_t * 1)(_lin(d_in=4352, lda=4352, d_out=4352, ldg=4352,
                                   algo=D.DP_NORM_DIRECT))
    need = L.dp_ghost_norm_linear_bias_workspace(big, None, 1, 8192, 1, D.DP_BF16)
    assert need == 8192 * 289 * 4
    assert need > (8 << 20)
    assert f(big, None, 1, 8192, 1, D.DP_BF16, 1 << 22, 0, None) == EUNSUP
    assert b"static scratch" in L.dp_last_error()


def test_embedding_rejects_bad_arguments(L):
    f = L.dp_ghost_norm_embedding
    args = dict(ids=1 << 20, dE=1 << 21, lde=64, B=4, T=16, V=512, d=64, dt=0, norm2=1 << 22,
                acc=0, seg=None, nu=None, ws=1 << 23, wsb=1 << 20, s=None)
    def call(**kw):
        a = dict(args, **kw)
        return f(*a.values())
    assert call(ids=None) == EINVAL
    assert call(lde=32) == EINVAL
    assert call(V=0) == EINVAL
    assert call(wsb=0) == EINVAL
    # past T = 4096 only rows of whole 8-byte units (here fp32 rows of 65)
    assert call(T=5000, lde=65, d=65) == EUNSUP
    assert b"8-byte" in L.dp_last_error()
    assert call(V=1 << 30, T=64) == EUNSUP     # 30 + 6 bits > 32
    assert L.dp_ghost_norm_embedding_workspace(4, 16, 64) == 256
    assert L.dp_ghost_norm_embedding_workspace(64, 256, 768) == 64 * 12 * 4


def test_cross_and_clip_reject_bad_arguments(L):
    f = L.dp_tied_cross_term
    ok = [1 << 20, 1 << 21, 64, 1 << 22, 64, 1 << 23, 512, 4, 16, 512, 64, 0, 2.0, 1 << 24, 1,
          1 << 25, 1 << 20, None]
    bad_ldz = list(ok); bad_ldz[6] = 100
    assert f(*bad_ldz) == EINVAL
    bad_scale = list(ok); bad_scale[12] = float("inf")
    assert f(*bad_scale) == EINVAL
    no_ws = list(ok); no_ws[16] = 0
    assert f(*no_ws) == EINVAL
    # T = 300: 5 x 5 blocks of 64 rows (direct-load kernel) > 3 x 3 tile pairs x 1 chunk
    assert L.dp_tied_cross_term_workspace(4, 300, 64) == 512
    # T = 128: 4 x 4 blocks of 32 rows (register-direct kernel) > 1 x 6 chunks > 2 x 2 blocks
    assert L.dp_tied_cross_term_workspace(32, 128, 768) == 32 * 16 * 4
    assert L.dp_clip_factors(1 << 20, 4, 0.0, 1 << 21, None) == EINVAL
    assert L.dp_clip_factors(1 << 20, 4, float("nan"), 1 << 21, None) == EINVAL
    assert L.dp_clip_factors(1 << 20, 0, 1.0, 1 << 21, None) == EINVAL
    g = L.dp_clip_factors_scaled
    assert g(1 << 20, 4, 1.0, 0.5, None, None, None) == EINVAL       # no c_scaled
    assert g(None, 4, 1.0, 0.5, None, 1 << 21, None) == EINVAL       # no norm2
    assert g(1 << 20, 0, 1.0, 0.5, None, 1 << 21, None) == EINVAL
    assert g(1 << 20, 4, -1.0, 0.5, None, 1 << 21, None) == EINVAL
    assert g(1 << 20, 4, 1.0, float("inf"), None, 1 << 21, None) == EINVAL
    g2 = L.dp_clip_factors_scaled2
    assert g2(1 << 20, None, 4, 1.0, 0.5, None, 1 << 21, None) == EINVAL  # no second array
    assert g2(None, 1 << 22, 4, 1.0, 0.5, None, 1 << 21, None) == EINVAL  # no first array
    assert g2(1 << 20, 1 << 22, 4, 1.0, 0.5, None, None, None) == EINVAL  # no c_scaled
    assert g2(1 << 20, 1 << 22, 0, 1.0, 0.5, None, 1 << 21, None) == EINVAL
    assert g2(1 << 20, 1 << 22, 4, 0.0, 0.5, None, 1 << 21, None) == EINVAL
    assert g2(1 << 20, 1 << 22, 4, 1.0, float("nan"), None, 1 << 21, None) == EINVAL


def test_clipped_sum_rejects_bad_arguments(L):
    f = L.dp_clipped_grad_sum
    # both A and ids
    assert f(1 << 20, 64, 1 << 21, 64, 1 << 22, 1 << 23, 4, 16, 512, 64, 0, 0, 1 << 24, 0,
             1 << 25, 1 << 20, None) == EINVAL
    # embedding form without workspace
    assert f(None, 0, 1 << 21, 64, 1 << 22, 1 << 23, 4, 16, 512, 64, 0, 0, 1 << 24, 0,
             None, 0, None) == EINVAL
    # a sort key would need more than 32 bits: 21 for ids up to V = 2^20, 15
    # for B*T = 32768 token indices
    assert f(None, 0, 1 << 21, 64, 1 << 22, 1 << 23, 64, 512, 1 << 20, 64, 0, 0, 1 << 24, 0,
             1 << 25, 1 << 30, None) == EUNSUP
    assert L.dp_clipped_grad_sum_workspace(4, 16, 64, 0) == 0
    assert L.dp_clipped_grad_sum_workspace(64, 256, 768, 1) > 2 * 512 * 768 * 4
    outs = (ctypes.c_void_p * 1)(None)
    arr = (D.dp_linear_t * 1)(_lin())
    assert L.dp_clipped_grad_sum_grouped(arr, outs, 1, 1 << 20, 4, 16, 0, 0, 0, None) == EINVAL


def _up(x):
    return (x + 255) // 256 * 256


def test_bias_norm_workspace_and_validation(L):
    """Fused biases (bf16, 16-byte rows, T <= 256) add nothing to the norm
    workspace; a bias the Gram launch cannot fuse (fp32 here, or T > 256)
    adds the vector kernel's partials: B x ceil(d / features per chunk)."""
    lay = (D.dp_linear_t * 2)(D.dp_linear_t(1 << 20, 768, 768, 1 << 21, 3072, 3072, 0),
                              D.dp_linear_t(1 << 22, 768, 768, 1 << 23, 768, 768, 0))
    bias = (ctypes.c_void_p * 2)(1 << 24, None)
    for T in (128, 256):
        plain = L.dp_ghost_norm_linear_workspace(lay, 2, 32, T, D.DP_BF16)
        assert L.dp_ghost_norm_linear_bias_workspace(lay, bias, 2, 32, T, D.DP_BF16) == plain
        assert L.dp_ghost_norm_linear_bias_workspace(lay, None, 2, 32, T, D.DP_BF16) == plain
    plain = L.dp_ghost_norm_linear_workspace(lay, 2, 32, 300, D.DP_BF16)
    assert L.dp_ghost_norm_linear_bias_workspace(lay, bias, 2, 32, 300, D.DP_BF16) == \
        plain + _up(32 * 6 * 4)                       # 3072 / 512 bf16 features per chunk
    plain = L.dp_ghost_norm_linear_workspace(lay, 2, 32, 64, D.DP_F32)
    assert L.dp_ghost_norm_linear_bias_workspace(lay, bias, 2, 32, 64, D.DP_F32) == \
        plain + _up(32 * 12 * 4)                      # 3072 / 256 fp32 features per chunk
    f = L.dp_ghost_norm_linear_bias_grouped
    assert f(lay, bias, 2, 32, 64, D.DP_BF16, None, 0, 1 << 25, 1 << 30, None) == EINVAL
    assert f(lay, bias, 2, 32, 64, D.DP_BF16, 1 << 26, 0, None, 0, None) == EINVAL
    assert f(lay, bias, 0, 32, 64, D.DP_BF16, 1 << 26, 0, 1 << 25, 1 << 30, None) == EINVAL


def test_embedding_rows_workspace_and_validation(L):
    """Two-call embedding form: workspace = the one-call form's (sorted keys,
    block partials) plus ranks, run starts, the run count and B*T rows of d
    floats, each 256-byte aligned; every bad argument fails before a launch."""
    for B, T, d in ((32, 128, 768), (3, 50, 70), (1, 1, 8)):
        K = B * T
        nb = -(-K // 32)
        want = (_up(K * 4) + 2 * _up(nb * d * 4) + _up(K * 4) + _up((K + 1) * 4) + _up(4)
                + _up(K * d * 4))
        assert L.dp_embedding_rows_workspace(B, T, d) == want
        assert L.dp_clipped_grad_sum_workspace(B, T, d, 1) == _up(K * 4) + 2 * _up(nb * d * 4)
    assert L.dp_embedding_rows_workspace(0, 16, 64) == 0
    ws = L.dp_embedding_rows_workspace(4, 16, 64)
    f = L.dp_embedding_rows
    args = [1 << 21, 64, 1 << 22, 1 << 23, 4, 16, 512, 64, D.DP_BF16, 1 << 25, ws, None]
    for i, bad in ((0, None), (2, None), (3, None), (1, 32), (4, 0), (6, 0), (8, 9), (9, None),
                   (10, ws - 1)):
        a = list(args)
        a[i] = bad
        assert f(*a) == EINVAL, (i, bad)
    big = list(args)
    big[4], big[5], big[6] = 64, 512, 1 << 20  # ids of 21 bits + 15 bits of B*T: no 32-bit key
    big[10] = 1 << 40
    assert f(*big) == EUNSUP
    g = L.dp_embedding_rows_add
    assert g(1 << 25, ws, 4, 16, 512, 64, 0, None, None) == EINVAL        # no out
    assert g(None, ws, 4, 16, 512, 64, 0, 1 << 24, None) == EINVAL        # no workspace
    assert g(1 << 25, ws - 1, 4, 16, 512, 64, 0, 1 << 24, None) == EINVAL
    assert g(1 << 25, ws, 4, 16, 0, 64, 0, 1 << 24, None) == EINVAL       # V = 0


def test_noised_sum_rejects_bad_arguments(L):
    """The fused clipped sum + noise validates everything on the host (no launch)."""
    f = L.dp_clipped_grad_sum_noised_grouped
    arr = (D.dp_linear_t * 1)(_lin())
    outs = (ctypes.c_void_p * 1)(1 << 24)
    tids = (ctypes.c_uint64 * 1)(3)
    acc = (ctypes.c_int32 * 1)(0)
    ok = dict(c=1 << 20, B=4, T=16, dt=D.DP_F32, tr=0, sigma=1.0, C=1.0, Bn=4, seed=1, step=2)

    def call(**kw):
        a = dict(ok, **kw)
        return f(arr, outs, kw.get("tids", tids), acc, 1, a["c"], a["B"], a["T"], a["dt"], a["tr"],
                 a["sigma"], a["C"], a["Bn"], a["seed"], a["step"], None)

    assert call(tids=None) == EINVAL
    assert call(tids=(ctypes.c_uint64 * 1)(1 << 32)) == EINVAL
    assert b"tensor_ids" in L.dp_last_error()
    assert call(sigma=-1.0) == EINVAL
    assert call(sigma=float("nan")) == EINVAL
    assert call(C=0.0) == EINVAL
    assert call(Bn=-1) == EINVAL
    assert call(step=1 << 32) == EINVAL
    assert call(c=None) == EINVAL
    assert f(arr, (ctypes.c_void_p * 1)(None), tids, acc, 1, 1 << 20, 4, 16, D.DP_F32, 0, 1.0,
             1.0, 4, 1, 2, None) == EINVAL
    assert call(B=0) == EINVAL


def test_noise_rejects_bad_arguments(L):
    f = L.dp_add_noise
    assert f(1 << 20, -1, 1.0, 1.0, 4, 0, 0, 0, None) == EINVAL
    assert f(None, 10, 1.0, 1.0, 4, 0, 0, 0, None) == EINVAL
    assert f(1 << 20, 10, -1.0, 1.0, 4, 0, 0, 0, None) == EINVAL
    assert f(1 << 20, 10, 1.0, 0.0, 4, 0, 0, 0, None) == EINVAL
    assert f(1 << 20, 10, 1.0, 1.0, -4, 0, 0, 0, None) == EINVAL
    assert f(1 << 20, 10, 1.0, 1.0, 4, 0, 1 << 32, 0, None) == EINVAL
    assert f(1 << 20, 10, 1.0, 1.0, 4, 0, 0, 1 << 32, None) == EINVAL
    # n = 0 is a no-op that launches nothing
    assert f(None, 0, 1.0, 1.0, 4, 0, 0, 0, None) == 0
    # the write-only form validates the same way
    g = L.dp_noise_fill
    assert g(None, 10, 1.0, 1.0, 4, 0, 0, 0, None) == EINVAL
    assert g(1 << 20, 10, float("nan"), 1.0, 4, 0, 0, 0, None) == EINVAL
    assert g(1 << 20, 10, 1.0, 1.0, 4, 0, 0, 1 << 32, None) == EINVAL
    assert g(None, 0, 1.0, 1.0, 4, 0, 0, 0, None) == 0


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.delenv("DPGHOST_LIBRARY", raising=False)
    monkeypatch.setattr(D, "_LIB", None)
    monkeypatch.setattr(D, "_HERE", str(tmp_path))
    with pytest.raises(D.DPError, match="not built"):
        D.lib()


def test_vector_and_positional_validation(L):
    vec = (D.dp_vector_t * 2)(D.dp_vector_t(None, 0, 1 << 21, 96, 96),
                              D.dp_vector_t(1 << 22, 64, 1 << 23, 64, 64))
    # workspace: one partial per 512-feature (bf16) or 256-feature (fp32) chunk per example
    assert L.dp_vector_grads_workspace(vec, 2, 4, 16, D.DP_BF16) == 256
    assert L.dp_vector_grads_workspace(vec, 2, 100, 16, D.DP_F32) == ((100 * 2 * 4 + 255) // 256) * 256
    grads = (ctypes.c_void_p * 2)(1 << 24, 1 << 25)
    ws, nws = 1 << 26, 1 << 20
    ok = lambda *a: L.dp_vector_grads_grouped(vec, 2, 4, 16, D.DP_BF16, *a)
    assert ok(None, None, 0, ws, nws, None) == EINVAL                    # grads NULL
    assert ok(grads, None, 0, None, 0, None) == EINVAL                   # no workspace
    assert L.dp_vector_grads_grouped(vec, 0, 4, 16, D.DP_BF16, grads, None, 0, ws, nws,
                                     None) == EINVAL                     # n = 0
    bad = (D.dp_vector_t * 1)(D.dp_vector_t(None, 0, 1 << 21, 90, 96))   # ldg < d
    assert L.dp_vector_grads_grouped(bad, 1, 4, 16, D.DP_BF16, grads, None, 0, ws, nws,
                                     None) == EINVAL
    bad = (D.dp_vector_t * 1)(D.dp_vector_t(None, 0, None, 96, 96))      # G NULL
    assert L.dp_vector_grads_grouped(bad, 1, 4, 16, D.DP_BF16, grads, None, 0, ws, nws,
                                     None) == EINVAL
    big = (D.dp_vector_t * 1)(D.dp_vector_t(None, 0, 1 << 21, 1 << 20, 64))
    assert L.dp_vector_grads_grouped(big, 1, 4096, 1024, D.DP_BF16, grads, None, 0, ws, nws,
                                     None) == EUNSUP                     # 8 TiB operand span
    d = (ctypes.c_int32 * 2)(96, 64)
    outs = (ctypes.c_void_p * 2)(1 << 27, 1 << 28)
    tids = (ctypes.c_uint64 * 2)(1, 2)
    vs = lambda *a: L.dp_vector_clipped_sum_noised_grouped(grads, d, 2, 4, 1 << 29, outs, tids,
                                                           None, *a)
    assert vs(-1.0, 1.0, 4, 0, 0, None) == EINVAL                        # sigma < 0
    assert vs(1.0, 0.0, 4, 0, 0, None) == EINVAL                         # C = 0
    assert vs(1.0, 1.0, -1, 0, 0, None) == EINVAL                        # B_norm < 0
    assert vs(1.0, 1.0, 4, 0, 1 << 32, None) == EINVAL                   # step >= 2^32
    tids_bad = (ctypes.c_uint64 * 2)(1, 1 << 33)
    assert L.dp_vector_clipped_sum_noised_grouped(grads, d, 2, 4, 1 << 29, outs, tids_bad, None,
                                                  1.0, 1.0, 4, 0, 0, None) == EINVAL
    # position table
    assert L.dp_ghost_norm_positional_workspace(4, 16, 768) == 256
    assert L.dp_ghost_norm_positional_workspace(0, 16, 768) == 0
    assert L.dp_ghost_norm_positional(None, 768, 4, 16, 768, D.DP_BF16, 1 << 20, 0, ws, nws,
                                      None) == EINVAL
    assert L.dp_ghost_norm_positional(1 << 21, 700, 4, 16, 768, D.DP_BF16, 1 << 20, 0, ws, nws,
                                      None) == EINVAL                    # lde < d
    ps = lambda T, n_pos, ldo: L.dp_clipped_grad_sum_positional_noised(
        1 << 21, 768, 1 << 22, 4, T, 768, D.DP_BF16, 1 << 23, n_pos, ldo, 3, 0, 1.0, 1.0, 4, 0, 0,
        None)
    assert ps(2048, 1024, 768) == EINVAL                                  # T > n_pos
    assert ps(16, 1024, 700) == EINVAL                                    # ldo < d
    assert L.dp_clipped_grad_sum_positional_noised(1 << 21, 768, 1 << 22, 4, 16, 768, D.DP_BF16,
                                                   1 << 23, 1024, 768, 1 << 32, 0, 1.0, 1.0, 4,
                                                   0, 0, None) == EINVAL  # tensor_id >= 2^32


def test_split_tail_workspace(L):
    """The clipped sum's split tail: 95 of GPT-2's 1887 tiles (256 CUs) split
    in 2 K ranges; a launch of whole rounds, or fp32, needs nothing."""
    body = [(768, 2304), (768, 768), (768, 3072), (3072, 768)] * 12
    ptr = [1 << 30]

    def lin(di, do):
        ptr[0] += 1 << 26
        return D.dp_linear_t(ptr[0], di, di, ptr[0] + (1 << 25), do, do, 0)
    # the head as the benchmark passes it: Gz rows padded to 50304 (16-byte aligned)
    descs = [lin(di, do) for di, do in body] + [D.dp_linear_t(1 << 40, 50304, 50257,
                                                              (1 << 40) + (1 << 35), 768, 768, 0)]
    arr = (D.dp_linear_t * len(descs))(*descs)
    ws = L.dp_clipped_grad_sum_noised_grouped_workspace(arr, len(descs), 32, 128, D.DP_BF16, 0)
    assert ws == 95 * 2 * 256 * 256 * 4
    # 48 body layers: 1296 tiles, 16 in the last round -> 8 K ranges each
    ws = L.dp_clipped_grad_sum_noised_grouped_workspace(arr, 48, 32, 128, D.DP_BF16, 0)
    assert ws == 16 * 8 * 256 * 256 * 4
    assert L.dp_clipped_grad_sum_noised_grouped_workspace(arr, 49, 32, 128, D.DP_F32, 0) == 0
    assert L.dp_clipped_grad_sum_noised_grouped_workspace(arr, 49, 32, 100, D.DP_BF16, 0) == 0
    # K = 64 rows = 2 stages: too short to split
    assert L.dp_clipped_grad_sum_noised_grouped_workspace(arr, 1, 2, 32, D.DP_BF16, 0) == 0
