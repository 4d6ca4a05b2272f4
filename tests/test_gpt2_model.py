"""End to end on a real PyTorch GPT-2 (transformers, random initial weights):
the operands captured from one forward/backward pass of the batch, pushed
through the oracle (CPU) and through the library (GPU), against the model's
true per-example gradients (one backward pass per example).

This checks, on the model itself, what the paper's method rests on: the
per-example norm of the whole tied model (eq. 6, eq. 11-13) and the clipped
sum as a reweighted second backward pass (Sec. "Ghost Clipping Mechanism")
over every parameter tensor, biases, LayerNorms and the position table
included.
"""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytest.importorskip("transformers")

import oracle as O  # noqa: E402
from workloads import gen  # noqa: E402
from tests import gpt2_capture as cap  # noqa: E402
from tests.helpers import TOL, assert_close, dev, fro_rel, host, rel  # noqa: E402


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _np(t, dtype):
    a = t.detach().float().cpu().numpy()
    return gen.f32_to_bf16_bits(a) if dtype == "bf16" else a


def _workload(c, ids, V, d, n_pos, dtype, C=1.0, sigma=1.0):
    """A Workload holding the captured operands (rounded to fp32 or bf16)."""
    B, T = ids.shape
    wl = gen.Workload(name="captured-gpt2", dtype=dtype, B=B, T=T, C=C, sigma=sigma)
    g_of = {}
    for name, A, G in c["linears"]:
        Gn = _np(G, dtype)
        g_of[name[:-len(".weight")]] = Gn
        wl.linears.append(gen.LinearInputs(name, A.shape[-1], G.shape[-1], _np(A, dtype), Gn))
    ln_g = {}
    for name, X, G in c["vectors"]:
        base = name.rsplit(".", 1)[0]
        if X is None and base in g_of:            # a Conv1D bias: that layer's G
            Gn = g_of[base]
        else:                                      # a LayerNorm: gain and bias share gy
            Gn = ln_g.setdefault(base, _np(G, dtype))
        wl.vectors.append(gen.VectorInputs(name, G.shape[-1], None if X is None else _np(X, dtype),
                                           Gn))
    wl.head = gen.HeadInputs(V=V, d=d, ids=ids.cpu().numpy().astype(np.int32), dE=_np(c["dE"], dtype),
                             H=_np(c["H"], dtype), Gz=_np(c["Gz"], dtype), ldz=V, tied=True)
    wl.n_pos = n_pos
    return wl


def _true_norm2(true):
    return sum((g.reshape(g.shape[0], -1) ** 2).sum(axis=1) for g in true.values())


def _names(wl):
    return ([l.name for l in wl.linears] + ["wte"] + [v.name for v in wl.vectors] + ["wpe"])


def test_oracle_on_captured_gpt2():
    """CPU, fp64 model: the oracle's flat norm and clipped sums from the
    captured operands equal the model's true per-example gradients."""
    V, n_pos, d, T, B = 97, 24, 32, 12, 3
    m = cap.tiny_gpt2(3, V, n_pos, d, 2, 2)
    ids = torch.randint(0, V, (B, T), generator=torch.Generator().manual_seed(4))
    c = cap.capture(m, ids)
    true = cap.per_example_grads(m, ids)
    wl = _workload(c, ids, V, d, n_pos, "f32", C=0.05)
    assert wl.n_coordinates() == sum(p.numel() for p in m.parameters())
    n2 = O.per_example_norms(wl)["total"]
    np.testing.assert_allclose(n2, _true_norm2(true), rtol=1e-5)
    r = O.step(wl, noise=False)
    assert (r["c"] < 1).all()  # C small enough that every example is clipped
    for name in _names(wl):
        ref = np.tensordot(r["c"], true[cap.hf_name(name)], axes=(0, 0))
        assert_close(r["sums"][name], ref, 1e-5, name)


def _library_step(dp, wl, seed=5, step=2, sigma=None):
    """The whole step through the C ABI on device copies of wl's operands.
    Returns (norm2, c, {name: noised sum})."""
    B, h = wl.B, wl.head
    d_ = lambda a: dev(a, wl.dtype)
    lin = [(d_(l.A), d_(l.G)) for l in wl.linears]
    same = {id(l.G): g for l, (_, g) in zip(wl.linears, lin)}

    def shared(a):
        if id(a) not in same:
            same[id(a)] = d_(a)
        return same[id(a)]
    ids, dE, H, Gz = dev(h.ids), d_(h.dE), d_(h.H), d_(h.Gz)
    sigma = wl.sigma if sigma is None else sigma
    n2 = torch.zeros(B, device="cuda")
    dp.dp_ghost_norm_linear_grouped(lin + [(H, Gz)], n2)
    dp.dp_ghost_norm_embedding(ids, dE, h.V, n2, accumulate=True)
    dp.dp_tied_cross_term(ids, dE, H, Gz, h.V, n2, scale=2.0, accumulate=True)
    vg = dp.VectorGroup([(None if v.X is None else d_(v.X), shared(v.G)) for v in wl.vectors])
    vg.grads_and_norm(n2, accumulate=True)
    dp.dp_ghost_norm_positional(dE, n2, accumulate=True)
    c = torch.empty(B, device="cuda")
    c_b = torch.empty(B, device="cuda")
    dp.dp_clip_factors_scaled(n2, wl.C, 1.0 / B, c_b, c=c)
    names = _names(wl)
    tid = {n: k for k, n in enumerate(names)}
    outs = {l.name: torch.empty(l.d_in, l.d_out, device="cuda") for l in wl.linears}
    outs["wte"] = torch.empty(h.V, h.d, device="cuda")
    dp.dp_clipped_grad_sum_noised_grouped(lin + [(Gz, H)], [outs[l.name] for l in wl.linears] +
                                          [outs["wte"]], c, [tid[l.name] for l in wl.linears] +
                                          [tid["wte"]], sigma, wl.C, B, seed, step)
    dp.dp_clipped_grad_sum(None, dE, c_b, outs["wte"], ids=ids, V=h.V, accumulate=True)
    vouts = [torch.empty(v.d, device="cuda") for v in wl.vectors]
    vg.clipped_sum_noised(c, vouts, [tid[v.name] for v in wl.vectors], sigma, wl.C, B, seed, step)
    outs.update({v.name: o for v, o in zip(wl.vectors, vouts)})
    outs["wpe"] = torch.empty(wl.n_pos, h.d, device="cuda")
    dp.dp_clipped_grad_sum_positional_noised(dE, c, outs["wpe"], tid["wpe"], sigma, wl.C, B,
                                             seed, step)
    torch.cuda.synchronize()
    return host(n2), host(c), {k: host(v) for k, v in outs.items()}


@pytest.fixture(scope="module")
def dp():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_40335_amd.dpghost as d
    d.lib()
    return d


@pytest.mark.gpu
def test_library_on_captured_gpt2_fp32(dp):
    """fp32 operands of a tiny GPT-2: norms, clip factors and noised sums of
    every parameter tensor against the true per-example gradients (the noise
    against the oracle's stream)."""
    V, n_pos, d, T, B = 97, 24, 32, 12, 3
    m = cap.tiny_gpt2(3, V, n_pos, d, 2, 2)
    ids = torch.randint(0, V, (B, T), generator=torch.Generator().manual_seed(4))
    c_ = cap.capture(m, ids)
    true = cap.per_example_grads(m, ids)
    wl = _workload(c_, ids, V, d, n_pos, "f32", C=0.05, sigma=0.5)
    n2, c, outs = _library_step(dp, wl)
    assert rel(n2, _true_norm2(true)).max() <= TOL["f32"]
    c_ref = O.clip_factors(_true_norm2(true), wl.C)
    assert rel(c, c_ref).max() <= TOL["f32"]
    for tid, name in enumerate(_names(wl)):
        S = np.tensordot(c_ref, true[cap.hf_name(name)], axes=(0, 0))
        ref = O.add_noise(S, wl.sigma, wl.C, B, 5, tid, 2)
        assert_close(outs[name], ref, TOL["f32"], name)


@pytest.mark.gpu
def test_library_on_captured_gpt2_widths_bf16(dp):
    """Two blocks at GPT-2-small widths (d = 768, V = 50257, 12 heads), fp32
    model on the GPU, operands rounded to bf16: per-example norms and clipped
    sums (noise off) of every parameter tensor against the true per-example
    gradients of the fp32 model."""
    V, n_pos, d, T, B = 50257, 1024, 768, 64, 4
    m = cap.tiny_gpt2(7, V, n_pos, d, 2, 12, dtype=torch.float32, device="cuda")
    ids = torch.randint(0, V, (B, T), generator=torch.Generator().manual_seed(8)).cuda()
    _say(f"captured GPT-2 widths: 2 blocks, d={d}, V={V}, B={B}, T={T}")
    c_ = cap.capture(m, ids)
    true = cap.per_example_grads(m, ids)
    wl = _workload(c_, ids.cpu(), V, d, n_pos, "bf16", C=0.5)
    n2, c, outs = _library_step(dp, wl, sigma=0.0)
    tn = _true_norm2(true)
    _say(f"  norm2 max rel err {rel(n2, tn).max():.2e}")
    assert rel(n2, tn).max() <= TOL["bf16"]
    c_ref = O.clip_factors(tn, wl.C)
    worst = 0.0
    for name in _names(wl):
        S = np.tensordot(c_ref, true[cap.hf_name(name)], axes=(0, 0)) / B
        # Against the model's true fp32 per-example gradients, from operands
        # the library received rounded to bf16: a whole-tensor bar (the
        # element-wise parity with the oracle on identical operands is in
        # the parity tests).
        err = fro_rel(outs[name], S)
        worst = max(worst, err)
        assert err <= TOL["bf16"], (name, err)
    _say(f"  worst clipped-sum rel err {worst:.2e}")


@pytest.mark.gpu
def test_dp_adam_steps_on_captured_gpt2(dp):
    """Two DP-Adam steps (the paper trains with Adam, lr 2e-4 for GPT-2) on a
    tiny GPT-2: one copy takes the library's noised clipped sums as p.grad
    (operands captured afresh after each update), the other the mean of the
    true per-example gradients clipped with the true norms plus the oracle's
    noise. The parameter updates agree to the fp32 tolerance."""
    import copy
    V, n_pos, d, T, B = 97, 24, 32, 12, 3
    C, sigma, seed, lr = 0.05, 0.5, 5, 2e-4
    m_lib = cap.tiny_gpt2(3, V, n_pos, d, 2, 2)
    m_ref = copy.deepcopy(m_lib)
    p0 = {n: p.detach().clone() for n, p in m_ref.named_parameters()}
    opt_lib = torch.optim.Adam(m_lib.parameters(), lr=lr)
    opt_ref = torch.optim.Adam(m_ref.parameters(), lr=lr)
    lib_params, ref_params = dict(m_lib.named_parameters()), dict(m_ref.named_parameters())
    for step in range(2):
        ids = torch.randint(0, V, (B, T), generator=torch.Generator().manual_seed(10 + step))
        wl = _workload(cap.capture(m_lib, ids), ids, V, d, n_pos, "f32", C=C, sigma=sigma)
        _, _, outs = _library_step(dp, wl, seed=seed, step=step)
        names = _names(wl)
        for name in names:
            p = lib_params[cap.hf_name(name)]
            p.grad = torch.from_numpy(outs[name].astype(np.float64)).reshape(p.shape)
        opt_lib.step()
        true = cap.per_example_grads(m_ref, ids)
        c_ref = O.clip_factors(_true_norm2(true), C)
        for tid, name in enumerate(names):
            p = ref_params[cap.hf_name(name)]
            S = np.tensordot(c_ref, true[cap.hf_name(name)], axes=(0, 0))
            p.grad = torch.from_numpy(O.add_noise(S, sigma, C, B, seed, tid, step)).reshape(p.shape)
        opt_ref.step()
    worst = 0.0
    for n, p in ref_params.items():
        du_ref = (p.detach() - p0[n]).numpy()
        du_lib = (lib_params[n].detach() - p0[n]).numpy()
        worst = max(worst, fro_rel(du_lib, du_ref))
    _say(f"  worst parameter-update rel err after 2 DP-Adam steps {worst:.2e}")
    assert worst <= TOL["f32"]
