"""Test plumbing: the operands of the DP-SGD hot path taken from a real PyTorch
GPT-2 (transformers, random initial weights, dropout off), and the true
per-example gradients of all its parameters, one backward pass per example.

The per-example loss is the causal-LM cross-entropy of that example (mean
over its predicted tokens); the batch loss is their sum, so example i's
activations and gradients depend on example i alone. Hooks record, for one
backward pass of the batch loss:
  * every Conv1D layer (attn.c_attn, attn.c_proj, mlp.c_fc, mlp.c_proj): its
    input A and the gradient G w.r.t. its output (weight [d_in, d_out]);
  * every LayerNorm: its normalised input xhat and the gradient gy w.r.t. its
    output (gain and bias);
  * the token-embedding output: dE (the position table reads the same
    gradient, as the two embeddings are added);
  * the tied output head: its input H and the logit gradients Gz.
Nothing here computes a norm, a clip factor or a clipped sum.
"""
from __future__ import annotations

from typing import Dict

import numpy as np
import torch


def tiny_gpt2(seed: int, V: int, n_pos: int, d: int, n_layer: int, n_head: int,
              dtype=torch.float64, device="cpu"):
    from transformers import GPT2Config, GPT2LMHeadModel
    torch.manual_seed(seed)
    cfg = GPT2Config(vocab_size=V, n_positions=n_pos, n_embd=d, n_layer=n_layer, n_head=n_head,
                     resid_pdrop=0.0, embd_pdrop=0.0, attn_pdrop=0.0, tie_word_embeddings=True,
                     bos_token_id=V - 1, eos_token_id=V - 1)
    m = GPT2LMHeadModel(cfg).to(device=device, dtype=dtype)
    m.eval()  # dropout off (the rates are 0 anyway); gradients still flow
    assert m.lm_head.weight is m.transformer.wte.weight
    return m


def _example_losses(model, ids):
    logits = model(input_ids=ids).logits
    B = ids.shape[0]
    return [torch.nn.functional.cross_entropy(logits[i, :-1], ids[i, 1:], reduction="mean")
            for i in range(B)]


def capture(model, ids) -> Dict[str, object]:
    """Operands of every parameter tensor for one backward pass of the batch."""
    tr = model.transformer
    acts: Dict[str, torch.Tensor] = {}
    grads: Dict[str, torch.Tensor] = {}
    hooks = []

    def grab_grad(name):
        def h(g):
            grads[name] = g.detach()
        return h

    def conv_hook(name):
        def f(mod, inp, out):
            acts[name] = inp[0].detach()
            out.register_hook(grab_grad(name))
        return f

    def ln_hook(name):
        def f(mod, inp, out):
            x = inp[0].detach()
            acts[name] = torch.nn.functional.layer_norm(x, mod.normalized_shape, eps=mod.eps)
            out.register_hook(grab_grad(name))
        return f

    def emb_hook(mod, inp, out):
        out.register_hook(grab_grad("wte"))

    def head_hook(mod, inp, out):
        acts["lm_head"] = inp[0].detach()
        out.register_hook(grab_grad("lm_head"))

    for b, blk in enumerate(tr.h):
        for name in ("attn.c_attn", "attn.c_proj", "mlp.c_fc", "mlp.c_proj"):
            mod = blk.get_submodule(name)
            hooks.append(mod.register_forward_hook(conv_hook(f"h.{b}.{name}")))
        hooks.append(blk.ln_1.register_forward_hook(ln_hook(f"h.{b}.ln_1")))
        hooks.append(blk.ln_2.register_forward_hook(ln_hook(f"h.{b}.ln_2")))
    hooks.append(tr.ln_f.register_forward_hook(ln_hook("ln_f")))
    hooks.append(tr.wte.register_forward_hook(emb_hook))
    hooks.append(model.lm_head.register_forward_hook(head_hook))
    try:
        model.zero_grad(set_to_none=True)
        sum(_example_losses(model, ids)).backward()
    finally:
        for h in hooks:
            h.remove()
    model.zero_grad(set_to_none=True)
    out = {"linears": [], "vectors": []}
    for b in range(len(tr.h)):
        for ln, convs in (("ln_1", ("attn.c_attn", "attn.c_proj")), ("ln_2", ("mlp.c_fc", "mlp.c_proj"))):
            n = f"h.{b}.{ln}"
            out["vectors"].append((n + ".weight", acts[n], grads[n]))
            out["vectors"].append((n + ".bias", None, grads[n]))
            for c in convs:
                n = f"h.{b}.{c}"
                out["linears"].append((n + ".weight", acts[n], grads[n]))
                out["vectors"].append((n + ".bias", None, grads[n]))
    out["vectors"].append(("ln_f.weight", acts["ln_f"], grads["ln_f"]))
    out["vectors"].append(("ln_f.bias", None, grads["ln_f"]))
    out["dE"], out["H"], out["Gz"] = grads["wte"], acts["lm_head"], grads["lm_head"]
    return out


def hf_name(name: str) -> str:
    """Our parameter name -> the model's parameter name."""
    if name in ("wte", "wpe"):
        return f"transformer.{name}.weight"
    return "transformer." + name


def per_example_grads(model, ids) -> Dict[str, np.ndarray]:
    """True per-example gradients: name -> [B, *shape] fp64 (wte is the tied matrix)."""
    names = dict(model.named_parameters())
    out: Dict[str, list] = {n: [] for n in names}
    for i in range(ids.shape[0]):
        model.zero_grad(set_to_none=True)
        _example_losses(model, ids[i:i + 1])[0].backward()
        for n, p in names.items():
            out[n].append(p.grad.detach().double().cpu().numpy().copy())
    model.zero_grad(set_to_none=True)
    return {n: np.stack(v) for n, v in out.items()}
