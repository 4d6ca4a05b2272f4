#!/usr/bin/env python3
"""DP-SGD ghost-clipping step on one MI355X: examples/s, roofline, CPU baseline.

    python bench.py [--gpus 1] [--steps 20] [--warmup 30] [--workload gpt2-step]

One step is the whole hot path on one batch, through the C ABI:
  1. squared per-example norms of every linear layer and of the output head
     (grouped T x T Gram kernel; eq. 4-6)
  2. input-embedding norm and token buckets, and the tied cross term
     + 2 <g_in, g_out> (eq. 11, eq. 13), on a second stream beside step 1
     into a second norm array
  3. clip factors from both norm arrays (eq. 2, eq. 7)
  4. clipped sums of all linears and of the head (one grouped GEMM, K = B*T),
     with Gaussian noise and the division by B fused into the GEMM's store
     (eq. 3); one generator stream per parameter tensor
  5. the input-embedding part of the tied gradient: its rows (sorted
     segment sums) are formed on the second stream beside the GEMM and
     added onto the matrix the head's tiles wrote once the GEMM is done;
     the other sums that do not read the GEMM's outputs (an untied
     embedding's, the vectors', the position table's) also run there
With every parameter (--workload gpt2-full), the biases, LayerNorm gains and
biases and the position table join: a linear layer's bias gradient is summed
inside that layer's Gram launch (which streams its G anyway), the LayerNorm
and position terms on the second stream; their noised clipped sums run on
the second stream beside the GEMM.
Inputs are resident in HBM before the timed region starts. Prints one JSON
line; per-phase times go to stderr.
"""
from __future__ import annotations

import argparse
import gc
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "examples/sec for ghost-norm + clipped grad sum (GPT-2-small shapes); % MFMA peak"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
PEAK_FP32_MFMA_TFLOPS = 157.3  # MI355X dense fp32 matrix
# HBM bytes per launch of the clipped-sum kernel: rocprofv3 FETCH_SIZE x 2 +
# WRITE_SIZE x 1 (factors from a plain 1 GiB copy), recorded for the kernel
# source with this SHA-256; any other source reports null.
GEMM_TRAFFIC = {"gemm.hip sha256": "7a91e1ae131f658f382149bc039c08b59f6395901af6ec1a497ba5057e6b5138",
                "bytes": 2698230107}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    # The GPU needs ~40 ms of this load to settle: after 5 warm-up steps a GPT-2
    # step still times 5 % slower than after 30 or 100.
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--workload", default="gpt2-step",
                    choices=["gpt2-step", "gpt2-full", "c2", "c3", "c4", "c5"])
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--ldz-multiple", type=int, default=64,
                    help="pad logit-gradient rows to a multiple of this many columns")
    ap.add_argument("--cpu-budget", type=float, default=25.0,
                    help="seconds of oracle work for the CPU baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--configs", default="c2,c3,c4,c5",
                    help="further workloads measured after the headline one, each with the "
                         "same warm-up and steps, reported under \"configs\" ('none': skip)")
    ap.add_argument("--crossover", action="store_true",
                    help="instead of the step: time each distinct layer shape's grouped norm "
                         "with the Gram kernel and with the direct kernel (one JSON line)")
    ap.add_argument("--no-grad-store", action="store_true",
                    help="form the clipped sums by the GEMM even where every norm layer takes "
                         "the direct form (default: from the per-example gradient store)")
    ap.add_argument("--crossover-shape", default=None, metavar="B,T",
                    help="with --crossover: the workload's layer shapes at this batch size and "
                         "sequence length instead of its own")
    ap.add_argument("--token-kernels", action="store_true",
                    help="instead of the step: time the token-keyed norm calls (embedding norm "
                         "with buckets, tied cross term) alone on the workload's inputs, "
                         "one after another on an idle GPU (one JSON line)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="instead of the step: three plain 1 GiB device copies, the reference "
                         "for scaling the FETCH_SIZE / WRITE_SIZE counters to bytes")
    return ap.parse_args(argv)


def gemm_traffic():
    src = os.path.join(ROOT, "paper_2609_40335_amd", "csrc", "gemm.hip")
    with open(src, "rb") as f:
        h = hashlib.sha256(f.read()).hexdigest()
    return GEMM_TRAFFIC["bytes"] if h == GEMM_TRAFFIC["gemm.hip sha256"] else None


def round_up(x, m):
    return (x + m - 1) // m * m


class Step:
    """Device inputs, outputs and the prepared calls of one DP-SGD step.
    grad_store: when every norm layer takes the direct form, keep the
    examples' gradient tiles in HBM and form the clipped sums from them
    (dp_ghost_norm_linear_store, dp_clipped_grad_sum_noised_store)."""

    def __init__(self, wl, dp, torch, grad_store=True):
        self.wl, self.dp, self.torch = wl, dp, torch
        B, T = wl.B, wl.T
        def dev(a):  # bf16 bit patterns or fp32 values
            if a.dtype.kind == "u":
                return torch.from_numpy(a.view("int16")).view(torch.bfloat16).cuda()
            return torch.from_numpy(a).cuda()
        self.lin = [(dev(l.A), dev(l.G)) for l in wl.linears]
        h = wl.head
        self.h = h
        # one flat fp32 gradient vector; every parameter tensor is a view of it
        n_lin = sum(l.d_in * l.d_out for l in wl.linears)
        n_head = 0 if h is None or h.H is None else h.V * h.d * (1 if h.tied else 1)
        n_emb = 0 if h is None else (h.V * h.d if (h.H is None or not h.tied) else 0)
        n_vec = sum(v.d for v in wl.vectors)
        n_pos = wl.n_pos * h.d if wl.n_pos else 0
        self.n_coords = n_lin + n_head + n_emb + n_vec + n_pos
        self.flat = torch.zeros(self.n_coords, device="cuda")
        off = 0
        self.outs = []
        for l in wl.linears:
            self.outs.append(self.flat[off:off + l.d_in * l.d_out].view(l.d_in, l.d_out))
            off += l.d_in * l.d_out
        norm_layers = list(self.lin)
        sum_layers, sum_outs = list(self.lin), list(self.outs)
        if h is not None:
            self.ids = torch.from_numpy(h.ids).cuda()
            self.dE = dev(h.dE)
            if h.H is not None:
                self.H = dev(h.H)
                self.Gz = dev(h.Gz)[:, :, :h.V]
                self.W = self.flat[off:off + h.V * h.d].view(h.V, h.d)   # W_out (= E if tied)
                off += h.V * h.d
                norm_layers.append((self.H, self.Gz))
                sum_layers.append((self.Gz, self.H))                    # Gz^T H -> [V, d]
                sum_outs.append(self.W)
            if h.H is None or not h.tied:
                self.E = self.flat[off:off + h.V * h.d].view(h.V, h.d)
                off += h.V * h.d
            else:
                self.E = self.W
            self.seg = torch.empty((B, T), dtype=torch.int32, device="cuda")
            self.nu = torch.empty(B, dtype=torch.int32, device="cuda")
        # biases, LayerNorm gains/biases and the position table (full-parameter workloads)
        self.vec_outs, self.vg, self.P = [], None, None
        self.vec_grads = []
        bias_grads = [None] * len(norm_layers)
        if wl.vectors:
            # One device buffer per host array: a LayerNorm's gain and bias share
            # theirs (one pass over it). A linear layer's bias (no X, the layer's
            # own G) is fused into that layer's norm launch, which streams G
            # anyway; the LayerNorm parameters go to the vector kernel.
            same = {id(l.G): g for l, (_, g) in zip(wl.linears, self.lin)}
            lin_of = {id(l.G): k for k, l in enumerate(wl.linears)}

            def shared(a):
                if id(a) not in same:
                    same[id(a)] = dev(a)
                return same[id(a)]
            self.vec_grads = [None] * len(wl.vectors)
            rest = []
            for j, v in enumerate(wl.vectors):
                k = lin_of.get(id(v.G)) if v.X is None else None
                if k is not None and bias_grads[k] is None:
                    bias_grads[k] = torch.empty(B, v.d, device="cuda")
                    self.vec_grads[j] = bias_grads[k]
                else:
                    rest.append(j)
            if rest:
                self.vg = dp.VectorGroup([(None if wl.vectors[j].X is None
                                           else dev(wl.vectors[j].X), shared(wl.vectors[j].G))
                                          for j in rest])
                for j, g in zip(rest, self.vg.grads):
                    self.vec_grads[j] = g
            for v in wl.vectors:
                self.vec_outs.append(self.flat[off:off + v.d])
                off += v.d
        if wl.n_pos:
            self.P = self.flat[off:off + wl.n_pos * h.d].view(wl.n_pos, h.d)
            off += wl.n_pos * h.d
        assert off == self.n_coords
        self.norm_layers = norm_layers
        self.n_fused_biases = sum(g is not None for g in bias_grads)
        self.norm_group = dp.LinearGroup(norm_layers,
                                         bias_grads=bias_grads if self.n_fused_biases else None)
        # Noise generator ids per parameter tensor, as in the oracle's step:
        # linear l -> l, the input embedding (or tied matrix) -> L, an untied
        # head -> L + 1. Every GEMM-shaped output is written once with its
        # noise; the embedding part is then added onto the (tied or untied)
        # embedding matrix with the factors c/B, so that matrix is noised once
        # and never zero-filled.
        L = len(wl.linears)
        self.sum_tids = list(range(L))
        self.tied = h is not None and h.H is not None and h.tied
        if h is not None and h.H is not None:
            self.sum_tids.append(L if h.tied else L + 1)
        self.e_tid = L
        # One grouped launch for every GEMM-shaped clipped sum (split in two, the
        # second launch waits for the first to drain and costs more than any
        # work it lets overlap). The sums that do not read the GEMM's outputs
        # (an untied embedding's noise and sum, the vector and position sums)
        # run on a second stream (default priority) beside it; a tied
        # embedding sum adds onto the matrix the head's tiles write, so only
        # its rows are formed there and their addition follows the GEMM.
        self.sum_groups = [(dp.LinearGroup(sum_layers, sum_outs), list(self.sum_tids))] \
            if sum_layers else []
        side_work = h is not None or bool(wl.vectors) or bool(wl.n_pos)
        self.emb_rows = dp.EmbeddingRows(B, T, h.V, h.d) if self.tied else None
        # The norm terms other than the weight matrices' (embedding, cross
        # term, vectors, position table) go to the side stream into a second
        # array, beside the HBM-bound Gram launch; the clip adds both parts.
        self.side_norms = h is not None or bool(wl.vectors) or bool(wl.n_pos)
        self.side = torch.cuda.Stream() if (side_work or self.side_norms) else None
        self.ev_start = torch.cuda.Event()
        self.ev_norms = torch.cuda.Event()
        self.ev_clip = torch.cuda.Event()
        self.ev_side = torch.cuda.Event()
        self.side_sums = side_work
        # after the weight matrices (and an untied head): the vectors, then the position table
        t0 = L + (2 if (h is not None and h.H is not None and not h.tied) else 1)
        self.vec_tids = list(range(t0, t0 + len(wl.vectors)))
        self.pos_tid = t0 + len(wl.vectors)
        self.vsum = dp.VectorSums(self.vec_grads, self.vec_outs, self.vec_tids) \
            if wl.vectors else None
        self.n2 = torch.zeros(B, device="cuda")
        self.n2b = torch.zeros(B, device="cuda")   # the side stream's norm terms
        self.c = torch.zeros(B, device="cuda")
        self.c_b = torch.zeros(B, device="cuda")   # c / B
        # algorithmic work of the grouped clipped-sum GEMM (the dominant kernel)
        K = B * T
        es = 2 if wl.dtype == "bf16" else 4
        self.gemm_flops = 2.0 * K * sum(a.shape[2] * g.shape[2] for a, g in sum_layers)
        self.gemm_bytes = K * es * sum(a.shape[2] + g.shape[2] for a, g in sum_layers) + \
            4.0 * sum(a.shape[2] * g.shape[2] for a, g in sum_layers)
        # algorithmic work of the grouped norm launch: every A and G element read
        # once; flops of the form the library's AUTO rule picks per layer (the
        # symmetric T x T Gram counted once, or the direct per-example GEMM)
        self.norm_bytes = float(K * es * sum(a.shape[2] + g.shape[2] for a, g in norm_layers))
        self.norm_flops, self.norm_direct = 0.0, 0
        for a, g in norm_layers:
            di, do = a.shape[2], g.shape[2]
            r = 0.38 if do > 4096 else 0.49   # the library's throughput ratios (AUTO)
            if T + 1 > r * 2.0 * di * do / (di + do):
                self.norm_flops += 2.0 * K * di * do
                self.norm_direct += 1
            else:
                self.norm_flops += float(B) * T * (T + 1) * (di + do)
        self.step_id = 0
        # Long sequences: every norm layer takes the direct form, which forms
        # each example's gradient tiles anyway. Kept in HBM (B * tiles * 256 KB,
        # 7.9 GB for GPT-2 small at B = 16) they give the clipped sums as a
        # weighted sum instead of a second GEMM. The norm table is the sum
        # table: the linears' outputs [d_in, d_out], a head (H, Gz) written
        # transposed into its [V, d] matrix.
        self.store = None
        if grad_store and self.norm_direct == len(norm_layers) and not self.n_fused_biases:
            nbytes = self.norm_group.store_bytes()
            free, _ = torch.cuda.mem_get_info()
            if nbytes and nbytes < 0.8 * free:
                self.store = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
                head = h is not None and h.H is not None
                self.norm_group.set_outputs(list(self.outs) + ([self.W] if head else []))
                self.store_tr = [False] * len(self.lin) + ([True] if head else [])
                tiles = sum(-(-a.shape[2] // 256) * -(-g.shape[2] // 256) for a, g in norm_layers)
                self.store_bytes_read = float(B) * tiles * 256 * 256 * 4
                self.store_out_bytes = 4.0 * sum(a.shape[2] * g.shape[2] for a, g in norm_layers)

    def total_norm2(self):
        """Per-example squared norms of the last step (both parts summed)."""
        return self.n2 + self.n2b if self.side_norms else self.n2.clone()

    def run(self, marks=None):
        """One step; marks(name) records an event after each phase if given."""
        dp, wl, h = self.dp, self.wl, self.h
        mark = marks or (lambda name: None)
        main = self.torch.cuda.current_stream()
        if self.side_norms:
            # after everything enqueued so far (the previous step's clip read n2b)
            self.ev_start.record(main)
            self.side.wait_event(self.ev_start)
            with self.torch.cuda.stream(self.side):
                # the first term writes n2b, the others add to it
                acc = False
                if h is not None:
                    dp.dp_ghost_norm_embedding(self.ids, self.dE, h.V, self.n2b, accumulate=acc,
                                               seg_id=self.seg, n_unique=self.nu)
                    acc = True
                    if h.H is not None and h.tied:
                        dp.dp_tied_cross_term(self.ids, self.dE, self.H, self.Gz, h.V, self.n2b,
                                              scale=2.0, accumulate=True)
                if self.vg is not None:
                    self.vg.grads_and_norm(self.n2b, accumulate=acc)
                    acc = True
                if self.P is not None:
                    dp.dp_ghost_norm_positional(self.dE, self.n2b, accumulate=acc)
            self.ev_norms.record(self.side)
            if h is not None and not self.tied:
                # An untied embedding's noise needs no clip factor: it is written
                # beside the norm launch (after the event the clip waits for),
                # and its clipped sum follows on the same stream.
                with self.torch.cuda.stream(self.side):
                    dp.dp_noise_fill(self.E, wl.sigma, wl.C, wl.B, tensor_id=self.e_tid,
                                     seed=1234, step=self.step_id)
        if self.store is not None:
            self.norm_group.ghost_norm_store(self.n2, self.store)
        else:
            self.norm_group.ghost_norm(self.n2, accumulate=False)
        mark("norms")
        if self.side_norms:
            main.wait_event(self.ev_norms)
            mark("side_norms_join")
            dp.dp_clip_factors_scaled2(self.n2, self.n2b, wl.C, 1.0 / wl.B, self.c_b, c=self.c)
        else:
            dp.dp_clip_factors_scaled(self.n2, wl.C, 1.0 / wl.B, self.c_b, c=self.c)
        mark("clip")
        # clipped sums with the Gaussian mechanism fused into their store
        # (eq. 3): (S + sigma C z) / B
        kw = dict(seed=1234, step=self.step_id)
        if self.side_sums:
            self.ev_clip.record(main)
            self.side.wait_event(self.ev_clip)
            with self.torch.cuda.stream(self.side):
                if h is not None and not self.tied:
                    dp.dp_clipped_grad_sum(None, self.dE, self.c_b, self.E, ids=self.ids, V=h.V,
                                           accumulate=True)
                if self.vsum is not None:
                    self.vsum.noised(self.c, wl.sigma, wl.C, wl.B, **kw)
                if self.P is not None:
                    dp.dp_clipped_grad_sum_positional_noised(self.dE, self.c, self.P,
                                                             self.pos_tid, wl.sigma, wl.C, wl.B,
                                                             **kw)
                # last, so that one wait covers the whole second stream: every
                # wait across streams costs ~10 us, even on a finished event
                if self.emb_rows is not None:
                    self.emb_rows.compute(self.dE, self.ids, self.c_b)
            self.ev_side.record(self.side)
        if self.store is not None:
            self.norm_group.clipped_sum_noised_store(self.c, self.store, self.sum_tids, wl.sigma,
                                                     wl.C, wl.B, transpose_out=self.store_tr,
                                                     **kw)
            mark("clipped_sum_noise")
        else:
            for grp, tids in self.sum_groups:
                grp.clipped_sum_noised(self.c, tids, wl.sigma, wl.C, wl.B, **kw)
                mark("clipped_sum_noise")
        if self.side_sums:
            main.wait_event(self.ev_side)
            mark("side_sums_join")
        if self.emb_rows is not None:
            self.emb_rows.add_to(self.E)
            mark("embedding_sum")
        self.step_id += 1


def crossover(st, dp, torch, reps=10):
    """Row a10: per distinct (d_in, d_out) of the workload, the grouped norm of
    all layers of that shape with the T x T Gram kernel and with the direct
    per-example GEMM, next to the flop-count rule T + 1 > 2 d_in d_out / (d_in + d_out)."""
    B, T = st.wl.B, st.wl.T
    by_shape = {}
    for A, G in st.norm_layers:
        by_shape.setdefault((A.shape[2], G.shape[2]), []).append((A, G))
    rows = []
    for (d_in, d_out), layers in by_shape.items():
        us = {}
        for name, algo in (("gram", dp.DP_NORM_GRAM), ("direct", dp.DP_NORM_DIRECT)):
            grp = dp.LinearGroup([(a, g, algo) for a, g in layers])
            n2 = torch.zeros(B, device="cuda")
            for _ in range(2):
                grp.ghost_norm(n2)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                grp.ghost_norm(n2)
            e1.record()
            torch.cuda.synchronize()
            us[name] = e0.elapsed_time(e1) / reps * 1e3
        rule = "direct" if T + 1 > 2.0 * d_in * d_out / (d_in + d_out) else "gram"
        gram_flop = float(len(layers)) * B * T * (T + 1) * (d_in + d_out)
        direct_flop = float(len(layers)) * B * 2.0 * T * d_in * d_out
        rows.append({"d_in": d_in, "d_out": d_out, "layers": len(layers),
                     "gram_us": round(us["gram"], 1), "direct_us": round(us["direct"], 1),
                     "gram_tflops": round(gram_flop / us["gram"] / 1e6, 1),
                     "direct_tflops": round(direct_flop / us["direct"] / 1e6, 1),
                     "flop_rule": rule,
                     "faster": "direct" if us["direct"] < us["gram"] else "gram"})
        log(f"[bench] crossover d_in={d_in} d_out={d_out} x{len(layers)}: gram {us['gram']:.1f} us, "
            f"direct {us['direct']:.1f} us (rule: {rule})")
    return rows


def token_kernels(st, dp, torch, reps=30):
    """The embedding norm (with bucket ids) and the tied cross term alone, each
    call timed by HIP events around it on the main stream (kernel plus the
    partials' reduction launch), medians over `reps` calls after 5 warm-ups."""
    import numpy as np
    h = st.h
    if h is None:
        return {}
    calls = {"embedding_norm": lambda n2: dp.dp_ghost_norm_embedding(
        st.ids, st.dE, h.V, n2, seg_id=st.seg, n_unique=st.nu)}
    if h.H is not None and h.tied:
        calls["tied_cross"] = lambda n2: dp.dp_tied_cross_term(st.ids, st.dE, st.H, st.Gz, h.V, n2)
    n2 = torch.zeros(st.wl.B, device="cuda")
    out = {}
    for name, fn in calls.items():
        for _ in range(5):
            fn(n2)
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn(n2)
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e3)
        out[name] = {"median_us": round(float(np.median(ts)), 1), "min_us": round(min(ts), 1)}
        log(f"[bench] {name}: median {out[name]['median_us']} us, min {out[name]['min_us']} us")
    return out


def cpu_baseline(wl, n_coords, budget):
    """The fp64 oracle on the host: per-example work on a sample of examples,
    noise on a slice of coordinates, extrapolated to one full step."""
    import numpy as np
    import oracle
    blas = "unknown"
    try:
        from threadpoolctl import threadpool_info
        libs = [p for p in threadpool_info() if p.get("user_api") == "blas"]
        threads = max([p.get("num_threads", 1) for p in libs] or [os.cpu_count() or 1])
        if libs:
            blas = " ".join(str(libs[0].get(k, "")) for k in ("internal_api", "version")).strip()
    except Exception:
        threads = os.cpu_count() or 1
    t0 = time.perf_counter()
    oracle.step(wl, examples=[0], noise=False)
    per_ex = time.perf_counter() - t0
    n_ex = int(max(1, min(wl.B - 1, budget * 0.7 / max(per_ex, 1e-9))))
    if n_ex > 1:
        t0 = time.perf_counter()
        oracle.step(wl, examples=list(range(1, 1 + n_ex)), noise=False)
        per_ex = (time.perf_counter() - t0) / n_ex
    n_slice = 1 << 22
    S = np.zeros(n_slice)
    t0 = time.perf_counter()
    oracle.add_noise(S, wl.sigma, wl.C, wl.B, 1234, 0, 0)
    per_coord = (time.perf_counter() - t0) / n_slice
    t_step = wl.B * per_ex + n_coords * per_coord
    return {
        "value": wl.B / t_step, "unit": "examples/s", "cores": int(threads), "kind": "oracle",
        "sample": (f"fp64 oracle (materialised per-example gradients): norms, clip factors and "
                   f"clipped sums on {1 + n_ex} example(s) of this workload, noise on "
                   f"{n_slice} coordinates; extrapolated to B={wl.B} examples and "
                   f"{n_coords} coordinates per step"),
        "seconds_per_example": per_ex, "seconds_noise_per_step": n_coords * per_coord,
        "host": host_cpu(), "blas": blas,
    }


def host_cpu():
    """CPU model name and socket count from /proc/cpuinfo (Linux)."""
    model, sockets = "unknown", set()
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                key, _, val = line.partition(":")
                key = key.strip()
                if key == "model name" and model == "unknown":
                    model = val.strip()
                elif key == "physical id":
                    sockets.add(val.strip())
    except OSError:
        pass
    return {"model": model, "sockets": max(1, len(sockets))}


def timed_run(st, torch, steps, warmup):
    """warmup untimed steps, then `steps` steps bracketed by HIP events on the
    main stream (the one every main-stream kernel is launched on), recording
    only the two events around the clipped-sum launch inside them; then up to
    10 more steps with every phase marked. Returns (ms per step, clipped-sum
    launch us, {phase: us})."""
    # A full garbage collection first, so that none falls due in the steps
    # below: a full pass over this process's objects stalls the host for tens
    # of milliseconds, and early in the timed loop the host is only a step
    # ahead of the GPU, which would idle. It runs before the warm-up, because
    # the GPU lowers its clock while idle and the warm-up brings it back.
    gc.collect()
    for _ in range(warmup):
        st.run()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = []

    def marks(name):
        e = torch.cuda.Event(enable_timing=True)
        e.record(stream)
        ev[-1].append((name, e))

    # every timing event costs the stream a few microseconds (all the phase
    # marks together add ~20 us to a GPT-2 step), so the timed steps record
    # only the two around the clipped-sum launch
    def gemm_marks(name):
        if name in ("clip", "clipped_sum_noise"):
            marks(name)

    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(steps):
        ev.append([])
        st.run(gemm_marks)
    end.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / steps
    gemm_us = sum(step[0][1].elapsed_time(step[-1][1]) for step in ev) / len(ev) * 1e3
    ev.clear()
    for _ in range(min(steps, 10)):
        e0 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        ev.append([("start", e0)])
        st.run(marks)
    torch.cuda.synchronize()
    phases = {}
    for step_ev in ev:
        for (_, a), (n1, b) in zip(step_ev[:-1], step_ev[1:]):
            phases.setdefault(n1, []).append(a.elapsed_time(b) * 1e3)
    return ms, gemm_us, {k: sum(v) / len(v) for k, v in phases.items()}


def rooflines(st, gemm_us, phase_us):
    """The clipped-sum GEMM against the MFMA peak of its dtype, and the grouped
    norm launch (the norms phase of the main stream) against HBM when it is
    the Gram form and against the MFMA peak when every layer takes the direct
    form."""
    peak = PEAK_BF16_TFLOPS if st.wl.dtype == "bf16" else PEAK_FP32_MFMA_TFLOPS
    if st.store is not None:
        # the clipped sums from the per-example gradient store: read every
        # example's tiles once, write every output once
        q = st.store_bytes_read + st.store_out_bytes
        achieved = q / (gemm_us * 1e-6) / 1e9
        gemm = {"bound": "hbm", "kernel": "store_sum_kernel (clipped sums from the per-example "
                                          "gradient store, noise fused)",
                "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": achieved / PEAK_HBM_GBS,
                "timed": "HIP events on the main stream around the clipped-sum call, inside "
                         "the timed steps (one launch), beside the second stream's sums",
                "algorithmic_flop_per_launch": st.gemm_flops,
                "algorithmic_bytes_per_launch": q}
    else:
        achieved = st.gemm_flops / (gemm_us * 1e-6) / 1e12
        gemm = {"bound": "mfma", "kernel": "dl_gemm_kernel (clipped sum with fused noise)",
                "achieved": achieved, "peak": peak, "unit": "TFLOP/s", "frac": achieved / peak,
                "timed": "HIP events on the main stream around the grouped clipped-sum call, "
                         "inside the timed steps: the GEMM launch and the split-tail fix-up "
                         "kernel that follows it (~16 us at the GPT-2 step), beside the second "
                         "stream's embedding rows",
                "algorithmic_flop_per_launch": st.gemm_flops,
                "algorithmic_bytes_per_launch": st.gemm_bytes}
    norm_us = phase_us["norms"]
    n_layers = len(st.norm_layers)
    if st.norm_direct == n_layers:
        ach = st.norm_flops / (norm_us * 1e-6) / 1e12
        norm = {"bound": "mfma", "achieved": ach, "peak": peak, "unit": "TFLOP/s",
                "frac": ach / peak}
    else:
        ach = st.norm_bytes / (norm_us * 1e-6) / 1e9
        norm = {"bound": "hbm", "achieved": ach, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": ach / PEAK_HBM_GBS}
    norm.update({"kernel": f"grouped norm launch ({n_layers - st.norm_direct} Gram, "
                           f"{st.norm_direct} direct layers"
                           + (", each example's gradient tiles written to the store)"
                              if st.store is not None else ")"),
                 "timed": "the norms phase of the phase-marked steps",
                 "algorithmic_bytes_per_launch": st.norm_bytes,
                 "algorithmic_flop_per_launch": st.norm_flops})
    return gemm, norm


def main(argv=None) -> int:
    args = parse(argv)
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the library has no "
              f"multi-GPU path. Run with --gpus 1.", file=sys.stderr)
        return 2
    import numpy as np  # noqa: F401
    import torch

    from paper_2609_40335_amd import dpghost as dp
    from workloads import gen

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    if args.copy_calibration:
        n = 256 << 20  # 256 Mi floats = 1 GiB
        src = torch.ones(n, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": src.numel() * 4, "copies": 3}), flush=True)
        return 0
    dp.lib()
    V = gen.GPT2_VOCAB
    ldz = round_up(V, args.ldz_multiple)

    bt = {}
    if args.crossover_shape:
        if not args.crossover:
            raise SystemExit("--crossover-shape applies to --crossover only")
        b_, t_ = (int(x) for x in args.crossover_shape.split(","))
        bt = {"B": b_, "T": t_}

    def load(name):
        t0 = time.perf_counter()
        wl = gen.make_workload(name, seed=args.seed, ldz=ldz, **bt)
        log(f"[bench] generated {name}: {wl.description} in {time.perf_counter() - t0:.1f}s")
        return wl, Step(wl, dp, torch, grad_store=not args.no_grad_store)

    wl, st = load(args.workload)
    log(f"[bench] {len(wl.linears)} linear layers, head={'none' if wl.head is None else ('tied' if wl.head.tied else 'untied')}, "
        f"{st.n_coords} gradient coordinates")

    if args.crossover:
        rows = crossover(st, dp, torch)
        print(json.dumps({"crossover": rows, "workload": args.workload, "B": wl.B, "T": wl.T}),
              flush=True)
        return 0

    if args.token_kernels:
        print(json.dumps({"token_kernels": token_kernels(st, dp, torch),
                          "workload": args.workload, "B": wl.B, "T": wl.T}), flush=True)
        return 0

    ms, gemm_us, phase_us = timed_run(st, torch, args.steps, args.warmup)
    for k, v in phase_us.items():
        log(f"[bench]   {k:16s} {v:9.1f} us")
    gemm_rf, norm_rf = rooflines(st, gemm_us, phase_us)
    gemm_rf["traffic"] = gemm_traffic() if args.workload == "gpt2-step" and st.store is None \
        else None
    gemm_rf["traffic_source"] = (
        "rocprofv3 FETCH_SIZE and WRITE_SIZE of this kernel source at the GPT-2 step, scaled "
        "by a 1 GiB copy (profiles/hbm_traffic_gpt2_step_B32_T128.md); null for another "
        "workload or when the source differs from the one measured")
    log(f"[bench] clipped sum ({gemm_rf['kernel'].split(' ')[0]}) in {gemm_us:.1f} us = "
        f"{gemm_rf['achieved']:.1f} {gemm_rf['unit']} ({gemm_rf['frac']:.3f}); grouped norm "
        f"{st.norm_bytes / 1e9:.3f} GB in {phase_us['norms']:.1f} us: {norm_rf['frac']:.3f} of "
        f"its {norm_rf['bound']} peak")

    h = wl.head
    config = {"workload": f"{args.workload}: {wl.description}", "B": wl.B, "T": wl.T,
              "linear_layers": len(wl.linears),
              "head": None if h is None else ("tied" if h.tied else ("untied" if h.H is not None
                                                                   else "embedding-only")),
              "V": None if h is None else h.V, "ldz": None if h is None else h.ldz,
              "gradient_coordinates": st.n_coords, "C": wl.C, "sigma": wl.sigma,
              "phase_us": {k: round(v, 1) for k, v in phase_us.items()}}
    out = {
        "metric": METRIC, "value": wl.B / (ms / 1e3), "unit": "examples/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype,
        "data": "synthetic", "config": config, "roofline": gemm_rf, "norm_roofline": norm_rf,
    }
    del st
    torch.cuda.empty_cache()

    # The other workloads of the metric (GPT-2 body alone, tied head alone,
    # DistilGPT2 tied at T = 256, GPT-2 untied at T = 1024): the same step,
    # warm-up and timing, one after another.
    extra = [c for c in args.configs.split(",") if c and c != "none" and c != args.workload]
    if extra:
        out["configs"] = {}
    for name in extra:
        wl_c, st_c = load(name)
        ms_c, gemm_c, ph_c = timed_run(st_c, torch, args.steps, args.warmup)
        g_c, n_c = rooflines(st_c, gemm_c, ph_c)
        hc = wl_c.head
        out["configs"][name] = {
            "workload": wl_c.description, "B": wl_c.B, "T": wl_c.T, "dtype": wl_c.dtype,
            "head": None if hc is None else ("tied" if hc.tied else "untied"),
            "ms_per_step": ms_c, "examples_per_s": wl_c.B / (ms_c / 1e3),
            "clipped_sum_us": gemm_c, "clipped_sum_form": "gradient store" if st_c.store
            is not None else "GEMM", "clipped_sum_bound": g_c["bound"],
            "clipped_sum_frac": g_c["frac"],
            "norms_us": ph_c["norms"], "norms_bound": n_c["bound"], "norms_frac": n_c["frac"],
            "phase_us": {k: round(v, 1) for k, v in ph_c.items()}}
        log(f"[bench] {name}: {ms_c:.3f} ms/step, {wl_c.B / (ms_c / 1e3):.0f} ex/s, clipped sum "
            f"{gemm_c:.1f} us ({g_c['frac']:.3f} of {g_c['bound']}), norms {ph_c['norms']:.1f} us "
            f"({n_c['frac']:.3f} of {n_c['bound']})")
        del st_c, wl_c
        torch.cuda.empty_cache()

    if not args.no_cpu_baseline:
        t0 = time.perf_counter()
        out["cpu_baseline"] = cpu_baseline(wl, out["config"]["gradient_coordinates"],
                                           args.cpu_budget)
        log(f"[bench] cpu baseline took {time.perf_counter() - t0:.1f}s")
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
