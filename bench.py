#!/usr/bin/env python3
"""Bench of the GliDe + CaPE decoding hot path on one MI355X.

One step = one pass of the whole hot path over one batch of synthetic input,
in the order a decoding round runs it:
  1. cape_expand        draft distributions -> expanded proposal tree;
  2. glide_tree_attn    one verification attention launch per target layer,
                        with the tree just built (tree mode);
  3. glide_verify_commit  the target's greedy token per tree row, accept
                        length, last node and bonus token, and the commit of
                        the accepted path's K/V rows in every layer;
  4. glide_tree_attn    the GliDe cross-attention of the draft's query rows
                        into the top target layer's cache (cross mode), for
                        workloads that have one.
Inputs are generated and resident in HBM before timing starts.

Default workload: Vicuna-7B verify step (32 layers x 32 heads, head_dim 128,
batch 1, prefix 2048, 16-node CaPE tree of depth 5 with top-k 3) plus one
5-query GliDe cross-attention layer.

Prints one JSON line.  `value` is the attention bytes per step (K/V rows read,
Q read, O written in every attention call of the step; the algorithmic count,
split partials excluded) divided by the GPU time of the whole step, replayed
as a HIP graph so that host launch overhead is not timed.  `roofline` is the
verification attention call (attention kernel + split merge): HIP events
around graph replays of the verification step, divided by its call count.
`other_configs` repeats the measurement for every other workload, and
`stream_probe` gives the streaming rates of plain torch kernels for context.
"""

import argparse
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import paper_2402_02082_amd as glide  # noqa: E402
from synth import workloads as W  # noqa: E402

HBM_PEAK_GBPS = 8000.0
METRIC = "tree-attn KV-read GB/s (% of HBM peak); µs per verify step at 7B shape"
SEED = 2


def attn_bytes(lens, n_q, heads, elem, tree):
    """Algorithmic HBM bytes of one attention launch: every visible K/V row
    once, the query rows once, the output rows once."""
    keys = sum(int(l) + (n_q if tree else 0) for l in lens)
    return heads * (2 * keys * 128 * elem + 2 * len(lens) * n_q * 128 * elem)


class Step:
    """Device-resident inputs and outputs of one workload, and its step."""

    def __init__(self, wl, dtype, seed, max_splits=0):
        dev = torch.device("cuda")
        self.wl, self.dev, self.max_splits = wl, dev, max_splits
        B, N, V = wl.batch, wl.nodes, wl.vocab
        self.lens_np = W.prefix_lengths(wl, seed)
        self.lens = torch.from_numpy(self.lens_np).to(dev)
        if wl.tree == "cape":
            probs, chain, leaf = W.draft_probs(wl, seed)
            logits, self.planted, _ = W.planted_logits_cape(wl, seed, chain, leaf, probs)
            self.probs_np = probs
            self.probs = torch.from_numpy(probs).to(dev)
        else:
            cand = W.chain_tokens(wl, seed)
            logits, self.planted = W.planted_logits_chain(wl, seed, cand)
            self.probs = None
            self.chain_tokens = torch.from_numpy(cand).to(dev)
            self.chain_parents = torch.from_numpy(
                np.tile(np.arange(-1, N - 1, dtype=np.int32), (B, 1))).to(dev)
        self.logits_np = logits
        self.logits = torch.from_numpy(logits).to(dev)
        self.layers = [W.attention_layer(wl, seed, l, dtype, dev) for l in range(wl.layers)]
        self.outs = [torch.empty_like(q) for q, _, _ in self.layers]
        self.cross_q = W.cross_queries(wl, seed, dtype, dev) if wl.cross else None
        self.cross_out = torch.empty_like(self.cross_q) if wl.cross else None
        self.tokens = torch.empty((B, N), dtype=torch.int32, device=dev)
        self.parents = torch.empty((B, N), dtype=torch.int32, device=dev)
        self.n_nodes = torch.empty((B,), dtype=torch.int32, device=dev)
        self.ta = torch.empty((B, N + 1), dtype=torch.int32, device=dev)
        self.acc = torch.empty((B,), dtype=torch.int32, device=dev)
        self.last = torch.empty((B,), dtype=torch.int32, device=dev)
        self.bonus = torch.empty((B,), dtype=torch.int32, device=dev)
        self.path = torch.empty((B, N), dtype=torch.int32, device=dev)
        self.seq_out = torch.empty((B,), dtype=torch.int32, device=dev)
        self.k_caches = [k for _, k, _ in self.layers]
        self.v_caches = [v for _, _, v in self.layers]
        L_cap = wl.l_cap
        self.ws = glide.attn_workspace(B, N, wl.heads, L_cap, max_splits, dev)
        self.xws = (glide.attn_workspace(B, wl.cross_queries, wl.heads, L_cap, max_splits, dev)
                    if wl.cross else None)
        self.cape_ws = torch.empty(max(glide.load().cape_expand_workspace(B, wl.depth, V), 1),
                                   dtype=torch.uint8, device=dev)
        elem = 2 if dtype == torch.bfloat16 else 4
        self.verify_bytes = attn_bytes(self.lens_np, N, wl.heads, elem, True)
        self.cross_bytes = attn_bytes(self.lens_np, wl.cross_queries, wl.heads, elem, False) \
            if wl.cross else 0

    def tree(self):
        if self.probs is not None:
            return self.tokens, self.parents
        return self.chain_tokens, self.chain_parents

    def run_verify_layers(self):
        """The verification pass's attention: one call per target layer."""
        _, parents = self.tree()
        for (q, k, v), o in zip(self.layers, self.outs):
            glide.glide_tree_attn(q, k, v, self.lens, parents, o, max_splits=self.max_splits,
                                  workspace=self.ws)

    def commit(self):
        """Argmax, acceptance and the cache commit of every layer."""
        tokens, parents = self.tree()
        glide.glide_verify_commit(self.logits, tokens, parents, self.k_caches, self.v_caches,
                                  self.lens, self.seq_out, self.ta, self.acc, self.last,
                                  self.bonus, self.path)

    def commit_bytes(self):
        """Algorithmic bytes of one commit: the logits read once, and every
        moved K/V row of every layer and head read and written once."""
        wl = self.wl
        acc, path = self.acc.cpu().numpy(), self.path.cpu().numpy()
        moved = sum(int(np.sum(path[b, :acc[b]] != np.arange(acc[b]))) for b in range(wl.batch))
        row = 128 * self.layers[0][1].element_size()
        return self.logits.numel() * 4 + 2 * 2 * moved * wl.heads * wl.layers * row, moved

    def run(self):
        wl = self.wl
        if self.probs is not None:
            glide.cape_expand(self.probs, wl.k, wl.nodes, self.tokens, self.parents, self.n_nodes,
                              workspace=self.cape_ws)
        self.run_verify_layers()
        self.commit()
        if wl.cross:
            _, k, v = self.layers[-1]
            glide.glide_tree_attn(self.cross_q, k, v, self.lens, None, self.cross_out,
                                  max_splits=self.max_splits, workspace=self.xws)


def host_cores():
    """Host threads the oracle may use on this machine: the CPUs this process
    may run on, capped by the OMP_NUM_THREADS share the machine sets (a GPU
    box gives each GPU's jobs a share of its cores), and the CPU model."""
    affinity = len(os.sched_getaffinity(0))
    share = int(os.environ.get("OMP_NUM_THREADS", "0") or 0)
    threads = min(affinity, share) if share > 0 else affinity
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"threads": threads, "affinity_cores": affinity, "omp_num_threads": share or None,
            "cpu_model": model}


def _bits(t):
    return t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32).cpu().numpy()


def _f64(t):
    return t.float().cpu().numpy().astype(np.float64)


def oracle_integer_steps(step):
    """The float64 oracle's CaPE expansion and verification epilogue (argmax,
    acceptance, commit of every layer's cache), in full; returns (seconds,
    parents the attention uses)."""
    from oracle import cape as OC
    from oracle import commit as OCm
    wl = step.wl
    k_bits = [_bits(k) for k in step.k_caches]
    v_bits = [_bits(v) for v in step.v_caches]
    t0 = time.perf_counter()
    if wl.tree == "cape":
        tokens, parents, _ = OC.cape_expand(step.probs_np, wl.k, wl.nodes)
    else:
        tokens = step.chain_tokens.cpu().numpy()
        parents = step.chain_parents.cpu().numpy()
    OCm.verify_commit(step.logits_np, tokens, parents, step.lens_np, k_bits, v_bits)
    return time.perf_counter() - t0, parents


def cpu_baseline(step, threads, budget_s=12.0):
    """The float64 oracle on a bounded sample of the same step: the CaPE
    expansion and the verification epilogue (argmax, acceptance, commit of
    every layer's cache) in full, then verification-attention layers (all
    heads) until ~budget_s, then the cross-attention layer; at `threads`
    BLAS threads.  Reported in the metric's unit (attention GB/s)."""
    import threadpoolctl

    from oracle import attention as OA

    wl = step.wl
    with threadpoolctl.threadpool_limits(threads):
        t_int, parents = oracle_integer_steps(step)
        t_attn, nbytes, layers_done = 0.0, 0, 0
        for (q, k, v) in step.layers:
            qh, kh, vh = _f64(q), _f64(k), _f64(v)
            t1 = time.perf_counter()
            OA.tree_attention(qh, kh, vh, step.lens_np, parents)
            t_attn += time.perf_counter() - t1
            nbytes += step.verify_bytes
            layers_done += 1
            if t_attn + t_int > budget_s:
                break
        if wl.cross:
            _, k, v = step.layers[-1]
            t1 = time.perf_counter()
            OA.tree_attention(_f64(step.cross_q), _f64(k), _f64(v), step.lens_np, None)
            t_attn += time.perf_counter() - t1
            nbytes += step.cross_bytes
    total = t_attn + t_int
    return {"value": round(nbytes / total / 1e9, 6), "unit": "GB/s", "cores": threads,
            "kind": "oracle",
            "sample": "%s: CaPE expansion and the verification epilogue (argmax, acceptance, "
                      "commit of every layer) in full, %d of %d verification-attention layers "
                      "(all heads)%s, float64 NumPy, %d BLAS thread(s), %.1f s"
                      % (wl.name, layers_done, wl.layers, " + the cross-attention layer"
                         if wl.cross else "", threads, total)}


def oracle_sampled(step, threads, budget_s=5.0):
    """The oracle's time for a workload too large to run in full on the host:
    the integer steps in full, and verification attention on the
    deterministic sample of (sequence, head) units -- every sequence, the
    first and last layer, heads 0, H/2 and H - 1, in that order until
    ~budget_s of attention time -- extrapolated to the whole step (mean time
    per unit x sequences x layers x heads, and the cross layer's units
    likewise).  Labelled extrapolated."""
    import threadpoolctl

    from oracle import attention as OA

    wl = step.wl
    heads = sorted({0, wl.heads // 2, wl.heads - 1})
    layers = sorted({0, wl.layers - 1})
    units = [(b, l, h) for l in layers for h in heads for b in range(wl.batch)]
    with threadpoolctl.threadpool_limits(threads):
        t_int, parents = oracle_integer_steps(step)
        t_units, done = 0.0, 0
        for b, l, h in units:
            q, k, v = step.layers[l]
            L = int(step.lens_np[b])
            rows = L + wl.nodes
            qh, kh, vh = _f64(q[b, :, h]), _f64(k[b, h, :rows]), _f64(v[b, h, :rows])
            t1 = time.perf_counter()
            OA.tree_attention_head(qh, kh, vh, L, parents[b])
            t_units += time.perf_counter() - t1
            done += 1
            if t_units > budget_s:
                break
        per_unit = t_units / done
        total_units = wl.batch * wl.layers * wl.heads
        t_cross, cross_done = 0.0, 0
        if wl.cross:
            _, k, v = step.layers[-1]
            for b, _, h in [u for u in units if u[1] == layers[-1]]:
                L = int(step.lens_np[b])
                qh, kh, vh = _f64(step.cross_q[b, :, h]), _f64(k[b, h, :L]), _f64(v[b, h, :L])
                t1 = time.perf_counter()
                OA.tree_attention_head(qh, kh, vh, L, None)
                t_cross += time.perf_counter() - t1
                cross_done += 1
                if t_cross > budget_s / 2:
                    break
    seconds = t_int + per_unit * total_units
    nbytes = step.verify_bytes * wl.layers
    if cross_done:
        seconds += t_cross / cross_done * wl.batch * wl.heads
        nbytes += step.cross_bytes
    return {"value": round(nbytes / seconds / 1e9, 6), "unit": "GB/s", "cores": threads,
            "kind": "oracle", "extrapolated": True, "seconds_per_step": round(seconds, 3),
            "sample": "%s: integer steps in full (%.2f s); verification attention on %d of "
                      "%d (sequence, layer, head) units (every sequence x first/last layer x "
                      "heads 0, H/2, H-1), %.3f s per unit, extrapolated to %d units%s"
                      % (wl.name, t_int, done, len(units), per_unit, total_units,
                         "; cross attention %d units" % cross_done if cross_done else "")}


def kernel_source_hash():
    """Hash of the attention kernels' code (comments and whitespace removed,
    so that editing a comment does not orphan the counter summaries)."""
    import hashlib
    import re
    code = []
    for n in ("tree_attn.hip", "attn.h"):
        text = open(os.path.join(ROOT, "paper_2402_02082_amd", "csrc", n)).read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        code.append(" ".join(text.split()))
    return hashlib.sha256("\n".join(code).encode()).hexdigest()[:16]


# Stem of each workload's profile summaries under profiles/.
PROFILE_STEM = {"7b-1layer-chain5": "chain5", "vicuna7b-cape16": "vicuna7b",
                "vicuna13b-cape32": "vicuna13b", "vicuna33b-cape64": "vicuna33b",
                "7b-longctx-cape64": "longctx"}


def verify_kernels(wl):
    """The launches one verification call of the workload makes, as the
    library plans them (bf16)."""
    ws = glide.load().glide_tree_attn_workspace(wl.batch, wl.nodes, wl.heads, wl.head_dim, wl.l_cap, 0)
    main = "tree_attn_kernel" if wl.nodes <= 16 else "tree_attn_shared_kernel"
    if ws == 0:
        return main + ", one split per sequence"
    if wl.batch == 1 and wl.nodes <= 16:
        return main + ", split merge inside the kernel"
    return main + " + tree_attn_combine"


def load_traffic(wl_name="vicuna7b-cape16"):
    """HBM bytes per verification attention call of a workload from the
    committed rocprofv3 counter summary, or None when there is none or the
    kernel source changed since it was taken."""
    path = os.path.join(ROOT, "profiles", "tree_attn_%s_pmc.json" % PROFILE_STEM.get(wl_name, wl_name))
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_sha256_16") != kernel_source_hash():
        return None
    return rec.get("traffic_bytes_per_launch")


def measure(wl, steps, warmup, max_splits):
    """Builds a workload's step, captures it (and its verification layers
    alone, and its verification epilogue alone) as HIP graphs, and times
    them with HIP events around the replays.  Short calls are captured
    several times per graph so that a replay outlasts the host's cost of
    launching it; times are per repetition."""
    step = Step(wl, torch.bfloat16, SEED, max_splits)
    torch.cuda.synchronize()
    rep = max(1, 16 // wl.layers)   # steps / verification passes per graph
    rep_commit = 16                 # verification epilogues per graph
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for _ in range(max(warmup, 1)):
            step.run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g_step, g_verify, g_commit = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_step):
        for _ in range(rep):
            step.run()
    with torch.cuda.graph(g_verify):
        for _ in range(rep):
            step.run_verify_layers()
    with torch.cuda.graph(g_commit):
        for _ in range(rep_commit):
            step.commit()
    torch.cuda.synchronize()
    for _ in range(warmup):
        g_step.replay()
    torch.cuda.synchronize()

    def timed(graph, per):
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record()
        for _ in range(steps):
            graph.replay()
        stop.record()
        torch.cuda.synchronize()
        return start.elapsed_time(stop) / (steps * per)

    # Timed region 1: whole steps.
    ms_step = timed(g_step, rep)
    planted_ok = bool(np.array_equal(step.acc.cpu().numpy(), step.planted))
    # Timed region 2: the verification step alone (the L attention calls).
    verify_us = timed(g_verify, rep) * 1e3
    # Timed region 3: the verification epilogue alone (argmax, acceptance,
    # commit of every layer).
    commit_us = timed(g_commit, rep_commit) * 1e3
    del g_step, g_verify, g_commit
    return step, {"ms_step": ms_step, "verify_us": verify_us, "planted_ok": planted_ok,
                  "commit_us": commit_us, "graph_reps": rep}


def commit_record(step, t):
    nbytes, moved = step.commit_bytes()
    return {"us": round(t["commit_us"], 2), "bytes": nbytes,
            "gbps": round(nbytes / (t["commit_us"] * 1e-6) / 1e9, 1),
            "rows_moved": moved, "layers": step.wl.layers,
            "launches": "argmax + acceptance/commit"}


def cross_block_record(step, steps, copies=8):
    """The GliDe cross-attention block (query projection, cross attention,
    output projection) at d_D = H * 128 on the workload's caches: `copies`
    distinct weight sets and layers per graph, so the working set (over
    256 MB) cannot be served from the last-level cache; also the query
    projection alone.  Random bf16 weights scaled 1/sqrt(d_D), packed once
    before timing (a load-time transformation of static weights); the
    row-major figures are reported beside them."""
    wl = step.wl
    dev = step.dev
    B, Nq, H = wl.batch, wl.cross_queries, wl.heads
    d_D = H * 128
    copies = min(copies, wl.layers)
    g = torch.Generator(device=dev)
    g.manual_seed(SEED)
    mk = lambda *shape: (torch.randn(shape, generator=g, device=dev) / np.sqrt(shape[-1])).to(torch.bfloat16)  # noqa: E731
    hidden = torch.randn((B, Nq, d_D), generator=g, device=dev).to(torch.bfloat16)
    wq = [mk(H * 128, d_D) for _ in range(copies)]
    wo = [mk(d_D, H * 128) for _ in range(copies)]
    wq_p = [glide.pack_rows_weights(w) for w in wq]
    wo_p = [glide.pack_rows_weights(w) for w in wo]
    outs = [torch.empty_like(hidden) for _ in range(copies)]
    q_out = torch.empty((B * Nq, H * 128), dtype=torch.bfloat16, device=dev)
    ws = glide.cross_block_workspace(B, Nq, d_D, H, wl.l_cap, dev)

    def blocks():
        for i in range(copies):
            _, k, v = step.layers[i]
            glide.glide_cross_block_packed(hidden, wq_p[i], k, v, step.lens, wo_p[i], outs[i], workspace=ws)

    def projections():
        for i in range(copies):
            glide.glide_rows_matmul_packed(hidden.view(B * Nq, d_D), wq_p[i], q_out)

    def blocks_row_major():
        for i in range(copies):
            _, k, v = step.layers[i]
            glide.glide_cross_block(hidden, wq[i], k, v, step.lens, wo[i], outs[i], workspace=ws)

    def projections_row_major():
        for i in range(copies):
            glide.glide_rows_matmul(hidden.view(B * Nq, d_D), wq[i], q_out)

    res = {}
    for name, fn in (("block", blocks), ("projection", projections),
                     ("block_row_major", blocks_row_major), ("projection_row_major", projections_row_major)):
        fn()
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            fn()
        for _ in range(steps):  # untimed warm-up, as many replays as are timed
            graph.replay()
        torch.cuda.synchronize()
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record()
        for _ in range(steps):
            graph.replay()
        stop.record()
        torch.cuda.synchronize()
        res[name] = start.elapsed_time(stop) * 1e3 / (steps * copies)
        del graph
    act = B * Nq * d_D * 2
    proj_bytes = H * 128 * d_D * 2 + act + B * Nq * H * 128 * 2
    block_bytes = 2 * proj_bytes + step.cross_bytes
    return {"us": round(res["block"], 2), "bytes": block_bytes,
            "gbps": round(block_bytes / (res["block"] * 1e-6) / 1e9, 1),
            "projection_us": round(res["projection"], 2), "projection_bytes": proj_bytes,
            "projection_gbps": round(proj_bytes / (res["projection"] * 1e-6) / 1e9, 1),
            "weights": "packed per 16-row operand tile",
            "row_major_us": round(res["block_row_major"], 2),
            "row_major_projection_us": round(res["projection_row_major"], 2),
            "d_D": d_D, "query_rows": B * Nq, "copies_per_graph": copies}


def spec_sampling_record(steps, gamma=5, V=32000):
    """Chain verification with speculative sampling (gamma = 5, the GliDe-only
    experiments' setting) for batch 1 and 16: seeded Dirichlet(0.3) draft
    rows, target rows blended from them and noise, uniforms as inputs; 16
    calls per graph (the call is launch-sized)."""
    dev = torch.device("cuda")
    rng = np.random.default_rng(SEED)
    out = {}
    for B in (1, 16):
        pd = rng.dirichlet(np.full(V, 0.3), size=(B, gamma)).astype(np.float32)
        noise = rng.dirichlet(np.full(V, 0.3), size=(B, gamma + 1)).astype(np.float32)
        pt = noise.copy()
        pt[:, :gamma] = 0.7 * pd + 0.3 * noise[:, :gamma]
        tokens = pd.argmax(axis=2).astype(np.int32)
        u = rng.random((B, gamma + 1)).astype(np.float32)
        args = [torch.from_numpy(a).to(dev) for a in (tokens, pd, pt, u)]
        acc = torch.empty((B,), dtype=torch.int32, device=dev)
        tok = torch.empty((B,), dtype=torch.int32, device=dev)
        reps = 16
        glide.spec_sample_verify(*args, acc, tok)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for _ in range(reps):
                glide.spec_sample_verify(*args, acc, tok)
        for _ in range(steps):  # untimed warm-up, as many replays as are timed
            graph.replay()
        torch.cuda.synchronize()
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record()
        for _ in range(steps):
            graph.replay()
        stop.record()
        torch.cuda.synchronize()
        us = start.elapsed_time(stop) * 1e3 / (steps * reps)
        # one draw row (the residual reads the draft row as well) per sequence
        nbytes = B * (2 * V * 4 + gamma * 12 + (gamma + 1) * 4)
        out["batch_%d" % B] = {"us": round(us, 2), "bytes": nbytes,
                               "gbps": round(nbytes / (us * 1e-6) / 1e9, 1),
                               "mean_accept_len": float(acc.float().mean().item())}
        del graph
    out.update({"gamma": gamma, "vocab": V})
    return out


def block_attention_record(steps, B=4, T=2048, H=32, block=5, copies=4, eager_only=0):
    """The block-masked cross attention of draft training at a 7B-head
    training shape (4 sequences of 2048 positions, blocks of 5): `copies`
    distinct inputs per graph (1 GB, beyond the last-level cache).  Bound:
    MFMA (4 * 128 flops per visible key per query and head)."""
    dev = torch.device("cuda")
    g = torch.Generator(device=dev)
    g.manual_seed(SEED)
    mk = lambda *shape: torch.randn(shape, generator=g, device=dev).to(torch.bfloat16)  # noqa: E731
    qs = [mk(B, T, H, 128) for _ in range(copies)]
    ks = [mk(B, H, T, 128) for _ in range(copies)]
    vs = [mk(B, H, T, 128) for _ in range(copies)]
    outs = [torch.empty_like(q) for q in qs]

    def fn():
        for i in range(copies):
            glide.glide_block_attn(qs[i], ks[i], vs[i], outs[i], block)
    if eager_only:
        for _ in range(eager_only):
            fn()
        torch.cuda.synchronize()
        print(json.dumps({"only": "block", "passes": eager_only, "calls": eager_only * copies}),
              flush=True)
        return None
    fn()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        fn()
    # Untimed warm-up of three times the timed replays (about 25 ms): the
    # first replays after other work run up to 15 % slower than sustained
    # MFMA load settles to.
    for _ in range(3 * steps):
        graph.replay()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        graph.replay()
    stop.record()
    torch.cuda.synchronize()
    us = start.elapsed_time(stop) * 1e3 / (steps * copies)
    flops = B * H * sum(4 * 128 * block * (p // block) for p in range(T))
    nbytes = 2 * B * T * H * 128 * 2 + 2 * B * H * T * 128 * 2
    del graph, qs, ks, vs, outs
    torch.cuda.empty_cache()
    return {"us": round(us, 1), "flops": flops, "tflops": round(flops / (us * 1e-6) / 1e12, 1),
            "frac_of_bf16_mfma_peak": round(flops / (us * 1e-6) / 2.5e15, 4),
            "bytes": nbytes, "gbps": round(nbytes / (us * 1e-6) / 1e9, 1),
            "shape": {"batch": B, "positions": T, "heads": H, "block": block}}


def speedup_model(verify_us, cross_block):
    """E(Spd) = (1 - a^(g+1)) / ((1 - a)(g c + 1)) at gamma = 5 with GliDe's
    acceptance rate on Vicuna-7B / GSM8K (Table 1: 64.8 %), once with the
    paper's cost coefficient (6.7 %) and once with an attention-only proxy
    measured here: one cross-attention block (a draft step's cross layer) over
    one verification step's attention."""
    alpha, gamma, c_paper = 0.648, 5, 0.067
    rec = {"alpha": alpha, "gamma": gamma, "c_paper": c_paper,
           "expected_speedup_paper_c": round(glide.glide_expected_speedup(alpha, gamma, c_paper), 4)}
    if cross_block:
        c = cross_block["us"] / verify_us
        rec["c_attention_proxy"] = round(c, 4)
        rec["expected_speedup_proxy_c"] = round(glide.glide_expected_speedup(alpha, gamma, c), 4)
    return rec


def other_configs(skip, steps, warmup, max_splits, oracle_threads=None):
    """The verification step and the whole step of every other workload,
    measured as the headline one (same seed, graphs, events); with
    oracle_threads, the float64 oracle's time beside it (the one-layer
    workload in full at that many threads and at one, the others on their
    extrapolated sample)."""
    out = []
    for i in sorted(W.WORKLOADS):
        if i == skip:
            continue
        wl = W.WORKLOADS[i]
        step, t = measure(wl, steps, warmup, max_splits)
        vgbps = step.verify_bytes * wl.layers / (t["verify_us"] * 1e-6) / 1e9
        sbytes = step.verify_bytes * wl.layers + step.cross_bytes
        traffic = load_traffic(wl.name)
        oracle = None
        if oracle_threads:
            if wl.layers == 1:
                oracle = cpu_baseline(step, oracle_threads, budget_s=30.0)
                oracle["one_thread"] = cpu_baseline(step, 1, budget_s=30.0)
            else:
                oracle = oracle_sampled(step, oracle_threads)
        out.append({"workload": wl.name, "layers": wl.layers, "batch": wl.batch,
                    "tree_nodes": wl.nodes,
                    "us_per_verify_step": round(t["verify_us"], 2),
                    "us_per_verify_call": round(t["verify_us"] / wl.layers, 2),
                    "verify_step_gbps": round(vgbps, 1),
                    "verify_frac_of_hbm_peak": round(vgbps / HBM_PEAK_GBPS, 4),
                    "ms_per_step": round(t["ms_step"], 4),
                    "step_gbps": round(sbytes / (t["ms_step"] * 1e-3) / 1e9, 1),
                    "planted_accept_len_ok": t["planted_ok"],
                    "verify_call_bytes": step.verify_bytes,
                    "verify_call_traffic": traffic,
                    "verify_call_traffic_ratio": round(traffic / step.verify_bytes, 4) if traffic else None,
                    "verify_commit": commit_record(step, t),
                    "cross_block": cross_block_record(step, steps) if wl.cross else None,
                    "oracle": oracle})
        del step
        torch.cuda.empty_cache()
    return out


def stream_probe():
    """Measured streaming rates of plain torch kernels, for context: a
    reduction that reads 4 GiB, and a 2 GiB device-to-device copy."""
    x = torch.zeros(2 << 30, dtype=torch.bfloat16, device="cuda")
    y = torch.empty(1 << 30, dtype=torch.bfloat16, device="cuda")
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    x.sum()
    torch.cuda.synchronize()
    start.record()
    for _ in range(10):
        x.sum()
    stop.record()
    torch.cuda.synchronize()
    read = x.numel() * 2 * 10 / (start.elapsed_time(stop) * 1e-3) / 1e9
    src = x[: y.numel()]
    y.copy_(src)
    start.record()
    for _ in range(10):
        y.copy_(src)
    stop.record()
    torch.cuda.synchronize()
    copy = 2 * y.numel() * 2 * 10 / (start.elapsed_time(stop) * 1e-3) / 1e9
    del x, y
    torch.cuda.empty_cache()
    return {"read_gbps": round(read, 1), "copy_gbps": round(copy, 1),
            "kernels": "torch sum over 4 GiB bf16 (read), torch copy of 2 GiB (read + write)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=2, choices=sorted(W.WORKLOADS))
    ap.add_argument("--max-splits", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--headline-only", action="store_true",
                    help="skip the other workloads and the streaming probe")
    ap.add_argument("--only", choices=["verify", "block"], default=None,
                    help="only run warmup + steps eager passes of one part (no timing, no JSON "
                         "record), for counter and trace passes of a profiler: 'verify' = the "
                         "workload's verification attention calls, 'block' = the block-masked "
                         "training attention at the bench's shape")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="only run a plain device-to-device copy of this many MiB (five times), "
                         "for scaling HBM traffic counters; prints nothing else")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the hot path here is a single-GPU kernel set and "
              "no multi-GPU figure is produced (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    if args.calibrate_copy_mib:
        n = args.calibrate_copy_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n, "copies": 5}), flush=True)
        return
    glide.load()

    wl = W.WORKLOADS[args.workload]
    if args.only == "block":
        block_attention_record(args.steps, eager_only=args.warmup + args.steps)
        return
    if args.only == "verify":
        step = Step(wl, torch.bfloat16, SEED, args.max_splits)
        if step.probs is not None:
            glide.cape_expand(step.probs, wl.k, wl.nodes, step.tokens, step.parents, step.n_nodes,
                              workspace=step.cape_ws)
        for _ in range(args.warmup + args.steps):
            step.run_verify_layers()
        torch.cuda.synchronize()
        print(json.dumps({"only": "verify", "workload": wl.name, "passes": args.warmup + args.steps,
                          "calls": (args.warmup + args.steps) * wl.layers}), flush=True)
        return
    step, t = measure(wl, args.steps, args.warmup, args.max_splits)
    ms_step, verify_us, planted_ok = t["ms_step"], t["verify_us"], t["planted_ok"]

    # The dominant kernel's launch: one glide_tree_attn call (attention kernel
    # + split merge) of the verification pass, averaged over the calls of
    # timed region 2 (events on the stream the graph replays on).
    call_ms = verify_us * 1e-3 / wl.layers

    step_bytes = step.verify_bytes * wl.layers + step.cross_bytes
    value = step_bytes / (ms_step * 1e-3) / 1e9
    achieved = step.verify_bytes / (call_ms * 1e-3) / 1e9
    rec = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "layers": wl.layers, "heads": wl.heads,
                   "head_dim": wl.head_dim, "batch": wl.batch,
                   "prefix": [int(x) for x in step.lens_np], "tree_nodes": wl.nodes,
                   "tree_depth": wl.depth, "top_k": wl.k, "vocab": wl.vocab,
                   "cross_attn_queries": wl.cross_queries, "seed": SEED},
        "us_per_verify_step": round(verify_us, 2),
        "verify_step_gbps": round(step.verify_bytes * wl.layers / (verify_us * 1e-6) / 1e9, 2),
        "hbm_frac_of_step": round(value / HBM_PEAK_GBPS, 4),
        "planted_accept_len_ok": planted_ok,
        "verify_commit": commit_record(step, t),
        "cross_block": cross_block_record(step, args.steps) if wl.cross else None,
        "spec_sampling": spec_sampling_record(args.steps),
        "block_attention": block_attention_record(max(3, min(args.steps, 10))),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": load_traffic(wl.name),
                     "kernel": "glide_tree_attn call (%s), verification layer" % verify_kernels(wl),
                     "bytes_per_launch": step.verify_bytes,
                     "avg_launch_us": round(call_ms * 1e3, 3),
                     "timing": "HIP events around graph replays of the verification "
                               "step's calls, divided by the call count"},
    }
    rec["speedup_model"] = speedup_model(verify_us, rec["cross_block"])
    host = host_cores()
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(step, host["threads"])
        rec["cpu_baseline"]["host"] = host
        rec["cpu_baseline"]["one_thread"] = cpu_baseline(step, 1)
    if not args.headline_only:
        del step
        torch.cuda.empty_cache()
        rec["other_configs"] = other_configs(args.workload, max(3, min(args.steps, 10)),
                                             max(1, min(args.warmup, 2)), args.max_splits,
                                             None if args.no_cpu_baseline else host["threads"])
        rec["stream_probe"] = stream_probe()
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
