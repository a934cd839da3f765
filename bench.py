#!/usr/bin/env python3
"""Benchmark of the Dustin sparse verification step on one MI355X.

One step is every stage of the hot path on one batch of synthetic input, with the inputs
resident in HBM:
    target scoring-head importance        (Eq. 5, target half)
    draft scoring-head importance x 3     (Eq. 5, draft half, one call per draft layer)
    tiered hybrid selection               (Eq. 6)
    sparse verification attention x L     (one global index set reused by all L layers)
    dense full-cache verification x L     (the comparison the paper normalises against)
HIP events on the launch stream separate the stages.  Prints ONE JSON line; every other
message goes to stderr.

    python bench.py [--gpus 1] [--steps 30] [--warmup 5] [--workload qwen72b] [--k 2048]
"""
import argparse
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0           # MI355X HBM3E, vendor figure
SPARSE_KERNEL = "verify_attn_kernel"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=30)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--workload", default="qwen72b",
                   choices=["tiny", "qwen7b", "qwen72b", "ragged", "long131k"])
    p.add_argument("--k", type=int, default=None, help="override the budget k (e.g. 512)")
    p.add_argument("--layers", type=int, default=None, help="override the stacked layer count")
    p.add_argument("--groups", choices=["1", "hkv"], default="1",
                   help="index sets per sequence: one (the paper's global set) or one per KV head")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-sample-seqs", type=int, default=16)
    p.add_argument("--no-secondary", action="store_true",
                   help="skip the other workloads (ragged, 131k, k = 512) that the default run also times")
    p.add_argument("--no-digit-hist", action="store_true",
                   help="the top-k makes its own first pass over each row instead of taking the score calls' "
                        "first-digit histograms")
    p.add_argument("--copy-probe", action="store_true",
                   help="also run one plain 1 GiB device copy (counter calibration)")
    p.add_argument("--only", choices=["all", "sparse", "dense", "estimate", "page"], default="all",
                   help="restrict the timed step (profiling runs)")
    return p.parse_args()


# ----------------------------------------------------------------------------- bytes

def sparse_bytes(s):
    """Algorithmic HBM bytes of one sparse layer: gathered K and V rows of every KV head
    (selected + verification window), Q read, O written, the index list read (+ one page
    table entry per gathered token when paged)."""
    tot = 0
    for n, t, k in zip(s.seq_lens, s.n_query, s.budget):
        kk = min(k, n)
        tot += s.num_kv_heads * (kk + t) * s.head_dim * 2 * 2
        tot += 2 * t * s.num_q_heads * s.head_dim * 2
        tot += s.groups * kk * 4
        if s.page_size:
            tot += s.num_kv_heads * (kk + t) * 4
    return tot


def dense_bytes(s):
    tot = 0
    for n, t in zip(s.seq_lens, s.n_query):
        tot += s.num_kv_heads * (n + t) * s.head_dim * 2 * 2
        tot += 2 * t * s.num_q_heads * s.head_dim * 2
        if s.page_size:
            tot += s.num_kv_heads * (n + t) * 4
    return tot


def score_bytes(s, target=True):
    """Distinct KV heads touched by the scoring heads, read once, plus S written (and the
    historical init read)."""
    if target:
        gs = s.num_q_heads // s.num_kv_heads
        kvh = len({h // gs for h in s.target_heads})
        return sum(kvh * n * s.head_dim * 2 + 4 * n * (1 + (s.init_kind is not None))
                   for n in s.seq_lens)
    d = s.draft
    gs = d.num_q_heads // d.num_kv_heads
    kvh = len({h // gs for h in d.heads})
    per_layer = sum(kvh * n * d.head_dim * 2 for n in s.seq_lens)
    return d.layers * per_layer + sum(4 * n for n in s.seq_lens) * (2 * d.layers - 1)


def topk_bytes(s):
    return sum(2 * 4 * n + 4 * min(k, n) for n, k in zip(s.seq_lens, s.budget))


def page_bytes(s, ps):
    """Page estimator: statistics rows (2d bf16 per page and KV head) built from K; page
    scores read the rows of the KV heads their heads use and write S (4 B per position)."""
    pages = [-(-n // ps) for n in s.seq_lens]
    row = 2 * s.head_dim * 2
    meta = sum(s.num_kv_heads * p * row for p in pages)
    build = sum(s.num_kv_heads * n * s.head_dim * 2 for n in s.seq_lens) + meta
    q_all = sum(t * s.num_q_heads * s.head_dim * 2 for t in s.n_query)
    score_all = meta + q_all + sum(4 * n for n in s.seq_lens)
    gs = s.num_q_heads // s.num_kv_heads
    kvh = len({h // gs for h in s.target_heads})
    score_srh = sum(kvh * p * row + 4 * n for p, n in zip(pages, s.seq_lens))
    return {"build": build, "score_all_heads": score_all, "score_scoring_heads": score_srh}


# ----------------------------------------------------------------------------- traffic

def measured_traffic(workload, k):
    """HBM bytes per sparse launch from the committed rocprofv3 counter summary, or None
    when it is missing or was taken on different kernel sources."""
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_sparse_verify_attn_{workload}_k{k}.md")
    if not os.path.exists(path):
        return None
    m = re.search(r"<!--\s*traffic:\s*(\{.*?\})\s*-->", open(path).read(), re.S)
    if not m:
        return None
    from paper_2606_24957_amd.rocprof_summary import kernel_sources_sha
    rec = json.loads(m.group(1))
    if rec.get("source_sha256") != kernel_sources_sha():
        return None
    return rec.get("bytes_per_launch")


# ----------------------------------------------------------------------------- timing

def med(x):
    x = sorted(x)
    return x[len(x) // 2] if x else float("nan")


def mean(x):
    return sum(x) / len(x) if x else float("nan")


class StepTimer:
    """The prepared launches of one step of a workload -- target score, draft scores, top-k,
    then L sparse layers and L dense layers with the one index set -- and their timing with
    HIP events recorded on the launch stream (around each stage; the L layers of a block run
    back to back, as in a forward pass, since an event between launches adds an end-of-pipe
    wait of its own)."""

    def __init__(self, s, layers, est, dev, digit_hist=True):
        import torch
        import paper_2606_24957_amd as D
        self.s, self.L = s, len(layers)
        B, N, G = s.B, s.n_max, s.groups
        i32 = lambda x: torch.tensor(list(x), dtype=torch.int32, device=dev)
        self.seq, self.nq, self.gam = i32(s.seq_lens), i32(s.n_query), i32(s.draft_gamma)
        self.bud, self.mm = i32(s.budget), i32(s.m)
        self.s_t = torch.zeros((B, G, N), dtype=torch.float32, device=dev)
        self.s_d = torch.zeros((B, 1, N), dtype=torch.float32, device=dev)
        self.idx = torch.zeros((B, G, s.k_max), dtype=torch.int32, device=dev)
        self.cnt = torch.zeros((B, G), dtype=torch.int32, device=dev)
        self.outs = [torch.empty_like(l.q) for l in layers]
        self.outs_d = [torch.empty_like(l.q) for l in layers]
        init_t = est.init_target
        if init_t is not None and G > 1:  # one historical row, the same for every group
            init_t = init_t.expand(B, G, N)
        self.score_t = D.plan_score(est.q_target, layers[0].k, self.seq, s.target_heads, groups=G, init=init_t,
                                    out=self.s_t, max_len=N, page_table=layers[0].page_table)
        self.score_d = []
        if est.s_draft_given is not None:
            self.s_d.copy_(est.s_draft_given)
        else:
            self.score_d.append(D.plan_score_layers(est.draft_q, est.draft_k, self.seq, s.draft.heads,
                                                    n_query=self.gam, out=self.s_d, max_len=N,
                                                    ws_tag="score_draft"))
        # the target's and the draft's scores in one dustin_score_calls (one launch where both
        # take the single-pass form); with one selection group they count their outputs by top
        # key digit, and the top-k takes those counts in place of its first pass
        self.hist_t = D.digit_hist(B, dev) if G == 1 and digit_hist else None
        self.hist_d = D.digit_hist(B, dev) if G == 1 and self.score_d and digit_hist else None
        self.scores = D.plan_score_calls([self.score_t] + self.score_d,
                                         digit_hists=[self.hist_t] + [self.hist_d] * len(self.score_d))
        self.sel = D.plan_topk(self.s_d, self.s_t, self.seq, s.k_max, budget=self.bud, m=self.mm, n_sink=s.n_sink,
                               n_window=s.n_window, groups=G, idx=self.idx, count=self.cnt, hist_d=self.hist_d,
                               hist_t=self.hist_t)
        self.sparse = [D.plan_sparse_verify_attn(l.q, l.k, l.v, self.idx, self.cnt, self.seq, n_query=self.nq,
                                                 page_table=l.page_table, out=o)
                       for l, o in zip(layers, self.outs)]
        self.dense = [D.plan_dense_verify_attn(l.q, l.k, l.v, self.seq, n_query=self.nq, page_table=l.page_table,
                                               out=o) for l, o in zip(layers, self.outs_d)]

    @staticmethod
    def _ev():
        import torch
        e = torch.cuda.Event(enable_timing=True)
        e.record()
        return e

    def step(self, rec, only="all"):
        marks = [self._ev()] if rec else None
        if only in ("all", "estimate", "sparse"):
            self.scores()
            if rec: marks.append(self._ev())
            self.sel()
            if rec: marks.append(self._ev())
        if only in ("all", "sparse"):
            for c in self.sparse:
                c()
            if rec: marks.append(self._ev())
        if only in ("all", "dense"):
            for c in self.dense:
                c()
            if rec: marks.append(self._ev())
        return marks

    def run(self, steps, warmup, only="all", copy_probe=False):
        """Stage durations (ms) of `steps` timed steps after `warmup` untimed ones."""
        import torch
        for _ in range(warmup):
            self.step(False, only)
        torch.cuda.synchronize()
        if copy_probe:
            a = torch.empty(1 << 30, dtype=torch.uint8, device=self.seq.device)
            b_ = torch.empty_like(a)
            b_.copy_(a)
            torch.cuda.synchronize()
            del a, b_
        all_marks = []
        t_start = time.perf_counter()
        for _ in range(steps):
            all_marks.append(self.step(True, only))
        torch.cuda.synchronize()
        wall = time.perf_counter() - t_start
        out = {"est_s": [], "est_k": [], "sp": [], "dn": [], "ms_per_step": wall * 1e3 / steps}
        for m in all_marks:
            i = 0
            if only in ("all", "estimate", "sparse"):
                out["est_s"].append(m[0].elapsed_time(m[1]))
                out["est_k"].append(m[1].elapsed_time(m[2]))
                i = 2
            if only in ("all", "sparse"):
                out["sp"].append(m[i].elapsed_time(m[i + 1]) / self.L)
                i += 1
            if only in ("all", "dense"):
                out["dn"].append(m[i].elapsed_time(m[i + 1]) / self.L)
        return out

    def score_parts(self, reps):
        """Mean event times (ms) of the target's and the draft's score calls as separate
        launches (context for the one-launch figure the step uses)."""
        import torch
        t, d = [], []
        for _ in range(reps + 2):
            e = [self._ev()]
            self.score_t()
            e.append(self._ev())
            for c in self.score_d:
                c()
            e.append(self._ev())
            torch.cuda.synchronize()
            t.append(e[0].elapsed_time(e[1]))
            d.append(e[1].elapsed_time(e[2]))
        return mean(t[2:]), mean(d[2:])

    def sparse_with_events(self, reps):
        """Per-launch event times (ms) of the sparse layers with an event between launches."""
        import torch
        sp_ev = []
        for _ in range(reps):
            es = [self._ev()]
            for c in self.sparse:
                c()
                es.append(self._ev())
            torch.cuda.synchronize()
            sp_ev += [es[j].elapsed_time(es[j + 1]) for j in range(self.L)]
        return sp_ev


# ----------------------------------------------------------------------------- page estimator

def page_estimator(s, layers, est, seq, nq, bud, steps, warmup, ps=16):
    """The page estimator (Quest with 16-position pages) on the same layers: statistics
    built once per layer (prefill) and refreshed for the newest T_b positions (per layer
    and step), page scores of every query head of a layer (Quest-16) and of the target's
    scoring heads only.  Each figure is the event time of `steps` launches cycling over
    the stacked layers, divided by `steps`."""
    import torch
    import paper_2606_24957_amd as D
    dev = seq.device
    B, N = s.B, s.n_max
    metas = [D.page_meta_empty(B, N, s.num_kv_heads, s.head_dim, ps, dev) for _ in layers]
    build = [D.plan_page_meta(l.k, seq, ps, m, max_len=N, page_table=l.page_table)
             for l, m in zip(layers, metas)]
    newest = (seq - nq).clamp(min=0)  # the last T_b positions stand for the newest append
    update = [D.plan_page_meta(l.k, seq, ps, m, from_=newest, max_span=s.t_max, max_len=N,
                               page_table=l.page_table) for l, m in zip(layers, metas)]
    s_q = torch.zeros((B, 1, N), dtype=torch.float32, device=dev)
    s_h = torch.zeros((B, 1, N), dtype=torch.float32, device=dev)
    quest = [D.plan_page_score(l.q, m, seq, list(range(s.num_q_heads)), ps, max_len=N, n_query=nq,
                               out=s_q) for l, m in zip(layers, metas)]
    srh = [D.plan_page_score(est.q_target, m, seq, s.target_heads, ps, max_len=N, out=s_h) for m in metas]
    idx = torch.zeros((B, 1, s.k_max), dtype=torch.int32, device=dev)
    cnt = torch.zeros((B, 1), dtype=torch.int32, device=dev)
    sel = [D.plan_topk(None, s_q, seq, s.k_max, budget=bud, m_scalar=0, n_sink=s.n_sink,
                       n_window=s.n_window, idx=idx, count=cnt)]

    def timed(calls):
        for i in range(warmup):
            calls[i % len(calls)]()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(steps):
            calls[i % len(calls)]()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / steps

    t_build = timed(build)
    t_update = timed(update)
    t_quest = timed(quest)
    t_srh = timed(srh)
    t_sel = timed(sel)
    nb = page_bytes(s, ps)

    def gbps(b, us):
        return round(b / (us * 1e-6) / 1e9, 1)

    per_layer = t_update + t_quest + t_sel
    rec = {
        "page_size": ps,
        "build_us_per_layer": round(t_build, 2), "build_GBps": gbps(nb["build"], t_build),
        "update_us_per_layer": round(t_update, 2),
        "score_all_heads_us_per_layer": round(t_quest, 2),
        "score_all_heads_GBps": gbps(nb["score_all_heads"], t_quest),
        "score_all_heads_frac": round(nb["score_all_heads"] / (t_quest * 1e-6) / 1e9 / PEAK_HBM_GBPS, 4),
        "score_all_heads_bytes": nb["score_all_heads"],
        "score_scoring_heads_us": round(t_srh, 2),
        "score_scoring_heads_GBps": gbps(nb["score_scoring_heads"], t_srh),
        "topk_us": round(t_sel, 2),
        "quest16_estimation_us_per_step_L80": round(80 * per_layer, 1),
    }
    log(f"[bench] page estimator (page {ps}): build {t_build:.1f} us/layer, update {t_update:.1f}, "
        f"all-heads score {t_quest:.1f} us/layer ({rec['score_all_heads_GBps']} GB/s), scoring-heads "
        f"score {t_srh:.1f} us, top-k {t_sel:.1f} us; Quest-16 estimation at L=80 {80 * per_layer:.0f} us/step")
    del metas
    return rec


# ----------------------------------------------------------------------------- selection fidelity

def arr_eval(s, layer, s_t, s_d, idx, cnt, seq, nq, bud, mm):
    """Windowed attention recovery rate (Eqs. 1-4) of the step's selection and of its
    variants on the first layer: A-bar from every query head over the 5 verification queries
    (dustin_score), then dustin_arr per set, averaged over the batch.  Also the event time
    of one evaluation (A-bar plus the oracle's selection and both ARRs)."""
    import torch
    import paper_2606_24957_amd as D
    N, k, P, G = s.n_max, s.k_max, s.n_sink + s.n_window, s.groups
    heads = list(range(s.num_q_heads))
    hpg = s.num_q_heads // G
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    abar = D.score(layer.q, layer.k, seq, heads, n_query=nq, groups=G, max_len=N, page_table=layer.page_table)
    oidx, ocnt = D.topk(None, abar, seq, k, budget=bud, n_sink=0, n_window=0, m_scalar=0, groups=G)
    orc = D.arr(abar, oidx, ocnt, seq, hpg, window=nq)
    hyb = D.arr(abar, idx, cnt, seq, hpg, window=nq)
    e1.record()
    torch.cuda.synchronize()
    eval_us = e0.elapsed_time(e1) * 1e3
    res = {"sd_oracle": orc, "dustin": hyb}
    ti, tc = D.topk(None, s_t, seq, k, budget=bud, m_scalar=0, n_sink=s.n_sink, n_window=s.n_window, groups=G)
    res["dustin_t"] = D.arr(abar, ti, tc, seq, hpg, window=nq)
    di, dc = D.topk(s_d, None, seq, k, budget=bud, n_sink=s.n_sink, n_window=s.n_window, groups=G)
    res["dustin_d"] = D.arr(abar, di, dc, seq, hpg, window=nq)
    if len(set(s.budget)) == 1:  # StreamingLLM-like: the whole budget on sinks and the recent window
        si, sc = D.topk(None, s_t, seq, k, budget=bud, m_scalar=0, n_sink=s.n_sink, n_window=k - s.n_sink,
                        groups=G)
        res["sinks_and_recent"] = D.arr(abar, si, sc, seq, hpg, window=nq)
    torch.cuda.synchronize()
    rec = {name: round(float(v.mean()), 5) for name, v in res.items()}
    rec["eval_us"] = round(eval_us, 1)
    rec["budget_k"] = k
    log(f"[bench] windowed ARR at k={k} (mean over the batch): " +
        ", ".join(f"{n} {v:.4f}" for n, v in rec.items() if n not in ("eval_us", "budget_k")) +
        f"; evaluation {eval_us:.0f} us")
    del abar
    return rec


# ----------------------------------------------------------------------------- SpecAttn-style step

def per_layer_selection(s, layers, dev, steps, warmup, sparse_us, dense_us, dustin_est_us, draft_layers=24):
    """The per-layer, all-draft-head selection of the paper's SpecAttn comparison: relevance
    from all 14 heads of each of the draft model's 24 layers (synthetic, planted like the
    draft scoring layers), one index set per draft layer, target layers matched by depth.
    Its estimation (the per-layer scores and the top-k) is timed with events; per-step
    speedups use the sparse and dense per-layer times measured above."""
    import torch
    from paper_2606_24957_amd import step as S
    from paper_2606_24957_amd import workloads as W
    s24 = s.replace(draft=W.DraftShape(layers=draft_layers))
    est24 = W.make_estimation(s24, layers[0], dev)
    st = S.PerLayerSelectionStep(s24, layers, est24, dev, n_target=80)
    for _ in range(warmup):
        st.run()
    torch.cuda.synchronize()
    e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    e0.record()
    for _ in range(steps):
        st.ops[0]()
        st.ops[1]()
    e1.record()
    for _ in range(steps):
        st.run()
    e2.record()
    torch.cuda.synchronize()
    est_us = e0.elapsed_time(e1) * 1e3 / steps
    step_us = e1.elapsed_time(e2) * 1e3 / steps
    rec = {
        "draft_layers": draft_layers, "draft_heads": s.draft.num_q_heads,
        "estimation_us_per_step": round(est_us, 1),
        f"step_us_L{len(layers)}": round(step_us, 1),
        "per_step_speedup_L80": round(80 * dense_us / (est_us + 80 * sparse_us), 3),
        "dustin_per_step_speedup_L80": round(80 * dense_us / (dustin_est_us + 80 * sparse_us), 3),
    }
    log(f"[bench] per-layer all-draft-head selection ({draft_layers} draft layers x "
        f"{s.draft.num_q_heads} heads): estimation {est_us:.0f} us/step, step over {len(layers)} layers "
        f"{step_us:.0f} us; per-step speedup at L=80 {rec['per_step_speedup_L80']}x vs Dustin "
        f"{rec['dustin_per_step_speedup_L80']}x")
    del st, est24
    return rec


# ----------------------------------------------------------------------------- CPU baseline

def cpu_baseline(s, layer0, est, n_seq):
    """The oracle as it stands, on the host cores, for the first n_seq sequences of the same
    synthetic batch: target + draft scoring, selection, one sparse layer, one dense layer;
    times scaled to the whole batch."""
    import numpy as np
    import oracle as O
    from paper_2606_24957_amd.workloads import bf16_bits

    nb = min(n_seq, s.B)
    sl = slice(0, nb)
    seq = list(s.seq_lens[:nb])
    nq = list(s.n_query[:nb])
    scale = 1.0 / (s.head_dim ** 0.5)
    kk, vv = layer0.contiguous_kv(s)
    q = bf16_bits(layer0.q[sl])
    k = bf16_bits(kk[sl])
    v = bf16_bits(vv[sl])
    times = {}
    t0 = time.perf_counter()
    init = None if est.init_target is None else np.ascontiguousarray(
        np.broadcast_to(est.init_target[sl].cpu().numpy(), (nb, s.groups, s.n_max)))
    st = O.score(bf16_bits(est.q_target[sl]), k, seq, [1] * nb, s.target_heads, scale,
                 num_kv_heads=s.num_kv_heads, groups=s.groups, init=init)
    times["score_target"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    if est.s_draft_given is not None:
        sd = est.s_draft_given[sl].cpu().numpy()
    else:
        sd = None
        dscale = 1.0 / (s.draft.head_dim ** 0.5)
        for l in range(s.draft.layers):
            sd = O.score(bf16_bits(est.draft_q[l][sl]), bf16_bits(est.draft_k[l][sl]), seq,
                         [t - 1 for t in nq], s.draft.heads, dscale, init=sd)
    times["score_draft"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    idx, cnt = O.select(sd, st, seq, s.k_max, budget=s.budget[:nb], m=s.m[:nb], groups=s.groups)
    times["select"] = time.perf_counter() - t0
    rows = O.all_rows(nb, nq, s.num_q_heads)
    t0 = time.perf_counter()
    O.attention(q, k, v, seq, scale, rows, idx=idx, count=cnt)
    times["sparse_layer"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    O.attention(q, k, v, seq, scale, rows)
    times["dense_layer"] = time.perf_counter() - t0
    f = s.B / nb
    us = {key: val * f * 1e6 for key, val in times.items()}
    # one thread, one sequence: the sparse layer and the scores of sequence 0
    threads = O.max_threads()
    O.set_threads(1)
    try:
        s0 = slice(0, 1)
        t0 = time.perf_counter()
        O.attention(q[s0], k[s0], v[s0], seq[:1], scale, O.all_rows(1, nq[:1], s.num_q_heads),
                    idx=idx[s0], count=cnt[s0])
        one_sparse = (time.perf_counter() - t0) * s.B * 1e6
        t0 = time.perf_counter()
        O.score(bf16_bits(est.q_target[s0]), k[s0], seq[:1], [1], s.target_heads, scale,
                num_kv_heads=s.num_kv_heads, groups=s.groups,
                init=None if init is None else init[s0])
        one_score = (time.perf_counter() - t0) * s.B * 1e6
    finally:
        O.set_threads(threads)
    return {
        "value": round(us["sparse_layer"], 1),
        "unit": "us/layer",
        "cores": O.max_threads(),
        "kind": "oracle",
        "sample": (f"sequences 0..{nb - 1} of {s.B} of layer 0 (same synthetic bytes), full "
                   f"oracle step: target+draft scoring, selection, one sparse and one dense "
                   f"layer; times scaled x{f:g} to the batch"),
        "dense_us_per_layer": round(us["dense_layer"], 1),
        "estimation_us_per_step": round(us["score_target"] + us["score_draft"] + us["select"], 1),
        "one_thread": {"sparse_us_per_layer": round(one_sparse, 1), "target_score_us": round(one_score, 1),
                       "sample": f"sequence 0 on one thread, times scaled x{s.B} to the batch"},
        "wall_s": round(sum(times.values()), 2),
    }


# ----------------------------------------------------------------------------- other workloads

SECONDARY = (("qwen72b", 512), ("ragged", None), ("long131k", None))


def secondary(name, k, steps, warmup, dev):
    """One more workload through the same timed step as the main workload (estimation, then its L
    sparse and L dense layers back to back): per-layer and per-step figures."""
    import torch
    from paper_2606_24957_amd import workloads as W
    s = W.config(name)
    if k is not None:
        s = s.replace(budget=(k,) * s.B, m=((k - s.n_sink - s.n_window) // 2,) * s.B)
    t0 = time.perf_counter()
    layers = [W.make_layer(s, l, dev) for l in range(s.layers)]
    est = W.make_estimation(s, layers[0], dev)
    torch.cuda.synchronize()
    gen_s = time.perf_counter() - t0
    T = StepTimer(s, layers, est, dev)
    r = T.run(steps, warmup)
    L = s.layers
    sp_us, dn_us = mean(r["sp"]) * 1e3, mean(r["dn"]) * 1e3
    est_s, est_k = (mean(r[x]) * 1e3 for x in ("est_s", "est_k"))
    est_t, est_d = (x * 1e3 for x in T.score_parts(5))
    est_us = est_s + est_k
    sb, db = sparse_bytes(s), dense_bytes(s)
    eb = score_bytes(s, True) + score_bytes(s, False) + topk_bytes(s)
    rec = {
        "config": {"batch": s.B, "context": list(s.seq_lens) if len(set(s.seq_lens)) > 1 else s.n_max,
                   "verify_queries": list(s.n_query) if len(set(s.n_query)) > 1 else s.t_max,
                   "budget_k": list(s.budget) if len(set(s.budget)) > 1 else s.k_max,
                   "stacked_layers": L, "paged": bool(s.page_size)},
        "sparse_us_per_layer": round(sp_us, 3), "sparse_GBps": round(sb / (sp_us * 1e-6) / 1e9, 1),
        "sparse_frac": round(sb / (sp_us * 1e-6) / 1e9 / PEAK_HBM_GBPS, 4), "sparse_bytes": sb,
        "dense_us_per_layer": round(dn_us, 3), "dense_GBps": round(db / (dn_us * 1e-6) / 1e9, 1),
        "dense_bytes": db,
        "estimation_us_per_step": round(est_us, 3), "scores_one_launch_us": round(est_s, 3),
        "target_score_us": round(est_t, 3), "draft_score_us": round(est_d, 3), "topk_us": round(est_k, 3),
        "estimation_GBps": round(eb / (est_us * 1e-6) / 1e9, 1),
        "speedup": {"per_layer": round(dn_us / sp_us, 3),
                    f"per_step_L{L}": round(L * dn_us / (est_us + L * sp_us), 3),
                    "per_step_L80": round(80 * dn_us / (est_us + 80 * sp_us), 3)},
        "steps": steps, "warmup": warmup,
    }
    tag = name + ("" if k is None else f"_k{k}")
    log(f"[bench] {tag}: sparse {sp_us:.2f} us/layer ({rec['sparse_GBps']} GB/s), dense {dn_us:.1f} us/layer, "
        f"estimation {est_us:.1f} us/step (scores in one launch {est_s:.1f}; alone target {est_t:.1f}, "
        f"draft {est_d:.1f}; topk {est_k:.1f}); "
        f"speedup per layer {rec['speedup']['per_layer']}x, per step L={L} {rec['speedup'][f'per_step_L{L}']}x, "
        f"L=80 {rec['speedup']['per_step_L80']}x (inputs {gen_s:.1f}s)")
    del T, layers, est
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return tag, rec


# ----------------------------------------------------------------------------- main

def main():
    args = parse()
    if args.gpus != 1:
        log(f"bench.py measures one GPU only (asked for --gpus {args.gpus}): the path would shard by "
            "sequence or by KV head, with no exchange inside a layer, and that is not built here")
        sys.exit(2)
    import torch
    import paper_2606_24957_amd as D
    from paper_2606_24957_amd import workloads as W

    if not torch.cuda.is_available():
        log("no GPU visible: bench.py needs an MI355X")
        sys.exit(3)
    D.lib()  # fails loudly when libdustin.so is missing
    dev = "cuda"
    s = W.config(args.workload)
    if args.k is not None:
        s = s.replace(budget=(args.k,) * s.B, m=((args.k - s.n_sink - s.n_window) // 2,) * s.B)
    if args.layers is not None:
        s = s.replace(layers=args.layers)
    if args.groups == "hkv":
        s = W.per_kv_head(s)
    L = s.layers
    log(f"[bench] workload {s.name}: B={s.B} N={s.n_max} Hq={s.num_q_heads} Hkv={s.num_kv_heads} "
        f"T={s.t_max} k={s.k_max} layers={L} paged={bool(s.page_size)}")
    t0 = time.perf_counter()
    layers = [W.make_layer(s, l, dev) for l in range(L)]
    est = W.make_estimation(s, layers[0], dev)
    torch.cuda.synchronize()
    log(f"[bench] inputs generated in {time.perf_counter() - t0:.1f}s")

    T = StepTimer(s, layers, est, dev, digit_hist=not args.no_digit_hist)
    seq, nq, bud, mm = T.seq, T.nq, T.bud, T.mm
    s_t, s_d, idx, cnt = T.s_t, T.s_d, T.idx, T.cnt
    r = T.run(args.steps, args.warmup, args.only, copy_probe=args.copy_probe)
    est_s, est_k, sp, dn = r["est_s"], r["est_k"], r["sp"], r["dn"]
    est_t, est_d = T.score_parts(10) if args.only in ("all", "estimate", "sparse") else (float("nan"),) * 2
    ms_per_step = r["ms_per_step"]
    # the same sparse launches with an event between each (for comparison only)
    sp_ev = T.sparse_with_events(max(1, args.steps // 3)) if args.only in ("all", "sparse") else []
    sp_us, dn_us = mean(sp) * 1e3, mean(dn) * 1e3
    est_us = (mean(est_s) + mean(est_k)) * 1e3
    sb, db = sparse_bytes(s), dense_bytes(s)
    est_sd_given = est.s_draft_given is not None
    eb = score_bytes(s, True) + (0 if est_sd_given else score_bytes(s, False)) + topk_bytes(s)
    achieved = sb / (sp_us * 1e-6) / 1e9 if sp else float("nan")
    dense_gbps = db / (dn_us * 1e-6) / 1e9 if dn else float("nan")
    log(f"[bench] sparse {sp_us:.2f} us/layer (median {med(sp) * 1e3:.2f}; with an event between launches "
        f"{mean(sp_ev) * 1e3:.2f}) = {achieved:.0f} GB/s on "
        f"{sb / 1e6:.1f} MB; dense {dn_us:.1f} us/layer = {dense_gbps:.0f} GB/s; estimation "
        f"{est_us:.1f} us/step (scores in one launch {mean(est_s) * 1e3:.1f}; alone target {est_t * 1e3:.1f}, "
        f"draft {est_d * 1e3:.1f}; topk {mean(est_k) * 1e3:.1f}); {ms_per_step:.3f} ms/step wall")

    # the whole step (estimation, then per layer the window append and the sparse attention)
    # enqueued eagerly and replayed as one HIP graph, timed over K steps without events
    # between launches
    vstep = None
    if args.only == "all":
        from paper_2606_24957_amd import step as S
        try:
            st = S.VerifyStep(s, layers, est, dev)
            st.run()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(args.steps):
                st.run()
            e1.record()
            torch.cuda.synchronize()
            eager_us = e0.elapsed_time(e1) * 1e3 / args.steps
            st.capture()
            for _ in range(args.warmup):
                st.replay()
            torch.cuda.synchronize()
            e0.record()
            for _ in range(args.steps):
                st.replay()
            e1.record()
            torch.cuda.synchronize()
            graph_us = e0.elapsed_time(e1) * 1e3 / args.steps
            vstep = {"layers": L, "launches": len(st.ops), "eager_us": round(eager_us, 2),
                     "graph_us": round(graph_us, 2)}
            log(f"[bench] verify step ({len(st.ops)} launches): eager {eager_us:.1f} us, "
                f"graph {graph_us:.1f} us")
            del st
        except Exception as exc:  # reported, not fatal: the per-layer figures stand
            vstep = {"error": str(exc)[:200]}
            log(f"[bench] verify step graph: {exc}")

    per_layer = None
    if args.only == "all" and s.draft is not None and s.groups == 1:
        try:
            per_layer = per_layer_selection(s, layers, dev, args.steps, args.warmup, sp_us, dn_us, est_us)
        except Exception as exc:  # reported, not fatal
            per_layer = {"error": str(exc)[:200]}
            log(f"[bench] per-layer selection: {exc}")

    fidelity = None
    if args.only == "all":
        fidelity = arr_eval(s, layers[0], s_t, s_d, idx, cnt, seq, nq, bud, mm)

    page = None
    if args.only in ("all", "page"):
        page = page_estimator(s, layers, est, seq, nq, bud, args.steps, args.warmup)
        if est_us == est_us:
            page["dustin_estimation_us_per_step"] = round(est_us, 1)
            page["quest16_over_dustin_L80"] = round(page["quest16_estimation_us_per_step_L80"] / est_us, 2)

    cpu = None
    if not args.no_cpu_baseline and args.only == "all":
        log("[bench] timing the oracle on the host cores ...")
        cpu = cpu_baseline(s, layers[0], est, args.cpu_sample_seqs)
        log(f"[bench] oracle: {cpu}")

    # context for the roofline: what a plain 1 GiB device copy reaches on this machine
    copy_gbps = None
    if args.only == "all":
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        c0.record()
        for _ in range(5):
            dst.copy_(src)
        c1.record()
        torch.cuda.synchronize()
        copy_gbps = round(2 * (1 << 30) * 5 / (c0.elapsed_time(c1) * 1e-3) / 1e9, 1)
        del src, dst
        log(f"[bench] 1 GiB device copy: {copy_gbps} GB/s (read + write)")
    # ... and what a plain streaming read of 2 GiB reaches (the library's read probe), the
    # practical ceiling of the read-only kernels
    read_gbps = None
    if args.only == "all":
        buf = torch.zeros(1 << 31, dtype=torch.uint8, device=dev)
        probe = D.plan_read_probe(buf, blocks=1024)
        probe()
        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        c0.record()
        for _ in range(5):
            probe()
        c1.record()
        torch.cuda.synchronize()
        read_gbps = round((1 << 31) * 5 / (c0.elapsed_time(c1) * 1e-3) / 1e9, 1)
        del buf, probe
        log(f"[bench] 2 GiB streaming read: {read_gbps} GB/s")

    # the other workloads through the same timed step, after the main workload's buffers are gone
    others = None
    if args.only == "all" and not args.no_secondary and args.workload == "qwen72b" and args.k is None \
            and args.layers is None and args.groups == "1":
        del T, layers, est, s_t, s_d, idx, cnt
        D.release_workspaces()
        torch.cuda.empty_cache()
        others = {}
        for name, k in SECONDARY:
            tag, r2 = secondary(name, k, min(args.steps, 10), min(args.warmup, 2), dev)
            others[tag] = r2

    traffic = measured_traffic(s.name, s.k_max)
    sc_bytes = score_bytes(s, True) + (0 if est_sd_given else score_bytes(s, False))
    scores_gbps = round(sc_bytes / (mean(est_s) * 1e-3) / 1e9, 1) if est_s and mean(est_s) > 0 else None
    rec = {
        "metric": "sparse verify-attention us/layer + achieved HBM GB/s, B=16 ctx=32k 72B-shape",
        "value": round(sp_us, 3),
        "unit": "us/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded; Qwen2.5-72B/0.5B-shaped attention, planted salient keys)",
        "config": {
            "workload": s.name, "batch": s.B, "context": s.n_max, "num_q_heads": s.num_q_heads,
            "num_kv_heads": s.num_kv_heads, "head_dim": s.head_dim, "verify_queries": s.t_max,
            "budget_k": s.k_max, "draft_share_m": s.m[0], "sinks": s.n_sink, "window": s.n_window,
            "scoring_heads": list(s.target_heads),
            "draft_scoring": None if s.draft is None else
            {"layers": s.draft.layers, "heads": list(s.draft.heads), "kv_heads": s.draft.num_kv_heads,
             "head_dim": s.draft.head_dim},
            "stacked_layers": L, "paged": bool(s.page_size), "selection_groups": s.groups,
        },
        "achieved_GBps": round(achieved, 1),
        "roofline": {
            "bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBPS, 4), "traffic": traffic,
            "kernel": SPARSE_KERNEL + " (sparse)", "bytes_per_launch": sb,
            "avg_launch_us": round(sp_us, 3),
            "timing": f"events around {L} back-to-back launches per step, divided by {L}",
            "avg_launch_us_with_event_between_launches": round(mean(sp_ev) * 1e3, 3) if sp_ev else None,
            "overfetch": round(traffic / sb, 4) if traffic else None,
            "measured_copy_GBps": copy_gbps,
            "frac_of_measured_copy": round(achieved / copy_gbps, 4) if copy_gbps else None,
            "measured_read_GBps": read_gbps,
            "frac_of_measured_read": round(achieved / read_gbps, 4) if read_gbps else None,
        },
        "dense": {"us_per_layer": round(dn_us, 3), "GBps": round(dense_gbps, 1), "bytes_per_launch": db,
                  "frac": round(dense_gbps / PEAK_HBM_GBPS, 4)},
        "estimation": {"us_per_step": round(est_us, 3), "scores_one_launch_us": round(mean(est_s) * 1e3, 3),
                       "target_score_us": round(est_t * 1e3, 3), "draft_score_us": round(est_d * 1e3, 3),
                       "topk_us": round(mean(est_k) * 1e3, 3),
                       "bytes": eb, "GBps": round(eb / (est_us * 1e-6) / 1e9, 1) if est_us == est_us else None,
                       "scores_GBps": scores_gbps,
                       "scores_frac_of_measured_read": round(scores_gbps / read_gbps, 4)
                       if scores_gbps and read_gbps else None},
        "speedup": {
            "per_layer": round(dn_us / sp_us, 3) if sp else None,
            f"per_step_L{L}": round(L * dn_us / (est_us + L * sp_us), 3) if sp else None,
            "per_step_L80": round(80 * dn_us / (est_us + 80 * sp_us), 3) if sp else None,
        },
        "verify_step": vstep,
        "page_estimator": page,
        "selection_arr": fidelity,
        "per_layer_selection": per_layer,
        "cpu_baseline": cpu,
        "other_workloads": others,
    }
    print(json.dumps(_finite(rec)), flush=True)
    # Release every device buffer while the HIP runtime is whole: the prepared calls, the
    # stacked layers, the cached workspaces, then torch's cached blocks.  (A run under
    # rocprofv3 once died in exit() inside the runtime's teardown, after the profiler had
    # finalised, with all of these still held.)
    if others is None:
        del T, layers, est, s_t, s_d, idx, cnt
    D.release_workspaces()
    import gc
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _finite(x):
    """The record with every non-finite float (a stage left out by --only) as null."""
    if isinstance(x, float):
        return x if x == x and abs(x) != float("inf") else None
    if isinstance(x, dict):
        return {k: _finite(v) for k, v in x.items()}
    if isinstance(x, (list, tuple)):
        return [_finite(v) for v in x]
    return x


if __name__ == "__main__":
    main()
