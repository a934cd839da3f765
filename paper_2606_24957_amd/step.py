"""One verification step of long-context speculative decoding on the GPU, planned once and
replayed: the target scoring-head score, the draft scores (accumulated over the draft
layers), the tiered top-k, and for every target layer the window's K/V append followed by
the sparse verification attention with the one index set (Sec. 3.2: a global, layer-invariant
selection; accepted tokens are appended to the cache).  Every launch is a prepared libdustin
call on one stream, so the whole step can be captured in a HIP graph and replayed.
"""
from typing import List, Optional

import torch

from . import (digit_hist, plan_kv_append, plan_kv_commit, plan_score, plan_score_calls, plan_score_layers,
               plan_score_per_layer, plan_sparse_verify_attn, plan_topk)


def window_kv(s, layer) -> tuple:
    """K and V of the verification window, [B, T_max, Hkv, d] each: the rows the layer's cache
    holds at [N_b, N_b + T_b) (what the target model's projections of the window tokens give)."""
    kk, vv = layer.contiguous_kv(s)
    B, T = s.B, s.t_max
    k_new = torch.zeros((B, T, s.num_kv_heads, s.head_dim), dtype=torch.bfloat16, device=kk.device)
    v_new = torch.zeros_like(k_new)
    for b in range(B):
        n, t = s.seq_lens[b], s.n_query[b]
        k_new[b, :t] = kk[b, n:n + t]
        v_new[b, :t] = vv[b, n:n + t]
    return k_new, v_new


class VerifyStep:
    """The step's launches over fixed buffers: run() enqueues them eagerly, capture() records
    them in a HIP graph and replay() launches the graph."""

    def __init__(self, s, layers, est, device, windows: Optional[list] = None, append: bool = True):
        self.s, self.layers, self.est, self.append = s, layers, est, append
        i32 = lambda x: torch.tensor(list(x), dtype=torch.int32, device=device)
        self.seq, self.nq, self.gam = i32(s.seq_lens), i32(s.n_query), i32(s.draft_gamma)
        self.bud, self.mm = i32(s.budget), i32(s.m)
        N = s.n_max
        self.s_t = torch.zeros((s.B, s.groups, N), dtype=torch.float32, device=device)
        self.s_d = torch.zeros((s.B, 1, N), dtype=torch.float32, device=device)
        self.idx = torch.zeros((s.B, s.groups, s.k_max), dtype=torch.int32, device=device)
        self.cnt = torch.zeros((s.B, s.groups), dtype=torch.int32, device=device)
        self.outs = [torch.empty_like(l.q) for l in layers]
        self.windows = windows if windows is not None else [window_kv(s, l) for l in layers]
        # with one selection group, the score calls count their outputs by top key digit and
        # the top-k takes those counts in place of its first pass over each row
        self.hist_t = digit_hist(s.B, device) if s.groups == 1 else None
        self.hist_d = digit_hist(s.B, device) if s.groups == 1 and est.s_draft_given is None else None
        self.graph = None
        self.ops = self._plan()

    def _plan(self, stream=None) -> List:
        """The step's operations, bound to `stream` (None: the current stream)."""
        s, est, N = self.s, self.est, self.s.n_max
        init = est.init_target
        if init is not None and s.groups > 1:  # one historical row, the same for every group
            init = init.expand(s.B, s.groups, N)
        target = plan_score(est.q_target, self.layers[0].k, self.seq, s.target_heads, groups=s.groups,
                            init=init, out=self.s_t, max_len=N, page_table=self.layers[0].page_table,
                            stream=stream)
        if est.s_draft_given is not None:
            given = est.s_draft_given
            ops = [plan_score_calls([target], stream=stream, digit_hists=[self.hist_t]),
                   lambda: self.s_d.copy_(given)]
        else:
            # the target's and the draft's scores in one call (one launch where the library can)
            draft = plan_score_layers(est.draft_q, est.draft_k, self.seq, s.draft.heads, n_query=self.gam,
                                      out=self.s_d, max_len=N, stream=stream, ws_tag="score_draft")
            ops = [plan_score_calls([target, draft], stream=stream, digit_hists=[self.hist_t, self.hist_d])]
        ops.append(plan_topk(self.s_d, self.s_t, self.seq, s.k_max, budget=self.bud, m=self.mm,
                             n_sink=s.n_sink, n_window=s.n_window, groups=s.groups, idx=self.idx,
                             count=self.cnt, hist_d=self.hist_d, hist_t=self.hist_t, stream=stream))
        for L, o, (k_new, v_new) in zip(self.layers, self.outs, self.windows):
            if self.append:
                ops.append(plan_kv_append(k_new, v_new, L.k, L.v, self.seq, n_query=self.nq,
                                          page_table=L.page_table, max_len=N, stream=stream))
            ops.append(plan_sparse_verify_attn(L.q, L.k, L.v, self.idx, self.cnt, self.seq,
                                               n_query=self.nq, page_table=L.page_table, out=o,
                                               stream=stream))
        return ops

    def run(self):
        for op in self.ops:
            op()

    def capture(self):
        """Records the step in a HIP graph on a capture stream of its own.  The capture
        stream's workspaces are allocated (zeroed) by a planning pass before the capture
        starts, so nothing is allocated or cleared while recording."""
        self.run()
        cs = torch.cuda.Stream()
        self._plan(stream=cs)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cs):
            ops = self._plan(stream=cs)
            for op in ops:
                op()
        self._graph_ops = ops  # keeps the marshalled arguments alive
        self._capture_stream = cs
        self.graph = g
        return g

    def replay(self):
        self.graph.replay()

    def commit(self, accepted: torch.Tensor):
        """After verification: N_b += accepted_b (clamped to [0, T_b])."""
        plan_kv_commit(self.seq, accepted, n_query=self.nq, nq_max=self.s.t_max)()


def draft_layer_of(layer: int, n_target: int, n_draft: int) -> int:
    """The draft layer whose relevance selects the tokens of target layer `layer`: layers
    matched by depth, target layer l to draft layer floor(l * n_draft / n_target)."""
    return min(n_draft - 1, layer * n_draft // n_target)


class PerLayerSelectionStep:
    """The SpecAttn-style step the paper compares with (appendix on SpecAttn): token relevance
    from every head of every draft layer, one index set per draft layer (no aggregation
    across layers), each target layer attending with the set of its depth-matched draft
    layer.  Launches: the per-layer draft scores (two), one top-k over (draft layer, sequence)
    rows, then per target layer the sparse attention.  est holds the draft model's layers
    (draft_q, draft_k); n_target is the target model's depth for the layer matching."""

    def __init__(self, s, layers, est, device, n_target: Optional[int] = None):
        self.s, self.layers, self.est = s, layers, est
        i32 = lambda x: torch.tensor(list(x), dtype=torch.int32, device=device)
        self.seq, self.nq, self.gam = i32(s.seq_lens), i32(s.n_query), i32(s.draft_gamma)
        self.bud = i32(s.budget)
        Ld, B, N = len(est.draft_q), s.B, s.n_max
        self.n_draft = Ld
        self.n_target = len(layers) if n_target is None else n_target
        # selection rows are (draft layer, sequence), layer-major: layer j's sets and counts
        # are the contiguous rows [j B, (j + 1) B)
        self.seq_rows, self.bud_rows = self.seq.repeat(Ld), self.bud.repeat(Ld)
        self.rel = torch.zeros((Ld, B, 1, N), dtype=torch.float32, device=device)
        self.idx = torch.zeros((Ld * B, 1, s.k_max), dtype=torch.int32, device=device)
        self.cnt = torch.zeros((Ld * B, 1), dtype=torch.int32, device=device)
        self.outs = [torch.empty_like(l.q) for l in layers]
        self.ops = self._plan()

    def _plan(self) -> List:
        s, est, N, B = self.s, self.est, self.s.n_max, self.s.B
        heads = list(range(s.draft.num_q_heads))
        ops = [plan_score_per_layer(est.draft_q, est.draft_k, self.seq, heads, n_query=self.gam,
                                    out=self.rel, max_len=N)]
        ops.append(plan_topk(self.rel.view(self.n_draft * B, 1, N), None, self.seq_rows, s.k_max,
                             budget=self.bud_rows, n_sink=s.n_sink, n_window=s.n_window,
                             idx=self.idx, count=self.cnt))
        for i, (L, o) in enumerate(zip(self.layers, self.outs)):
            j = draft_layer_of(i, self.n_target, self.n_draft)
            ops.append(plan_sparse_verify_attn(L.q, L.k, L.v, self.idx[j * B:(j + 1) * B],
                                               self.cnt[j * B:(j + 1) * B], self.seq, n_query=self.nq,
                                               page_table=L.page_table, out=o))
        return ops

    def run(self):
        for op in self.ops:
            op()
