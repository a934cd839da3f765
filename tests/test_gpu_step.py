"""The whole step on the GPU (scores, tiered top-k, sparse attention: VerifyStep) against the
oracle running the whole step on its own: its fp64 scores, its selection on them, its
attention.  The two index sets may differ only at near ties, positions whose score lies
within the score tolerance of the last score its tier took (fp32 on the GPU, fp64 in the
oracle: a near tie can order either way); the attention rows are checked against the
oracle's attention over the GPU's set."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2606_24957_amd import step as S
from paper_2606_24957_amd import workloads as W
from tests.gpu_util import SCORE_REL, bits, check_attention, gpu_rows, scale_of

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _oracle_tiers(d, t, N, k, m, n_sink, n_window):
    """The oracle's two tiers rebuilt with a library sort: the draft tier is the first m free
    positions by (S_D desc, position asc), the target tier the next k - m - |P| of the rest by
    (S_T desc, position asc)."""
    free = np.arange(n_sink, N - n_window)
    D = free[np.lexsort((free, -d[free]))][:m]
    rest = np.setdiff1d(free, D)
    T = rest[np.lexsort((rest, -t[rest]))][:k - m - n_sink - n_window]
    return D, T


@pytest.mark.parametrize("preset,B,n,k", [("qwen72b", 3, 4096, 384), ("qwen7b", 2, 6000, 512)])
def test_step_end_to_end_matches_the_oracle_up_to_near_ties(preset, B, n, k):
    s = W.shrink(W.config(preset), B=B, n=n, k=k, layers=1)
    L = W.make_layer(s, 0, DEV)
    est = W.make_estimation(s, L, DEV)
    st = S.VerifyStep(s, [L], est, DEV, append=False)
    st.run()
    torch.cuda.synchronize()
    seq = list(s.seq_lens)
    kk, vv = L.contiguous_kv(s)
    qb, kb, vb = bits(L.q), bits(kk), bits(vv)

    # the oracle's own step
    init = None if est.init_target is None else est.init_target.cpu().numpy()
    ref_t = O.score(bits(est.q_target), kb, seq, [1] * s.B, s.target_heads, scale_of(s.head_dim), init=init)
    ref_d = None
    dscale = scale_of(s.draft.head_dim)
    for l in range(s.draft.layers):
        ref_d = O.score(bits(est.draft_q[l]), bits(est.draft_k[l]), seq, list(s.draft_gamma), s.draft.heads,
                        dscale, init=ref_d)
    ri, rc = O.select(ref_d, ref_t, seq, s.k_max, budget=s.budget, m=s.m)

    gi, gc = st.idx.cpu().numpy(), st.cnt.cpu().numpy()
    for b in range(s.B):
        N = seq[b]
        assert gc[b, 0] == rc[b, 0] == min(s.budget[b], N)
        g_set, r_set = set(gi[b, 0, :gc[b, 0]].tolist()), set(ri[b, 0, :rc[b, 0]].tolist())
        diff = sorted(g_set ^ r_set)
        if not diff:
            continue
        # each differing position lies within twice the score tolerance of the last pick of
        # the draft tier or of the target tier (a swap in the draft tier moves the target
        # tier's boundary pick, which sits at that tier's last score)
        d, t = ref_d[b, 0].astype(np.float64), ref_t[b, 0].astype(np.float64)
        D, T = _oracle_tiers(d, t, N, s.budget[b], s.m[b], s.n_sink, s.n_window)
        assert set(D.tolist()) | set(T.tolist()) <= r_set
        tau_d = d[D].min() if len(D) else np.inf
        tau_t = t[T].min() if len(T) else np.inf
        for x in diff:
            near_d = abs(d[x] - tau_d) <= 2 * SCORE_REL * max(abs(tau_d), 1.0 / N)
            near_t = abs(t[x] - tau_t) <= 2 * SCORE_REL * max(abs(tau_t), 1.0 / N)
            assert near_d or near_t, f"b={b}: position {x} differs but is no near tie"
        assert len(diff) <= 8, f"b={b}: {len(diff)} positions differ"

    # attention rows against the oracle over the GPU's own set
    rows = O.all_rows(s.B, s.n_query, s.num_q_heads)[::7]
    ref = O.attention(qb, kb, vb, seq, scale_of(s.head_dim), rows, idx=gi, count=gc)
    check_attention(gpu_rows(st.outs[0], rows), ref, f"{preset} step")
