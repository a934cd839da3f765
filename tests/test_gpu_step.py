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
from tests.gpu_util import SCORE_REL, bits, check_attention, check_score, gpu_rows, scale_of

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


def _fresh_windows(s, n_layers, seed):
    """Window K/V rows per layer, drawn independently of the caches (so that the append
    inside the step writes values the caches did not hold)."""
    g = torch.Generator(device=DEV).manual_seed(seed)
    shape = (s.B, s.t_max, s.num_kv_heads, s.head_dim)
    return [(torch.randn(shape, generator=g, device=DEV, dtype=torch.bfloat16),
             torch.randn(shape, generator=g, device=DEV, dtype=torch.bfloat16)) for _ in range(n_layers)]


def _ragged_small():
    base = W.config("ragged")
    n, t = (3000, 1234, 5000), (3, 9, 6)
    k = tuple(max(64, x // 16) for x in n)
    return base.replace(name="ragged_small", B=3, seq_lens=n, n_query=t, budget=k,
                        m=tuple((x - 20) // 2 for x in k), planted=tuple(round(0.01 * x) for x in n), layers=3)


@pytest.mark.parametrize("preset", ["qwen72b", "ragged"])
def test_multi_layer_step_reuses_one_index_set_with_fresh_window_rows(preset):
    """Three stacked target layers in one VerifyStep (Sec. 4.1: one selection per step,
    reused by every layer): the scores against the oracle's, the index set bit-exact against
    the oracle's Eq. 6 on the GPU's scores, the caches after the in-step append equal to the
    oracle's append of the fresh window rows, and every layer's attention rows against the
    oracle over that single set and the appended rows."""
    s = W.shrink(W.config("qwen72b"), B=3, n=4000, k=384, layers=3) if preset == "qwen72b" else _ragged_small()
    layers = [W.make_layer(s, l, DEV) for l in range(s.layers)]
    est = W.make_estimation(s, layers[0], DEV)
    windows = _fresh_windows(s, s.layers, 77)
    seq = list(s.seq_lens)
    # host copies of the caches before the step (the oracle's inputs)
    before = []
    for L in layers:
        before.append((bits(L.k), bits(L.v)))
    st = S.VerifyStep(s, layers, est, DEV, windows=windows, append=True)
    st.run()
    torch.cuda.synchronize()

    # scores and the one selection
    k0, _ = layers[0].contiguous_kv(s)
    init = None if est.init_target is None else est.init_target.cpu().numpy()
    ref_t = O.score(bits(est.q_target), bits(k0), seq, [1] * s.B, s.target_heads, scale_of(s.head_dim), init=init)
    ref_d = None
    for l in range(s.draft.layers):
        ref_d = O.score(bits(est.draft_q[l]), bits(est.draft_k[l]), seq, list(s.draft_gamma), s.draft.heads,
                        scale_of(s.draft.head_dim), init=ref_d)
    s_t, s_d = st.s_t.cpu().numpy(), st.s_d.cpu().numpy()
    for b, n in enumerate(seq):
        check_score(s_t[b, 0, :n], ref_t[b, 0, :n], n, f"S_T b={b}")
        check_score(s_d[b, 0, :n], ref_d[b, 0, :n], n, f"S_D b={b}")
    ri, rc = O.select(s_d, s_t, seq, s.k_max, budget=s.budget, m=s.m)
    gi, gc = st.idx.cpu().numpy(), st.cnt.cpu().numpy()
    np.testing.assert_array_equal(gc, rc)
    for b in range(s.B):
        np.testing.assert_array_equal(gi[b, 0, :rc[b, 0]], ri[b, 0, :rc[b, 0]], err_msg=f"b={b}")

    rows = O.all_rows(s.B, s.n_query, s.num_q_heads)
    for l, (L, (kb, vb), (k_new, v_new)) in enumerate(zip(layers, before, windows)):
        pt = None if L.page_table is None else L.page_table.cpu().numpy()
        k_ref = O.kv_append(kb, bits(k_new), seq, s.n_query, page_table=pt)
        v_ref = O.kv_append(vb, bits(v_new), seq, s.n_query, page_table=pt)
        # the window rows really changed, and the step's append wrote exactly them
        for b in range(s.B):
            n, t = seq[b], s.n_query[b]
            assert not np.array_equal(bits(k_new[b, :t]), _logical_rows(kb, pt, s, b, n, t))
        np.testing.assert_array_equal(bits(L.k), k_ref, err_msg=f"layer {l} K after append")
        np.testing.assert_array_equal(bits(L.v), v_ref, err_msg=f"layer {l} V after append")
        kc = _contiguous(k_ref, pt, s)
        vc = _contiguous(v_ref, pt, s)
        ref = O.attention(bits(L.q), kc, vc, seq, scale_of(s.head_dim), rows, idx=ri, count=rc)
        check_attention(gpu_rows(st.outs[l], rows), ref, f"{preset} layer {l}")


def _contiguous(cache, pt, s):
    """[B, N_cap, Hkv, d] host view of a (possibly paged) host cache: input plumbing only."""
    if pt is None:
        return cache
    ps = s.page_size
    n_pages = (s.n_cap + ps - 1) // ps
    return cache[pt[:, :n_pages]].reshape(s.B, n_pages * ps, s.num_kv_heads, s.head_dim)


def _logical_rows(cache, pt, s, b, n, t):
    return _contiguous(cache, pt, s)[b, n:n + t]
