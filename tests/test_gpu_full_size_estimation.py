"""Estimation at full size on the ragged paged batch and on the 131k stress layer, against
the oracle: the step's target score (Eq. 5 over the scoring heads, on the paged cache, with
the handed-in historical score for the 131k layer) and its draft score (three draft layers,
per-sequence Gamma_b) on sampled sequences, within 1e-4 * max(|S_ref|, 1/N_b); the tiered
top-k (Eq. 6, one set per sequence) on the GPU's own scores bit-exact against the oracle's
selection for every sequence; and sampled attention rows over the step's set."""
import os

import numpy as np
import pytest
import torch

import oracle as O
from paper_2606_24957_amd import step as S
from paper_2606_24957_amd import workloads as W
from tests.gpu_util import bits, check_attention, check_score, gpu_rows, scale_of

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _run(preset, sample):
    s = W.config(preset).replace(layers=1)
    L = W.make_layer(s, 0, DEV)
    est = W.make_estimation(s, L, DEV)
    st = S.VerifyStep(s, [L], est, DEV, append=False)
    st.run()
    torch.cuda.synchronize()
    seq = list(s.seq_lens)
    s_t, s_d = st.s_t.cpu().numpy(), st.s_d.cpu().numpy()
    gi, gc = st.idx.cpu().numpy(), st.cnt.cpu().numpy()

    # Eq. 6 on the GPU's scores, every sequence, bit for bit
    ri, rc = O.select(s_d, s_t, seq, s.k_max, budget=s.budget, m=s.m)
    np.testing.assert_array_equal(gc, rc)
    for b in range(s.B):
        np.testing.assert_array_equal(gi[b, 0, :rc[b, 0]], ri[b, 0, :rc[b, 0]], err_msg=f"{preset} b={b}")
        assert rc[b, 0] == min(s.budget[b], seq[b])

    kk, vv = L.contiguous_kv(s)
    init = None if est.init_target is None else est.init_target.cpu().numpy()
    for b in sample:
        n = seq[b]
        ref_t = O.score(bits(est.q_target[b:b + 1]), bits(kk[b:b + 1, :n]), [n], [1], s.target_heads,
                        scale_of(s.head_dim), num_kv_heads=s.num_kv_heads,
                        init=None if init is None else np.ascontiguousarray(init[b:b + 1, :, :n]))
        check_score(s_t[b, 0, :n], ref_t[0, 0, :n], n, f"{preset} S_T b={b}")
        ref_d = None
        for l in range(s.draft.layers):
            ref_d = O.score(bits(est.draft_q[l][b:b + 1]), bits(est.draft_k[l][b:b + 1, :n]), [n],
                            [s.draft_gamma[b]], s.draft.heads, scale_of(s.draft.head_dim),
                            num_kv_heads=s.draft.num_kv_heads, init=ref_d)
        check_score(s_d[b, 0, :n], ref_d[0, 0, :n], n, f"{preset} S_D b={b} (Gamma_b={s.draft_gamma[b]})")
        # sampled attention rows of this sequence over the step's set
        rng = np.random.default_rng(b)
        rows = np.asarray([(0, int(rng.integers(s.n_query[b])), int(rng.integers(s.num_q_heads)))
                           for _ in range(6)] + [(0, s.n_query[b] - 1, s.num_q_heads - 1)], dtype=np.int32)
        ref = O.attention(bits(L.q[b:b + 1]), bits(kk[b:b + 1]), bits(vv[b:b + 1]), [n], scale_of(s.head_dim),
                          rows, idx=gi[b:b + 1], count=gc[b:b + 1])
        got = rows.copy()
        got[:, 0] = b
        check_attention(gpu_rows(st.outs[0], got), ref, f"{preset} attention b={b}")


def test_full_size_ragged_paged_estimation():
    """B = 16, N_b from 4096 to 65536, paged by 16, per-sequence gamma_b, k_b and m_b."""
    s = W.config("ragged")
    order = np.argsort(s.seq_lens)
    _run("ragged", [int(order[0]), int(order[len(order) // 2]), int(order[-1])])


@pytest.mark.skipif(os.environ.get("DUSTIN_SKIP_131K") == "1", reason="131k layer skipped by request")
def test_full_size_131k_estimation():
    """B = 8, N = 131072, Gamma = 6, k = 4096, heavy-tailed historical score."""
    _run("long131k", [0, 7])
