"""GPU windowed attention recovery rate (Eqs. 1-4) against the oracle, which computes it
from the attention rows step by step: dustin_score over every head and the window's
queries, then dustin_arr over index sets (Dustin's selection, the SD oracle's TopK of A-bar,
the full set).  Tolerance: 2e-4 absolute on an ARR in [0, 1] (fp32 scores summed in fp64)."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_24957_amd as D
from paper_2606_24957_amd import workloads as W
from tests.gpu_util import bits, host, scale_of

pytestmark = pytest.mark.gpu
DEV = "cuda"
ARR_ABS = 2e-4


def _window_scores(q, k, seq, win, groups, max_len):
    Hq = q.shape[2]
    return D.score(q, k, torch.tensor(seq, dtype=torch.int32, device=DEV), list(range(Hq)),
                   n_query=torch.tensor(win, dtype=torch.int32, device=DEV), groups=groups, max_len=max_len)


@pytest.mark.parametrize("groups", [1, 2])
def test_arr_of_selections_and_sd_oracle(groups):
    B, Hq, Hkv, d = 2, 8, 2, 128
    seq, win, kb = [3000, 1200], [5, 3], 256
    N = max(seq)
    g = torch.Generator(device=DEV).manual_seed(21)
    q = torch.randn((B, max(win), Hq, d), generator=g, device=DEV).to(torch.bfloat16)
    k = torch.randn((B, N + 8, Hkv, d), generator=g, device=DEV).to(torch.bfloat16)
    for p in (17, 500, 1100):                        # positions the window attends strongly
        k[:, p] = (2.0 * q[:, 0, ::Hq // Hkv]).to(torch.bfloat16)
    s = _window_scores(q, k, seq, win, groups, N)
    seq_t = torch.tensor(seq, dtype=torch.int32, device=DEV)
    hpg = Hq // groups
    # Dustin-style set: sinks, window and the top of a noisy copy of the score
    noisy = s + torch.rand(s.shape, generator=g, device=DEV) * s.mean()
    idx, cnt = D.topk(None, noisy, seq_t, kb, groups=groups, m_scalar=0)
    got = host(D.arr(s, idx, cnt, seq_t, hpg, window=win))
    # SD oracle: TopK_k of A-bar, no protected positions
    oidx, ocnt = D.topk(None, s, seq_t, kb, groups=groups, n_sink=0, n_window=0, m_scalar=0)
    got_orc = host(D.arr(s, oidx, ocnt, seq_t, hpg, window=win))
    # the full set
    fidx, fcnt = D.topk(None, s, seq_t, N, groups=groups, n_sink=0, n_window=0, m_scalar=0)
    got_full = host(D.arr(s, fidx, fcnt, seq_t, hpg, window=win))
    torch.cuda.synchronize()
    qb, kbits = bits(q), bits(k[:, :N])
    ref = O.arr(qb, kbits, seq, win, scale_of(d), groups=groups, idx=host(idx), count=host(cnt))
    ref_orc, abar = O.arr(qb, kbits, seq, win, scale_of(d), groups=groups, idx=host(oidx), count=host(ocnt),
                          with_abar=True, length=N)
    np.testing.assert_allclose(got, ref, atol=ARR_ABS)
    np.testing.assert_allclose(got_orc, ref_orc, atol=ARR_ABS)
    np.testing.assert_allclose(got_full, 1.0, atol=ARR_ABS)
    for b, n in enumerate(seq):
        for go in range(groups):
            best = np.sort(abar[b, go, :n])[::-1][:kb].sum()          # Eq. 4 on the oracle's A-bar
            assert ref_orc[b, go] == pytest.approx(best, abs=ARR_ABS)
            assert got_orc[b, go] >= got[b, go] - 1e-12                # the oracle bounds any k-set
    # deterministic: the same call gives the same bits
    again = host(D.arr(s, idx, cnt, seq_t, hpg, window=win))
    assert np.array_equal(again, got)


def test_arr_full_size_qwen72b():
    """B = 16, N = 32768: A-bar from all 64 heads and 5 verification queries, ARR of the
    method's selection (target scoring heads, draft scoring, tiered top-k) and of the SD
    oracle; the oracle recomputes sequences 0 and 9 from Q and K."""
    s = W.config("qwen72b").replace(layers=1)
    L = W.make_layer(s, 0, DEV)
    E = W.make_estimation(s, L, DEV)
    seq = torch.tensor(s.seq_lens, dtype=torch.int32, device=DEV)
    nq = torch.tensor(s.n_query, dtype=torch.int32, device=DEV)
    st = D.score(E.q_target, L.k, seq, s.target_heads, init=E.init_target, max_len=s.n_max)
    sd = D.score_layers(E.draft_q, E.draft_k, seq, s.draft.heads,
                        n_query=torch.tensor(s.draft_gamma, dtype=torch.int32, device=DEV), max_len=s.n_max)
    idx, cnt = D.topk(sd, st, seq, s.k_max, m=torch.tensor(s.m, dtype=torch.int32, device=DEV),
                      n_sink=s.n_sink, n_window=s.n_window)
    a = D.score(L.q, L.k, seq, list(range(s.num_q_heads)), n_query=nq, max_len=s.n_max)
    got = host(D.arr(a, idx, cnt, seq, s.num_q_heads, window=nq))
    oidx, ocnt = D.topk(None, a, seq, s.k_max, n_sink=0, n_window=0, m_scalar=0)
    got_orc = host(D.arr(a, oidx, ocnt, seq, s.num_q_heads, window=nq))
    torch.cuda.synchronize()
    assert np.all(got_orc >= got - 1e-12) and np.all(got > 0) and np.all(got_orc <= 1 + ARR_ABS)
    sel = [0, 9]                                         # one oracle call per set, two sequences
    n = max(s.seq_lens[b] for b in sel)
    qb, kb = bits(L.q[sel]), bits(L.k[sel, :n])
    lens, wins = [s.seq_lens[b] for b in sel], [s.n_query[b] for b in sel]
    ref = O.arr(qb, kb, lens, wins, scale_of(128), idx=host(idx)[sel], count=host(cnt)[sel])
    np.testing.assert_allclose(got[sel], ref, atol=ARR_ABS)
    ref_o = O.arr(qb, kb, lens, wins, scale_of(128), idx=host(oidx)[sel], count=host(ocnt)[sel])
    np.testing.assert_allclose(got_orc[sel], ref_o, atol=ARR_ABS)


def test_arr_degenerate_lengths():
    """ARR of an empty sequence is 0, of a one-position sequence with that position is 1."""
    B, Hq, Hkv, d = 3, 4, 1, 128
    seq = [0, 1, 300]
    g = torch.Generator(device=DEV).manual_seed(10)
    q = torch.randn((B, 3, Hq, d), generator=g, device=DEV).to(torch.bfloat16)
    k = torch.randn((B, 320, Hkv, d), generator=g, device=DEV).to(torch.bfloat16)
    seq_t = torch.tensor(seq, dtype=torch.int32, device=DEV)
    s = D.score(q, k, seq_t, list(range(Hq)), n_query=torch.tensor([3, 3, 3], dtype=torch.int32, device=DEV),
                max_len=320)
    s[0].fill_(7.0)                                                # never read: N_0 = 0
    idx, cnt = D.topk(None, s, seq_t, 64, n_sink=0, n_window=0, m_scalar=0)
    a = host(D.arr(s, idx, cnt, seq_t, Hq, window=3))
    torch.cuda.synchronize()
    assert a[0, 0] == 0.0 and abs(a[1, 0] - 1.0) < 2e-4 and 0.0 < a[2, 0] < 1.0
    ref = O.arr(bits(q), bits(k[:, :300]), seq, [3, 3, 3], scale_of(d), idx=host(idx), count=host(cnt))
    np.testing.assert_allclose(a, ref, atol=2e-4)
