"""GPU parity of the window K/V append and the commit (through the C ABI) against the
oracle, bit for bit; and a HIP-graph capture of a whole verification step replayed
against its eager run."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_24957_amd as D
from paper_2606_24957_amd import step as S
from paper_2606_24957_amd import workloads as W
from tests.gpu_util import bits

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _rand_bf16(shape, seed):
    g = torch.Generator(device=DEV).manual_seed(seed)
    return torch.randn(shape, generator=g, device=DEV, dtype=torch.bfloat16)


@pytest.mark.parametrize("strided", [False, True])
def test_kv_append_contiguous(strided):
    B, cap, H, d, T = 3, 300, 4, 128, 7
    k, v = _rand_bf16((B, cap, H, d), 1), _rand_bf16((B, cap, H, d), 2)
    if strided:  # window rows as a view into a wider projection output
        big = _rand_bf16((B, T, 3 * H, d), 3)
        k_new, v_new = big[:, :, :H], big[:, :, H:2 * H]
    else:
        k_new, v_new = _rand_bf16((B, T, H, d), 4), _rand_bf16((B, T, H, d), 5)
    seq, nq = [100, 0, cap - T], [7, 3, 7]        # the last one ends at the last cache row
    kb, vb = bits(k), bits(v)
    D.kv_append(k_new, v_new, k, v, torch.tensor(seq, dtype=torch.int32, device=DEV),
                n_query=torch.tensor(nq, dtype=torch.int32, device=DEV), max_len=cap - T)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(bits(k), O.kv_append(kb, bits(k_new), seq, nq))
    np.testing.assert_array_equal(bits(v), O.kv_append(vb, bits(v_new), seq, nq))


def test_kv_append_paged():
    B, ps, H, d, T, maxp = 4, 16, 2, 128, 9, 12
    rng = np.random.default_rng(6)
    pt = torch.from_numpy(rng.permutation(B * maxp).astype(np.int32).reshape(B, maxp)).to(DEV)
    k, v = _rand_bf16((B * maxp, ps, H, d), 7), _rand_bf16((B * maxp, ps, H, d), 8)
    k_new, v_new = _rand_bf16((B, T, H, d), 9), _rand_bf16((B, T, H, d), 10)
    seq, nq = [0, 15, 100, 181], [9, 9, 4, 9]
    kb, vb = bits(k), bits(v)
    D.kv_append(k_new, v_new, k, v, torch.tensor(seq, dtype=torch.int32, device=DEV),
                n_query=torch.tensor(nq, dtype=torch.int32, device=DEV), page_table=pt,
                max_len=maxp * ps - T)
    torch.cuda.synchronize()
    ptn = pt.cpu().numpy()
    np.testing.assert_array_equal(bits(k), O.kv_append(kb, bits(k_new), seq, nq, page_table=ptn))
    np.testing.assert_array_equal(bits(v), O.kv_append(vb, bits(v_new), seq, nq, page_table=ptn))


def test_kv_commit():
    seq = torch.tensor([100, 0, 7, 9, 50], dtype=torch.int32, device=DEV)
    acc = torch.tensor([3, -2, 9, 0, 5], dtype=torch.int32, device=DEV)
    nq = torch.tensor([5, 4, 6, 2, 5], dtype=torch.int32, device=DEV)
    want = O.kv_commit(seq.cpu().numpy(), acc.cpu().numpy(), nq.cpu().numpy())
    D.kv_commit(seq, acc, n_query=nq)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(seq.cpu().numpy(), want)


@pytest.mark.parametrize("preset", ["qwen7b", "ragged_small"])
def test_graph_replays_match_the_eager_step(preset):
    """The whole step (scores, top-k, per layer append + sparse attention) captured in one
    graph: every replay gives the eager step's index set and outputs, bit for bit, with
    eager work (clearing the outputs) between the replays."""
    if preset == "ragged_small":
        s = W.config("ragged").replace(B=4, seq_lens=(5000, 9000, 4100, 12000), n_query=(3, 9, 5, 7),
                                       budget=(312, 562, 256, 750), m=(146, 271, 118, 365),
                                       planted=(50, 90, 41, 120), layers=2)
    else:
        s = W.config(preset).replace(layers=2)
    layers = [W.make_layer(s, l, DEV) for l in range(s.layers)]
    est = W.make_estimation(s, layers[0], DEV)
    st = S.VerifyStep(s, layers, est, DEV)
    st.run()
    torch.cuda.synchronize()
    ref = [o.clone() for o in st.outs], st.idx.clone(), st.cnt.clone()
    st.capture()
    for r in range(3):
        for o in st.outs:
            o.fill_(float("nan"))
        st.idx.fill_(-1)
        torch.cuda.synchronize()
        st.replay()
        torch.cuda.synchronize()
        assert torch.equal(st.cnt, ref[2]), f"replay {r}"
        for b in range(s.B):
            c = int(ref[2][b, 0])
            assert torch.equal(st.idx[b, :, :c], ref[1][b, :, :c]), f"replay {r} b={b}"
        for o, oref in zip(st.outs, ref[0]):
            for b, t in enumerate(s.n_query):
                assert torch.equal(o[b, :t].view(torch.int16), oref[b, :t].view(torch.int16)), f"replay {r}"


def test_per_layer_selection_step():
    """The SpecAttn-style step: draft layer j's relevance is dustin_score over all 14 draft
    heads of that layer (bit-identical), its index set is the oracle's Eq. 6 selection on that
    relevance with the draft tier only (bit-exact), and target layer i attends with the set of
    draft layer floor(i * L_d / L_t)."""
    s = W.config("qwen7b").replace(layers=4, draft=W.DraftShape(layers=6))
    layers = [W.make_layer(s, l, DEV) for l in range(s.layers)]
    est = W.make_estimation(s, layers[0], DEV)
    st = S.PerLayerSelectionStep(s, layers, est, DEV, n_target=12)
    st.run()
    torch.cuda.synchronize()
    B, N = s.B, s.n_max
    seq = torch.tensor(s.seq_lens, dtype=torch.int32, device=DEV)
    gam = torch.tensor(s.draft_gamma, dtype=torch.int32, device=DEV)
    nq = torch.tensor(s.n_query, dtype=torch.int32, device=DEV)
    for j in range(6):
        one = D.score(est.draft_q[j], est.draft_k[j], seq, list(range(14)), n_query=gam, max_len=N)
        torch.cuda.synchronize()
        for b, n in enumerate(s.seq_lens):
            assert torch.equal(st.rel[j, b, 0, :n], one[b, 0, :n]), f"layer {j} b={b}"
        rel = st.rel[j].cpu().numpy()
        ri, rc = O.select(rel, None, s.seq_lens, s.k_max, budget=s.budget, m_scalar=s.k_max - 20)
        for b in range(B):
            c = int(st.cnt[j * B + b, 0])
            assert c == int(rc[b, 0]), f"layer {j} b={b}"
            np.testing.assert_array_equal(st.idx[j * B + b, 0, :c].cpu().numpy(), ri[b, 0, :c])
    for i, L in enumerate(layers):
        j = S.draft_layer_of(i, 12, 6)
        assert j == i * 6 // 12
        ref = D.sparse_verify_attn(L.q, L.k, L.v, st.idx[j * B:(j + 1) * B], st.cnt[j * B:(j + 1) * B], seq,
                                   n_query=nq)
        torch.cuda.synchronize()
        for b, t in enumerate(s.n_query):
            assert torch.equal(st.outs[i][b, :t].view(torch.int16), ref[b, :t].view(torch.int16)), f"layer {i}"
