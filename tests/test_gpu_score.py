"""GPU scoring-head importance (Eq. 5) against the oracle: every score within
1e-4 * max(|S_ref|, 1/N_b), plus the row-sum invariant sum_n (S - init) = nq_b * |H|."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_24957_amd as D
from paper_2606_24957_amd import workloads as W
from tests.gpu_util import bits, check_score, host, scale_of

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _case(B, N, nq, Hq, Hkv, d, heads, groups=1, with_init=True, seed=0, n_list=None):
    g = torch.Generator(device=DEV).manual_seed(seed)
    ncap = max(n_list) if n_list else N
    q = torch.randn((B, nq, Hq, d), generator=g, device=DEV).to(torch.bfloat16)
    k = torch.randn((B, ncap, Hkv, d), generator=g, device=DEV).to(torch.bfloat16)
    k[:, 7] = (3.0 * q[:, 0, 0]).to(torch.bfloat16).unsqueeze(1).expand(B, Hkv, d)  # a salient key
    seq = n_list or [N] * B
    init = None
    if with_init:
        init = torch.rand((B, groups, ncap), generator=g, device=DEV) / ncap
    out = torch.full((B, groups, ncap), -5.0, device=DEV)
    D.score(q, k, torch.tensor(seq, dtype=torch.int32, device=DEV), heads, groups=groups,
            init=init, out=out, n_query=torch.tensor([nq] * B, dtype=torch.int32, device=DEV))
    torch.cuda.synchronize()
    ref = O.score(bits(q), bits(k), seq, [nq] * B, heads, scale_of(d), num_kv_heads=Hkv,
                  groups=groups, init=None if init is None else host(init))
    got = host(out)
    for b in range(B):
        for go in range(groups):
            n = seq[b]
            check_score(got[b, go, :n], ref[b, go, :n], n, f"b={b} g={go}")
            assert np.all(got[b, go, n:] == -5.0)          # positions >= N_b untouched
            base = 0 if init is None else host(init)[b, go, :n].astype(np.float64).sum()
            hs = [h for h in heads if groups == 1 or h // (Hq // Hkv) == go]
            assert abs(got[b, go, :n].astype(np.float64).sum() - base - nq * len(hs)) <= 1e-4 * nq * max(1, len(hs))
    return got


def test_score_target_shape():
    """Target scoring: last token's query, 4 heads in 4 distinct KV heads, d = 128."""
    _case(3, 5000, 1, 64, 8, 128, [0, 17, 34, 51], with_init=True)


def test_score_draft_shape():
    """Draft scoring: Gamma = 4 queries, heads {0, 4, 7, 11} over 2 KV heads, d = 64."""
    _case(2, 4100, 4, 14, 2, 64, [0, 4, 7, 11], with_init=False)


def test_score_per_group_and_ragged():
    _case(3, 0, 2, 64, 8, 128, [0, 9, 63], groups=8, n_list=[3000, 1025, 17])


def test_score_layer_chaining_accumulates():
    """init aliasing out accumulates draft layers like a sum over layers in Eq. 5."""
    B, N, nq, Hq, Hkv, d, heads = 2, 2048, 4, 14, 2, 64, [0, 4, 7, 11]
    g = torch.Generator(device=DEV).manual_seed(3)
    seq = torch.tensor([N, N - 100], dtype=torch.int32, device=DEV)
    acc = torch.zeros((B, 1, N), device=DEV)
    ref = np.zeros((B, 1, N), dtype=np.float32)
    for _ in range(3):
        q = torch.randn((B, nq, Hq, d), generator=g, device=DEV).to(torch.bfloat16)
        k = torch.randn((B, N, Hkv, d), generator=g, device=DEV).to(torch.bfloat16)
        D.score(q, k, seq, heads, init=acc, out=acc)
        ref = O.score(bits(q), bits(k), [N, N - 100], [nq] * B, heads, scale_of(d), init=ref.copy())
    torch.cuda.synchronize()
    got = host(acc)
    for b, n in enumerate([N, N - 100]):
        check_score(got[b, 0, :n], ref[b, 0, :n], n, f"chain b={b}")


def test_score_full_size_target_and_draft():
    """Qwen2.5-72B-shaped target scoring layer and one Qwen2.5-0.5B-shaped draft layer at
    B = 16, N = 32768; the oracle checks four sequences."""
    s = W.config("qwen72b").replace(layers=1)
    L = W.make_layer(s, 0, DEV)
    E = W.make_estimation(s, L, DEV)
    seq = torch.tensor(s.seq_lens, dtype=torch.int32, device=DEV)
    st = D.score(E.q_target, L.k, seq, s.target_heads, max_len=s.n_max)
    sd = D.score(E.draft_q[0], E.draft_k[0], seq, s.draft.heads, max_len=s.n_max,
                 n_query=torch.tensor(s.draft_gamma, dtype=torch.int32, device=DEV))
    torch.cuda.synchronize()
    for b in (0, 5, 10, 15):
        rt = O.score(bits(E.q_target[b:b + 1]), bits(L.k[b:b + 1]), [s.seq_lens[b]], [1],
                     s.target_heads, scale_of(128), num_kv_heads=8)
        check_score(host(st)[b, 0, :s.seq_lens[b]], rt[0, 0, :s.seq_lens[b]], s.seq_lens[b], f"target b={b}")
        rd = O.score(bits(E.draft_q[0][b:b + 1]), bits(E.draft_k[0][b:b + 1]), [s.seq_lens[b]],
                     [s.draft_gamma[b]], s.draft.heads, scale_of(64), num_kv_heads=2)
        check_score(host(sd)[b, 0, :s.seq_lens[b]], rd[0, 0, :s.seq_lens[b]], s.seq_lens[b], f"draft b={b}")


@pytest.mark.parametrize("n_layers,with_init,paged", [(3, False, False), (2, True, False), (3, False, True),
                                                       (32, True, False)])
def test_score_layers_sums_layers_in_one_call(n_layers, with_init, paged):
    """dustin_score_layers: Eq. 5 summed over layers in two launches equals init plus the
    oracle's per-layer scores, summed in fp64."""
    B, N, nq, Hq, Hkv, d, heads = 3, 3000, 4, 14, 2, 64, [0, 4, 7, 11]
    g = torch.Generator(device=DEV).manual_seed(11)
    seq_l = [N, N - 777, 1500]
    seq = torch.tensor(seq_l, dtype=torch.int32, device=DEV)
    nqt = torch.tensor([nq, 2, 3], dtype=torch.int32, device=DEV)
    qs = [torch.randn((B, nq, Hq, d), generator=g, device=DEV).to(torch.bfloat16) for _ in range(n_layers)]
    ks = [torch.randn((B, N, Hkv, d), generator=g, device=DEV).to(torch.bfloat16) for _ in range(n_layers)]
    pt = None
    if paged:  # the same page table for every layer, pages permuted
        ps, maxp = 16, (N + 15) // 16
        perm = torch.randperm(B * maxp, generator=torch.Generator().manual_seed(5)).to(torch.int32)
        pt = perm.reshape(B, maxp).to(DEV)
        kp = []
        for k in ks:
            pages = torch.zeros((B * maxp, ps, Hkv, d), dtype=torch.bfloat16, device=DEV)
            pages[pt.reshape(-1).long()] = torch.nn.functional.pad(k, (0, 0, 0, 0, 0, maxp * ps - N)).reshape(
                B * maxp, ps, Hkv, d)
            kp.append(pages)
        kin = kp
    else:
        kin = ks
    init = torch.rand((B, 1, N), generator=g, device=DEV) / N if with_init else None
    out = torch.full((B, 1, N), -5.0, device=DEV)
    D.score_layers(qs, kin, seq, heads, n_query=nqt, init=init, out=out, max_len=N, page_table=pt)
    torch.cuda.synchronize()
    ref = np.zeros((B, 1, N), dtype=np.float64) if init is None else host(init).astype(np.float64)
    for q, k in zip(qs, ks):
        ref += O.score(bits(q), bits(k), seq_l, nqt.cpu().tolist(), heads, scale_of(d)).astype(np.float64)
    got = host(out)
    for b, n in enumerate(seq_l):
        check_score(got[b, 0, :n], ref[b, 0, :n], n, f"layers b={b}")
        assert np.all(got[b, 0, n:] == -5.0)


def test_score_layers_one_layer_is_dustin_score():
    B, N, nq, Hq, Hkv, d, heads = 2, 2100, 1, 64, 8, 128, [0, 17, 34, 51]
    g = torch.Generator(device=DEV).manual_seed(12)
    q = torch.randn((B, nq, Hq, d), generator=g, device=DEV).to(torch.bfloat16)
    k = torch.randn((B, N, Hkv, d), generator=g, device=DEV).to(torch.bfloat16)
    init = torch.rand((B, 1, N), generator=g, device=DEV) / N
    seq = torch.tensor([N, 1000], dtype=torch.int32, device=DEV)
    a = D.score(q, k, seq, heads, init=init, max_len=N).clone()
    b = D.score_layers([q], [k], seq, heads, init=init, max_len=N)
    torch.cuda.synchronize()
    assert torch.equal(a[:, :, :1000], b[:, :, :1000]) and torch.equal(a[0], b[0])


def test_score_twelve_draft_heads_share_a_workgroup():
    """Dustin-D's 12 draft heads: 24 (head, query) pairs per KV head span two column tiles,
    which one pass-1 workgroup computes from a single read of each K row."""
    _case(3, 0, 4, 14, 2, 64, list(range(12)), n_list=[3000, 1025, 40], with_init=True, seed=5)
    _case(2, 0, 4, 14, 2, 64, list(range(12)), groups=2, n_list=[2100, 700], seed=6)


def test_score_all_target_heads():
    """Every head of a Qwen2.5-72B-shaped layer (the naive estimator's per-layer work):
    64 heads, 2 queries, 16 pairs per KV head."""
    _case(2, 0, 2, 64, 8, 128, list(range(64)), n_list=[2000, 555], seed=7)


def test_score_maximum_rows():
    """The largest score call: 64 heads times 16 queries, 1024 (head, query) rows, eight
    column tiles per KV head."""
    _case(2, 0, 16, 64, 8, 128, list(range(64)), n_list=[1500, 301], seed=8)


@pytest.mark.parametrize("groups", [1, 2])
def test_score_per_layer_outputs_equal_single_layer_calls(groups):
    """dustin_score_per_layer: every layer into its own row, bit-identical to dustin_score
    on that layer alone (all 14 draft heads x 4 queries: two column tiles per KV head); one
    layer also against the oracle."""
    B, N, nq, Hq, Hkv, d = 2, 2500, 4, 14, 2, 64
    heads = list(range(Hq))
    g = torch.Generator(device=DEV).manual_seed(13)
    seq = torch.tensor([N, 1700], dtype=torch.int32, device=DEV)
    nqt = torch.tensor([4, 3], dtype=torch.int32, device=DEV)
    qs = [torch.randn((B, nq, Hq, d), generator=g, device=DEV).to(torch.bfloat16) for _ in range(5)]
    ks = [torch.randn((B, N, Hkv, d), generator=g, device=DEV).to(torch.bfloat16) for _ in range(5)]
    out = D.score_per_layer(qs, ks, seq, heads, n_query=nqt, groups=groups, max_len=N)
    singles = [D.score(q, k, seq, heads, n_query=nqt, groups=groups, max_len=N).clone() for q, k in zip(qs, ks)]
    torch.cuda.synchronize()
    for l, one in enumerate(singles):
        assert torch.equal(out[l, 0, :, :N], one[0, :, :N]) and torch.equal(out[l, 1, :, :1700], one[1, :, :1700])
    ref = O.score(bits(qs[3]), bits(ks[3]), [N, 1700], [4, 3], heads, scale_of(d), num_kv_heads=Hkv, groups=groups)
    for b, n in enumerate([N, 1700]):
        for go in range(groups):
            check_score(host(out[3])[b, go, :n], ref[b, go, :n], n, f"layer 3 b={b} go={go}")
