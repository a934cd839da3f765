"""GPU page estimator against the oracle: page statistics bit-exact (they are bf16 values
of K), page-level importance within 1e-4 * max(|S_ref|, 1/P_b), plus the properties that
hold at any size (page-constant scores, the row-sum invariant, whole-page selections)."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_24957_amd as D
from paper_2606_24957_amd import workloads as W
from tests.gpu_util import bits, check_score, host, scale_of

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _k(B, N, Hkv, d, seed, seq=None):
    g = torch.Generator(device=DEV).manual_seed(seed)
    k = torch.randn((B, N, Hkv, d), generator=g, device=DEV).to(torch.bfloat16)
    k[:, 3::7, 0, 5] = 0.0                       # zeros of both signs inside pages
    k[:, 4::7, 0, 5] = -0.0
    if seq is not None:
        for b, n in enumerate(seq):
            k[b, n:] = 1e30                      # past N_b: never part of a page
    return k


def _meta_host(meta):
    return bits(meta)


@pytest.mark.parametrize("d,ps,seq", [(128, 16, [1000, 17, 1]), (64, 16, [333, 2048]), (128, 1, [50, 9]),
                                      (128, 64, [4100, 64, 65])])
def test_page_meta_bit_exact(d, ps, seq):
    B, Hkv = len(seq), 4
    N = max(seq) + 5
    k = _k(B, N, Hkv, d, 1, seq)
    meta = D.page_meta(k, seq, ps, max_len=N)
    torch.cuda.synchronize()
    ref = O.page_meta(bits(k), seq, ps, num_pages=meta.shape[1])
    got = _meta_host(meta)
    for b, n in enumerate(seq):
        P = -(-n // ps)
        np.testing.assert_array_equal(got[b, :P], ref[b, :P], err_msg=f"b={b}")
        assert not got[b, P:].any()              # pages past N_b stay as they were (zero)


def test_page_meta_paged_cache_matches_contiguous():
    B, Hkv, d, ps, N = 3, 2, 128, 16, 700
    seq = [700, 300, 31]
    k = _k(B, N, Hkv, d, 2)
    page = 16
    maxp = -(-N // page)
    perm = torch.randperm(B * maxp, generator=torch.Generator().manual_seed(3)).to(torch.int32)
    pt = perm.reshape(B, maxp).to(DEV)
    pool = torch.zeros((B * maxp, page, Hkv, d), dtype=torch.bfloat16, device=DEV)
    pool[pt.reshape(-1).long()] = torch.nn.functional.pad(k, (0, 0, 0, 0, 0, maxp * page - N)).reshape(
        B * maxp, page, Hkv, d)
    a = D.page_meta(k, seq, ps, max_len=N)
    b = D.page_meta(pool, seq, ps, max_len=N, page_table=pt)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    ref = O.page_meta(bits(k), seq, ps, num_pages=a.shape[1])
    np.testing.assert_array_equal(_meta_host(a), ref)


def test_page_meta_update_after_append_equals_rebuild():
    """After T_b new positions, rebuilding from the old lengths rewrites exactly the pages
    that changed: the result equals a full rebuild, earlier pages are not written."""
    B, Hkv, d, ps, N = 3, 2, 128, 16, 600
    old = [300, 47, 16]
    T = [5, 9, 16]
    k = _k(B, N, Hkv, d, 4)
    meta = D.page_meta(k, old, ps, max_len=N)
    sentinel = 0x7F7F
    untouched = []
    for b, n in enumerate(old):                  # mark every page that must not be written
        first = n // ps
        meta.view(torch.int16)[b, :first] = sentinel
        untouched.append(first)
    new = [n + t for n, t in zip(old, T)]
    D.page_meta(k, new, ps, meta=meta, max_len=N, from_=torch.tensor(old, dtype=torch.int32, device=DEV),
                max_span=max(T))
    full = D.page_meta(k, new, ps, max_len=N)
    torch.cuda.synchronize()
    got, ref = _meta_host(meta), _meta_host(full)
    for b, n in enumerate(new):
        f, P = untouched[b], -(-n // ps)
        assert np.all(got[b, :f].view(np.int16) == sentinel), f"b={b}: a page before the append was written"
        np.testing.assert_array_equal(got[b, f:P], ref[b, f:P], err_msg=f"b={b}")


def _score_case(B, seq, nq, Hq, Hkv, d, heads, ps, groups=1, with_init=True, seed=0):
    g = torch.Generator(device=DEV).manual_seed(seed)
    N = max(seq)
    q = torch.randn((B, max(nq), Hq, d), generator=g, device=DEV).to(torch.bfloat16)
    k = torch.randn((B, N, Hkv, d), generator=g, device=DEV).to(torch.bfloat16)
    k[:, 40] = (3.0 * q[:, 0, 0]).to(torch.bfloat16).unsqueeze(1).expand(B, Hkv, d)  # a salient page
    init = torch.rand((B, groups, N), generator=g, device=DEV) / N if with_init else None
    meta = D.page_meta(k, seq, ps, max_len=N)
    out = torch.full((B, groups, N), -5.0, device=DEV)
    nqt = torch.tensor(nq, dtype=torch.int32, device=DEV)
    D.page_score(q, meta, seq, heads, ps, max_len=N, n_query=nqt, groups=groups, init=init, out=out)
    torch.cuda.synchronize()
    ref = O.page_score(bits(q), bits(meta), seq, nq, heads, scale_of(d), ps, groups=groups,
                       init=None if init is None else host(init), length=N)
    got = host(out)
    for b, n in enumerate(seq):
        P = -(-n // ps)
        for go in range(groups):
            check_score(got[b, go, :n], ref[b, go, :n], P, f"b={b} go={go}")
            assert np.all(got[b, go, n:] == -5.0)
            if init is None:                        # every position carries its page's value
                row = got[b, go, :n]
                for p in range(P):
                    assert np.all(row[p * ps:min(n, (p + 1) * ps)] == row[p * ps])
    return got


def test_page_score_all_heads_target_shape():
    """Quest's estimator: every query head of a Qwen2.5-72B-shaped layer (64 heads over 8 KV
    heads, 5 verification queries: 40 pairs per KV head, three column tiles)."""
    _score_case(2, [3000, 1234], [5, 3], 64, 8, 128, list(range(64)), 16, with_init=False)
    _score_case(2, [3000, 1234], [5, 3], 64, 8, 128, list(range(64)), 16, seed=1)


def test_page_score_scoring_heads_per_group_and_draft_shape():
    _score_case(3, [2000, 777, 20], [1, 1, 1], 64, 8, 128, [0, 17, 34, 51], 16, groups=8)
    _score_case(2, [4100, 1500], [4, 2], 14, 2, 64, [0, 4, 7, 11], 16, with_init=False)


def test_page_score_page_size_one_is_dustin_score():
    B, N, Hq, Hkv, d, heads = 2, 1500, 64, 8, 128, [0, 17, 34, 51]
    g = torch.Generator(device=DEV).manual_seed(7)
    q = torch.randn((B, 1, Hq, d), generator=g, device=DEV).to(torch.bfloat16)
    k = torch.randn((B, N, Hkv, d), generator=g, device=DEV).to(torch.bfloat16)
    seq = [1500, 999]
    a = D.score(q, k, torch.tensor(seq, dtype=torch.int32, device=DEV), heads, max_len=N)
    meta = D.page_meta(k, seq, 1, max_len=N)
    b = D.page_score(q, meta, seq, heads, 1, max_len=N)
    torch.cuda.synchronize()
    for i, n in enumerate(seq):
        check_score(host(b)[i, 0, :n], host(a)[i, 0, :n].astype(np.float64), n, f"b={i}")


def test_page_score_full_size_qwen72b():
    """B = 16, N = 32768: page statistics of the layer's K, then Quest-16's all-heads page
    score over the 5 verification queries and the scoring-head page score of the last
    token; the oracle checks sequences 0, 7 and 15.  Top-k over the page scores keeps whole
    pages (bit-exact against the oracle's selection on the same scores)."""
    s = W.config("qwen72b").replace(layers=1)
    L = W.make_layer(s, 0, DEV)
    E = W.make_estimation(s, L, DEV)
    seq = torch.tensor(s.seq_lens, dtype=torch.int32, device=DEV)
    nq = torch.tensor(s.n_query, dtype=torch.int32, device=DEV)
    ps = 16
    meta = D.page_meta(L.k, seq, ps, max_len=s.n_max)
    quest = D.page_score(L.q, meta, seq, list(range(64)), ps, max_len=s.n_max, n_query=nq)
    srh = D.page_score(E.q_target, meta, seq, s.target_heads, ps, max_len=s.n_max)
    idx, cnt = D.topk(None, quest, seq, s.k_max, m_scalar=0)
    torch.cuda.synchronize()
    for b in (0, 7, 15):
        n = s.seq_lens[b]
        kb = bits(L.k[b:b + 1, :n])
        mb = O.page_meta(kb, [n], ps)
        np.testing.assert_array_equal(bits(meta[b:b + 1, :mb.shape[1]]), mb, err_msg=f"meta b={b}")
        rq = O.page_score(bits(L.q[b:b + 1]), mb, [n], [s.n_query[b]], list(range(64)), scale_of(128), ps)
        check_score(host(quest)[b, 0, :n], rq[0, 0, :n], -(-n // ps), f"quest b={b}")
        rs = O.page_score(bits(E.q_target[b:b + 1]), mb, [n], [1], s.target_heads, scale_of(128), ps)
        check_score(host(srh)[b, 0, :n], rs[0, 0, :n], -(-n // ps), f"srh b={b}")
        ri, rc = O.select(None, host(quest)[b:b + 1], [n], s.k_max, m_scalar=0)
        c = int(host(cnt)[b, 0])
        assert c == int(rc[0, 0])
        got_idx = host(idx)[b, 0, :c]
        np.testing.assert_array_equal(got_idx, ri[0, 0, :c])
        # outside the sinks and the window, at most one page is taken in part
        inner = got_idx[(got_idx >= s.n_sink) & (got_idx < n - s.n_window)]
        pages, per = np.unique(inner // ps, return_counts=True)
        full = [p for p, c_ in zip(pages, per) if c_ == min(ps, n - s.n_window - p * ps) or p * ps < s.n_sink]
        assert len(pages) - len(full) <= 1


def test_page_estimator_degenerate_lengths():
    """Empty sequences get no page and no output; a sequence shorter than one page has one
    page whose score is the whole softmax (1 per (head, query)); a page size above every
    length gives one page per sequence."""
    B, Hq, Hkv, d, ps = 3, 8, 2, 128, 16
    seq = [0, 5, 40]
    N = 48
    k = _k(B, N, Hkv, d, 9)
    g = torch.Generator(device=DEV).manual_seed(9)
    q = torch.randn((B, 2, Hq, d), generator=g, device=DEV).to(torch.bfloat16)
    meta = torch.full((B, 3, Hkv, 2 * d), -3.0, dtype=torch.bfloat16, device=DEV)
    D.page_meta(k, seq, ps, meta=meta, max_len=N)
    out = torch.full((B, 1, N), -5.0, device=DEV)
    D.page_score(q, meta, seq, [0, 5], ps, max_len=N, n_query=torch.tensor([2, 2, 1], dtype=torch.int32,
                                                                           device=DEV), out=out)
    big = D.page_meta(k, seq, 64, max_len=N)
    out64 = D.page_score(q, big, seq, [0, 5], 64, max_len=N)
    torch.cuda.synchronize()
    m = meta.float().cpu()
    assert torch.all(m[0] == -3.0)                                 # N_b = 0: no page written
    assert torch.all(m[1, 1:] == -3.0) and torch.all(m[2, 3:] == -3.0)
    o = host(out)
    assert np.all(o[0] == -5.0)                                    # no output for N_b = 0
    np.testing.assert_allclose(o[1, 0, :5], 2 * 2, rtol=1e-6)       # one page: 2 heads x 2 queries
    assert np.all(o[1, 0, 5:] == -5.0)
    ref = O.page_score(bits(q), bits(meta), seq, [2, 2, 1], [0, 5], scale_of(d), ps, length=N)
    check_score(o[2, 0, :40], ref[2, 0, :40], 3, "b=2")
    o64 = host(out64)
    np.testing.assert_allclose(o64[2, 0, :40], 2 * 2, rtol=1e-6)    # one page of 64 holds all 40

