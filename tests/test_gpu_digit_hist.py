"""First-digit histograms: the score calls count their outputs by top key digit
(digit_hist), and the top-k takes those counts in place of its first pass over a row.  The
counts must equal those of the written outputs' order keys (the key's definition is written
out here on the host), the top-k's result must be the oracle's bit for bit whether or not
the histograms are given, and every histogram must be left at zero."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_24957_amd as D
from tests.gpu_util import bits, host
from tests.test_gpu_score_single_pass import _step_scores
from tests.test_gpu_topk import _scores

pytestmark = pytest.mark.gpu
DEV = "cuda"


def host_keys(x: np.ndarray) -> np.ndarray:
    """The order-preserving uint32 of fp32 values: -0 as +0, negatives bit-inverted, the sign
    bit set on the rest."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).copy()
    u[u == 0x80000000] = 0
    return np.where(u & 0x80000000, ~u, u | 0x80000000).astype(np.uint32)


def ref_hist(out: np.ndarray, lens) -> np.ndarray:
    """[B * G, 4096] counts of the rows' first N_b order keys by their top 12 bits."""
    B, G, _ = out.shape
    return np.stack([np.bincount(host_keys(out[b, g, :lens[b]]) >> 20, minlength=4096)
                     for b in range(B) for g in range(G)]).astype(np.int64)


@pytest.mark.parametrize("B,N,page_size", [(16, 32768, 0), (5, 3000, 0), (5, 3000, 4)])
def test_score_calls_count_their_outputs(B, N, page_size):
    """Both calls of a step (one launch at the full shape, the single-pass form in two below
    it, paged too): each histogram holds its call's outputs' key digits; a second call adds
    the same counts again."""
    lens = [N - 37 * b for b in range(B)]
    pt_, pd_, st, sd = _step_scores(B, N, lens, 4, page_size)
    ht, hd = D.digit_hist(B, DEV), D.digit_hist(B, DEV)
    both = D.plan_score_calls([pt_, pd_], digit_hists=[ht, hd])
    both()
    torch.cuda.synchronize()
    rt, rd = ref_hist(host(st), lens), ref_hist(host(sd), lens)
    assert np.array_equal(host(ht).astype(np.int64), rt)
    assert np.array_equal(host(hd).astype(np.int64), rd)
    both()
    torch.cuda.synchronize()
    assert np.array_equal(host(ht).astype(np.int64), 2 * rt)


def test_two_pass_score_counts_per_group():
    """The two-pass form (one output row per KV head) counts each output row on its own."""
    B, N, Hkv = 3, 2500, 4
    g = torch.Generator(device=DEV).manual_seed(5)
    q = torch.randn((B, 2, 16, 64), generator=g, device=DEV).to(torch.bfloat16)
    k = torch.randn((B, N, Hkv, 64), generator=g, device=DEV).to(torch.bfloat16)
    lens = [N, 1000, 1]
    seq = torch.tensor(lens, dtype=torch.int32, device=DEV)
    call = D.plan_score(q, k, seq, [0, 5, 10], groups=Hkv, max_len=N)
    h = D.digit_hist(B * Hkv, DEV)
    D.plan_score_calls([call], digit_hists=[h])()
    torch.cuda.synchronize()
    assert np.array_equal(host(h).astype(np.int64), ref_hist(host(call.result), lens))


def _topk_case(sd, st, lens, k, budget=None, m=None, m_scalar=None, use_hist=True):
    """dustin_topk on host score arrays, with their histograms given or not; checks the
    oracle's set and that the histograms are zero afterwards."""
    B = len(lens)
    P = 20
    if m_scalar is None:
        m_scalar = 0 if sd is None else (k - P if st is None else (k - P) // 2)
    idx_ref, cnt_ref = O.select(sd, st, lens, k, budget=budget, m=m, m_scalar=m_scalar, n_sink=4, n_window=16)
    dev = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    hist = lambda a: None if a is None or not use_hist else \
        torch.from_numpy(ref_hist(a, lens).astype(np.int32)).to(DEV)
    hd, ht = hist(sd), hist(st)
    idx, cnt = D.topk(dev(sd), dev(st), dev(np.asarray(lens, np.int32)), k,
                      budget=dev(None if budget is None else np.asarray(budget, np.int32)),
                      m=dev(None if m is None else np.asarray(m, np.int32)), m_scalar=m_scalar,
                      n_sink=4, n_window=16, hist_d=hd, hist_t=ht)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(cnt), cnt_ref)
    for b in range(B):
        c = cnt_ref[b, 0]
        np.testing.assert_array_equal(host(idx)[b, 0, :c], idx_ref[b, 0, :c], err_msg=f"b={b}")
    for h in (hd, ht):
        if h is not None:
            assert int(h.count_nonzero()) == 0, "a histogram was left non-zero"


@pytest.mark.parametrize("kind", ["uniform", "dirichlet", "quantized", "zeros", "special"])
def test_topk_with_histograms_matches_the_oracle(kind):
    B, N, k = 4, 40000, 2048
    lens = [N, N - 1, 20000, 9000]
    _topk_case(_scores(kind, B, N, 11), _scores(kind, B, N, 12), lens, k)


def test_topk_histograms_with_single_tiers_and_short_rows():
    """Per-sequence k and m: a row shorter than its budget, a target-only row (m = 0), a
    draft-only row (m = k - |P|), a row of both tiers; and each score array alone."""
    B, N = 4, 30000
    lens = [30000, 500, 25000, 12000]
    budget = [2048, 1024, 1000, 1536]
    m = [1014, 100, 0, 1536 - 20]
    sd, st = _scores("dirichlet", B, N, 21), _scores("uniform", B, N, 22)
    _topk_case(sd, st, lens, 2048, budget=budget, m=m)
    _topk_case(None, st, lens, 2048, m_scalar=0)
    _topk_case(sd, None, lens, 2048, m_scalar=2048 - 20)


def test_topk_histograms_when_the_tiers_run_in_turn():
    """Beyond 4096 rows (no hand-off workspace) a row's tiers run one after the other: the
    draft tier takes its histogram, the target tier (with I_D taken too) cannot and makes its
    own first pass, and both histograms are still cleared."""
    B, N, k = 4100, 300, 64
    lens = [N - (b % 50) for b in range(B)]
    assert D.lib().dustin_topk_workspace(B, 1, N) == 0
    _topk_case(_scores("dirichlet", B, N, 31), _scores("uniform", B, N, 32), lens, k)
