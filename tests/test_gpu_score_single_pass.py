"""The single-pass form of Eq. 5 (score_sync.hip) against the oracle: every number of
used KV heads, both row lengths, ragged batches with empty and one-position sequences,
sequences of one chunk and of several, per-sequence query counts, paged caches with pages
smaller and larger than a 16-position tile, several layers in one call, and the counter
region returned to zero with no timeout after every call."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_24957_amd as D
from tests.gpu_util import bits, check_score, host, scale_of

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _sync_region_clear():
    reg = D.score_sync_region()
    assert reg is not None
    assert int(reg.count_nonzero()) == 0, "counters or timeout flag left non-zero"


def _paged(k: torch.Tensor, page_size: int, seed: int):
    """The cache rows of k [B, N, Hkv, d] scattered over permuted pages."""
    B, N, Hkv, d = k.shape
    maxp = (N + page_size - 1) // page_size
    perm = torch.randperm(B * maxp, generator=torch.Generator().manual_seed(seed)).to(torch.int32)
    pt = perm.reshape(B, maxp).to(k.device)
    pages = torch.zeros((B * maxp, page_size, Hkv, d), dtype=torch.bfloat16, device=k.device)
    padded = torch.nn.functional.pad(k, (0, 0, 0, 0, 0, maxp * page_size - N))
    pages[pt.reshape(-1).long()] = padded.reshape(B * maxp, page_size, Hkv, d)
    return pages, pt


def _run(seq_l, nq_l, Hq, Hkv, d, heads, n_layers=1, with_init=True, page_size=0, seed=0):
    B, N = len(seq_l), max(max(seq_l), 1)
    nq = max(nq_l)
    assert len(heads) * nq <= 16  # the single-pass form's limit
    g = torch.Generator(device=DEV).manual_seed(seed)
    qs = [torch.randn((B, nq, Hq, d), generator=g, device=DEV).to(torch.bfloat16) for _ in range(n_layers)]
    ks = [torch.randn((B, N, Hkv, d), generator=g, device=DEV).to(torch.bfloat16) for _ in range(n_layers)]
    for q, k in zip(qs, ks):  # a salient key per sequence
        k[:, min(7, N - 1)] = (3.0 * q[:, 0, heads[0]]).to(torch.bfloat16).unsqueeze(1).expand(B, Hkv, d)
    pt = None
    kin = ks
    if page_size:
        pairs = [_paged(k, page_size, seed + 1) for k in ks]
        kin, pt = [p for p, _ in pairs], pairs[0][1]
    seq = torch.tensor(seq_l, dtype=torch.int32, device=DEV)
    nqt = torch.tensor(nq_l, dtype=torch.int32, device=DEV)
    init = torch.rand((B, 1, N), generator=g, device=DEV) / N if with_init else None
    out = torch.full((B, 1, N), -5.0, device=DEV)
    if n_layers == 1:
        D.score(qs[0], kin[0], seq, heads, n_query=nqt, init=init, out=out, max_len=N, page_table=pt)
    else:
        D.score_layers(qs, kin, seq, heads, n_query=nqt, init=init, out=out, max_len=N, page_table=pt)
    torch.cuda.synchronize()
    _sync_region_clear()
    ref = np.zeros((B, 1, N)) if init is None else host(init).astype(np.float64)
    for q, k in zip(qs, ks):
        ref = ref + O.score(bits(q), bits(k), seq_l, nq_l, heads, scale_of(d), num_kv_heads=Hkv)[:, :, :N]
    got = host(out)
    for b, n in enumerate(seq_l):
        check_score(got[b, 0, :n], ref[b, 0, :n], n, f"b={b} N_b={n}")
        assert np.all(got[b, 0, n:] == -5.0)  # positions >= N_b untouched
        base = 0.0 if init is None else host(init)[b, 0, :n].astype(np.float64).sum()
        if n:
            assert abs(got[b, 0, :n].astype(np.float64).sum() - base - n_layers * nq_l[b] * len(heads)) <= \
                1e-4 * n_layers * nq_l[b] * len(heads)
    return out


# ragged lengths: empty, one position, under one tile, a chunk and one more, several chunks
RAGGED = [0, 1, 15, 17, 512, 513, 1500, 2048]


@pytest.mark.parametrize("Hq,Hkv,d,heads,nq", [
    (64, 8, 128, [0], 16),               # one KV head, 16 queries
    (64, 8, 128, [0, 17], 2),            # two KV heads
    (64, 8, 128, [0, 17, 34], 1),        # three
    (64, 8, 128, [0, 17, 34, 51], 4),    # four: 16 pairs (the target's heads, four queries)
    (64, 8, 128, [0, 1, 9], 5),          # two heads on one KV head, one on another: 15 pairs
    (14, 2, 64, [0, 4, 7, 11], 4),       # the draft's scoring heads: 16 pairs over 2 KV heads
    (14, 2, 64, [0, 4], 3),              # one KV head
    (16, 4, 64, [0, 5, 10], 2),          # three KV heads of 64-element rows
    (16, 4, 64, [0, 5, 10, 15], 4),      # four
])
def test_single_pass_matches_oracle(Hq, Hkv, d, heads, nq):
    nq_l = [max(1, nq - (b % 3)) for b in range(len(RAGGED))]  # per-sequence query counts
    _run(RAGGED, nq_l, Hq, Hkv, d, heads, seed=len(heads) * 7 + nq)


@pytest.mark.parametrize("page_size", [4, 16, 64])
def test_single_pass_paged(page_size):
    _run([3000, 1, 777, 2049], [1, 1, 1, 1], 64, 8, 128, [0, 17, 34, 51], page_size=page_size, seed=21)
    _run([3000, 1, 777, 2049], [4, 3, 2, 4], 14, 2, 64, [0, 4, 7, 11], page_size=page_size, seed=22)


@pytest.mark.parametrize("n_layers,d", [(3, 64), (5, 64), (2, 128)])
def test_single_pass_layers(n_layers, d):
    """Several layers in one launch: each layer's softmax over its own statistics, summed."""
    if d == 64:
        _run([2500, 700, 0, 513], [4, 2, 1, 3], 14, 2, 64, [0, 4, 7, 11], n_layers=n_layers, seed=30 + n_layers)
    else:
        _run([2500, 700, 0, 513], [1, 1, 1, 1], 64, 8, 128, [0, 17, 34, 51], n_layers=n_layers, seed=40)


def test_single_pass_is_deterministic_and_reusable():
    """Calls in a row (the counters returned to zero by each) give the same bits; init may
    alias out."""
    B, N, d, heads = 4, 5000, 128, [0, 17, 34, 51]
    g = torch.Generator(device=DEV).manual_seed(50)
    q = torch.randn((B, 1, 64, d), generator=g, device=DEV).to(torch.bfloat16)
    k = torch.randn((B, N, 8, d), generator=g, device=DEV).to(torch.bfloat16)
    seq = torch.tensor([N, 4000, 3333, 1], dtype=torch.int32, device=DEV)
    outs = [D.score(q, k, seq, heads, max_len=N).clone() for _ in range(3)]
    acc = torch.zeros((B, 1, N), device=DEV)
    for _ in range(2):
        D.score(q, k, seq, heads, init=acc, out=acc, max_len=N)
    torch.cuda.synchronize()
    _sync_region_clear()
    for o in outs[1:]:
        assert torch.equal(o[0, 0, :N], outs[0][0, 0, :N]) and torch.equal(o[3, 0, :1], outs[0][3, 0, :1])
    lens = [N, 4000, 3333, 1]
    for b, n in enumerate(lens):
        np.testing.assert_allclose(host(acc)[b, 0, :n], 2 * host(outs[0])[b, 0, :n], rtol=1e-6, atol=0)


def test_single_pass_many_chunks_per_sequence():
    """Sequences of many chunks, spread over every XCD (64 chunks of 2048 positions do not
    fit one): B = 2 of N = 131072 with the draft's shape."""
    B, N, d, heads = 2, 131072, 64, [0, 4, 7, 11]
    g = torch.Generator(device=DEV).manual_seed(60)
    q = torch.randn((B, 4, 14, d), generator=g, device=DEV).to(torch.bfloat16)
    k = torch.randn((B, N, 2, d), generator=g, device=DEV).to(torch.bfloat16)
    lens = [N, 77777]
    seq = torch.tensor(lens, dtype=torch.int32, device=DEV)
    out = D.score(q, k, seq, heads, max_len=N)
    torch.cuda.synchronize()
    _sync_region_clear()
    for b in (0, 1):
        n = lens[b]
        ref = O.score(bits(q[b:b + 1]), bits(k[b:b + 1]), [n], [4], heads, scale_of(d), num_kv_heads=2)
        check_score(host(out)[b, 0, :n], ref[0, 0, :n], n, f"b={b}")


def _step_scores(B, N, lens, gamma, page_size=0, seed=70):
    """A target call (last token, heads {0, 17, 34, 51} over 8 KV heads of 128) and a draft
    call (Gamma queries, heads {0, 4, 7, 11} over 2 KV heads of 64, three layers)."""
    g = torch.Generator(device=DEV).manual_seed(seed)
    qt = torch.randn((B, 1, 64, 128), generator=g, device=DEV).to(torch.bfloat16)
    kt = torch.randn((B, N, 8, 128), generator=g, device=DEV).to(torch.bfloat16)
    qd = [torch.randn((B, gamma, 14, 64), generator=g, device=DEV).to(torch.bfloat16) for _ in range(3)]
    kd = [torch.randn((B, N, 2, 64), generator=g, device=DEV).to(torch.bfloat16) for _ in range(3)]
    init = torch.rand((B, 1, N), generator=g, device=DEV) / N
    pt = None
    if page_size:
        kt, pt = _paged(kt, page_size, seed)
        kd = [_paged(k, page_size, seed)[0] for k in kd]
    seq = torch.tensor(lens, dtype=torch.int32, device=DEV)
    nq = torch.tensor([max(1, gamma - b % 2) for b in range(B)], dtype=torch.int32, device=DEV)
    st, sd = torch.full((B, 1, N), -5.0, device=DEV), torch.full((B, 1, N), -5.0, device=DEV)
    pt_ = D.plan_score(qt, kt, seq, [0, 17, 34, 51], init=init, out=st, max_len=N, page_table=pt)
    pd_ = D.plan_score_layers(qd, kd, seq, [0, 4, 7, 11], n_query=nq, out=sd, max_len=N, page_table=pt,
                              ws_tag="score_draft")
    return pt_, pd_, st, sd


@pytest.mark.parametrize("B,N,page_size", [(16, 32768, 0), (16, 32768, 16), (5, 3000, 0), (5, 3000, 4)])
def test_two_calls_in_one_launch_equal_the_separate_calls(B, N, page_size):
    """dustin_score_calls with the target's and the draft's calls of a step: the outputs have
    the bits of the two calls made one after the other (one launch at the full shape, where
    both take the single-pass form with eight tiles per wave; two tiles per wave below)."""
    lens = [N - 37 * b for b in range(B)]
    pt_, pd_, st, sd = _step_scores(B, N, lens, 4, page_size)
    pt_()
    pd_()
    torch.cuda.synchronize()
    ref_t, ref_d = st.clone(), sd.clone()
    st.fill_(-5.0)
    sd.fill_(-5.0)
    both = D.plan_score_calls([pt_, pd_])
    for _ in range(2):  # twice in a row: the counters return to zero
        both()
    torch.cuda.synchronize()
    assert torch.equal(st, ref_t) and torch.equal(sd, ref_d)
    for tag in ("score", "score_draft"):
        reg = D.score_sync_region(tag=tag)
        assert int(reg.count_nonzero()) == 0
    if not page_size:  # and the target against the oracle for the last sequence
        b, n = B - 1, lens[-1]
        q, k, init = pt_._keep[0], pt_._keep[1], pt_._keep[2]
        ref = O.score(bits(q[b:b + 1]), bits(k[b:b + 1]), [n], [1], [0, 17, 34, 51], scale_of(128),
                      num_kv_heads=8, init=host(init)[b:b + 1])
        check_score(host(st)[b, 0, :n], ref[0, 0, :n], n, f"target b={b}")


def test_two_calls_fall_back_to_one_after_the_other():
    """A pair of shapes the fused launch does not cover (a draft call of three KV heads)
    still gives the separate calls' bits."""
    B, N = 3, 2500
    g = torch.Generator(device=DEV).manual_seed(80)
    qt = torch.randn((B, 1, 64, 128), generator=g, device=DEV).to(torch.bfloat16)
    kt = torch.randn((B, N, 8, 128), generator=g, device=DEV).to(torch.bfloat16)
    qd = torch.randn((B, 2, 16, 64), generator=g, device=DEV).to(torch.bfloat16)
    kd = torch.randn((B, N, 4, 64), generator=g, device=DEV).to(torch.bfloat16)
    seq = torch.tensor([N, 1000, 1], dtype=torch.int32, device=DEV)
    a = D.plan_score(qt, kt, seq, [0, 17, 34, 51], max_len=N)
    b_ = D.plan_score(qd, kd, seq, [0, 5, 10], max_len=N, ws_tag="score_draft")
    a()
    b_()
    torch.cuda.synchronize()
    ra, rb = a.result.clone(), b_.result.clone()
    D.plan_score_calls([a, b_])()
    torch.cuda.synchronize()
    assert torch.equal(a.result[0, 0, :N], ra[0, 0, :N]) and torch.equal(b_.result[1, 0, :1000], rb[1, 0, :1000])
