"""GPU tiered selection (Eq. 6) against the oracle: on identical fp32 score vectors the
index set, its ascending order and the count must match bit for bit."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_24957_amd as D

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _compare(sd, st, seq, k_max, budget=None, m=None, m_scalar=None, groups=1, ns=4, nw=16):
    B = len(seq)
    P = ns + nw
    if m_scalar is None:
        m_scalar = 0 if sd is None else (k_max - P if st is None else (k_max - P) // 2)
    idx_ref, cnt_ref = O.select(sd, st, seq, k_max, budget=budget, m=m, m_scalar=m_scalar,
                                n_sink=ns, n_window=nw, groups=groups)
    tdev = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    idx = torch.full((B, groups, k_max), -7, dtype=torch.int32, device=DEV)
    idx_g, cnt_g = D.topk(tdev(sd), tdev(st), tdev(np.asarray(seq, np.int32)), k_max,
                          budget=tdev(None if budget is None else np.asarray(budget, np.int32)),
                          m=tdev(None if m is None else np.asarray(m, np.int32)),
                          m_scalar=m_scalar, n_sink=ns, n_window=nw, groups=groups, idx=idx)
    torch.cuda.synchronize()
    cnt_g = cnt_g.cpu().numpy()
    idx_g = idx_g.cpu().numpy()
    np.testing.assert_array_equal(cnt_g, cnt_ref)
    for b in range(B):
        for g in range(groups):
            c = cnt_ref[b, g]
            np.testing.assert_array_equal(idx_g[b, g, :c], idx_ref[b, g, :c], err_msg=f"b={b} g={g}")
            assert np.all(idx_g[b, g, c:] == -7)          # entries past count untouched
    return idx_g, cnt_g


def _scores(kind, B, N, seed):
    rng = np.random.default_rng(seed)
    if kind == "uniform":
        x = rng.random((B, 1, N))
    elif kind == "dirichlet":
        x = rng.gamma(0.1, size=(B, 1, N))
        x /= x.sum(-1, keepdims=True)
    elif kind == "quantized":
        x = rng.integers(0, 7, (B, 1, N)) / 7.0
    elif kind == "equal":
        x = np.full((B, 1, N), 0.25)
    elif kind == "zeros":
        x = np.where(rng.random((B, 1, N)) < 0.97, 0.0, rng.random((B, 1, N)))
        x = np.where(rng.random((B, 1, N)) < 0.5, -0.0, x)
    elif kind == "signed":
        x = rng.standard_normal((B, 1, N)) * 1e3
    elif kind == "special":
        x = rng.standard_normal((B, 1, N))
        for v in (np.inf, -np.inf, np.nan, -np.nan, 1e-45, -1e-45, 3.4e38):
            x[:, :, rng.integers(0, N, 20)] = v
    else:
        raise KeyError(kind)
    return x.astype(np.float32)


@pytest.mark.parametrize("kind", ["uniform", "dirichlet", "quantized", "equal", "zeros", "signed", "special"])
def test_topk_bit_exact(kind):
    B, N, k = 4, 5000, 512
    _compare(_scores(kind, B, N, 1), _scores(kind, B, N, 2), [N] * B, k)


@pytest.mark.parametrize("N", [21, 33, 1000, 4097, 32768, 131072, 1 << 19])
def test_topk_lengths(N):
    k = min(2048, max(20, N // 8))
    _compare(_scores("uniform", 2, N, N), _scores("dirichlet", 2, N, N + 1), [N, N - 1], k)


def test_topk_short_sequences_take_all():
    N = 600
    _compare(_scores("uniform", 3, N, 3), _scores("uniform", 3, N, 4), [600, 100, 0], 256)


def test_topk_variants_target_only_and_draft_only():
    B, N, k = 2, 3000, 300
    sd, st = _scores("uniform", B, N, 5), _scores("uniform", B, N, 6)
    _compare(None, st, [N] * B, k, m_scalar=0)
    _compare(sd, None, [N] * B, k, m_scalar=k - 20)
    _compare(sd, st, [N] * B, k, m_scalar=0)
    _compare(sd, st, [N] * B, k, m_scalar=k - 20)


def test_topk_per_sequence_budget_m_and_groups():
    B, G, N = 3, 8, 4096
    rng = np.random.default_rng(9)
    sd = _scores("uniform", B, N, 7)                           # broadcast over groups
    st = rng.random((B, G, N)).astype(np.float32)
    seq = [4096, 3000, 50]
    budget = [256, 300, 64]
    m = [100, 0, 22]
    _compare(sd, st, seq, 320, budget=budget, m=m, groups=G)


def test_topk_streaming_llm_closed_form():
    """n_window = k - 4 with m = 0 gives sinks + the most recent k - 4 positions."""
    N, k = 10000, 256
    idx, cnt = _compare(None, _scores("uniform", 1, N, 8), [N], k, m_scalar=0, nw=k - 4)
    assert idx[0, 0, :k].tolist() == list(range(4)) + list(range(N - k + 4, N))


def test_topk_deterministic_repeat():
    B, N, k = 16, 32768, 2048
    sd, st = _scores("quantized", B, N, 10), _scores("zeros", B, N, 11)
    a, _ = _compare(sd, st, [N] * B, k)
    b, _ = _compare(sd, st, [N] * B, k)
    assert np.array_equal(a, b)


def test_topk_calls_of_different_shapes_in_turn():
    """Calls of different (batch, groups, length) in turn each match the oracle."""
    shapes = [(2, 1, 40000, 1500), (5, 4, 6000, 300), (2, 1, 40000, 1500), (1, 2, 3000, 64)]
    for t, (B, G, N, k) in enumerate(shapes):
        sd = _scores("uniform", B, N, 30 + t)
        st = np.random.default_rng(40 + t).random((B, G, N)).astype(np.float32)
        _compare(sd, st, [N - b for b in range(B)], k, groups=G)


def test_topk_workspace_reused_by_a_call_with_more_rows():
    """A workspace that served long rows (its bitmaps written) serves a later call with
    more rows and a smaller total size: the arrival counters of every row still start at
    zero (they live in a region of fixed size at the start)."""
    shapes = [(4, 1, 131072, 2048), (16, 8, 1000, 128), (4, 1, 131072, 2048), (16, 8, 1000, 128)]
    sizes = [D.lib().dustin_topk_workspace(B, G, N) for B, G, N, _ in shapes]
    assert sizes[1] < sizes[0]          # the second call reuses the first call's buffer
    for t, (B, G, N, k) in enumerate(shapes):
        sd = _scores("uniform", B, N, 80 + t)
        st = np.random.default_rng(90 + t).random((B, G, N)).astype(np.float32)
        _compare(sd, st, [N - b for b in range(B)], k, groups=G)


def test_topk_many_rows_run_the_tiers_in_turn():
    """Beyond 4096 (sequence, group) rows there is no hand-off workspace: each row's two
    tiers run one after the other in one workgroup."""
    B, G, N, k = 520, 8, 300, 64
    assert D.lib().dustin_topk_workspace(B, G, N) == 0
    sd = _scores("dirichlet", B, N, 95)
    st = np.random.default_rng(96).random((B, G, N)).astype(np.float32)
    _compare(sd, st, [N - (b % 50) for b in range(B)], k, groups=G)


def test_topk_rows_whose_low_address_word_is_above_two_gib():
    """Score rows placed where the low 32 bits of their address have bit 31 set: the kernel
    rebuilds each row's address from two 32-bit halves, and the low half must not be
    sign-extended into the high one."""
    B, N, k = 2, 40000, 1024
    sd, st = _scores("uniform", B, N, 97), _scores("dirichlet", B, N, 98)
    span = B * N * 4
    pool = torch.empty((1 << 32) + 2 * span + 4096, dtype=torch.uint8, device=DEV)
    base = pool.data_ptr()
    off = ((0x80000100 - (base & 0xFFFFFFFF)) % (1 << 32))  # low word 0x80000100, 256-byte aligned
    assert (base + off) % 256 == 0 and ((base + off) & 0xFFFFFFFF) >= 0x80000000
    views = []
    for j, a in enumerate((sd, st)):
        v = pool[off + j * span: off + (j + 1) * span].view(torch.float32).view(B, 1, N)
        v.copy_(torch.from_numpy(a))
        views.append(v)
    P = 20
    idx_ref, cnt_ref = O.select(sd, st, [N, N - 7], k, m_scalar=(k - P) // 2, n_sink=4, n_window=16)
    idx_g, cnt_g = D.topk(views[0], views[1], torch.tensor([N, N - 7], dtype=torch.int32, device=DEV), k,
                          m_scalar=(k - P) // 2, n_sink=4, n_window=16)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(cnt_g.cpu().numpy(), cnt_ref)
    for b in range(B):
        c = cnt_ref[b, 0]
        np.testing.assert_array_equal(idx_g.cpu().numpy()[b, 0, :c], idx_ref[b, 0, :c])
    del pool, views
