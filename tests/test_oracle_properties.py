"""Property tests of the oracle on random tiny inputs (hypothesis): facts that hold for every
input, checked over many shapes, lengths, budgets, ties and groupings rather than at fixed
seeds.  CPU only; the fixed-value pins are in test_oracle_pins.py."""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle as O

SETTINGS = settings(max_examples=40, deadline=None, suppress_health_check=[HealthCheck.too_slow])


def bits_of(x):
    """float array -> bf16 patterns (round to nearest even, finite inputs)."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return r.astype(np.uint16)


def val(b):
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


@st.composite
def selection_case(draw):
    B = draw(st.integers(1, 3))
    G = draw(st.sampled_from([1, 2]))
    ns, nw = draw(st.integers(0, 4)), draw(st.integers(0, 6))
    N = draw(st.integers(1, 96))
    k = draw(st.integers(ns + nw, ns + nw + 40))
    m = draw(st.integers(0, k - ns - nw))
    levels = draw(st.sampled_from([3, 17, 1000]))  # few levels: many exact ties
    seed = draw(st.integers(0, 2**31 - 1))
    rng = np.random.default_rng(seed)
    sd = (rng.integers(0, levels, (B, G, N)) / levels).astype(np.float32)
    stg = (rng.integers(0, levels, (B, G, N)) / levels).astype(np.float32)
    lens = [int(rng.integers(1, N + 1)) for _ in range(B)]
    return sd, stg, lens, k, m, ns, nw, G


def _sel(sd, stg, lens, k, m, ns, nw, G):
    return O.select(sd, stg, lens, k, m_scalar=m, n_sink=ns, n_window=nw, groups=G)


@SETTINGS
@given(selection_case())
def test_selection_shape_protected_set_and_order(case):
    sd, stg, lens, k, m, ns, nw, G = case
    idx, cnt = _sel(*case)
    for b, N in enumerate(lens):
        for g in range(G):
            c = int(cnt[b, g])
            assert c == min(k, N)
            sel = idx[b, g, :c]
            assert np.all(np.diff(sel) > 0) and (c == 0 or (sel[0] >= 0 and sel[-1] < N))
            prot = set(range(min(ns, N))) | set(range(max(0, N - nw), N))
            assert prot <= set(sel.tolist())


@SETTINGS
@given(selection_case(), st.sampled_from([0.25, 2.0, 8.0]))
def test_selection_is_invariant_to_exact_positive_rescaling(case, f):
    sd, stg, lens, k, m, ns, nw, G = case
    a = _sel(*case)
    b = _sel((sd * f).astype(np.float32), (stg * np.float32(f)).astype(np.float32), lens, k, m, ns, nw, G)
    assert np.array_equal(a[1], b[1])
    for bb, N in enumerate(lens):
        for g in range(G):
            c = int(a[1][bb, g])
            assert np.array_equal(a[0][bb, g, :c], b[0][bb, g, :c])


@SETTINGS
@given(selection_case())
def test_selection_grows_with_the_budget(case):
    """With m fixed, one more unit of budget adds exactly one position (the next of the
    target tier) and removes none."""
    sd, stg, lens, k, m, ns, nw, G = case
    a_idx, a_cnt = _sel(*case)
    b_idx, b_cnt = _sel(sd, stg, lens, k + 1, m, ns, nw, G)
    for b, N in enumerate(lens):
        for g in range(G):
            sa = set(a_idx[b, g, :a_cnt[b, g]].tolist())
            sb = set(b_idx[b, g, :b_cnt[b, g]].tolist())
            assert sa <= sb and len(sb) - len(sa) == (1 if N > k else 0)


@SETTINGS
@given(selection_case())
def test_target_only_selection_is_a_library_sort(case):
    """m = 0 without a draft score: the protected set plus the best free positions by
    (S_T desc, position asc), taken from numpy's lexsort."""
    _, stg, lens, k, _, ns, nw, G = case
    idx, cnt = O.select(None, stg, lens, k, m_scalar=0, n_sink=ns, n_window=nw, groups=G)
    for b, N in enumerate(lens):
        for g in range(G):
            if N <= k:
                want = list(range(N))
            else:
                prot = sorted(set(range(min(ns, N))) | set(range(max(0, N - nw), N)))
                free = np.array([n for n in range(N) if n not in prot], dtype=np.int64)
                order = free[np.lexsort((free, -stg[b, g, free].astype(np.float64)))]
                want = sorted(prot + order[:k - len(prot)].tolist())
            assert idx[b, g, :cnt[b, g]].tolist() == want


@st.composite
def attention_case(draw):
    Hkv = draw(st.sampled_from([1, 2]))
    G = draw(st.sampled_from([1, 2, 4]))
    Hq = Hkv * G
    d = draw(st.sampled_from([8, 16]))
    N = draw(st.integers(1, 40))
    T = draw(st.integers(1, 4))
    seed = draw(st.integers(0, 2**31 - 1))
    rng = np.random.default_rng(seed)
    q = bits_of(rng.standard_normal((1, T, Hq, d)) * draw(st.sampled_from([0.0, 0.5, 3.0])))
    k = bits_of(rng.standard_normal((1, N + T, Hkv, d)))
    v = bits_of(rng.standard_normal((1, N + T, Hkv, d)))
    return q, k, v, N, T, Hq, Hkv, d, rng


@SETTINGS
@given(attention_case())
def test_score_row_sums_and_uniform_for_zero_queries(case):
    q, k, _, N, T, Hq, Hkv, d, rng = case
    heads = sorted(set(rng.integers(0, Hq, 2).tolist()))
    s = O.score(q, k[:, :N], [N], [T], heads, 0.7)[0, 0]
    assert abs(s.astype(np.float64).sum() - T * len(heads)) <= 1e-5 * T * len(heads)
    if not val(q).any():  # all-zero queries: every position gets exactly nq |H| / N
        assert np.allclose(s, T * len(heads) / N, rtol=1e-6)


@SETTINGS
@given(attention_case())
def test_attention_output_is_a_convex_combination(case):
    """Each output channel lies between the smallest and largest value of that channel over
    the attended rows (selected set plus the causal window)."""
    q, k, v, N, T, Hq, Hkv, d, rng = case
    c = int(rng.integers(0, N + 1))
    sel = np.sort(rng.choice(N, c, replace=False)).astype(np.int32)
    idx = np.full((1, 1, max(c, 1)), -1, dtype=np.int32)
    idx[0, 0, :c] = sel
    rows = O.all_rows(1, [T], Hq)
    out = O.attention(q, k, v, [N], 0.5, rows, idx=idx, count=np.array([[c]], dtype=np.int32))
    vv = val(v)[0]
    for (_, t, h), o in zip(rows, out):
        g = h // (Hq // Hkv)
        att = np.concatenate([sel, np.arange(N, N + t + 1)])
        lo, hi = vv[att, g].min(axis=0), vv[att, g].max(axis=0)
        assert np.all(o >= lo - 1e-9) and np.all(o <= hi + 1e-9)


@SETTINGS
@given(attention_case(), st.sampled_from([1, 2, 4, 8]))
def test_page_bound_dominates_every_key(case, ps):
    q, k, _, N, T, Hq, Hkv, d, _ = case
    meta = O.page_meta(k[:, :N], [N], ps)
    qv, kv, mv = val(q)[0], val(k)[0], val(meta)[0]
    for t in range(T):
        for h in range(Hq):
            g = h // (Hq // Hkv)
            for n in range(N):
                p = n // ps
                u = np.maximum(qv[t, h] * mv[p, g, :d], qv[t, h] * mv[p, g, d:]).sum()
                assert kv[n, g] @ qv[t, h] <= u + 1e-9


@SETTINGS
@given(attention_case())
def test_arr_is_a_fraction_and_grows_with_the_set(case):
    q, k, _, N, T, Hq, Hkv, d, rng = case
    a = np.sort(rng.choice(N, int(rng.integers(0, N + 1)), replace=False))
    extra = rng.choice(N, int(rng.integers(0, N + 1)), replace=False)
    b = np.union1d(a, extra)

    def arr_of(s_):
        ix = np.full((1, 1, max(len(s_), 1)), -1, dtype=np.int32)
        ix[0, 0, :len(s_)] = s_
        return O.arr(q, k[:, :N], [N], [T], 0.5, idx=ix, count=np.array([[len(s_)]], dtype=np.int32))[0, 0]

    ra, rb = arr_of(a), arr_of(b)
    assert -1e-12 <= ra <= rb + 1e-12 and rb <= 1 + 1e-12
    if len(b) == N:
        assert rb == pytest.approx(1.0, abs=1e-12)
