"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

Each test checks the oracle against something other than itself: the paper's printed
worked example, closed forms, invariants, special cases that reduce to a library routine,
brute-force enumeration on tiny inputs.  They are chosen so that a plausible mistake in the
oracle (a dropped term, a wrong sign or scale, a wrong head-to-KV-head index, a transposed
operand, a wrong tie or tier order, an off-by-one in the causal window) fails at least one.
"""
import itertools
import math
import os

import numpy as np
import pytest
import torch

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def bits(x):
    """float array -> bf16 bit patterns (round to nearest even)."""
    t = torch.as_tensor(np.asarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def val(b):
    return torch.from_numpy(b.view(np.int16).copy()).view(torch.bfloat16).double().numpy()


def rand_bits(rng, shape, scale=1.0):
    return bits(rng.standard_normal(shape) * scale)


# ----------------------------------------------------------------------------- basics

def test_bf16_decode_known_patterns():
    assert O.bf16_to_float(0x3F80) == 1.0
    assert O.bf16_to_float(0xC000) == -2.0
    assert O.bf16_to_float(0x0000) == 0.0
    assert math.copysign(1.0, O.bf16_to_float(0x8000)) == -1.0
    assert O.bf16_to_float(0x7F80) == math.inf
    assert O.bf16_to_float(0x0001) == 2.0 ** -133          # smallest bf16 subnormal
    assert O.bf16_to_float(0x4049) == 3.140625


def test_order_key_matches_float_order():
    rng = np.random.default_rng(0)
    vals = list(rng.standard_normal(300).astype(np.float32)) + [
        0.0, -0.0, np.inf, -np.inf, 1e-45, -1e-45, 1e-38, -1e-38, 3.4e38, -3.4e38]
    vals = [np.float32(v) for v in vals]
    for a, b in itertools.product(vals[:60] + vals[-10:], repeat=2):
        ka, kb = O.order_key(a), O.order_key(b)
        if a > b:
            assert ka > kb
        elif a < b:
            assert ka < kb
        else:                                   # includes +0 == -0
            assert ka == kb
    nan = np.float32(np.nan)
    assert O.order_key(nan) > O.order_key(np.float32(np.inf))
    assert O.order_key(-nan) < O.order_key(np.float32(-np.inf))


def test_overhead_ratio_worked_example():
    """Appendix A: (4*3*4 + 4*1*1) / (14*24*4 + 64*80*1) = 52 / 6464 ~ 0.8 %."""
    row = [ln for ln in open(os.path.join(GOLDEN, "overhead_ratio.txt")) if not ln.startswith("#")]
    f = row[0].split()
    args = [int(x) for x in f[:9]]
    num, den, pct = int(f[9]), int(f[10]), float(f[11])
    r = O.overhead_ratio(*args)
    assert r == num / den
    assert round(100 * r, 1) == pct


# ----------------------------------------------------------------------------- score (Eq. 5)

def _score_one(q, k, N, nq, heads, scale, Hkv=None, groups=1, init=None):
    B = q.shape[0]
    return O.score(q, k, [N] * B, [nq] * B, heads, scale, num_kv_heads=Hkv, groups=groups,
                   init=init)


def test_score_equal_keys_closed_form():
    """All keys equal: each softmax is exactly 1/N, so S = init + nq * |H| / N."""
    rng = np.random.default_rng(1)
    B, nq, Hq, Hkv, d, N = 2, 3, 4, 2, 16, 37
    q = rand_bits(rng, (B, nq, Hq, d))
    k = np.repeat(rand_bits(rng, (B, 1, Hkv, d)), N, axis=1)
    init = rng.random((B, 1, N)).astype(np.float32)
    heads = [0, 3]
    s = _score_one(q, k, N, nq, heads, 0.25, init=init.copy())
    want = (init.astype(np.float64) + nq * len(heads) / N).astype(np.float32)
    np.testing.assert_array_equal(s, want)


def test_score_two_tokens_is_logistic():
    """N = 2, one head, one query: S[0] = 1 / (1 + exp(l1 - l0))."""
    q = bits(np.array([1, 2, -1, 0], dtype=np.float64).reshape(1, 1, 1, 4))
    k = bits(np.array([[1, 0, 1, 2], [-2, 1, 0, 1]], dtype=np.float64).reshape(1, 2, 1, 4))
    s = _score_one(q, k, 2, 1, [0], 0.5)
    l0, l1 = 0.5 * (1 + 0 - 1 + 0), 0.5 * (-2 + 2 + 0 + 0)
    assert s[0, 0, 0] == np.float32(1 / (1 + math.exp(l1 - l0)))
    assert s[0, 0, 1] == np.float32(1 / (1 + math.exp(l0 - l1)))


def test_score_log_ratio_is_scaled_logit_difference():
    """One head, one query: log(S[a] / S[b]) = scale * q . (K[a] - K[b]).  Integer-valued
    q, K make the dot products exact, so the expected ratio is known independently."""
    rng = np.random.default_rng(2)
    d, N, Hq, Hkv, h = 8, 50, 4, 2, 3
    qi = rng.integers(-2, 3, (1, 1, Hq, d)).astype(np.float64)
    ki = rng.integers(-2, 3, (1, N, Hkv, d)).astype(np.float64)
    scale = 0.3
    s = _score_one(bits(qi), bits(ki), N, 1, [h], scale).astype(np.float64)[0, 0]
    g = h // (Hq // Hkv)
    dots = ki[0, :, g, :] @ qi[0, 0, h, :]
    for a, b in [(0, 1), (5, 17), (49, 3)]:
        assert math.log(s[a] / s[b]) == pytest.approx(scale * (dots[a] - dots[b]), abs=1e-6)


def test_score_row_sum_invariant_and_domain():
    """sum_n (S - init) = nq * |H| over [0, N_b); rows past N_b (set huge here) are neither
    read into the softmax nor written."""
    rng = np.random.default_rng(3)
    B, nq, Hq, Hkv, d, Ncap = 3, 4, 6, 3, 32, 64
    lens = [64, 40, 17]
    q = rand_bits(rng, (B, nq, Hq, d))
    kf = rng.standard_normal((B, Ncap, Hkv, d))
    for b, n in enumerate(lens):
        kf[b, n:] = 40.0
    k = bits(kf)
    out = np.full((B, 1, Ncap), -7.0, dtype=np.float32)
    heads = [1, 2, 5]
    O.score(q, k, lens, [nq] * B, heads, 1 / math.sqrt(d), out=out)
    for b, n in enumerate(lens):
        assert out[b, 0, :n].astype(np.float64).sum() == pytest.approx(nq * len(heads), rel=1e-6)
        assert np.all(out[b, 0, n:] == -7.0)
        assert np.all(out[b, 0, :n] > 0)


def test_score_query_count_per_sequence():
    """Each sequence sums over its own n_query[b] queries only."""
    rng = np.random.default_rng(4)
    B, Hq, d, N = 2, 2, 16, 30
    q = rand_bits(rng, (B, 5, Hq, d))
    k = rand_bits(rng, (B, N, 1, d))
    s = O.score(q, k, [N, N], [5, 2], [0, 1], 0.2)
    assert s[0, 0].astype(np.float64).sum() == pytest.approx(10, rel=1e-6)
    assert s[1, 0].astype(np.float64).sum() == pytest.approx(4, rel=1e-6)


def test_score_gqa_head_to_kv_head_map():
    """Query head h reads KV head h // (Hq/Hkv): plant one dominant key per KV head at a
    distinct position and check where each head's mass lands."""
    d, N, Hq, Hkv = 16, 40, 8, 4
    qf = np.ones((1, 1, Hq, d))
    kf = np.zeros((1, N, Hkv, d))
    for g in range(Hkv):
        kf[0, 10 + 5 * g, g, :] = 4.0
    q, k = bits(qf), bits(kf)
    for h in range(Hq):
        s = _score_one(q, k, N, 1, [h], 1.0)[0, 0]
        assert int(np.argmax(s)) == 10 + 5 * (h // (Hq // Hkv))
        assert s[10 + 5 * (h // 2)] > 0.999


def test_score_matches_library_softmax():
    """Tiny shapes: the same sum formed with torch's fp64 softmax over q K^T."""
    rng = np.random.default_rng(5)
    B, nq, Hq, Hkv, d, N = 2, 3, 6, 2, 16, 23
    q = rand_bits(rng, (B, nq, Hq, d))
    k = rand_bits(rng, (B, N, Hkv, d))
    heads, scale = [0, 4, 5], 0.3
    init = rng.random((B, 1, N)).astype(np.float32)
    s = _score_one(q, k, N, nq, heads, scale, init=init.copy())
    qv, kv = torch.from_numpy(val(q)), torch.from_numpy(val(k))
    for b in range(B):
        acc = torch.from_numpy(init[b, 0].astype(np.float64))
        for h in heads:
            g = h // (Hq // Hkv)
            acc = acc + torch.softmax(scale * (qv[b, :, h, :] @ kv[b, :, g, :].T), dim=-1).sum(0)
        np.testing.assert_allclose(s[b, 0], acc.numpy().astype(np.float32), rtol=2e-7, atol=0)


def test_score_heads_are_additive_and_init_chains():
    """Scoring {a, b} at once equals scoring {a} and feeding it as init to scoring {b}."""
    rng = np.random.default_rng(6)
    B, nq, Hq, d, N = 1, 2, 4, 16, 29
    q = rand_bits(rng, (B, nq, Hq, d))
    k = rand_bits(rng, (B, N, 2, d))
    both = _score_one(q, k, N, nq, [1, 3], 0.25)
    first = _score_one(q, k, N, nq, [1], 0.25)
    chained = _score_one(q, k, N, nq, [3], 0.25, init=first)
    np.testing.assert_allclose(both, chained, rtol=3e-7, atol=1e-9)


def test_score_per_group_output():
    """groups == Hkv: group go sums only the scoring heads whose KV head is go; a group
    with no scoring head keeps init."""
    rng = np.random.default_rng(7)
    B, nq, Hq, Hkv, d, N = 1, 2, 8, 4, 16, 33
    q = rand_bits(rng, (B, nq, Hq, d))
    k = rand_bits(rng, (B, N, Hkv, d))
    init = rng.random((B, Hkv, N)).astype(np.float32)
    heads = [0, 1, 6]                                   # KV heads 0, 0, 3
    s = _score_one(q, k, N, nq, heads, 0.25, Hkv=Hkv, groups=Hkv, init=init.copy())
    for go, hs in [(0, [0, 1]), (3, [6])]:
        ref = _score_one(q, k, N, nq, hs, 0.25, init=init[:, go:go + 1].copy())
        np.testing.assert_array_equal(s[:, go:go + 1], ref)
    for go in (1, 2):
        np.testing.assert_array_equal(s[0, go], init[0, go])


# ----------------------------------------------------------------------------- select (Eq. 6)

def _sel(sd, st, N, k, m, G=1, ns=4, nw=16):
    B = sd.shape[0] if sd is not None else st.shape[0]
    idx, cnt = O.select(sd, st, [N] * B, k, m_scalar=m, n_sink=ns, n_window=nw, groups=G)
    return [sorted(idx[b, g, :cnt[b, g]].tolist()) for b in range(B) for g in range(G)], cnt


def _full_sort_reference(sd, st, N, k, m, ns=4, nw=16):
    """Eq. 6 with Python's stable sort as the TopK."""
    if N <= k:
        return list(range(N))
    prot = set(range(ns)) | set(range(N - nw, N))
    cand = [n for n in range(N) if n not in prot]
    d_sel = sorted(cand, key=lambda n: (-float(sd[n]), n))[:m] if sd is not None else []
    rest = [n for n in cand if n not in set(d_sel)]
    t_sel = sorted(rest, key=lambda n: (-float(st[n]), n))[:k - m - len(prot)] if st is not None else []
    return sorted(prot | set(d_sel) | set(t_sel))


@pytest.mark.parametrize("kind", ["random", "quantized", "equal", "zeros", "negative"])
def test_select_matches_full_sort(kind):
    rng = np.random.default_rng(hash(kind) % 1000)
    B, N, k, m = 3, 300, 64, 17
    if kind == "random":
        sd, st = rng.random((B, 1, N)), rng.random((B, 1, N))
    elif kind == "quantized":
        sd, st = rng.integers(0, 4, (B, 1, N)) / 4, rng.integers(0, 3, (B, 1, N)) / 3
    elif kind == "equal":
        sd, st = np.ones((B, 1, N)), np.ones((B, 1, N))
    elif kind == "zeros":
        sd = np.where(rng.random((B, 1, N)) < 0.9, 0.0, rng.random((B, 1, N)))
        st = np.where(rng.random((B, 1, N)) < 0.95, -0.0, rng.random((B, 1, N)))
    else:
        sd, st = -rng.random((B, 1, N)), -np.abs(rng.standard_normal((B, 1, N)))
    sd, st = sd.astype(np.float32), st.astype(np.float32)
    got, cnt = _sel(sd, st, N, k, m)
    for b in range(B):
        assert got[b] == _full_sort_reference(sd[b, 0], st[b, 0], N, k, m)
        assert cnt[b, 0] == k


def test_select_brute_force_subsets():
    """Tiny N with distinct values: the draft tier is the m-subset of the unprotected
    positions with the largest S_D sum; the target tier is then the subset of what is left
    with the largest S_T sum (enumerated, no sorting involved)."""
    rng = np.random.default_rng(11)
    ns, nw = 2, 3
    for trial in range(20):
        N, k = 11, 8
        m = int(rng.integers(0, k - ns - nw + 1))
        sd = rng.permutation(N).astype(np.float32)[None, None, :] * 0.5 - 1
        st = rng.permutation(N).astype(np.float32)[None, None, :] * 0.25 + 3
        got, _ = _sel(sd, st, N, k, m, ns=ns, nw=nw)
        prot = set(range(ns)) | set(range(N - nw, N))
        cand = [n for n in range(N) if n not in prot]
        best_d = max(itertools.combinations(cand, m), key=lambda c: sum(sd[0, 0, list(c)]))
        rest = [n for n in cand if n not in best_d]
        nt = k - m - len(prot)
        best_t = max(itertools.combinations(rest, nt), key=lambda c: sum(st[0, 0, list(c)]))
        assert got[0] == sorted(prot | set(best_d) | set(best_t)), trial


def test_select_invariants_and_threshold():
    rng = np.random.default_rng(12)
    B, N, k, m, ns, nw = 4, 1000, 200, 70, 4, 16
    sd = rng.random((B, 1, N)).astype(np.float32)
    st = rng.integers(0, 50, (B, 1, N)).astype(np.float32)     # many ties
    idx, cnt = O.select(sd, st, [N] * B, k, m_scalar=m, n_sink=ns, n_window=nw)
    for b in range(B):
        sel = idx[b, 0, :cnt[b, 0]]
        assert cnt[b, 0] == k
        assert np.all(np.diff(sel) > 0)                           # ascending, distinct
        prot = set(range(ns)) | set(range(N - nw, N))
        assert prot <= set(sel.tolist())
        cand = [n for n in range(N) if n not in prot]
        chosen = set(sel.tolist()) - prot
        # draft tier = the m best candidates by (S_D desc, n asc)
        d_tier = sorted(chosen, key=lambda n: (-sd[b, 0, n], n))
        d_set = set(sorted(cand, key=lambda n: (-sd[b, 0, n], n))[:m])
        assert d_set <= chosen
        t_set = chosen - d_set
        assert len(t_set) == k - m - len(prot)
        unchosen = [n for n in cand if n not in chosen]
        tmin = min(st[b, 0, n] for n in t_set)
        for n in unchosen:                                        # threshold property
            assert st[b, 0, n] <= tmin
            if st[b, 0, n] == tmin:                               # ties go to lower index
                assert all(j < n for j in t_set if st[b, 0, j] == tmin)
        assert len(d_tier) == k - len(prot)


def test_select_streaming_llm_closed_form():
    """n_window = k - 4, m = 0 gives StreamingLLM's 4 sinks + the most recent k - 4 tokens
    (Appendix C)."""
    rng = np.random.default_rng(13)
    N, k = 500, 64
    st = rng.random((1, 1, N)).astype(np.float32)
    got, _ = _sel(None, st, N, k, 0, ns=4, nw=k - 4)
    assert got[0] == list(range(4)) + list(range(N - k + 4, N))


def test_select_variants_T_and_D():
    """m = 0 with no S_D is target-only selection; m = k - |P| with no S_T is draft-only;
    each equals a single TopK of its own signal over the unprotected positions."""
    rng = np.random.default_rng(14)
    N, k = 400, 100
    sd = rng.random((1, 1, N)).astype(np.float32)
    st = rng.random((1, 1, N)).astype(np.float32)
    got_t, _ = _sel(None, st, N, k, 0)
    assert got_t[0] == _full_sort_reference(None, st[0, 0], N, k, 0)
    got_d, _ = _sel(sd, None, N, k, k - 20)
    assert got_d[0] == _full_sort_reference(sd[0, 0], None, N, k, k - 20)
    both_t, _ = _sel(sd, st, N, k, 0)
    assert both_t == got_t
    both_d, _ = _sel(sd, st, N, k, k - 20)
    assert both_d == got_d


def test_select_short_sequences_take_everything():
    st = np.random.default_rng(15).random((3, 1, 64)).astype(np.float32)
    idx, cnt = O.select(st, st, [64, 30, 1], 64, m_scalar=10)
    assert cnt[:, 0].tolist() == [64, 30, 1]
    assert idx[1, 0, :30].tolist() == list(range(30))


def test_select_per_sequence_budget_and_broadcast_groups():
    rng = np.random.default_rng(16)
    B, G, N = 2, 3, 300
    sd = rng.random((B, 1, N)).astype(np.float32)                # broadcast over groups
    st = rng.random((B, G, N)).astype(np.float32)
    budget, m = [50, 80], [10, 30]
    idx, cnt = O.select(sd, st, [N, N], 80, budget=budget, m=m, groups=G)
    for b in range(B):
        for g in range(G):
            assert cnt[b, g] == budget[b]
            assert idx[b, g, :budget[b]].tolist() == _full_sort_reference(
                sd[b, 0], st[b, g], N, budget[b], m[b])


def test_select_rejects_invalid_budget():
    st = np.ones((1, 1, 100), dtype=np.float32)
    with pytest.raises(ValueError):
        O.select(st, st, [100], 19, m_scalar=0)                  # k < sinks + window
    with pytest.raises(ValueError):
        O.select(st, st, [100], 40, m_scalar=21)                 # m > k - |P|
    with pytest.raises(ValueError):
        O.select(None, st, [100], 40, m_scalar=3)                # no S_D needs m = 0


# ----------------------------------------------------------------------------- attention

def _attn(q, k, v, lens, scale, rows, idx=None, cnt=None):
    return O.attention(q, k, v, lens, scale, rows, idx=idx, count=cnt)


def test_attention_constant_values():
    """Constant V rows: every convex combination returns that row."""
    rng = np.random.default_rng(21)
    B, T, Hq, Hkv, d, N = 2, 3, 4, 2, 8, 20
    q = rand_bits(rng, (B, T, Hq, d))
    k = rand_bits(rng, (B, N + T, Hkv, d))
    row = rng.integers(-4, 5, d).astype(np.float64)
    v = bits(np.broadcast_to(row, (B, N + T, Hkv, d)))
    rows = O.all_rows(B, [T] * B, Hq)
    out = _attn(q, k, v, [N] * B, 0.5, rows)
    np.testing.assert_allclose(out, np.broadcast_to(row, out.shape), rtol=0, atol=1e-12)


def test_attention_equal_keys_is_mean_over_attended_set():
    """Equal keys: weights are uniform over J = selected set + causal window."""
    rng = np.random.default_rng(22)
    B, T, Hq, d, N = 1, 4, 2, 8, 30
    q = rand_bits(rng, (B, T, Hq, d))
    k = np.repeat(rand_bits(rng, (B, 1, 1, d)), N + T, axis=1)
    v = rand_bits(rng, (B, N + T, 1, d))
    vv = val(v)
    idx = np.array([[[1, 5, 9, 22]]], dtype=np.int32)
    cnt = np.array([[4]], dtype=np.int32)
    rows = O.all_rows(B, [T], Hq)
    out = _attn(q, k, v, [N], 0.7, rows, idx, cnt)
    for r, (b, t, h) in enumerate(rows):
        J = [1, 5, 9, 22] + [N + u for u in range(t + 1)]
        np.testing.assert_allclose(out[r], vv[0, J, 0].mean(0), rtol=0, atol=1e-12)


def test_attention_two_tokens_logistic():
    """Dense, N = 1, t = 0: J = {0, N}: weights are the logistic of the logit gap."""
    q = bits(np.array([1, -1, 2, 0.5]).reshape(1, 1, 1, 4))
    k = bits(np.array([[2, 0, 1, 0], [0, 1, -1, 2]]).reshape(1, 2, 1, 4))
    v = bits(np.array([[1, 2, 3, 4], [-4, 0, 8, 1]]).reshape(1, 2, 1, 4))
    out = _attn(q, k, v, [1], 0.5, [(0, 0, 0)])
    l0, l1 = 0.5 * (2 + 0 + 2 + 0), 0.5 * (0 - 1 - 2 + 1)
    w0 = 1 / (1 + math.exp(l1 - l0))
    want = w0 * np.array([1, 2, 3, 4]) + (1 - w0) * np.array([-4, 0, 8, 1])
    np.testing.assert_allclose(out[0], want, rtol=1e-14, atol=1e-14)


def test_attention_dominant_key_selects_its_value():
    rng = np.random.default_rng(23)
    d, N = 16, 50
    q = bits(np.ones((1, 1, 1, d)))
    kf = rng.standard_normal((1, N + 1, 1, d)) * 0.1
    kf[0, 17] = 8.0
    k, v = bits(kf), rand_bits(rng, (1, N + 1, 1, d))
    out = _attn(q, k, v, [N], 1.0, [(0, 0, 0)])
    np.testing.assert_allclose(out[0], val(v)[0, 17, 0], atol=1e-12)


def test_attention_causal_window():
    """Query t sees verification tokens N_b + u for u <= t only."""
    rng = np.random.default_rng(24)
    B, T, Hq, d, N = 1, 5, 2, 16, 40
    q = rand_bits(rng, (B, T, Hq, d))
    k = rand_bits(rng, (B, N + T, 1, d))
    v = rand_bits(rng, (B, N + T, 1, d))
    rows = O.all_rows(B, [T], Hq)
    base = _attn(q, k, v, [N], 0.25, rows)
    for u in range(T):
        v2 = v.copy()
        v2[0, N + u] = bits(np.full(d, 50.0))
        out = _attn(q, k, v2, [N], 0.25, rows)
        for r, (_, t, _) in enumerate(rows):
            if t < u:
                np.testing.assert_array_equal(out[r], base[r])
            else:
                assert np.abs(out[r] - base[r]).max() > 1e-3


def test_attention_full_budget_sparse_equals_dense_bitwise():
    rng = np.random.default_rng(25)
    B, T, Hq, Hkv, d, N = 2, 3, 4, 2, 16, 45
    q = rand_bits(rng, (B, T, Hq, d))
    k = rand_bits(rng, (B, N + T, Hkv, d))
    v = rand_bits(rng, (B, N + T, Hkv, d))
    rows = O.all_rows(B, [T] * B, Hq)
    dense = _attn(q, k, v, [N] * B, 0.2, rows)
    idx = np.broadcast_to(np.arange(N, dtype=np.int32), (B, Hkv, N)).copy()
    cnt = np.full((B, Hkv), N, dtype=np.int32)
    sparse = _attn(q, k, v, [N] * B, 0.2, rows, idx, cnt)
    np.testing.assert_array_equal(dense, sparse)


def test_attention_matches_library_sdpa():
    """Tiny shapes: torch's fp64 scaled_dot_product_attention over the gathered rows with
    an explicit causal mask on the verification tokens."""
    rng = np.random.default_rng(26)
    B, T, Hq, Hkv, d, N = 2, 4, 6, 2, 16, 33
    q = rand_bits(rng, (B, T, Hq, d))
    k = rand_bits(rng, (B, N + T, Hkv, d))
    v = rand_bits(rng, (B, N + T, Hkv, d))
    idx = np.zeros((B, Hkv, 12), dtype=np.int32)
    for b in range(B):
        for g in range(Hkv):
            idx[b, g] = np.sort(rng.choice(N, 12, replace=False))
    cnt = np.full((B, Hkv), 12, dtype=np.int32)
    rows = O.all_rows(B, [T] * B, Hq)
    scale = 1 / math.sqrt(d)
    got = _attn(q, k, v, [N] * B, scale, rows, idx, cnt).reshape(B, T, Hq, d)
    qv, kv, vv = (torch.from_numpy(val(x)) for x in (q, k, v))
    for b in range(B):
        for h in range(Hq):
            g = h // (Hq // Hkv)
            J = list(idx[b, g]) + [N + u for u in range(T)]
            mask = torch.ones((T, len(J)), dtype=torch.bool)
            for t in range(T):
                mask[t, 12 + t + 1:] = False
            ref = torch.nn.functional.scaled_dot_product_attention(
                qv[b, :, h][None], kv[b, J, g][None], vv[b, J, g][None], attn_mask=mask[None],
                scale=scale)[0]
            np.testing.assert_allclose(got[b, :, h], ref.numpy(), rtol=1e-12, atol=1e-13)


def test_attention_gqa_isolation():
    """Changing KV head g alters exactly the query heads h with h // (Hq/Hkv) == g."""
    rng = np.random.default_rng(27)
    B, T, Hq, Hkv, d, N = 1, 2, 8, 4, 16, 25
    q = rand_bits(rng, (B, T, Hq, d))
    k = rand_bits(rng, (B, N + T, Hkv, d))
    v = rand_bits(rng, (B, N + T, Hkv, d))
    rows = O.all_rows(B, [T], Hq)
    base = _attn(q, k, v, [N], 0.3, rows)
    v2 = v.copy()
    v2[0, :, 2] = rand_bits(rng, (N + T, d))
    out = _attn(q, k, v2, [N], 0.3, rows)
    for r, (_, _, h) in enumerate(rows):
        changed = np.abs(out[r] - base[r]).max() > 0
        assert changed == (h // 2 == 2)


def test_attention_group_index_source():
    """G == Hkv reads each KV head's own index row; G == 1 reads row 0 for every head."""
    rng = np.random.default_rng(28)
    B, T, Hq, Hkv, d, N = 1, 1, 4, 2, 8, 30
    q = rand_bits(rng, (B, T, Hq, d))
    k = rand_bits(rng, (B, N + T, Hkv, d))
    v = rand_bits(rng, (B, N + T, Hkv, d))
    vv = val(v)
    kq = bits(np.zeros((B, N + T, Hkv, d)))                 # equal keys -> plain means
    idx = np.array([[[1, 2, 3], [10, 11, 12]]], dtype=np.int32)
    cnt = np.array([[3, 3]], dtype=np.int32)
    rows = O.all_rows(B, [T], Hq)
    per_g = _attn(q, kq, v, [N], 1.0, rows, idx, cnt)
    one = _attn(q, kq, v, [N], 1.0, rows, idx[:, :1].copy(), cnt[:, :1].copy())
    for r, (_, _, h) in enumerate(rows):
        g = h // 2
        np.testing.assert_allclose(per_g[r], vv[0, list(idx[0, g]) + [N], g].mean(0), atol=1e-12)
        np.testing.assert_allclose(one[r], vv[0, [1, 2, 3, N], g].mean(0), atol=1e-12)
    del k


# ----------------------------------------------------------------------------- ARR (Eqs. 1-4)

def test_arr_full_set_is_one_and_oracle_policy_is_upper_bound():
    """Eq. ARR window def / K orc def: selecting every position recovers all mass, and for
    any index set of size k the windowed ARR is at most that of TopK of the
    window-averaged attention (Eq. ARR orc)."""
    rng = np.random.default_rng(31)
    w, n, k = 4, 60, 9
    A = rng.random((w, n)) ** 4
    A /= A.sum(1, keepdims=True)
    assert O.arr_window(A, np.arange(n)) == pytest.approx(1.0, abs=1e-14)
    top = np.argsort(-A.mean(0), kind="stable")[:k]
    best = O.arr_window(A, top)
    assert best == pytest.approx(A.mean(0)[top].sum(), abs=1e-14)
    for _ in range(300):
        assert O.arr_window(A, rng.choice(n, k, replace=False)) <= best + 1e-15


def _softmax_rows(logits):
    z = torch.softmax(torch.from_numpy(logits), dim=-1)  # library softmax, fp64
    return z.numpy()


def test_arr_of_qk_matches_library_softmax_and_arr_window():
    """oracle_arr against the attention rows built with torch.softmax in fp64 and the
    separately pinned arr_window, per head, then the mean over the heads of each group."""
    rng = np.random.default_rng(44)
    B, w, Hq, Hkv, d, N = 2, 3, 4, 2, 8, 40
    q = rand_bits(rng, (B, w, Hq, d))
    k = rand_bits(rng, (B, N, Hkv, d))
    seq, win = [40, 23], [3, 2]
    idx = np.zeros((B, Hkv, 10), dtype=np.int32)
    cnt = np.zeros((B, Hkv), dtype=np.int32)
    for b in range(B):
        for g in range(Hkv):
            sel = np.sort(rng.choice(seq[b], 7, replace=False))
            idx[b, g, :7], cnt[b, g] = sel, 7
    got, abar = O.arr(q, k, seq, win, 0.3, groups=Hkv, idx=idx, count=cnt, with_abar=True, length=N)
    qv, kv = val(q), val(k)
    for b in range(B):
        n, t = seq[b], win[b]
        for g in range(Hkv):
            heads = [h for h in range(Hq) if h // (Hq // Hkv) == g]
            per_head, mean_rows = [], np.zeros(n)
            for h in heads:
                A = _softmax_rows(0.3 * qv[b, :t, h] @ kv[b, :n, g].T)
                per_head.append(O.arr_window(A, idx[b, g, :cnt[b, g]]))
                mean_rows += A.mean(0) / len(heads)
            assert got[b, g] == pytest.approx(np.mean(per_head), abs=1e-12)
            np.testing.assert_allclose(abar[b, g, :n], mean_rows, atol=1e-14)


def test_arr_closed_forms_and_oracle_bound():
    """The full set recovers everything; the empty set nothing; A-bar sums to one; windowed
    ARR is linear in the set (sum of A-bar over it); and no set of size k beats TopK_k of
    A-bar (Eq. 4), checked over every subset of a tiny row."""
    rng = np.random.default_rng(45)
    B, w, Hq, Hkv, d, N, k = 1, 4, 2, 1, 8, 9, 3
    q = rand_bits(rng, (B, w, Hq, d), 2.0)
    kk = rand_bits(rng, (B, N, Hkv, d))
    full = np.arange(N, dtype=np.int32).reshape(1, 1, N)
    one, abar = O.arr(q, kk, [N], [w], 0.5, idx=full, count=[[N]], with_abar=True)
    assert one[0, 0] == pytest.approx(1.0, abs=1e-12)
    assert abar[0, 0].sum() == pytest.approx(1.0, abs=1e-12)
    assert O.arr(q, kk, [N], [w], 0.5)[0, 0] == 0.0
    best = -1.0
    for sub in itertools.combinations(range(N), k):
        ix = np.array(sub, dtype=np.int32).reshape(1, 1, k)
        v = O.arr(q, kk, [N], [w], 0.5, idx=ix, count=[[k]])[0, 0]
        assert v == pytest.approx(abar[0, 0, list(sub)].sum(), abs=1e-12)
        best = max(best, v)
    top = np.argsort(-abar[0, 0], kind="stable")[:k]
    assert best == pytest.approx(abar[0, 0, top].sum(), abs=1e-12)


def test_arr_dominant_key():
    """A key aligned with every window query takes nearly all mass: ARR is about 1 with it
    and about 0 without it."""
    rng = np.random.default_rng(46)
    w, d, N = 2, 16, 30
    qf = rng.standard_normal((1, w, 1, d))
    kf = rng.standard_normal((1, N, 1, d)) * 0.1
    kf[0, 11, 0] = 8.0 * qf[0].mean(0)[0]
    q, kk = bits(qf), bits(kf)
    with_key = O.arr(q, kk, [N], [w], 1.0, idx=np.array([[[11]]], dtype=np.int32), count=[[1]])[0, 0]
    others = np.array([[list(range(11)) + list(range(12, N))]], dtype=np.int32)
    without = O.arr(q, kk, [N], [w], 1.0, idx=others, count=[[N - 1]])[0, 0]
    assert with_key > 0.999 and without < 1e-3
    assert with_key + without == pytest.approx(1.0, abs=1e-12)


# ----------------------------------------------------------------------------- KV append / commit

def _kv_case(rng, B=3, cap=40, H=2, d=16, T=5):
    cache = rng.integers(0, 1 << 16, (B, cap, H, d), dtype=np.uint16)
    new = rng.integers(0, 1 << 16, (B, T, H, d), dtype=np.uint16)
    return cache, new


def test_kv_append_contiguous_is_a_splice():
    """Rows [N_b, N_b + T_b) become the window rows; every other row is unchanged (checked
    against a splice built from slices)."""
    rng = np.random.default_rng(1)
    cache, new = _kv_case(rng)
    seq, nq = [10, 0, 35], [5, 3, 5]     # the last sequence runs past the capacity (40)
    got = O.kv_append(cache, new, seq, nq)
    for b in range(3):
        N, T = seq[b], nq[b]
        keep = min(T, cache.shape[1] - N)
        want = np.concatenate([cache[b, :N], new[b, :keep], cache[b, N + keep:]])
        np.testing.assert_array_equal(got[b], want)


def test_kv_append_paged_matches_contiguous_through_the_page_table():
    rng = np.random.default_rng(2)
    B, ps, H, d, T = 3, 8, 2, 16, 6
    maxp = 5
    cache, new = _kv_case(rng, B=B, cap=maxp * ps, H=H, d=d, T=T)
    perm = rng.permutation(B * maxp).astype(np.int32)
    pt = perm.reshape(B, maxp)
    paged = np.zeros((B * maxp, ps, H, d), dtype=np.uint16)
    for b in range(B):
        for j in range(maxp):
            paged[pt[b, j]] = cache[b, j * ps:(j + 1) * ps]
    seq, nq = [7, 30, 16], [6, 6, 0]
    got = O.kv_append(paged, new, seq, nq, page_table=pt)
    want = O.kv_append(cache, new, seq, nq)
    for b in range(B):
        back = np.concatenate([got[pt[b, j]] for j in range(maxp)])
        np.testing.assert_array_equal(back, want[b])


def test_kv_commit_closed_form():
    seq = np.array([100, 0, 7, 9], np.int32)
    acc = np.array([3, -2, 9, 0], np.int32)
    nq = np.array([5, 4, 6, 2], np.int32)
    np.testing.assert_array_equal(O.kv_commit(seq, acc, nq), [103, 0, 13, 9])


# ----------------------------------------------------------------------------- page estimator

def test_page_meta_is_library_min_max_over_valid_positions():
    """Channel-wise max and min of K per page over positions < N_b, checked against numpy's
    max/min on the reshaped valid prefix; positions >= N_b hold huge values that must not leak."""
    rng = np.random.default_rng(40)
    B, N, Hkv, d, ps = 3, 70, 2, 8, 16
    kf = rng.standard_normal((B, N, Hkv, d))
    seq = [70, 33, 16]
    for b, n in enumerate(seq):
        kf[b, n:] = 1e30 * np.sign(rng.standard_normal((N - n, Hkv, d)))
    k = bits(kf)
    meta = O.page_meta(k, seq, ps)
    kv = val(k)
    for b, n in enumerate(seq):
        P = -(-n // ps)
        for p in range(P):
            blk = kv[b, p * ps:min(n, (p + 1) * ps)]
            np.testing.assert_array_equal(val(meta[b, p, :, :d]), blk.max(axis=0))
            np.testing.assert_array_equal(val(meta[b, p, :, d:]), blk.min(axis=0))
        assert not meta[b, P:].any()


def test_page_meta_earliest_pattern_of_equal_values():
    """-0 and +0 compare equal: the earliest position's pattern is kept, for max and min."""
    k = np.array([0x8000, 0x0000, 0x0000, 0x8000], dtype=np.uint16).reshape(1, 4, 1, 1)
    meta = O.page_meta(k, [4], 2)
    assert meta[0, 0, 0].tolist() == [0x8000, 0x8000] and meta[0, 1, 0].tolist() == [0x0000, 0x0000]


def test_page_score_hand_worked_example():
    """d = 2, page size 2, N = 3.  Page 0 holds keys (1, -2) and (3, 0.5): max (3, 0.5),
    min (1, -2).  For q = (1, -1): u0 = max(3, 1) + max(-0.5, 2) = 5.  Page 1 holds (-1, 1)
    alone: u1 = q . k = -2.  Softmax over the two pages at scale 1."""
    q = bits(np.array([1, -1], dtype=np.float64).reshape(1, 1, 1, 2))
    k = bits(np.array([[1, -2], [3, 0.5], [-1, 1]], dtype=np.float64).reshape(1, 3, 1, 2))
    meta = O.page_meta(k, [3], 2)
    s = O.page_score(q, meta, [3], [1], [0], 1.0, 2)[0, 0]
    p0 = 1 / (1 + math.exp(-2 - 5))
    assert s.tolist() == [np.float32(p0), np.float32(p0), np.float32(1 - p0)]


def test_page_score_page_size_one_is_eq5():
    """With one position per page min = max = K, the bound is q . k, and the page score is
    Eq. 5 itself: bit-identical to oracle.score (same fp64 sums, one rounding)."""
    rng = np.random.default_rng(41)
    B, nq, Hq, Hkv, d, N = 2, 3, 8, 2, 32, 45
    q = rand_bits(rng, (B, nq, Hq, d))
    k = rand_bits(rng, (B, N, Hkv, d))
    init = rng.random((B, Hkv, N)).astype(np.float32)
    seq, nqs, heads = [45, 20], [3, 2], [1, 4, 6]
    want = O.score(q, k, seq, nqs, heads, 0.2, groups=Hkv, init=init.copy())
    got = O.page_score(q, O.page_meta(k, seq, 1), seq, nqs, heads, 0.2, 1, groups=Hkv,
                       init=init.copy(), length=N)
    for b, n in enumerate(seq):
        np.testing.assert_array_equal(got[b, :, :n], want[b, :, :n])


def test_page_bound_dominates_every_key_of_its_page():
    """The page bound is an upper bound: q . k_n <= u(page of n) for every position, by
    brute force over the keys, with equality for a page whose keys are all equal."""
    rng = np.random.default_rng(42)
    N, d, ps = 64, 16, 8
    q = rand_bits(rng, (1, 1, 1, d))
    kf = rng.standard_normal((1, N, 1, d))
    kf[0, 8:16] = kf[0, 8]  # page 1: eight equal keys
    k = bits(kf)
    meta = O.page_meta(k, [N], ps)
    qv, kv, mv = val(q)[0, 0, 0], val(k)[0, :, 0], val(meta)[0, :, 0]
    u = np.array([np.maximum(qv * mv[p, :d], qv * mv[p, d:]).sum() for p in range(N // ps)])
    assert np.all(kv @ qv <= u[np.arange(N) // ps] + 1e-12)
    assert u[1] == pytest.approx(kv[8] @ qv, abs=1e-12)
    # the page scores are the softmax of u: log-ratios are differences of u
    s = O.page_score(q, meta, [N], [1], [0], 1.0, ps)[0, 0].astype(np.float64)
    assert math.log(s[0] / s[ps * 5]) == pytest.approx(u[0] - u[5], abs=1e-6)


def test_page_score_row_sum_and_broadcast():
    """Every position of a page carries the page's value; summing one position per page
    gives nq * |H(go)| per output group; positions past N_b are not written."""
    rng = np.random.default_rng(43)
    B, nq, Hq, Hkv, d, N, ps = 2, 2, 4, 2, 16, 50, 8
    q = rand_bits(rng, (B, nq, Hq, d))
    k = rand_bits(rng, (B, N, Hkv, d))
    seq = [50, 9]
    meta = O.page_meta(k, seq, ps)
    out = np.full((B, Hkv, N), -7.0, dtype=np.float32)
    O.page_score(q, meta, seq, [nq, 1], [0, 1, 3], 0.3, ps, groups=Hkv, out=out)
    for b, n in enumerate(seq):
        P = -(-n // ps)
        for go, nh in enumerate([2, 1]):  # heads 0, 1 read KV head 0; head 3 reads KV head 1
            row = out[b, go, :n].reshape(-1)
            for p in range(P):
                assert np.all(row[p * ps:min(n, (p + 1) * ps)] == row[p * ps])
            tot = sum(float(row[p * ps]) for p in range(P))
            assert tot == pytest.approx([nq, 1][b] * nh, abs=1e-5)
            assert np.all(out[b, go, n:] == -7.0)
