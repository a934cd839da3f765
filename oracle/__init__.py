"""ctypes front end of the CPU oracle (oracle.c).

TEST INFRASTRUCTURE ONLY: the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline
leg of ``bench.py`` are its only users.  The product library never imports this package,
and this package imports nothing from the product.

All inputs are numpy arrays.  bf16 tensors are passed as their raw uint16 bit patterns
(``torch_bf16.view(torch.int16).numpy().view(numpy.uint16)``).  Arrays may be strided
views as long as the innermost axis is contiguous.
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# DUSTIN_ORACLE_LIB selects another build of oracle.c (the sanitizer build of the CPU suite)
_LIB_PATH = os.environ.get("DUSTIN_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
_lib = None

_i64 = ctypes.c_int64
_i32 = ctypes.c_int
_ptr = ctypes.c_void_p


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _build  # the checker may be compiled on demand
            _build.build()
        lib = ctypes.CDLL(_LIB_PATH)
        lib.oracle_score.restype = _i32
        lib.oracle_score.argtypes = [_ptr, _i64, _i64, _i64, _ptr, _i64, _i64, _i64,
                                     _i32, _ptr, _ptr, _i32, _i32, _i32, _ptr, _i32, _i32,
                                     ctypes.c_double, _ptr, _i64, _i64, _ptr, _i64, _i64]
        lib.oracle_select.restype = _i32
        lib.oracle_select.argtypes = [_ptr, _i64, _i64, _ptr, _i64, _i64, _i32, _i32, _ptr,
                                      _ptr, _i32, _ptr, _i32, _i32, _i32, _ptr, _i64, _i64, _ptr]
        lib.oracle_attention.restype = _i32
        lib.oracle_attention.argtypes = [_ptr, _i64, _i64, _i64, _ptr, _i64, _i64, _i64,
                                         _ptr, _i64, _i64, _i64, _i32, _i32, _i32, _ptr,
                                         _ptr, _i64, _i64, _ptr, _i32, ctypes.c_double,
                                         _i32, _ptr, _ptr, _ptr, _ptr]
        lib.oracle_order_key.restype = ctypes.c_uint32
        lib.oracle_order_key.argtypes = [ctypes.c_float]
        lib.oracle_bf16_to_double.restype = ctypes.c_double
        lib.oracle_bf16_to_double.argtypes = [ctypes.c_uint16]
        lib.oracle_arr_window.restype = ctypes.c_double
        lib.oracle_arr_window.argtypes = [_ptr, _i32, _i32, _ptr, _i32]
        lib.oracle_overhead_ratio.restype = ctypes.c_double
        lib.oracle_overhead_ratio.argtypes = [_i32] * 9
        lib.oracle_page_meta.restype = _i32
        lib.oracle_page_meta.argtypes = [_ptr, _i64, _i64, _i64, _i32, _ptr, _i32, _i32, _i32,
                                         _ptr, _i64, _i64, _i64]
        lib.oracle_page_score.restype = _i32
        lib.oracle_page_score.argtypes = [_ptr, _i64, _i64, _i64, _ptr, _i64, _i64, _i64, _i32,
                                          _ptr, _ptr, _i32, _i32, _i32, _i32, _ptr, _i32, _i32,
                                          ctypes.c_double, _ptr, _i64, _i64, _ptr, _i64, _i64]
        lib.oracle_arr.restype = _i32
        lib.oracle_arr.argtypes = [_ptr, _i64, _i64, _i64, _ptr, _i64, _i64, _i64, _i32, _ptr, _ptr,
                                   _i32, _i32, _i32, _i32, ctypes.c_double, _ptr, _i64, _i64, _ptr,
                                   _ptr, _ptr, _i64, _i64]
        lib.oracle_max_threads.restype = _i32
        lib.oracle_set_threads.argtypes = [_i32]
        _lib = lib
    return _lib


def _p(a):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def _st(a):
    """Element strides of a numpy array."""
    return [s // a.itemsize for s in a.strides]


def _check_inner(a, name):
    if a.strides[-1] != a.itemsize:
        raise ValueError(f"{name}: innermost axis must be contiguous")


def _i32arr(x, n=None):
    a = np.ascontiguousarray(np.asarray(x, dtype=np.int32))
    if n is not None and a.shape != (n,):
        raise ValueError(f"expected {n} entries, got shape {a.shape}")
    return a


def max_threads() -> int:
    return _load().oracle_max_threads()


def set_threads(n: int) -> None:
    _load().oracle_set_threads(int(n))


def order_key(x: float) -> int:
    return int(_load().oracle_order_key(float(x)))


def bf16_to_float(bits: int) -> float:
    return float(_load().oracle_bf16_to_double(int(bits)))


def score(q, k, seq_lens, n_query, heads, scale, num_kv_heads=None, groups=1, init=None,
          out=None):
    """Eq. 5 over the scoring heads.  q: uint16 [B, nq, Hq, d]; k: uint16 [B, N, Hkv, d];
    init/out: float32 [B, G, N] (out is created when None).  Returns out."""
    lib = _load()
    B, _, Hq, d = q.shape
    Hkv = k.shape[2] if num_kv_heads is None else num_kv_heads
    _check_inner(q, "q")
    _check_inner(k, "k")
    seq = _i32arr(seq_lens, B)
    nqa = _i32arr(n_query, B)
    hd = _i32arr(heads)
    if out is None:
        out = np.zeros((B, groups, k.shape[1]), dtype=np.float32)
    if init is not None:
        _check_inner(init, "init")
    _check_inner(out, "out")
    qs, ks, os_ = _st(q), _st(k), _st(out)
    ins = _st(init) if init is not None else [0, 0, 0]
    rc = lib.oracle_score(_p(q), qs[0], qs[1], qs[2], _p(k), ks[0], ks[1], ks[2],
                          B, _p(seq), _p(nqa), Hq, Hkv, d, _p(hd), len(hd), groups,
                          float(scale), _p(init), ins[0], ins[1], _p(out), os_[0], os_[1])
    if rc:
        raise ValueError(f"oracle_score rejected its arguments ({rc})")
    return out


def page_meta(k, seq_lens, page_size, num_pages=None):
    """Page key statistics (the Quest-style page estimator).  k: uint16 [B, N, Hkv, d].
    Returns uint16 [B, num_pages, Hkv, 2d]: per page, the channel-wise maximum then minimum
    of K over the page's positions below N_b; rows of pages past N_b stay zero."""
    lib = _load()
    B, N, Hkv, d = k.shape
    _check_inner(k, "k")
    seq = _i32arr(seq_lens, B)
    if num_pages is None:
        num_pages = (N + page_size - 1) // page_size
    meta = np.zeros((B, num_pages, Hkv, 2 * d), dtype=np.uint16)
    ks, ms = _st(k), _st(meta)
    rc = lib.oracle_page_meta(_p(k), ks[0], ks[1], ks[2], B, _p(seq), Hkv, d, int(page_size),
                              _p(meta), ms[0], ms[1], ms[2])
    if rc:
        raise ValueError(f"oracle_page_meta rejected its arguments ({rc})")
    return meta


def page_score(q, meta, seq_lens, n_query, heads, scale, page_size, groups=1, init=None,
               out=None, length=None):
    """Page-estimator importance: Eq. 5 over pages with each page's key bound in place of
    q . k, broadcast to the page's positions.  q: uint16 [B, nq, Hq, d]; meta: uint16
    [B, P, Hkv, 2d] from page_meta; init/out float32 [B, G, >= max N_b]."""
    lib = _load()
    B, _, Hq, d = q.shape
    Hkv = meta.shape[2]
    _check_inner(q, "q")
    _check_inner(meta, "meta")
    seq = _i32arr(seq_lens, B)
    nqa = _i32arr(n_query, B)
    hd = _i32arr(heads)
    if out is None:
        n_out = length if length is not None else max(int(seq.max(initial=0)), 1)
        out = np.zeros((B, groups, n_out), dtype=np.float32)
    if init is not None:
        _check_inner(init, "init")
    _check_inner(out, "out")
    qs, ms, os_ = _st(q), _st(meta), _st(out)
    ins = _st(init) if init is not None else [0, 0, 0]
    rc = lib.oracle_page_score(_p(q), qs[0], qs[1], qs[2], _p(meta), ms[0], ms[1], ms[2], B,
                               _p(seq), _p(nqa), Hq, Hkv, d, int(page_size), _p(hd), len(hd),
                               groups, float(scale), _p(init), ins[0], ins[1], _p(out), os_[0],
                               os_[1])
    if rc:
        raise ValueError(f"oracle_page_score rejected its arguments ({rc})")
    return out


def select(s_draft, s_target, seq_lens, k_max, budget=None, m=None, m_scalar=0,
           n_sink=4, n_window=16, groups=1):
    """Eq. 6 tiered selection.  s_draft / s_target: float32 [B, G or 1, N] (an axis of
    length 1 over groups broadcasts) or None.  Returns (idx int32 [B, G, k_max] padded
    with -1, count int32 [B, G])."""
    lib = _load()
    B = len(seq_lens)
    seq = _i32arr(seq_lens, B)
    bud = None if budget is None else _i32arr(budget, B)
    ma = None if m is None else _i32arr(m, B)

    def strides(s):
        if s is None:
            return 0, 0
        _check_inner(s, "score")
        st = _st(s)
        return st[0], (0 if s.shape[1] == 1 else st[1])

    dsb, dsg = strides(s_draft)
    tsb, tsg = strides(s_target)
    idx = np.full((B, groups, k_max), -1, dtype=np.int32)
    count = np.zeros((B, groups), dtype=np.int32)
    rc = lib.oracle_select(_p(s_draft), dsb, dsg, _p(s_target), tsb, tsg, B, groups,
                           _p(seq), _p(bud), int(k_max), _p(ma), int(m_scalar),
                           int(n_sink), int(n_window), _p(idx), k_max * groups, k_max,
                           _p(count))
    if rc:
        raise ValueError(f"oracle_select rejected its arguments ({rc})")
    return idx, count


def attention(q, k, v, seq_lens, scale, rows, idx=None, count=None, num_kv_heads=None):
    """Verification attention for the requested (b, t, h) rows.  q: uint16 [B, T, Hq, d];
    k, v: uint16 [B, N_cap, Hkv, d]; idx int32 [B, G, k_max] and count int32 [B, G] for
    the sparse form (None = dense).  Returns float64 [len(rows), d]."""
    lib = _load()
    for a, nm in ((q, "q"), (k, "k"), (v, "v")):
        _check_inner(a, nm)
    B, _, Hq, d = q.shape
    Hkv = k.shape[2] if num_kv_heads is None else num_kv_heads
    seq = _i32arr(seq_lens, B)
    rows = np.asarray(rows, dtype=np.int32).reshape(-1, 3)
    rb = np.ascontiguousarray(rows[:, 0])
    rt = np.ascontiguousarray(rows[:, 1])
    rh = np.ascontiguousarray(rows[:, 2])
    out = np.zeros((rows.shape[0], d), dtype=np.float64)
    G = 1
    isb = isg = 0
    if idx is not None:
        G = idx.shape[1]
        _check_inner(idx, "idx")
        isb, isg = _st(idx)[0], _st(idx)[1]
        count = np.ascontiguousarray(np.asarray(count, dtype=np.int32).reshape(B, G))
    qs, ks, vs = _st(q), _st(k), _st(v)
    rc = lib.oracle_attention(_p(q), qs[0], qs[1], qs[2], _p(k), ks[0], ks[1], ks[2],
                              _p(v), vs[0], vs[1], vs[2], Hq, Hkv, d, _p(seq),
                              _p(idx), isb, isg, _p(count), G, float(scale),
                              rows.shape[0], _p(rb), _p(rt), _p(rh), _p(out))
    if rc:
        raise ValueError(f"oracle_attention rejected its arguments ({rc})")
    return out


def all_rows(B, n_query, Hq):
    """Every (b, t, h) output row of a batch, in (b, t, h) order."""
    rows = [(b, t, h) for b in range(B) for t in range(int(n_query[b])) for h in range(Hq)]
    return np.asarray(rows, dtype=np.int32).reshape(-1, 3)


def arr_window(A, sel):
    """Windowed attention recovery rate of the index set sel over attention rows A
    (float64 [w, n])."""
    A = np.ascontiguousarray(A, dtype=np.float64)
    s = _i32arr(sel)
    return float(_load().oracle_arr_window(_p(A), A.shape[0], A.shape[1], _p(s), len(s)))


def arr(q, k, seq_lens, window, scale, groups=1, idx=None, count=None, num_kv_heads=None,
        with_abar=False, length=None):
    """Windowed attention recovery rate of the verification window (Eqs. 1-4), averaged over
    the heads each index set serves.  q: uint16 [B, w_max, Hq, d] (the w_b = window[b] queries);
    k: uint16 [B, N, Hkv, d]; idx int32 [B, G, >= count], count int32 [B, G] (None: the empty
    set).  Returns arr float64 [B, G], and with with_abar also A-bar float64 [B, G, length]."""
    lib = _load()
    B, _, Hq, d = q.shape
    Hkv = k.shape[2] if num_kv_heads is None else num_kv_heads
    _check_inner(q, "q")
    _check_inner(k, "k")
    seq = _i32arr(seq_lens, B)
    wa = _i32arr(window, B)
    out = np.zeros((B, groups), dtype=np.float64)
    ab = None
    if with_abar:
        n_out = length if length is not None else max(int(seq.max(initial=0)), 1)
        ab = np.zeros((B, groups, n_out), dtype=np.float64)
    ix = cn = None
    if idx is not None:
        ix = np.ascontiguousarray(idx, dtype=np.int32)
        cn = np.ascontiguousarray(count, dtype=np.int32)
    qs, ks = _st(q), _st(k)
    abs_ = _st(ab) if ab is not None else [0, 0, 0]
    ixs = _st(ix) if ix is not None else [0, 0, 0]
    rc = lib.oracle_arr(_p(q), qs[0], qs[1], qs[2], _p(k), ks[0], ks[1], ks[2], B, _p(seq), _p(wa),
                        Hq, Hkv, d, groups, float(scale), _p(ix), ixs[0], ixs[1], _p(cn), _p(out),
                        _p(ab), abs_[0], abs_[1])
    if rc:
        raise ValueError(f"oracle_arr rejected its arguments ({rc})")
    return (out, ab) if with_abar else out


def overhead_ratio(hd_sel, ld_sel, gamma, ht_sel, lt_sel, hd, ld, ht, lt):
    """Appendix A estimator cost ratio."""
    return float(_load().oracle_overhead_ratio(hd_sel, ld_sel, gamma, ht_sel, lt_sel,
                                               hd, ld, ht, lt))


# ----------------------------------------------------------------------------- KV append / commit
# Sec. 3.2 (sparse verification workflow): the verification window's target KV sits in the
# cache at positions [N_b, N_b + T_b) while it is verified; afterwards the accepted tokens
# are appended (kept) and the rejected draft tokens discarded.

def kv_append(cache, new, seq_lens, n_query, page_table=None):
    """The cache after writing the window rows: for every b and t < T_b, logical position
    N_b + t of sequence b holds new[b, t].  cache: uint16 [B, N_cap, Hkv, d] (contiguous) or
    [P, page_size, Hkv, d] with page_table int32 [B, max_pages] (paged); new: uint16
    [B, T_max, Hkv, d].  Positions past the capacity (or without a page) are not written.
    Returns a new array."""
    out = np.array(cache, copy=True)
    for b in range(new.shape[0]):
        for t in range(int(n_query[b])):
            pos = int(seq_lens[b]) + t
            if page_table is None:
                if pos < out.shape[1]:
                    out[b, pos] = new[b, t]
            else:
                ps = out.shape[1]
                if pos // ps < page_table.shape[1]:
                    out[int(page_table[b, pos // ps]), pos % ps] = new[b, t]
    return out


def kv_commit(seq_lens, accepted, n_query):
    """N_b + clamp(accepted_b, 0, T_b): the accepted window tokens become history."""
    seq = np.asarray(seq_lens, dtype=np.int64)
    acc = np.clip(np.asarray(accepted, dtype=np.int64), 0, np.asarray(n_query, dtype=np.int64))
    return (seq + acc).astype(np.int32)
