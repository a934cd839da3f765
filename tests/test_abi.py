"""The C ABI without a GPU: libdustin.so loads, exports every function include/dustin.h
declares, sizes its workspaces on the host, and rejects invalid arguments before any
launch (every call here fails validation, so no kernel is ever enqueued)."""
import ctypes
import os
import re

import pytest

import paper_2606_24957_amd as D

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dustin.h")

FAKE = 0x10000  # a non-null, 256-byte aligned address that validation never dereferences


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dustin_\w+|dense_verify_attn)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(D.LIB_PATH):
        pytest.skip("libdustin.so not built")
    return D.lib()


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert set(names) == set(D.EXPORTED)
    for n in names:
        assert hasattr(L, n), n


def test_status_strings_and_version(L):
    assert D.status_string(D.OK) == "ok"
    for s in range(1, 6):
        assert D.status_string(s) not in ("ok", "unknown status")
    assert D.status_string(99) == "unknown status"
    assert L.dustin_version() >> 16 == 1


def test_workspace_sizes(L):
    t = L.dustin_topk_workspace(16, 1, 32768)   # a fixed counter region, two bitmaps per row
    assert t == 4096 * 4 + 16 * 2 * 1024 * 4 and t % 256 == 0
    assert L.dustin_topk_workspace(0, 1, 32768) == 0
    assert L.dustin_topk_workspace(4097, 1, 1000) == 0   # no hand-off: no workspace
    s = L.dustin_score_workspace(16, 32768, 4, 4)
    assert s >= D.SCORE_SYNC_BYTES + 16 * 4 * 4 * 32768 * 4 and s % 256 == 0
    assert L.dustin_score_workspace(0, 10, 1, 1) == 0
    # attention: a split-K workspace once the batch leaves compute units idle
    w = L.dustin_attn_workspace(16, 64, 8, 5, 2048, 1)
    assert w == 0 or w > 4096
    assert L.dustin_attn_workspace(0, 64, 8, 5, 2048, 1) == 0


def test_score_sync_layout_matches_the_header():
    """The binding's copy of the score workspace's counter region and flag offset."""
    text = open(HEADER).read()
    got = {k: int(v) for k, v in re.findall(r"#define (DUSTIN_SCORE_SYNC_\w+) (\d+)u", text)}
    assert got == {"DUSTIN_SCORE_SYNC_BYTES": D.SCORE_SYNC_BYTES,
                   "DUSTIN_SCORE_SYNC_FLAG_OFFSET": D.SCORE_SYNC_FLAG_OFFSET}
    assert D.SCORE_SYNC_FLAG_OFFSET + 4 <= D.SCORE_SYNC_BYTES and D.SCORE_SYNC_BYTES % 256 == 0


def _batch(B=2, max_len=100, nq=4, k_max=40, m=10):
    bt = D.DustinBatch()
    bt.batch, bt.max_len, bt.nq_max, bt.k_max, bt.m_scalar = B, max_len, nq, k_max, m
    bt.seq_lens = FAKE
    return bt


def _kv(Hkv=2, d=128, cap=200):
    kv = D.DustinKV()
    kv.data = FAKE
    kv.num_kv_heads, kv.head_dim = Hkv, d
    kv.stride_n, kv.stride_h, kv.stride_b, kv.capacity = Hkv * d, d, cap * Hkv * d, cap
    return kv


def _topk(L, bt, sd=FAKE, st=FAKE, groups=1, ns=4, nw=16, idx=FAKE, cnt=FAKE, ws=FAKE, ws_bytes=1 << 30,
          hd=None, ht=None):
    return L.dustin_topk(sd, 0, 0, st, 0, 0, ctypes.byref(bt), groups, ns, nw, idx, 0, 0, cnt,
                         hd, ht, ws, ws_bytes, None)


def test_topk_rejects(L):
    assert _topk(L, _batch(k_max=19)) == D.ERR_INVALID_ARG              # k < sinks + window
    assert _topk(L, _batch(k_max=40, m=21)) == D.ERR_INVALID_ARG        # m > k - |P|
    assert _topk(L, _batch(m=-1)) == D.ERR_INVALID_ARG
    assert _topk(L, _batch(m=3), sd=None) == D.ERR_INVALID_ARG          # no S_D needs m = 0
    assert _topk(L, _batch(m=3), st=None) == D.ERR_INVALID_ARG          # no S_T needs m = k-|P|
    assert _topk(L, _batch(), sd=None, st=None) == D.ERR_INVALID_ARG
    assert _topk(L, _batch(), idx=None) == D.ERR_INVALID_ARG
    assert _topk(L, _batch(), groups=0) == D.ERR_INVALID_ARG
    assert _topk(L, _batch(max_len=(1 << 19) + 1)) == D.ERR_UNSUPPORTED
    # both tiers hand off through the workspace; one tier alone needs none
    assert _topk(L, _batch(), ws=None, ws_bytes=0) == D.ERR_WORKSPACE
    assert _topk(L, _batch(), ws=FAKE + 4) == D.ERR_WORKSPACE
    assert _topk(L, _batch(), ws_bytes=64) == D.ERR_WORKSPACE
    bt = _batch()
    bt.seq_lens = None
    assert _topk(L, bt) == D.ERR_INVALID_ARG
    assert L.dustin_topk(FAKE, 0, 0, FAKE, 0, 0, None, 1, 4, 16, FAKE, 0, 0, FAKE, None, None, None, 0,
                         None) == D.ERR_INVALID_ARG
    # the first-digit histograms: each with its score array, 16-byte aligned, distinct, one group
    assert _topk(L, _batch(m=0), sd=None, hd=FAKE) == D.ERR_INVALID_ARG
    assert _topk(L, _batch(m=20), st=None, ht=FAKE) == D.ERR_INVALID_ARG
    assert _topk(L, _batch(), hd=FAKE + 4) == D.ERR_INVALID_ARG
    assert _topk(L, _batch(), hd=FAKE, ht=FAKE) == D.ERR_INVALID_ARG
    assert _topk(L, _batch(), groups=2, ht=FAKE) == D.ERR_INVALID_ARG


def _attn(L, q=FAKE, kv=None, vv=None, bt=None, Hq=8, idx=FAKE, cnt=FAKE, groups=1, out=FAKE,
          qs=(800 * 8 * 128, 8 * 128, 128), scale=0.1, ws=None, ws_bytes=0):
    kv = kv or _kv()
    vv = vv or _kv()
    bt = bt or _batch()
    return L.dustin_sparse_verify_attn(q, *qs, Hq, ctypes.byref(kv), ctypes.byref(vv),
                                       ctypes.byref(bt), idx, 0, 0, cnt, groups, scale, out,
                                       *qs, ws, ws_bytes, None)


def test_attention_rejects(L):
    assert _attn(L, q=None) == D.ERR_INVALID_ARG
    assert _attn(L, out=None) == D.ERR_INVALID_ARG
    assert _attn(L, idx=None) == D.ERR_INVALID_ARG
    assert _attn(L, cnt=None) == D.ERR_INVALID_ARG
    assert _attn(L, Hq=7) == D.ERR_INVALID_ARG                        # Hq % Hkv
    assert _attn(L, groups=3) == D.ERR_INVALID_ARG                    # groups not in {1, Hkv}
    assert _attn(L, q=FAKE + 2) == D.ERR_INVALID_ARG                  # 16-byte rows
    assert _attn(L, qs=(4, 8 * 128, 128)) == D.ERR_INVALID_ARG
    assert _attn(L, scale=float("nan")) == D.ERR_INVALID_ARG
    assert _attn(L, kv=_kv(d=64), vv=_kv(d=64)) == D.ERR_UNSUPPORTED  # head_dim 128 only
    assert _attn(L, kv=_kv(cap=103)) == D.ERR_INVALID_ARG             # capacity < max_len + T
    assert _attn(L, vv=_kv(Hkv=4)) == D.ERR_INVALID_ARG
    assert _attn(L, Hq=64, kv=_kv(Hkv=2), vv=_kv(Hkv=2), bt=_batch(nq=5)) == D.ERR_UNSUPPORTED
    paged = _kv()
    paged.page_table, paged.page_size, paged.max_pages, paged.num_pages = FAKE, 12, 20, 40
    paged.stride_page = 12 * 256
    assert _attn(L, kv=paged, vv=paged) == D.ERR_INVALID_ARG          # page size not 2^k
    assert _attn(L, kv=paged) == D.ERR_INVALID_ARG                    # K paged, V not
    # a batch that needs the split-K workspace refuses to run without one
    need = L.dustin_attn_workspace(1, 8, 2, 4, 40, 1)
    if need:
        assert _attn(L, bt=_batch(B=1)) == D.ERR_WORKSPACE
        assert _attn(L, bt=_batch(B=1), ws=FAKE + 8, ws_bytes=need) == D.ERR_WORKSPACE


def test_dense_rejects(L):
    kv, bt = _kv(), _batch()
    qs = (800 * 8 * 128, 8 * 128, 128)
    assert L.dense_verify_attn(None, *qs, 8, ctypes.byref(kv), ctypes.byref(kv), ctypes.byref(bt),
                               0.1, FAKE, *qs, None, 0, None) == D.ERR_INVALID_ARG
    assert L.dense_verify_attn(FAKE, *qs, 8, ctypes.byref(kv), ctypes.byref(kv), None, 0.1, FAKE,
                               *qs, None, 0, None) == D.ERR_INVALID_ARG


def _score(L, heads=(0, 3), Hq=8, kv=None, bt=None, groups=1, q=FAKE, out=FAKE, ws=FAKE,
           ws_bytes=1 << 30):
    kv = kv or _kv()
    bt = bt or _batch()
    arr = (ctypes.c_int32 * max(1, len(heads)))(*heads)
    return L.dustin_score(q, 800 * 8 * 128, 8 * 128, 128, Hq, arr, len(heads), ctypes.byref(kv),
                          ctypes.byref(bt), 0.1, groups, None, 0, 0, out, 0, 0, ws, ws_bytes, None)


def test_score_rejects(L):
    assert _score(L, heads=(0, 8)) == D.ERR_INVALID_ARG               # head out of range
    assert _score(L, heads=(2, 2)) == D.ERR_INVALID_ARG               # duplicate head
    assert _score(L, heads=()) == D.ERR_UNSUPPORTED
    assert _score(L, heads=tuple(range(65)), Hq=128) == D.ERR_UNSUPPORTED  # at most 64 heads
    assert _score(L, groups=3) == D.ERR_INVALID_ARG
    assert _score(L, q=None) == D.ERR_INVALID_ARG
    assert _score(L, out=None) == D.ERR_INVALID_ARG
    assert _score(L, kv=_kv(d=96)) == D.ERR_UNSUPPORTED
    assert _score(L, bt=_batch(nq=17)) == D.ERR_UNSUPPORTED
    assert _score(L, ws=None, ws_bytes=0) == D.ERR_WORKSPACE
    assert _score(L, ws=FAKE + 4) == D.ERR_WORKSPACE
    assert _score(L, ws_bytes=16) == D.ERR_WORKSPACE


def _score_call(keep, heads=(0, 2), Hq=8, kv=None, bt=None, ws=FAKE, ws_bytes=1 << 30, out=FAKE):
    """A dustin_score_call descriptor; keep holds the ctypes objects it points at."""
    kv = kv or _kv(Hkv=4)
    bt = bt or _batch(nq=1)
    hd = (ctypes.c_int32 * max(len(heads), 1))(*heads)
    qh = (ctypes.c_void_p * 1)(FAKE)
    keep += [kv, bt, hd, qh]
    c = D.DustinScoreCall()
    c.n_layers, c.q_layers_host, c.q_sb, c.q_sj, c.q_sh = 1, ctypes.addressof(qh), 8 * 128, 8 * 128, 128
    c.num_q_heads, c.heads_host, c.n_heads = Hq, ctypes.addressof(hd), len(heads)
    c.k_layers_host, c.bt, c.scale, c.groups = ctypes.addressof(kv), ctypes.addressof(bt), 0.1, 1
    c.out, c.workspace, c.workspace_bytes = out, ws, ws_bytes
    return c


def test_score_calls_rejects(L):
    keep = []
    one = _score_call(keep)
    arr = (D.DustinScoreCall * 3)(one, _score_call(keep, ws=FAKE + 0x40000000), one)
    assert L.dustin_score_calls(0, arr, None) == D.ERR_INVALID_ARG
    assert L.dustin_score_calls(3, arr, None) == D.ERR_INVALID_ARG
    assert L.dustin_score_calls(1, None, None) == D.ERR_INVALID_ARG
    shared = (D.DustinScoreCall * 2)(one, one)
    assert L.dustin_score_calls(2, shared, None) == D.ERR_WORKSPACE    # one workspace for two calls
    bad = (D.DustinScoreCall * 2)(one, _score_call(keep, heads=(0, 8), ws=FAKE + 0x40000000))
    assert L.dustin_score_calls(2, bad, None) == D.ERR_INVALID_ARG     # the second call's head
    bad = (D.DustinScoreCall * 2)(_score_call(keep, out=None), one)
    assert L.dustin_score_calls(2, bad, None) == D.ERR_INVALID_ARG
    small = (D.DustinScoreCall * 1)(_score_call(keep, ws_bytes=16))
    assert L.dustin_score_calls(1, small, None) == D.ERR_WORKSPACE


def test_read_probe_rejects(L):
    f = ctypes.c_void_p(FAKE)
    assert L.dustin_read_probe(None, 4096, f, 4, None) == D.ERR_INVALID_ARG
    assert L.dustin_read_probe(f, 4096, None, 4, None) == D.ERR_INVALID_ARG
    assert L.dustin_read_probe(ctypes.c_void_p(FAKE + 8), 4096, f, 4, None) == D.ERR_INVALID_ARG
    assert L.dustin_read_probe(f, 4100, f, 4, None) == D.ERR_INVALID_ARG
    assert L.dustin_read_probe(f, 4096, f, 0, None) == D.ERR_INVALID_ARG
    assert L.dustin_read_probe(f, 4096, f, 65537, None) == D.ERR_INVALID_ARG
    assert L.dustin_read_probe(f, 1 << 32, f, 1, None) == D.ERR_UNSUPPORTED


def test_product_never_touches_the_oracle():
    """The HIP path has no CPU fallback and never imports the checker."""
    pkg = os.path.join(ROOT, "paper_2606_24957_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".hpp", ".cpp", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"^\s*(import|from)\s+oracle", text, re.M), f
                assert "liboracle" not in text, f


def test_page_workspace_sizes(L):
    s = L.dustin_page_score_workspace(16, 32768, 16, 5, 64)
    assert s >= 16 * 64 * 5 * 2048 * 4 and s % 256 == 0
    assert L.dustin_page_score_workspace(16, 32768, 12, 5, 64) == 0   # page size not 2^k
    assert L.dustin_page_score_workspace(0, 32768, 16, 5, 64) == 0


def _meta_call(L, kv=None, bt=None, frm=None, span=100, ps=16, meta=FAKE, sb=None, sp=None, pages=7):
    kv = kv or _kv()
    bt = bt or _batch()
    d, Hkv = kv.head_dim, kv.num_kv_heads
    sp = Hkv * 2 * d if sp is None else sp
    sb = pages * sp if sb is None else sb
    return L.dustin_page_meta(ctypes.byref(kv), ctypes.byref(bt), frm, span, ps, meta, sb, sp, pages, None)


def test_page_meta_rejects(L):
    assert _meta_call(L, ps=12) == D.ERR_INVALID_ARG                  # page size not 2^k
    assert _meta_call(L, ps=0) == D.ERR_INVALID_ARG
    assert _meta_call(L, ps=8192) == D.ERR_INVALID_ARG
    assert _meta_call(L, kv=_kv(d=96)) == D.ERR_UNSUPPORTED
    assert _meta_call(L, meta=None) == D.ERR_INVALID_ARG
    assert _meta_call(L, meta=FAKE + 4) == D.ERR_INVALID_ARG
    assert _meta_call(L, pages=6) == D.ERR_INVALID_ARG                # ceil(100 / 16) = 7 pages
    assert _meta_call(L, sp=2 * 128) == D.ERR_INVALID_ARG             # rows of 2 KV heads overlap
    assert _meta_call(L, span=101) == D.ERR_INVALID_ARG               # span > max_len
    assert _meta_call(L, span=-1) == D.ERR_INVALID_ARG
    assert _meta_call(L, frm=FAKE + 2) == D.ERR_INVALID_ARG
    assert _meta_call(L, kv=_kv(cap=99)) == D.ERR_INVALID_ARG         # cache shorter than max_len
    assert L.dustin_page_meta(None, ctypes.byref(_batch()), None, 10, 16, FAKE, 0, 512, 7,
                              None) == D.ERR_INVALID_ARG


def _pscore(L, heads=(0, 3), Hq=8, Hkv=2, d=128, ps=16, pages=7, bt=None, groups=1, q=FAKE, meta=FAKE,
            out=FAKE, ws=FAKE, ws_bytes=1 << 30, sp=None):
    bt = bt or _batch()
    arr = (ctypes.c_int32 * max(1, len(heads)))(*heads)
    sp = Hkv * 2 * d if sp is None else sp
    return L.dustin_page_score(q, 800 * 8 * d, 8 * d, d, Hq, arr, len(heads), meta, pages * sp, sp, pages, Hkv,
                               d, ps, ctypes.byref(bt), 0.1, groups, None, 0, 0, out, 0, 0, ws, ws_bytes, None)


def test_page_score_rejects(L):
    assert _pscore(L, heads=(0, 8)) == D.ERR_INVALID_ARG
    assert _pscore(L, heads=(1, 1)) == D.ERR_INVALID_ARG
    assert _pscore(L, heads=tuple(range(65)), Hq=128) == D.ERR_UNSUPPORTED
    assert _pscore(L, ps=3) == D.ERR_INVALID_ARG
    assert _pscore(L, d=96) == D.ERR_UNSUPPORTED
    assert _pscore(L, Hq=7) == D.ERR_INVALID_ARG
    assert _pscore(L, groups=3) == D.ERR_INVALID_ARG
    assert _pscore(L, pages=6) == D.ERR_INVALID_ARG
    assert _pscore(L, meta=None) == D.ERR_INVALID_ARG
    assert _pscore(L, q=None) == D.ERR_INVALID_ARG
    assert _pscore(L, out=None) == D.ERR_INVALID_ARG
    assert _pscore(L, bt=_batch(nq=17)) == D.ERR_UNSUPPORTED
    assert _pscore(L, ws=None, ws_bytes=0) == D.ERR_WORKSPACE
    assert _pscore(L, ws_bytes=64) == D.ERR_WORKSPACE


def test_arr_rejects(L):
    bt = _batch()

    def call(s=FAKE, idx=FAKE, cnt=FAKE, groups=1, hpg=8, out=FAKE, sb=100, b=bt):
        return L.dustin_arr(s, sb, 0, idx, 40, 40, cnt, ctypes.byref(b) if b else None, groups, hpg, out, None)

    assert call(s=None) == D.ERR_INVALID_ARG
    assert call(idx=None) == D.ERR_INVALID_ARG
    assert call(cnt=None) == D.ERR_INVALID_ARG
    assert call(out=None) == D.ERR_INVALID_ARG
    assert call(out=FAKE + 4) == D.ERR_INVALID_ARG                    # fp64 output
    assert call(groups=0) == D.ERR_INVALID_ARG
    assert call(hpg=0) == D.ERR_INVALID_ARG
    assert call(sb=-1) == D.ERR_INVALID_ARG
    assert call(b=None) == D.ERR_INVALID_ARG


def test_score_per_layer_rejects(L):
    kvs = (D.DustinKV * 2)(_kv(), _kv())
    qs = (ctypes.c_void_p * 2)(FAKE, FAKE)
    heads = (ctypes.c_int32 * 2)(0, 3)
    bt = _batch()

    def call(n=2, q=qs, kv=kvs, sl=1 << 20, out=FAKE, ws_bytes=1 << 30, nh=2, b=bt):
        return L.dustin_score_per_layer(n, q, 800 * 8 * 128, 8 * 128, 128, 8, heads, nh, kv, ctypes.byref(b), 0.1,
                                        1, out, sl, 0, 0, FAKE, ws_bytes, None)

    assert call(n=0) == D.ERR_UNSUPPORTED
    assert call(n=33) == D.ERR_UNSUPPORTED                            # at most 32 layers
    assert call(sl=-1) == D.ERR_INVALID_ARG
    assert call(out=None) == D.ERR_INVALID_ARG
    assert call(ws_bytes=16) == D.ERR_WORKSPACE
    other = (D.DustinKV * 2)(_kv(), _kv(cap=300))                     # layers must share the layout
    assert call(kv=other) == D.ERR_INVALID_ARG
    assert call(b=_batch(nq=17)) == D.ERR_UNSUPPORTED
