"""Python binding of libdustin, the MI355X (gfx950) hot path of Dustin's sparse verification.

Every function here only marshals arguments (torch tensors -> device pointers, strides,
the current HIP stream) and calls the C ABI declared in include/dustin.h; all arithmetic
runs in the HIP kernels.  There is no CPU fallback: when libdustin.so is missing or the
tensors are not on a GPU, the call raises.

Step of one speculative verification (paper: method section 4, Eqs. 5 and 6):
    s_t = score(q_last, k_layer, seq_lens, target_heads, init=history)       # S_Target
    s_d = score(q_draft[l], k_draft[l], seq_lens, draft_heads, init=s_d)     # S_Draft, per layer
    idx, cnt = topk(s_d, s_t, seq_lens, k_max, m_scalar=m)                   # I_verify
    o[l] = sparse_verify_attn(q[l], k[l], v[l], idx, cnt, seq_lens)          # every layer
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdustin.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_LAUNCH, ERR_SCRATCH_LIMIT = range(6)

EXPORTED = ("dustin_status_string", "dustin_version", "dustin_score_workspace", "dustin_score",
            "dustin_topk_workspace", "dustin_topk", "dustin_attn_workspace",
            "dustin_sparse_verify_attn", "dense_verify_attn", "dustin_kv_append", "dustin_kv_commit",
            "dustin_score_layers", "dustin_page_meta", "dustin_page_score_workspace",
            "dustin_page_score", "dustin_arr", "dustin_score_per_layer",
            "dustin_sparse_verify_attn_noalloc", "dustin_score_calls", "dustin_read_probe")


class DustinError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_string(status)} (status {status})")
        self.status = status


class DustinKV(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("stride_b", ctypes.c_int64),
                ("stride_n", ctypes.c_int64), ("stride_h", ctypes.c_int64),
                ("capacity", ctypes.c_int64), ("page_table", ctypes.c_void_p),
                ("page_size", ctypes.c_int32), ("max_pages", ctypes.c_int32),
                ("num_pages", ctypes.c_int32), ("stride_page", ctypes.c_int64)]


class DustinBatch(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("max_len", ctypes.c_int32),
                ("nq_max", ctypes.c_int32), ("k_max", ctypes.c_int32),
                ("seq_lens", ctypes.c_void_p), ("n_query", ctypes.c_void_p),
                ("budget", ctypes.c_void_p), ("m", ctypes.c_void_p),
                ("m_scalar", ctypes.c_int32)]


class DustinScoreCall(ctypes.Structure):
    """dustin_score_call: the arguments of one dustin_score_layers call."""
    _fields_ = [("n_layers", ctypes.c_int32), ("q_layers_host", ctypes.c_void_p),
                ("q_sb", ctypes.c_int64), ("q_sj", ctypes.c_int64), ("q_sh", ctypes.c_int64),
                ("num_q_heads", ctypes.c_int32), ("heads_host", ctypes.c_void_p),
                ("n_heads", ctypes.c_int32), ("k_layers_host", ctypes.c_void_p),
                ("bt", ctypes.c_void_p), ("scale", ctypes.c_float), ("groups", ctypes.c_int32),
                ("init", ctypes.c_void_p), ("init_sb", ctypes.c_int64), ("init_sg", ctypes.c_int64),
                ("out", ctypes.c_void_p), ("out_sb", ctypes.c_int64), ("out_sg", ctypes.c_int64),
                ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t),
                ("digit_hist", ctypes.c_void_p)]


_lib = None
_i64, _i32, _vp, _sz = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t


def lib():
    """The loaded libdustin.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -c 'import __graft_entry__ as g; g.build()'`")
        L = ctypes.CDLL(LIB_PATH)
        P_KV, P_BT = ctypes.POINTER(DustinKV), ctypes.POINTER(DustinBatch)
        L.dustin_status_string.restype = ctypes.c_char_p
        L.dustin_status_string.argtypes = [ctypes.c_int]
        L.dustin_version.restype = _i32
        L.dustin_score_workspace.restype = _sz
        L.dustin_score_workspace.argtypes = [_i32, _i32, _i32, _i32]
        L.dustin_score.restype = ctypes.c_int
        L.dustin_score.argtypes = [_vp, _i64, _i64, _i64, _i32, _vp, _i32, P_KV, P_BT,
                                   ctypes.c_float, _i32, _vp, _i64, _i64, _vp, _i64, _i64,
                                   _vp, _sz, _vp]
        L.dustin_topk_workspace.restype = _sz
        L.dustin_topk_workspace.argtypes = [_i32, _i32, _i32]
        L.dustin_topk.restype = ctypes.c_int
        L.dustin_topk.argtypes = [_vp, _i64, _i64, _vp, _i64, _i64, P_BT, _i32, _i32, _i32,
                                  _vp, _i64, _i64, _vp, _vp, _vp, _vp, _sz, _vp]
        L.dustin_attn_workspace.restype = _sz
        L.dustin_attn_workspace.argtypes = [_i32, _i32, _i32, _i32, _i32, _i32]
        L.dustin_sparse_verify_attn.restype = ctypes.c_int
        L.dustin_sparse_verify_attn.argtypes = [_vp, _i64, _i64, _i64, _i32, P_KV, P_KV, P_BT,
                                                _vp, _i64, _i64, _vp, _i32, ctypes.c_float,
                                                _vp, _i64, _i64, _i64, _vp, _sz, _vp]
        L.dustin_sparse_verify_attn_noalloc.restype = ctypes.c_int
        L.dustin_sparse_verify_attn_noalloc.argtypes = [_vp, _i64, _i64, _i64, _i32, P_KV, P_KV, P_BT,
                                                        _vp, _i64, _i64, _vp, _i32, ctypes.c_float,
                                                        _vp, _i64, _i64, _i64, _vp]
        L.dense_verify_attn.restype = ctypes.c_int
        L.dense_verify_attn.argtypes = [_vp, _i64, _i64, _i64, _i32, P_KV, P_KV, P_BT,
                                        ctypes.c_float, _vp, _i64, _i64, _i64, _vp, _sz, _vp]
        L.dustin_score_layers.restype = ctypes.c_int
        L.dustin_score_layers.argtypes = [_i32, _vp, _i64, _i64, _i64, _i32, _vp, _i32, P_KV, P_BT,
                                          ctypes.c_float, _i32, _vp, _i64, _i64, _vp, _i64, _i64,
                                          _vp, _sz, _vp]
        L.dustin_kv_append.restype = ctypes.c_int
        L.dustin_kv_append.argtypes = [_vp, _i64, _i64, _i64, _vp, _i64, _i64, _i64, P_KV, P_KV,
                                       P_BT, _vp]
        L.dustin_page_meta.restype = ctypes.c_int
        L.dustin_page_meta.argtypes = [P_KV, P_BT, _vp, _i32, _i32, _vp, _i64, _i64, _i32, _vp]
        L.dustin_page_score_workspace.restype = _sz
        L.dustin_page_score_workspace.argtypes = [_i32, _i32, _i32, _i32, _i32]
        L.dustin_page_score.restype = ctypes.c_int
        L.dustin_page_score.argtypes = [_vp, _i64, _i64, _i64, _i32, _vp, _i32, _vp, _i64, _i64, _i32,
                                        _i32, _i32, _i32, P_BT, ctypes.c_float, _i32, _vp, _i64, _i64,
                                        _vp, _i64, _i64, _vp, _sz, _vp]
        L.dustin_score_per_layer.restype = ctypes.c_int
        L.dustin_score_per_layer.argtypes = [_i32, _vp, _i64, _i64, _i64, _i32, _vp, _i32, P_KV, P_BT,
                                             ctypes.c_float, _i32, _vp, _i64, _i64, _i64, _vp, _sz, _vp]
        L.dustin_arr.restype = ctypes.c_int
        L.dustin_arr.argtypes = [_vp, _i64, _i64, _vp, _i64, _i64, _vp, P_BT, _i32, _i32, _vp, _vp]
        L.dustin_score_calls.restype = ctypes.c_int
        L.dustin_score_calls.argtypes = [_i32, ctypes.POINTER(DustinScoreCall), _vp]
        L.dustin_kv_commit.restype = ctypes.c_int
        L.dustin_kv_commit.argtypes = [_vp, _vp, _vp, _i32, _i32, _vp]
        L.dustin_read_probe.restype = ctypes.c_int
        L.dustin_read_probe.argtypes = [_vp, _sz, _vp, _i32, _vp]
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().dustin_status_string(int(status)).decode()


def _check(status: int, what: str):
    if status != OK:
        raise DustinError(status, what)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _on_gpu(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("libdustin runs on the GPU only: every tensor must be on a HIP device")


def _i32_dev(x, device) -> Optional[torch.Tensor]:
    if x is None:
        return None
    if isinstance(x, torch.Tensor):
        if x.dtype != torch.int32 or not x.is_cuda:
            raise ValueError("per-sequence arrays must be int32 device tensors")
        return x.contiguous()
    return torch.tensor(list(x), dtype=torch.int32, device=device)


class Call:
    """One prepared libdustin call: every argument marshalled once, replayed by calling
    the object (one C call per launch, on the stream captured when it was planned)."""

    def __init__(self, fn, args, what, keep, result):
        self._fn, self._args, self._what, self._keep = fn, args, what, keep
        self.result = result

    def __call__(self):
        _check(self._fn(*self._args), self._what)
        return self.result


_WS = {}


def workspace(nbytes: int, device, tag: str, stream=None) -> Optional[torch.Tensor]:
    """A cached, zero-initialised device scratch buffer per (device, stream, tag) of at
    least nbytes.  Calls that share a workspace must not overlap on the device (the split
    attention's counters and partials, the score's logits); keying by stream keeps calls
    planned on different streams apart, and calls on one stream run in order."""
    if nbytes == 0:
        return None
    s = torch.cuda.current_stream(device) if stream is None else stream
    key = (str(torch.device(device)), int(s.cuda_stream), tag)
    buf = _WS.get(key)
    if buf is None or buf.numel() < nbytes:
        buf = torch.zeros(int(nbytes) + 256, dtype=torch.uint8, device=device)
        _WS[key] = buf
    off = (-buf.data_ptr()) % 256
    return buf[off:off + nbytes]


# Layout of a score workspace's first bytes (include/dustin.h): per-sequence counters of
# the single-pass form, zero between calls, and its timeout flag.
SCORE_SYNC_BYTES = 16896
SCORE_SYNC_FLAG_OFFSET = 16384


def score_sync_region(device=None, stream=None, tag: str = "score") -> Optional[torch.Tensor]:
    """The counters and flag at the start of the cached score workspace of (device,
    stream), as uint8 (None if no score call has made one)."""
    dev = torch.device("cuda", torch.cuda.current_device()) if device is None else torch.device(device)
    s = torch.cuda.current_stream(dev) if stream is None else stream
    buf = _WS.get((str(dev), int(s.cuda_stream), tag))
    if buf is None:
        return None
    off = (-buf.data_ptr()) % 256
    return buf[off:off + SCORE_SYNC_BYTES]


def release_workspaces() -> None:
    """Drops the cached workspaces (after synchronising the device), so that a program can
    return their memory to the allocator before it exits."""
    if _WS:
        torch.cuda.synchronize()
    _WS.clear()


def kv_view(cache: torch.Tensor, page_table: Optional[torch.Tensor] = None) -> DustinKV:
    """dustin_kv of a bf16 cache: [B, N_cap, Hkv, d] (contiguous mode) or
    [num_pages, page_size, Hkv, d] with an int32 page table [B, max_pages] (paged)."""
    if cache.dtype != torch.bfloat16 or cache.dim() != 4 or cache.stride(3) != 1:
        raise ValueError("cache must be bf16 [B|pages, N|page_size, Hkv, d] with contiguous d")
    kv = DustinKV()
    kv.data = cache.data_ptr()
    kv.num_kv_heads = cache.shape[2]
    kv.head_dim = cache.shape[3]
    kv.stride_n = cache.stride(1)
    kv.stride_h = cache.stride(2)
    if page_table is None:
        kv.stride_b = cache.stride(0)
        kv.capacity = cache.shape[1]
    else:
        if page_table.dtype != torch.int32 or page_table.dim() != 2:
            raise ValueError("page_table must be int32 [B, max_pages]")
        page_table = page_table.contiguous()
        kv.page_table = page_table.data_ptr()
        kv.page_size = cache.shape[1]
        kv.max_pages = page_table.shape[1]
        kv.num_pages = cache.shape[0]
        kv.stride_page = cache.stride(0)
        kv._keep = page_table
    return kv


def _check_scores(t: torch.Tensor, B: int, groups: int, max_len: int, name: str):
    """An fp32 [>= B, >= groups (or 1 with stride 0), >= max_len] score array with
    contiguous positions."""
    if t.dtype != torch.float32 or t.dim() != 3 or t.stride(2) != 1:
        raise ValueError(f"{name} must be fp32 [B, G, N] with contiguous positions")
    if t.shape[0] < B or t.shape[2] < max_len or not (t.shape[1] >= groups or t.stride(1) == 0):
        raise ValueError(f"{name} {tuple(t.shape)} does not hold [{B}, {groups}, {max_len}]")


def _capacity(kv: DustinKV) -> int:
    return kv.max_pages * kv.page_size if kv.page_table else kv.capacity


def _batch(B, max_len, nq_max, k_max, seq_lens, n_query=None, budget=None, m=None, m_scalar=0):
    bt = DustinBatch()
    bt.batch, bt.max_len, bt.nq_max, bt.k_max = int(B), int(max_len), int(nq_max), int(k_max)
    bt.seq_lens = seq_lens.data_ptr()
    bt.n_query = None if n_query is None else n_query.data_ptr()
    bt.budget = None if budget is None else budget.data_ptr()
    bt.m = None if m is None else m.data_ptr()
    bt.m_scalar = int(m_scalar)
    bt._keep = (seq_lens, n_query, budget, m)
    return bt


# ----------------------------------------------------------------------------- score

def _score_desc(n_layers, q_host, q0, Hq, heads_host, n_heads, kv_addr, bt, scale, groups, init, ins, out, ws,
                nbytes) -> DustinScoreCall:
    """The dustin_score_call of a planned score call (its buffers are kept by the plan)."""
    c = DustinScoreCall()
    c.n_layers = n_layers
    c.q_layers_host = ctypes.addressof(q_host)
    c.q_sb, c.q_sj, c.q_sh = q0.stride(0), q0.stride(1), q0.stride(2)
    c.num_q_heads, c.heads_host, c.n_heads = Hq, ctypes.addressof(heads_host), n_heads
    c.k_layers_host, c.bt = kv_addr, ctypes.addressof(bt)
    c.scale, c.groups = float(scale), int(groups)
    c.init = None if init is None else init.data_ptr()
    c.init_sb, c.init_sg = ins
    c.out, c.out_sb, c.out_sg = out.data_ptr(), out.stride(0), out.stride(1)
    c.workspace, c.workspace_bytes = (None if ws is None else ws.data_ptr()), nbytes
    return c


def plan_score(q: torch.Tensor, k: torch.Tensor, seq_lens, heads: Sequence[int], *,
               n_query=None, scale: Optional[float] = None, groups: int = 1,
               init: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
               max_len: Optional[int] = None, page_table: Optional[torch.Tensor] = None,
               stream=None, ws_tag: str = "score") -> Call:
    """Prepared dustin_score (Eq. 5 over the scoring heads).  q bf16 [B, nq_max, Hq, d];
    k bf16 [B, N_cap, Hkv, d] (or paged with page_table); init / out fp32
    [B, groups, >= max_len].  ws_tag names the cached workspace (calls that are to run in
    one dustin_score_calls need different ones)."""
    _on_gpu(q, k, init, out, page_table)
    B, nq_max, Hq, d = q.shape
    dev = q.device
    seq = _i32_dev(seq_lens, dev)
    nqa = _i32_dev(n_query, dev)
    kv = kv_view(k, page_table)
    max_len = _capacity(kv) if max_len is None else int(max_len)
    if out is None:
        out = torch.empty((B, groups, max_len), dtype=torch.float32, device=dev)
    _check_scores(out, B, groups, max_len, "out")
    if init is not None:
        _check_scores(init, B, groups, max_len, "init")
    heads_host = (ctypes.c_int32 * len(heads))(*[int(h) for h in heads])
    bt = _batch(B, max_len, nq_max, 0, seq, nqa)
    nbytes = lib().dustin_score_workspace(B, max_len, nq_max, len(heads))
    ws = workspace(nbytes, dev, ws_tag, stream)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    ins = (init.stride(0), init.stride(1)) if init is not None else (0, 0)
    args = (_ptr(q), q.stride(0), q.stride(1), q.stride(2), Hq, heads_host, len(heads),
            ctypes.byref(kv), ctypes.byref(bt), float(scale), int(groups), _ptr(init), ins[0],
            ins[1], _ptr(out), out.stride(0), out.stride(1), _ptr(ws), nbytes, _stream(stream))
    q_host = (ctypes.c_void_p * 1)(q.data_ptr())
    desc = _score_desc(1, q_host, q, Hq, heads_host, len(heads), ctypes.addressof(kv), bt, scale, groups,
                       init, ins, out, ws, nbytes)
    c = Call(lib().dustin_score, args, "dustin_score", (q, k, init, kv, bt, ws, heads_host, q_host), out)
    c.desc = desc
    return c


def score(q, k, seq_lens, heads, **kw):
    """Eq. 5 over the scoring heads; returns out (positions >= N_b untouched)."""
    return plan_score(q, k, seq_lens, heads, **kw)()


def plan_score_layers(qs: Sequence[torch.Tensor], ks: Sequence[torch.Tensor], seq_lens,
                      heads: Sequence[int], *, n_query=None, scale: Optional[float] = None,
                      groups: int = 1, init: Optional[torch.Tensor] = None,
                      out: Optional[torch.Tensor] = None, max_len: Optional[int] = None,
                      page_table: Optional[torch.Tensor] = None, stream=None, ws_tag: str = "score") -> Call:
    """Prepared dustin_score_layers: Eq. 5 summed over layers (qs[l], ks[l]) that share every
    shape and stride, into one output, in one launch or two."""
    if len(qs) != len(ks) or not qs:
        raise ValueError("one query tensor per cache, at least one layer")
    _on_gpu(*qs, *ks, init, out, page_table)
    q0 = qs[0]
    B, nq_max, Hq, d = q0.shape
    for q in qs:
        if q.shape != q0.shape or q.stride() != q0.stride() or q.dtype != q0.dtype:
            raise ValueError("the layers' queries must share shape and strides")
    dev = q0.device
    seq = _i32_dev(seq_lens, dev)
    nqa = _i32_dev(n_query, dev)
    kvs = (DustinKV * len(ks))()
    for i, k in enumerate(ks):
        kvs[i] = kv_view(k, page_table)
    max_len = _capacity(kvs[0]) if max_len is None else int(max_len)
    if out is None:
        out = torch.empty((B, groups, max_len), dtype=torch.float32, device=dev)
    _check_scores(out, B, groups, max_len, "out")
    if init is not None:
        _check_scores(init, B, groups, max_len, "init")
    heads_host = (ctypes.c_int32 * len(heads))(*[int(h) for h in heads])
    q_host = (ctypes.c_void_p * len(qs))(*[q.data_ptr() for q in qs])
    bt = _batch(B, max_len, nq_max, 0, seq, nqa)
    nbytes = lib().dustin_score_workspace(B, max_len, nq_max, len(heads) * len(qs))
    ws = workspace(nbytes, dev, ws_tag, stream)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    ins = (init.stride(0), init.stride(1)) if init is not None else (0, 0)
    args = (len(qs), q_host, q0.stride(0), q0.stride(1), q0.stride(2), Hq, heads_host, len(heads),
            kvs, ctypes.byref(bt), float(scale), int(groups), _ptr(init), ins[0], ins[1], _ptr(out),
            out.stride(0), out.stride(1), _ptr(ws), nbytes, _stream(stream))
    c = Call(lib().dustin_score_layers, args, "dustin_score_layers",
             (tuple(qs), tuple(ks), init, kvs, bt, ws, heads_host, q_host), out)
    c.desc = _score_desc(len(qs), q_host, q0, Hq, heads_host, len(heads), ctypes.addressof(kvs), bt, scale,
                         groups, init, ins, out, ws, nbytes)
    return c


def score_layers(qs, ks, seq_lens, heads, **kw):
    """Eq. 5 summed over layers; returns out (positions >= N_b untouched)."""
    return plan_score_layers(qs, ks, seq_lens, heads, **kw)()


DIGIT_BINS = 4096


def digit_hist(rows: int, device) -> torch.Tensor:
    """A zeroed first-digit histogram for `rows` score rows (uint32 held as int32
    [rows, 4096]): what dustin_score_calls fills with digit_hist and dustin_topk consumes
    (and returns to zero)."""
    return torch.zeros((rows, DIGIT_BINS), dtype=torch.int32, device=device)


def plan_score_calls(calls: Sequence[Call], stream=None, digit_hists=None) -> Call:
    """Prepared dustin_score_calls: one or two planned score calls (plan_score or
    plan_score_layers, each with its own workspace tag) in one launch where the library can
    (the target's and the draft's scores of a step), else one after the other.  Returns the
    outputs of the calls.  digit_hists: per call None or a zeroed digit_hist of the call's
    output rows, into which the call counts its outputs by top key digit."""
    if not 1 <= len(calls) <= 2 or any(getattr(c, "desc", None) is None for c in calls):
        raise ValueError("one or two calls planned by plan_score or plan_score_layers")
    hists = list(digit_hists) if digit_hists is not None else [None] * len(calls)
    if len(hists) != len(calls):
        raise ValueError("one histogram (or None) per call")
    for h in hists:
        if h is not None and (h.dtype != torch.int32 or not h.is_contiguous() or h.shape[-1] != DIGIT_BINS):
            raise ValueError("a histogram is a contiguous int32 [rows, 4096] tensor")
    _on_gpu(*[h for h in hists if h is not None])
    descs = []
    for c, h in zip(calls, hists):
        d = DustinScoreCall.from_buffer_copy(c.desc)
        d.digit_hist = None if h is None else h.data_ptr()
        descs.append(d)
    arr = (DustinScoreCall * len(calls))(*descs)
    args = (len(calls), arr, _stream(stream))
    return Call(lib().dustin_score_calls, args, "dustin_score_calls", (tuple(calls), arr, tuple(hists)),
                tuple(c.result for c in calls))


def plan_score_per_layer(qs: Sequence[torch.Tensor], ks: Sequence[torch.Tensor], seq_lens,
                         heads: Sequence[int], *, n_query=None, scale: Optional[float] = None,
                         groups: int = 1, out: Optional[torch.Tensor] = None,
                         max_len: Optional[int] = None, page_table: Optional[torch.Tensor] = None,
                         stream=None) -> Call:
    """Prepared dustin_score_per_layer: Eq. 5 of each layer (qs[l], ks[l]) into out[l]
    (fp32 [L, B, groups, max_len]), in two launches."""
    if len(qs) != len(ks) or not qs:
        raise ValueError("one query tensor per cache, at least one layer")
    _on_gpu(*qs, *ks, out, page_table)
    q0 = qs[0]
    B, nq_max, Hq, d = q0.shape
    for q in qs:
        if q.shape != q0.shape or q.stride() != q0.stride() or q.dtype != q0.dtype:
            raise ValueError("the layers' queries must share shape and strides")
    dev = q0.device
    seq = _i32_dev(seq_lens, dev)
    nqa = _i32_dev(n_query, dev)
    kvs = (DustinKV * len(ks))()
    for i, k in enumerate(ks):
        kvs[i] = kv_view(k, page_table)
    max_len = _capacity(kvs[0]) if max_len is None else int(max_len)
    if out is None:
        out = torch.empty((len(qs), B, groups, max_len), dtype=torch.float32, device=dev)
    if (out.dtype != torch.float32 or out.dim() != 4 or out.shape[0] < len(qs) or out.shape[1] < B
            or out.shape[2] < groups or out.shape[3] < max_len or out.stride(3) != 1):
        raise ValueError(f"out must be fp32 [>= {len(qs)}, >= {B}, >= {groups}, >= {max_len}] with contiguous positions")
    heads_host = (ctypes.c_int32 * len(heads))(*[int(h) for h in heads])
    q_host = (ctypes.c_void_p * len(qs))(*[q.data_ptr() for q in qs])
    bt = _batch(B, max_len, nq_max, 0, seq, nqa)
    nbytes = lib().dustin_score_workspace(B, max_len, nq_max, len(heads) * len(qs))
    ws = workspace(nbytes, dev, "score", stream)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    args = (len(qs), q_host, q0.stride(0), q0.stride(1), q0.stride(2), Hq, heads_host, len(heads),
            kvs, ctypes.byref(bt), float(scale), int(groups), _ptr(out), out.stride(0), out.stride(1),
            out.stride(2), _ptr(ws), nbytes, _stream(stream))
    return Call(lib().dustin_score_per_layer, args, "dustin_score_per_layer",
                (tuple(qs), tuple(ks), kvs, bt, ws, heads_host, q_host), out)


def score_per_layer(qs, ks, seq_lens, heads, **kw):
    """Eq. 5 of each layer into its own output; returns out [L, B, groups, max_len]."""
    return plan_score_per_layer(qs, ks, seq_lens, heads, **kw)()


# ----------------------------------------------------------------------------- page estimator

def page_meta_empty(B: int, max_len: int, num_kv_heads: int, head_dim: int, page_size: int,
                    device) -> torch.Tensor:
    """A zeroed page-statistics array bf16 [B, ceil(max_len / page_size), Hkv, 2 d]."""
    P = (int(max_len) + page_size - 1) // page_size
    return torch.zeros((B, P, num_kv_heads, 2 * head_dim), dtype=torch.bfloat16, device=device)


def plan_page_meta(k: torch.Tensor, seq_lens, page_size: int, meta: torch.Tensor, *,
                   from_=None, max_span: Optional[int] = None, max_len: Optional[int] = None,
                   page_table: Optional[torch.Tensor] = None, stream=None) -> Call:
    """Prepared dustin_page_meta: per page of page_size positions and KV head, the channel
    max then min of K over the page's positions < N_b, into meta bf16 [B, P, Hkv, 2d].
    from_ (int32 [B]) limits the rebuild to pages holding a position >= from_b, with
    max_span bounding N_b - from_b (after an append: the old lengths and the largest T_b)."""
    _on_gpu(k, meta, page_table)
    dev = k.device
    seq = _i32_dev(seq_lens, dev)
    frm = _i32_dev(from_, dev)
    kv = kv_view(k, page_table)
    max_len = _capacity(kv) if max_len is None else int(max_len)
    max_span = max_len if max_span is None else int(max_span)
    if meta.dtype != torch.bfloat16 or meta.dim() != 4 or meta.stride(3) != 1 or meta.stride(2) != meta.shape[3]:
        raise ValueError("meta must be bf16 [B, pages, Hkv, 2d] with contiguous (Hkv, 2d) rows")
    B = seq.shape[0]
    pages = (max_len + int(page_size) - 1) // int(page_size)
    if (meta.shape[0] < B or meta.shape[1] < pages or meta.shape[2] != k.shape[2]
            or meta.shape[3] != 2 * k.shape[3]):
        raise ValueError(f"meta {tuple(meta.shape)} does not hold [{B}, {pages}, {k.shape[2]}, {2 * k.shape[3]}]")
    bt = _batch(B, max_len, 0, 0, seq)
    args = (ctypes.byref(kv), ctypes.byref(bt), _ptr(frm), max_span, int(page_size), _ptr(meta),
            meta.stride(0), meta.stride(1), meta.shape[1], _stream(stream))
    return Call(lib().dustin_page_meta, args, "dustin_page_meta", (k, meta, kv, bt, frm), meta)


def page_meta(k, seq_lens, page_size, meta=None, **kw):
    """Page statistics of K; returns meta (allocated when None)."""
    if meta is None:
        kv = kv_view(k, kw.get("page_table"))
        max_len = kw.get("max_len") or _capacity(kv)
        B = len(seq_lens) if not isinstance(seq_lens, torch.Tensor) else seq_lens.shape[0]
        meta = page_meta_empty(B, max_len, k.shape[2], k.shape[3], page_size, k.device)
    return plan_page_meta(k, seq_lens, page_size, meta, **kw)()


def plan_page_score(q: torch.Tensor, meta: torch.Tensor, seq_lens, heads: Sequence[int],
                    page_size: int, *, max_len: int, n_query=None, scale: Optional[float] = None,
                    groups: int = 1, init: Optional[torch.Tensor] = None,
                    out: Optional[torch.Tensor] = None, stream=None) -> Call:
    """Prepared dustin_page_score: Eq. 5 over pages with each page's bound on q . k, given
    to the page's positions.  q bf16 [B, nq_max, Hq, d]; meta from page_meta; init / out
    fp32 [B, groups, >= max_len]."""
    _on_gpu(q, meta, init, out)
    B, nq_max, Hq, d = q.shape
    dev = q.device
    Hkv = meta.shape[2]
    if meta.shape[3] != 2 * d or meta.dtype != torch.bfloat16 or meta.stride(3) != 1 or meta.stride(2) != 2 * d:
        raise ValueError("meta must be bf16 [B, pages, Hkv, 2d] matching q's head_dim")
    seq = _i32_dev(seq_lens, dev)
    nqa = _i32_dev(n_query, dev)
    max_len = int(max_len)
    pages = (max_len + int(page_size) - 1) // int(page_size)
    if meta.shape[0] < B or meta.shape[1] < pages:
        raise ValueError(f"meta {tuple(meta.shape)} holds fewer than {B} sequences or {pages} pages")
    if out is None:
        out = torch.empty((B, groups, max_len), dtype=torch.float32, device=dev)
    _check_scores(out, B, groups, max_len, "out")
    if init is not None:
        _check_scores(init, B, groups, max_len, "init")
    heads_host = (ctypes.c_int32 * len(heads))(*[int(h) for h in heads])
    bt = _batch(B, max_len, nq_max, 0, seq, nqa)
    nbytes = lib().dustin_page_score_workspace(B, max_len, int(page_size), nq_max, len(heads))
    ws = workspace(nbytes, dev, "page_score", stream)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    ins = (init.stride(0), init.stride(1)) if init is not None else (0, 0)
    args = (_ptr(q), q.stride(0), q.stride(1), q.stride(2), Hq, heads_host, len(heads), _ptr(meta),
            meta.stride(0), meta.stride(1), meta.shape[1], Hkv, d, int(page_size), ctypes.byref(bt),
            float(scale), int(groups), _ptr(init), ins[0], ins[1], _ptr(out), out.stride(0),
            out.stride(1), _ptr(ws), nbytes, _stream(stream))
    return Call(lib().dustin_page_score, args, "dustin_page_score", (q, meta, init, bt, ws, heads_host), out)


def page_score(q, meta, seq_lens, heads, page_size, **kw):
    """Page-estimator importance; returns out (positions >= N_b untouched)."""
    return plan_page_score(q, meta, seq_lens, heads, page_size, **kw)()


# ----------------------------------------------------------------------------- attention recovery rate

def plan_arr(s: torch.Tensor, idx: torch.Tensor, count: torch.Tensor, seq_lens, heads_per_group: int,
             *, window=None, max_len: Optional[int] = None, out: Optional[torch.Tensor] = None,
             stream=None) -> Call:
    """Prepared dustin_arr: windowed ARR (Eqs. 1-2) of the sets (idx, count) from s, the Eq. 5
    score over every served head and the window's queries.  Returns fp64 [B, groups]."""
    _on_gpu(s, idx, count, out)
    if s.dtype != torch.float32 or s.dim() != 3 or s.stride(2) != 1:
        raise ValueError("s must be fp32 [B, G or 1, N] with contiguous positions")
    if idx.dtype != torch.int32 or count.dtype != torch.int32 or idx.stride(2) != 1:
        raise ValueError("idx / count must be int32 (idx [B, G, k_max] contiguous in k)")
    B, G, k_max = idx.shape
    if count.shape != (B, G) or s.shape[0] < B or s.shape[1] not in (1, G):
        raise ValueError("count must be [B, G] and s [B, G or 1, N] for idx [B, G, k_max]")
    dev = s.device
    seq = _i32_dev(seq_lens, dev)
    if window is None:
        raise ValueError("window: the verification queries per sequence (an int or one per sequence)")
    if isinstance(window, int):
        win, w_max = None, int(window)
    else:
        win, w_max = _i32_dev(window, dev), 1 << 16
    count = count.contiguous()
    max_len = s.shape[2] if max_len is None else int(max_len)
    if out is None:
        out = torch.empty((B, G), dtype=torch.float64, device=dev)
    if out.dtype != torch.float64 or out.shape != (B, G) or not out.is_contiguous():
        raise ValueError("out must be a contiguous fp64 [B, G] tensor")
    if max_len > s.shape[2]:
        raise ValueError("max_len exceeds the score rows")
    bt = _batch(B, max_len, w_max, k_max, seq, win)
    s_sg = s.stride(1) if s.shape[1] > 1 else 0
    args = (_ptr(s), s.stride(0), s_sg, _ptr(idx), idx.stride(0), idx.stride(1), _ptr(count),
            ctypes.byref(bt), G, int(heads_per_group), _ptr(out), _stream(stream))
    return Call(lib().dustin_arr, args, "dustin_arr", (s, idx, count, bt), out)


def arr(s, idx, count, seq_lens, heads_per_group, **kw):
    """Windowed ARR of index sets; returns fp64 [B, groups]."""
    return plan_arr(s, idx, count, seq_lens, heads_per_group, **kw)()


# ----------------------------------------------------------------------------- top-k

def plan_topk(s_draft: Optional[torch.Tensor], s_target: Optional[torch.Tensor], seq_lens,
         k_max: int, *, budget=None, m=None, m_scalar: Optional[int] = None, n_sink: int = 4,
         n_window: int = 16, groups: int = 1, idx: Optional[torch.Tensor] = None,
         count: Optional[torch.Tensor] = None, hist_d: Optional[torch.Tensor] = None,
         hist_t: Optional[torch.Tensor] = None, stream=None) -> Call:
    """Prepared dustin_topk, Eq. 6.  s_draft / s_target fp32 [B, G' (1 = broadcast), N]; returns (idx int32
    [B, groups, k_max] ascending, only [:count] written; count int32 [B, groups]).  hist_d / hist_t: the
    rows' first-digit histograms (digit_hist [B, 4096], groups = 1) written with the scores; taken in place
    of a first pass and left at zero."""
    _on_gpu(s_draft, s_target, idx, count, hist_d, hist_t)
    for h in (hist_d, hist_t):
        if h is not None and (h.dtype != torch.int32 or not h.is_contiguous() or h.shape[-1] != DIGIT_BINS):
            raise ValueError("a histogram is a contiguous int32 [B, 4096] tensor")
    ref = s_target if s_target is not None else s_draft
    B, _, max_len = ref.shape
    dev = ref.device
    seq = _i32_dev(seq_lens, dev)
    bud = _i32_dev(budget, dev)
    ma = _i32_dev(m, dev)
    P = n_sink + n_window
    if m_scalar is None:
        m_scalar = 0 if s_draft is None else (k_max - P if s_target is None else (k_max - P) // 2)
    if idx is None:
        idx = torch.empty((B, groups, k_max), dtype=torch.int32, device=dev)
    if count is None:
        count = torch.empty((B, groups), dtype=torch.int32, device=dev)

    def st(s):
        if s is None:
            return 0, 0
        return s.stride(0), (0 if s.shape[1] == 1 else s.stride(1))

    dsb, dsg = st(s_draft)
    tsb, tsg = st(s_target)
    bt = _batch(B, max_len, 0, k_max, seq, None, bud, ma, m_scalar)
    nbytes = lib().dustin_topk_workspace(B, int(groups), max_len) if s_draft is not None and s_target is not None else 0
    ws = workspace(nbytes, dev, "topk", stream)
    args = (_ptr(s_draft), dsb, dsg, _ptr(s_target), tsb, tsg, ctypes.byref(bt), int(groups),
            int(n_sink), int(n_window), _ptr(idx), idx.stride(0), idx.stride(1), _ptr(count),
            _ptr(hist_d), _ptr(hist_t), _ptr(ws), nbytes, _stream(stream))
    return Call(lib().dustin_topk, args, "dustin_topk", (s_draft, s_target, bt, ws, hist_d, hist_t), (idx, count))


def topk(s_draft, s_target, seq_lens, k_max, **kw):
    """Eq. 6; returns (idx int32 [B, groups, k_max], count int32 [B, groups])."""
    return plan_topk(s_draft, s_target, seq_lens, k_max, **kw)()


def plan_read_probe(data: torch.Tensor, blocks: int = 1024, stream=None) -> "Call":
    """Prepared dustin_read_probe over a contiguous device tensor (its bytes, a multiple of
    16): a plain streaming read, for measuring the read rate.  Returns the per-workgroup
    wrapping sums of its 32-bit words, uint32 as int32 [blocks]."""
    if not data.is_cuda or not data.is_contiguous():
        raise ValueError("data must be a contiguous device tensor")
    nbytes = data.numel() * data.element_size()
    sums = torch.empty(int(blocks), dtype=torch.int32, device=data.device)
    args = (_ptr(data), nbytes, _ptr(sums), int(blocks), _stream(stream))
    return Call(lib().dustin_read_probe, args, "dustin_read_probe", (data,), sums)




# ----------------------------------------------------------------------------- attention

def _attn_common(q, k, v, seq_lens, n_query, page_table, max_len, out):
    _on_gpu(q, k, v, out, page_table)
    B, nq_max, Hq, d = q.shape
    dev = q.device
    kv, vv = kv_view(k, page_table), kv_view(v, page_table)
    if max_len is None:
        max_len = _capacity(kv) - nq_max
    if out is None:
        out = torch.empty_like(q)
    return B, nq_max, Hq, d, dev, kv, vv, int(max_len), out


def plan_sparse_verify_attn(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
                            idx: torch.Tensor, count: torch.Tensor, seq_lens, *, n_query=None,
                            page_table: Optional[torch.Tensor] = None,
                            scale: Optional[float] = None, out: Optional[torch.Tensor] = None,
                            max_len: Optional[int] = None, stream=None) -> Call:
    """Prepared verification attention over idx[b, g, :count] plus the causal verification window.
    q/out bf16 [B, T_max, Hq, 128]; idx int32 [B, G, k_max]; count int32 [B, G]."""
    B, nq_max, Hq, d, dev, kv, vv, max_len, out = _attn_common(q, k, v, seq_lens, n_query,
                                                                page_table, max_len, out)
    _on_gpu(idx, count)
    seq = _i32_dev(seq_lens, dev)
    nqa = _i32_dev(n_query, dev)
    G, k_max = idx.shape[1], idx.shape[2]
    bt = _batch(B, max_len, nq_max, k_max, seq, nqa)
    nbytes = lib().dustin_attn_workspace(B, Hq, kv.num_kv_heads, nq_max, k_max, 1)
    ws = workspace(nbytes, dev, "attn", stream)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    count = count.contiguous()
    args = (_ptr(q), q.stride(0), q.stride(1), q.stride(2), Hq, ctypes.byref(kv),
            ctypes.byref(vv), ctypes.byref(bt), _ptr(idx), idx.stride(0), idx.stride(1),
            _ptr(count), G, float(scale), _ptr(out), out.stride(0), out.stride(1), out.stride(2),
            _ptr(ws), nbytes, _stream(stream))
    return Call(lib().dustin_sparse_verify_attn, args, "dustin_sparse_verify_attn",
                (q, k, v, idx, count, kv, vv, bt, ws), out)


def plan_sparse_verify_attn_noalloc(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
                                    idx: torch.Tensor, count: torch.Tensor, seq_lens, *, out: torch.Tensor,
                                    n_query=None, page_table: Optional[torch.Tensor] = None,
                                    scale: Optional[float] = None, max_len: Optional[int] = None,
                                    stream=None) -> Call:
    """Prepared dustin_sparse_verify_attn_noalloc: the same attention with the split scratch
    taken from the library's fixed per-GPU array (no workspace; the caller passes out, and
    per-sequence arrays as int32 device tensors, so that calling the plan allocates nothing)."""
    B, nq_max, Hq, d, dev, kv, vv, max_len, out = _attn_common(q, k, v, seq_lens, n_query,
                                                                page_table, max_len, out)
    _on_gpu(idx, count)
    seq = _i32_dev(seq_lens, dev)
    nqa = _i32_dev(n_query, dev)
    G, k_max = idx.shape[1], idx.shape[2]
    bt = _batch(B, max_len, nq_max, k_max, seq, nqa)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    count = count.contiguous()
    args = (_ptr(q), q.stride(0), q.stride(1), q.stride(2), Hq, ctypes.byref(kv),
            ctypes.byref(vv), ctypes.byref(bt), _ptr(idx), idx.stride(0), idx.stride(1),
            _ptr(count), G, float(scale), _ptr(out), out.stride(0), out.stride(1), out.stride(2),
            _stream(stream))
    return Call(lib().dustin_sparse_verify_attn_noalloc, args, "dustin_sparse_verify_attn_noalloc",
                (q, k, v, idx, count, kv, vv, bt), out)


def sparse_verify_attn_noalloc(q, k, v, idx, count, seq_lens, **kw):
    """dustin_sparse_verify_attn_noalloc; returns out."""
    return plan_sparse_verify_attn_noalloc(q, k, v, idx, count, seq_lens, **kw)()


def sparse_verify_attn(q, k, v, idx, count, seq_lens, **kw):
    """Verification attention over idx[b, g, :count] plus the causal verification window;
    returns out bf16 [B, T_max, Hq, 128] (rows t >= T_b untouched)."""
    return plan_sparse_verify_attn(q, k, v, idx, count, seq_lens, **kw)()


def plan_dense_verify_attn(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, seq_lens, *,
                           n_query=None, page_table: Optional[torch.Tensor] = None,
                           scale: Optional[float] = None, out: Optional[torch.Tensor] = None,
                           max_len: Optional[int] = None, stream=None) -> Call:
    """Prepared full-cache verification attention over [0, N_b) plus the causal window."""
    B, nq_max, Hq, d, dev, kv, vv, max_len, out = _attn_common(q, k, v, seq_lens, n_query,
                                                                page_table, max_len, out)
    seq = _i32_dev(seq_lens, dev)
    nqa = _i32_dev(n_query, dev)
    bt = _batch(B, max_len, nq_max, 0, seq, nqa)
    nbytes = lib().dustin_attn_workspace(B, Hq, kv.num_kv_heads, nq_max, max_len, 0)
    ws = workspace(nbytes, dev, "attn", stream)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    args = (_ptr(q), q.stride(0), q.stride(1), q.stride(2), Hq, ctypes.byref(kv),
            ctypes.byref(vv), ctypes.byref(bt), float(scale), _ptr(out), out.stride(0),
            out.stride(1), out.stride(2), _ptr(ws), nbytes, _stream(stream))
    return Call(lib().dense_verify_attn, args, "dense_verify_attn", (q, k, v, kv, vv, bt, ws), out)


def dense_verify_attn(q, k, v, seq_lens, **kw):
    """Full-cache verification attention over [0, N_b) plus the causal window."""
    return plan_dense_verify_attn(q, k, v, seq_lens, **kw)()


# ----------------------------------------------------------------------------- KV append / commit

def plan_kv_append(k_new: torch.Tensor, v_new: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
                   seq_lens, *, n_query=None, page_table: Optional[torch.Tensor] = None,
                   max_len: Optional[int] = None, stream=None) -> Call:
    """Prepared dustin_kv_append: k_new / v_new bf16 [B, T_max, Hkv, d] go to cache
    positions [N_b, N_b + T_b) of k / v (contiguous [B, N_cap, Hkv, d] or paged)."""
    _on_gpu(k_new, v_new, k, v, page_table)
    B, nq_max = k_new.shape[0], k_new.shape[1]
    dev = k_new.device
    kv, vv = kv_view(k, page_table), kv_view(v, page_table)
    if max_len is None:
        max_len = _capacity(kv) - nq_max
    seq = _i32_dev(seq_lens, dev)
    nqa = _i32_dev(n_query, dev)
    bt = _batch(B, max_len, nq_max, 0, seq, nqa)
    args = (_ptr(k_new), k_new.stride(0), k_new.stride(1), k_new.stride(2), _ptr(v_new),
            v_new.stride(0), v_new.stride(1), v_new.stride(2), ctypes.byref(kv), ctypes.byref(vv),
            ctypes.byref(bt), _stream(stream))
    return Call(lib().dustin_kv_append, args, "dustin_kv_append", (k_new, v_new, k, v, kv, vv, bt), None)


def kv_append(k_new, v_new, k, v, seq_lens, **kw):
    """Writes the verification window's K and V into the caches at [N_b, N_b + T_b)."""
    return plan_kv_append(k_new, v_new, k, v, seq_lens, **kw)()


def plan_kv_commit(seq_lens: torch.Tensor, accepted: torch.Tensor, *, n_query=None,
                   nq_max: Optional[int] = None, stream=None) -> Call:
    """Prepared dustin_kv_commit: seq_lens += clamp(accepted, 0, T_b), in place."""
    _on_gpu(seq_lens, accepted, n_query)
    for t in (seq_lens, accepted) + (() if n_query is None else (n_query,)):
        if t.dtype != torch.int32 or not t.is_contiguous():
            raise ValueError("seq_lens, accepted and n_query must be contiguous int32 tensors")
    B = seq_lens.numel()
    if nq_max is None:
        if n_query is None:
            raise ValueError("kv_commit needs n_query or nq_max")
        nq_max = int(n_query.max().item())
    args = (_ptr(seq_lens), _ptr(accepted), _ptr(n_query), int(B), int(nq_max), _stream(stream))
    return Call(lib().dustin_kv_commit, args, "dustin_kv_commit", (seq_lens, accepted, n_query), seq_lens)


def kv_commit(seq_lens, accepted, **kw):
    """N_b += accepted_b (clamped to [0, T_b]); returns seq_lens."""
    return plan_kv_commit(seq_lens, accepted, **kw)()
