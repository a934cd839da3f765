"""dustin_sparse_verify_attn_noalloc (split scratch in the library's fixed per-GPU array)
against dustin_sparse_verify_attn (caller workspace): two calls in a row, the second
smaller and on a paged cache, each bit-identical to the workspace entry point's output and
within the attention tolerance of the oracle; a call needing more scratch than the array
holds is rejected before anything is enqueued."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_24957_amd as D
from paper_2606_24957_amd import workloads as W
from tests.gpu_util import bits, check_attention, gpu_rows, scale_of

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _shape(B, n, t, k, paged, name):
    n = tuple(n) if isinstance(n, (list, tuple)) else (n,) * B
    t = tuple(t) if isinstance(t, (list, tuple)) else (t,) * B
    return W.config("qwen72b").replace(name=name, B=B, seq_lens=n, n_query=t, budget=(k,) * B,
                                       m=((k - 20) // 2,) * B, layers=1, seed=31,
                                       planted=tuple(max(1, x // 100) for x in n), page_size=16 if paged else 0)


def _selection(s, seed):
    rng = np.random.default_rng(seed)
    idx = np.full((s.B, 1, s.k_max), -1, dtype=np.int32)
    cnt = np.zeros((s.B, 1), dtype=np.int32)
    for b in range(s.B):
        c = min(s.k_max, s.seq_lens[b])
        idx[b, 0, :c] = np.sort(rng.choice(s.seq_lens[b], c, replace=False))
        cnt[b, 0] = c
    return idx, cnt


def _compare(s, seed):
    L = W.make_layer(s, 0, DEV)
    seq = torch.tensor(s.seq_lens, dtype=torch.int32, device=DEV)
    nq = torch.tensor(s.n_query, dtype=torch.int32, device=DEV)
    idx_np, cnt_np = _selection(s, seed)
    idx, cnt = torch.from_numpy(idx_np).to(DEV), torch.from_numpy(cnt_np).to(DEV)
    ref = D.sparse_verify_attn(L.q, L.k, L.v, idx, cnt, seq, n_query=nq, page_table=L.page_table)
    out = torch.full_like(L.q, float("nan"))
    call = D.plan_sparse_verify_attn_noalloc(L.q, L.k, L.v, idx, cnt, seq, n_query=nq,
                                             page_table=L.page_table, out=out)
    call()
    torch.cuda.synchronize()
    for b, t in enumerate(s.n_query):
        assert torch.equal(out[b, :t].view(torch.int16), ref[b, :t].view(torch.int16)), f"{s.name} b={b}"
        assert torch.isnan(out[b, t:].float()).all()
    kk, vv = L.contiguous_kv(s)
    rows = O.all_rows(s.B, s.n_query, s.num_q_heads)[::3]
    oref = O.attention(bits(L.q), bits(kk), bits(vv), s.seq_lens, scale_of(s.head_dim), rows,
                       idx=idx_np, count=cnt_np)
    check_attention(gpu_rows(out, rows), oref, s.name + " noalloc")


def test_noalloc_equals_the_workspace_entry_point_on_two_calls_in_a_row():
    big = _shape(4, [6000, 5100, 4000, 6000], 5, 1024, False, "noalloc_first")
    small = _shape(2, [2500, 900], [9, 3], 300, True, "noalloc_second_smaller_paged")
    _compare(big, 1)
    _compare(small, 2)


def test_noalloc_rejects_a_call_beyond_its_scratch(monkeypatch):
    monkeypatch.setenv("DUSTIN_ATTN_SPLITS", "32")
    s = _shape(32, 300, 16, 256, False, "noalloc_too_big")
    assert D.lib().dustin_attn_workspace(32, 64, 8, 16, 256, 1) > (48 << 20)
    L = W.make_layer(s, 0, DEV)
    seq = torch.tensor(s.seq_lens, dtype=torch.int32, device=DEV)
    idx = torch.zeros((s.B, 1, 256), dtype=torch.int32, device=DEV)
    cnt = torch.full((s.B, 1), 256, dtype=torch.int32, device=DEV)
    out = torch.full_like(L.q, float("nan"))
    with pytest.raises(D.DustinError) as e:
        D.sparse_verify_attn_noalloc(L.q, L.k, L.v, idx, cnt, seq, out=out)
    assert e.value.status == D.ERR_SCRATCH_LIMIT
    torch.cuda.synchronize()
    assert torch.isnan(out.float()).all()
