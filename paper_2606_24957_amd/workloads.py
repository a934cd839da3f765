"""Seeded synthetic workloads for the sparse-verification step.

This module only draws inputs: random bf16 Q/K/V caches with planted salient keys, the
historical and draft-lookahead importance vectors a configuration hands in directly,
per-sequence lengths, budgets and page tables.  It holds none of the method's own
arithmetic (no scoring, no selection, no attention), so the HIP path and the CPU oracle
can both be fed from it without sharing code.

The shapes follow the paper's efficiency setting: Qwen2.5-72B-shaped target attention
(64 query heads, Appendix A) verified with a Qwen2.5-0.5B draft (14 query heads over 2 KV
heads of width 64), speculative depth 4 (Table sd_config), protected set of 4 sinks and
16 recent tokens (Appendix C).  The paper's own workload (PG-19 story continuation) is a
dataset; these seeded tensors stand in for it.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import Optional

import torch


@dataclass(frozen=True)
class DraftShape:
    """The draft model's scoring layers: query heads, KV heads, head width, number of
    scoring layers and the scoring heads used in each."""
    num_q_heads: int = 14
    num_kv_heads: int = 2
    head_dim: int = 64
    layers: int = 3
    heads: tuple = (0, 4, 7, 11)


@dataclass(frozen=True)
class Shape:
    name: str
    B: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    seq_lens: tuple           # N_b: committed context per sequence
    n_query: tuple            # T_b = gamma_b + 1 verification queries per sequence
    budget: tuple             # k_b, protected tokens included
    m: tuple                  # m_b, the draft share of the budget
    target_heads: tuple       # scoring heads of the target scoring layer
    draft: Optional[DraftShape]
    layers: int               # stacked target layers the attention runs over
    seed: int
    planted: tuple            # planted salient positions per (sequence, KV head)
    init_kind: Optional[str]  # historical target score handed in: None or a recipe name
    draft_given: bool = False  # S_draft handed in directly instead of recomputed
    page_size: int = 0        # 0 = contiguous [B, N_cap, Hkv, d] caches
    n_sink: int = 4
    n_window: int = 16
    groups: int = 1           # selection groups: 1 (one set per sequence) or Hkv

    @property
    def group_size(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def t_max(self) -> int:
        return max(self.n_query)

    @property
    def k_max(self) -> int:
        return max(self.budget)

    @property
    def n_max(self) -> int:
        return max(self.seq_lens)

    @property
    def n_cap(self) -> int:
        """Cache rows per sequence: the longest context plus the most verification tokens
        (the capacity every kernel call of the batch may address)."""
        return max(self.seq_lens) + max(self.n_query)

    @property
    def draft_gamma(self) -> tuple:
        """Draft queries per sequence (Gamma_b = T_b - 1)."""
        return tuple(t - 1 for t in self.n_query)

    def replace(self, **kw) -> "Shape":
        return dataclasses.replace(self, **kw)


def _default_m(k: int, n_sink: int = 4, n_window: int = 16) -> int:
    return (k - n_sink - n_window) // 2


def _uniform(B, v):
    return tuple([v] * B)


def config(name: str, **overrides) -> Shape:
    """Preset workloads.

    tiny        B=1, N=2048, Hq=8, Hkv=1, d=128, T=5, k=256, 1 scoring head, S_draft given
    qwen7b      B=4, N=8192, Hq=28, Hkv=4, T=5, k=1024, heads {0,14}, 3 draft layers
    qwen72b     B=16, N=32768, Hq=64, Hkv=8, T=5, k=2048, heads {0,17,34,51}, 8 layers
    ragged      B=16, N_b ~ U[4096, 65536], gamma_b ~ U{2..8}, k_b = N_b/16, paged by 16
    long131k    B=8, N=131072, T=7, k=4096, 24 layers, heavy-tailed history
    """
    if name == "tiny":
        B, k = 1, 256
        s = Shape(name, B, 8, 1, 128, _uniform(B, 2048), _uniform(B, 5), _uniform(B, k),
                  _uniform(B, _default_m(k)), (0,), None, 1, 1, (32,), "softmax_normal2",
                  draft_given=True)
    elif name == "qwen7b":
        B, k = 4, 1024
        s = Shape(name, B, 28, 4, 128, _uniform(B, 8192), _uniform(B, 5), _uniform(B, k),
                  _uniform(B, _default_m(k)), (0, 14), DraftShape(), 1, 2, (82,),
                  "dirichlet0.1")
    elif name == "qwen72b":
        B, k = 16, 2048
        s = Shape(name, B, 64, 8, 128, _uniform(B, 32768), _uniform(B, 5), _uniform(B, k),
                  _uniform(B, _default_m(k)), (0, 17, 34, 51), DraftShape(), 8, 3000, (328,),
                  None)
    elif name == "ragged":
        B = 16
        g = torch.Generator().manual_seed(4000)
        n = torch.randint(4096, 65537, (B,), generator=g).tolist()
        gam = torch.randint(2, 9, (B,), generator=g).tolist()
        k = [x // 16 for x in n]
        s = Shape(name, B, 64, 8, 128, tuple(n), tuple(x + 1 for x in gam), tuple(k),
                  tuple(_default_m(x) for x in k), (0, 17, 34, 51), DraftShape(), 8, 4000,
                  tuple(round(0.01 * x) for x in n), None, page_size=16)
    elif name == "long131k":
        B, k = 8, 4096
        s = Shape(name, B, 64, 8, 128, _uniform(B, 131072), _uniform(B, 7), _uniform(B, k),
                  _uniform(B, _default_m(k)), (0, 17, 34, 51), DraftShape(), 24, 5000,
                  (1311,), "pareto1.2")
    else:
        raise KeyError(f"unknown workload {name!r}")
    if overrides:
        s = s.replace(**overrides)
    return s


def per_kv_head(s: Shape) -> Shape:
    """The same workload with one index set per KV head (groups = Hkv): each KV head then
    needs target scoring heads of its own, so the preset takes one per KV head (head
    g * G + g mod G of group g, G = Hq / Hkv), in place of heads spread over half the groups."""
    gs = s.num_q_heads // s.num_kv_heads
    heads = tuple(g * gs + g % gs for g in range(s.num_kv_heads))
    return s.replace(name=s.name + "_per_kv_head", groups=s.num_kv_heads, target_heads=heads)


def shrink(s: Shape, B: int = None, n: int = None, k: int = None, layers: int = None,
           t: int = None, name: str = None) -> Shape:
    """A smaller copy of a preset with uniform per-sequence values, for oracle-sized tests."""
    B = s.B if B is None else B
    ns = s.seq_lens[:B] if n is None else _uniform(B, n)
    ts = s.n_query[:B] if t is None else _uniform(B, t)
    ks = s.budget[:B] if k is None else _uniform(B, k)
    ms = tuple(_default_m(x, s.n_sink, s.n_window) for x in ks)
    planted = tuple(max(1, round(0.01 * x)) for x in ns)
    return s.replace(name=name or (s.name + "_small"), B=B, seq_lens=tuple(ns),
                     n_query=tuple(ts), budget=tuple(ks), m=ms, planted=planted,
                     layers=s.layers if layers is None else layers)


def _gen(device, seed):
    return torch.Generator(device=device).manual_seed(int(seed))


def _planted_count(s: Shape, b: int) -> int:
    return s.planted[b] if len(s.planted) == s.B else s.planted[0]


def plant_positions(s: Shape, seed: int, device) -> list:
    """positions[b][g]: distinct planted salient positions in [n_sink, N_b - n_window)."""
    g = _gen("cpu", seed)
    out = []
    for b in range(s.B):
        row = []
        lo, hi = s.n_sink, max(s.n_sink, s.seq_lens[b] - s.n_window)
        cnt = min(_planted_count(s, b), hi - lo)
        for _ in range(s.num_kv_heads):
            row.append((torch.randperm(hi - lo, generator=g)[:cnt] + lo).to(device))
        out.append(row)
    return out


def _plant(kc, q, positions, n_query, group_size, gen):
    """K[b, p, g] = bf16(4 * mean(q over the group's rows) + N(0,1)) at the planted p."""
    Hkv, d = kc.shape[2], kc.shape[3]
    for b in range(len(positions)):
        for gi, pos in enumerate(positions[b]):
            if gi >= Hkv or pos.numel() == 0:
                continue
            rows = q[b, :n_query[b], gi * group_size:(gi + 1) * group_size, :].float()
            qbar = rows.reshape(-1, d).mean(dim=0)
            noise = torch.randn((pos.numel(), d), generator=gen, device=kc.device)
            kc[b, pos, gi, :] = (4.0 * qbar + noise).to(kc.dtype)


@dataclass
class Layer:
    """One target layer's verification inputs."""
    q: torch.Tensor                       # bf16 [B, T_max, Hq, d]
    k: torch.Tensor                       # bf16 [B, N_cap, Hkv, d] or [P, page, Hkv, d]
    v: torch.Tensor
    page_table: Optional[torch.Tensor] = None   # int32 [B, max_pages] (paged only)

    def contiguous_kv(self, s: Shape):
        """[B, N_cap, Hkv, d] views of a paged cache (a host-side gather for the checker)."""
        if self.page_table is None:
            return self.k, self.v
        ps = s.page_size
        n_pages = (s.n_cap + ps - 1) // ps
        pt = self.page_table[:, :n_pages].long()
        kk = self.k[pt].reshape(s.B, n_pages * ps, s.num_kv_heads, s.head_dim)
        vv = self.v[pt].reshape(s.B, n_pages * ps, s.num_kv_heads, s.head_dim)
        return kk, vv


def _pages_per_seq(s: Shape):
    return [(n + t + s.page_size - 1) // s.page_size for n, t in zip(s.seq_lens, s.n_query)]


def make_page_table(s: Shape, seed: int, device):
    """A random permutation of the physical pages, consecutive runs of it per sequence.
    Unused table entries are 0 (a valid page) so no read can leave the pool."""
    per = _pages_per_seq(s)
    total = sum(per)
    perm = torch.randperm(total, generator=_gen("cpu", seed)).to(torch.int32)
    maxp = (s.n_cap + s.page_size - 1) // s.page_size
    pt = torch.zeros((s.B, maxp), dtype=torch.int32)
    off = 0
    for b, c in enumerate(per):
        pt[b, :c] = perm[off:off + c]
        off += c
    return pt.to(device), total


def make_layer(s: Shape, layer: int, device) -> Layer:
    seed = s.seed + layer
    gen = _gen(device, seed)
    B, Hq, Hkv, d = s.B, s.num_q_heads, s.num_kv_heads, s.head_dim
    q = torch.randn((B, s.t_max, Hq, d), generator=gen, device=device, dtype=torch.bfloat16)
    kc = torch.randn((B, s.n_cap, Hkv, d), generator=gen, device=device, dtype=torch.bfloat16)
    vc = torch.randn((B, s.n_cap, Hkv, d), generator=gen, device=device, dtype=torch.bfloat16)
    pos = plant_positions(s, seed, device)
    _plant(kc, q, pos, s.n_query, s.group_size, gen)
    if not s.page_size:
        return Layer(q, kc, vc)
    pt, total = make_page_table(s, seed + 7919, device)
    ps = s.page_size
    kp = torch.zeros((total, ps, Hkv, d), device=device, dtype=torch.bfloat16)
    vp = torch.zeros_like(kp)
    for b, c in enumerate(_pages_per_seq(s)):
        pages = pt[b, :c].long()
        rows = min(c * ps, s.seq_lens[b] + s.n_query[b])
        src_k = torch.zeros((c * ps, Hkv, d), device=device, dtype=torch.bfloat16)
        src_v = torch.zeros_like(src_k)
        src_k[:rows] = kc[b, :rows]
        src_v[:rows] = vc[b, :rows]
        kp[pages] = src_k.reshape(c, ps, Hkv, d)
        vp[pages] = src_v.reshape(c, ps, Hkv, d)
    del kc, vc
    return Layer(q, kp, vp, pt)


@dataclass
class Estimation:
    """Inputs of the estimation half of a step."""
    q_target: torch.Tensor                 # bf16 [B, 1, Hq, d]: last accepted token's query
    init_target: Optional[torch.Tensor]    # fp32 [B, 1, N_max] historical score or None
    s_draft_given: Optional[torch.Tensor]  # fp32 [B, 1, N_max] (draft_given presets)
    draft_q: list = field(default_factory=list)   # per draft layer bf16 [B, Gmax, Hq_d, d_d]
    draft_k: list = field(default_factory=list)   # per draft layer bf16 [B, N_cap, Hkv_d, d_d]


def _history(kind, s: Shape, gen, device):
    B, N = s.B, s.n_max
    if kind is None:
        return None
    if kind == "softmax_normal2":       # exp-normalised N(0, sigma=2) logits
        z = torch.randn((B, 1, N), generator=gen, device=device) * 2.0
        return torch.softmax(z, dim=-1).float()
    if kind == "dirichlet0.1":          # Gamma(0.1) draws, normalised
        u = torch._standard_gamma(torch.full((B, 1, N), 0.1, device=device), generator=gen)
        return (u / u.sum(dim=-1, keepdim=True)).float()
    if kind == "pareto1.2":             # Pareto(alpha=1.2, x_m=1) draws, normalised
        u = torch.rand((B, 1, N), generator=gen, device=device)
        x = (1.0 - u).clamp_min(1e-30).pow(-1.0 / 1.2)
        return (x / x.sum(dim=-1, keepdim=True)).float()
    raise KeyError(kind)


def make_estimation(s: Shape, layer0: Layer, device) -> Estimation:
    gen = _gen(device, s.seed + 100003)
    q_target = layer0.q[:, :1].contiguous()
    init = _history(s.init_kind, s, gen, device)
    sd = None
    if s.draft_given:                   # four draft steps of exp-normalised 3*N(0,1) logits
        z = torch.randn((s.B, 4, s.n_max), generator=gen, device=device) * 3.0
        sd = torch.softmax(z, dim=-1).sum(dim=1, keepdim=True).float()
    est = Estimation(q_target, init, sd)
    if s.draft is not None:
        dr = s.draft
        gmax = max(s.draft_gamma)
        tpos = plant_positions(s, s.seed, device)
        step = max(1, s.num_kv_heads // dr.num_kv_heads)
        for l in range(dr.layers):
            qd = torch.randn((s.B, gmax, dr.num_q_heads, dr.head_dim), generator=gen,
                             device=device, dtype=torch.bfloat16)
            kd = torch.randn((s.B, s.n_cap, dr.num_kv_heads, dr.head_dim), generator=gen,
                             device=device, dtype=torch.bfloat16)
            dpos = [[tpos[b][gd * step] for gd in range(dr.num_kv_heads)] for b in range(s.B)]
            _plant(kd, qd, dpos, s.draft_gamma, dr.num_q_heads // dr.num_kv_heads, gen)
            est.draft_q.append(qd)
            est.draft_k.append(kd)
    return est


def bf16_bits(t: torch.Tensor):
    """Raw uint16 patterns of a bf16 tensor as a numpy array (host copy)."""
    import numpy as np
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def plant_ramp(s: Shape, layer: Layer, positions, coefs, window_coef: Optional[float] = None,
               window_slot: int = 1):
    """Peaked attention for the parity tests: K[b, p_j, g] = bf16(c_j * mean(q over the KV
    head's query rows)) for the positions p_j of positions[b] and the coefficients c_j
    (the same positions in every KV head), and, when window_coef is given, the same with
    window_coef at window position N_b + window_slot (seen by queries t >= window_slot).
    With queries scaled by a power of two beforehand, these keys' logits lie tens of units
    apart, so an online softmax meets its running maximum at many steps.  Writes through
    the page table when the layer is paged."""
    Hkv, d, gs = s.num_kv_heads, s.head_dim, s.group_size
    for b in range(s.B):
        t = s.n_query[b]
        if t == 0:
            continue
        rows = layer.q[b, :t].float()  # [t, Hq, d]
        qbar = rows.reshape(t, Hkv, gs, d).mean(dim=(0, 2))  # [Hkv, d]
        pos = list(positions[b]) if positions is not None else []
        coef = list(coefs)[:len(pos)]
        if window_coef is not None and window_slot < t:
            pos.append(s.seq_lens[b] + window_slot)
            coef.append(window_coef)
        for p, c in zip(pos, coef):
            row = (float(c) * qbar).to(torch.bfloat16)  # [Hkv, d]
            if layer.page_table is None:
                layer.k[b, int(p)] = row
            else:
                ps = s.page_size
                page = int(layer.page_table[b, int(p) // ps].item())
                layer.k[page, int(p) % ps] = row
