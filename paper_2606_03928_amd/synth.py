"""Seeded synthetic inputs for the eviction round (shared by tests, bench and smoke).

This module only draws random tensors; it holds none of the method's
arithmetic.  The shapes follow the Qwen3 family (8 KV heads, head_dim 128,
GQA groups of 2-8 query heads) and the distributions follow what the paper
reports about real caches:

* keys and queries are i.i.d. N(0, 1), rounded to the storage dtype;
* the first few slots of a trace are attention sinks whose key rows are scaled
  up (the paper's per-position Range analysis treats the first four tokens as
  sinks, Appendix D);
* a small fraction of value rows carry large magnitudes (the Range outliers of
  Sec. 3.1): each row independently, with probability ``out_p``, is scaled by a
  factor drawn log-uniformly from ``[out_lo, out_hi]`` (a fixed factor when the
  two are equal).

Cache layout: ``k``, ``v`` are ``[n_inst, N, d]`` with ``N = K + B`` slots per
head instance (instance = layer x batch x KV head, in that nesting order);
``q_win`` is ``[n_inst, G, w, d]`` (the G query heads of the group times the w
most recent queries); ``q_dec`` is ``[n_inst, G, d]``.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Optional

import torch


@dataclasses.dataclass(frozen=True)
class RoundConfig:
    name: str
    layers: int
    batch: int
    h_kv: int
    h_q: int
    d: int
    dtype: str          # "bf16" or "f32"
    K: int              # persistent budget
    B: int              # recency buffer
    w: int              # observation-window queries per query head
    Nv: int             # reserved value slots
    pool: int = 7       # average-pooling kernel (odd)
    sinks: int = 0      # leading key rows scaled by sink_scale
    sink_scale: float = 10.0
    out_p: float = 0.0  # probability that a value row is an outlier
    out_lo: float = 1.0
    out_hi: float = 1.0
    rounds: int = 1
    seed: int = 0

    @property
    def n_inst(self) -> int:
        return self.layers * self.batch * self.h_kv

    @property
    def G(self) -> int:
        return self.h_q // self.h_kv

    @property
    def N(self) -> int:
        return self.K + self.B

    @property
    def R(self) -> int:
        return self.G * self.w

    @property
    def torch_dtype(self) -> torch.dtype:
        return {"bf16": torch.bfloat16, "f32": torch.float32}[self.dtype]

    @property
    def elem_bytes(self) -> int:
        return 2 if self.dtype == "bf16" else 4

    def with_(self, **kw) -> "RoundConfig":
        return dataclasses.replace(self, **kw)


# The five workloads: a tiny CPU-checkable round and four Qwen3-shaped ones.
CONFIGS: Dict[str, RoundConfig] = {
    "tiny": RoundConfig(name="tiny", layers=1, batch=1, h_kv=2, h_q=4, d=64, dtype="f32",
                        K=128, B=32, w=8, Nv=8, pool=7, sinks=0, out_p=0.02, out_lo=50.0,
                        out_hi=50.0),
    "qwen3-1.7b": RoundConfig(name="qwen3-1.7b", layers=1, batch=1, h_kv=8, h_q=16, d=128,
                              dtype="bf16", K=2048, B=128, w=128, Nv=64, pool=7, sinks=4,
                              out_p=0.005, out_lo=20.0, out_hi=100.0, rounds=100),
    "qwen3-8b": RoundConfig(name="qwen3-8b", layers=36, batch=8, h_kv=8, h_q=32, d=128,
                            dtype="bf16", K=4096, B=128, w=128, Nv=128, pool=7, sinks=4,
                            out_p=0.005, out_lo=20.0, out_hi=100.0),
    "qwen3-14b": RoundConfig(name="qwen3-14b", layers=40, batch=32, h_kv=8, h_q=40, d=128,
                             dtype="bf16", K=8192, B=256, w=256, Nv=256, pool=7, sinks=4,
                             out_p=0.01, out_lo=50.0, out_hi=50.0),
    "qwen3-32b": RoundConfig(name="qwen3-32b", layers=64, batch=64, h_kv=8, h_q=64, d=128,
                             dtype="bf16", K=8192, B=128, w=128, Nv=256, pool=7, sinks=4,
                             out_p=0.005, out_lo=20.0, out_hi=100.0, rounds=192),
}


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def _fill_normal(out: torch.Tensor, gen: torch.Generator, chunk_rows: int) -> None:
    """Fill ``out`` ([n, ...]) with N(0,1) drawn in fp32, chunk by chunk."""
    n = out.shape[0]
    for s in range(0, n, chunk_rows):
        e = min(n, s + chunk_rows)
        t = torch.randn(out[s:e].shape, generator=gen, device=out.device, dtype=torch.float32)
        out[s:e].copy_(t)


def _outlier_scale(shape, cfg: RoundConfig, gen: torch.Generator, device) -> torch.Tensor:
    """Per-row scale factor: 1, or an outlier factor with probability out_p."""
    hit = torch.rand(shape, generator=gen, device=device) < cfg.out_p
    if cfg.out_hi > cfg.out_lo:
        u = torch.rand(shape, generator=gen, device=device)
        lo, hi = math.log(cfg.out_lo), math.log(cfg.out_hi)
        fac = torch.exp(lo + (hi - lo) * u)
    else:
        fac = torch.full(shape, float(cfg.out_lo), device=device)
    return torch.where(hit, fac, torch.ones_like(fac))


def make_round_inputs(cfg: RoundConfig, device="cpu", seed: Optional[int] = None,
                      n_inst: Optional[int] = None, chunk_inst: int = 256) -> dict:
    """Allocate and fill one round's cache, window queries and decode queries.

    ``n_inst`` overrides the instance count (a prefix of the full workload:
    the first instances of layer 0, batch 0, ...).  Drawing happens in chunks
    of ``chunk_inst`` instances so fp32 temporaries stay small.
    """
    seed = cfg.seed if seed is None else seed
    n = cfg.n_inst if n_inst is None else n_inst
    dt = cfg.torch_dtype
    N, d, G, w = cfg.N, cfg.d, cfg.G, cfg.w
    k = torch.empty((n, N, d), dtype=dt, device=device)
    v = torch.empty((n, N, d), dtype=dt, device=device)
    q_win = torch.empty((n, G, w, d), dtype=dt, device=device)
    q_dec = torch.empty((n, G, d), dtype=dt, device=device)
    gk, gv, gq, gs = (_gen(device, seed * 4 + i) for i in range(4))
    for s in range(0, n, chunk_inst):
        e = min(n, s + chunk_inst)
        kk = torch.randn((e - s, N, d), generator=gk, device=device, dtype=torch.float32)
        if cfg.sinks > 0:
            kk[:, :cfg.sinks, :] *= cfg.sink_scale
        k[s:e].copy_(kk)
        del kk
        vv = torch.randn((e - s, N, d), generator=gv, device=device, dtype=torch.float32)
        if cfg.out_p > 0:
            vv *= _outlier_scale((e - s, N, 1), cfg, gs, device)
        v[s:e].copy_(vv)
        del vv
    _fill_normal(q_win, gq, chunk_inst)
    _fill_normal(q_dec, gq, chunk_inst)
    return {"k": k, "v": v, "q_win": q_win, "q_dec": q_dec}


def refresh_buffer(inputs: dict, cfg: RoundConfig, step_seed: int) -> None:
    """Write B fresh token rows into the buffer slots [K, N) and a fresh window.

    Models what the decoder does between two rounds: B new (k, v) pairs are
    appended after the K survivors, and the window holds the newest queries.
    Sinks are not redrawn (they sit at the start of the trace).
    """
    k, v, q_win = inputs["k"], inputs["v"], inputs["q_win"]
    device = k.device
    n = k.shape[0]
    g = _gen(device, 1_000_003 * (step_seed + 1) + cfg.seed)
    kk = torch.randn((n, cfg.B, cfg.d), generator=g, device=device, dtype=torch.float32)
    k[:, cfg.K:, :].copy_(kk)
    del kk
    vv = torch.randn((n, cfg.B, cfg.d), generator=g, device=device, dtype=torch.float32)
    if cfg.out_p > 0:
        vv *= _outlier_scale((n, cfg.B, 1), cfg, g, device)
    v[:, cfg.K:, :].copy_(vv)
    del vv
    _fill_normal(q_win, g, 256)


def draw_round_tokens(cfg: RoundConfig, device, n_inst: int, step_seed: int) -> dict:
    """The tokens of one period between two rounds, drawn without touching a cache.

    Returns ``k_new``, ``v_new`` ([n_inst, B, d]: the B rows the decoder appends
    to the buffer slots [K, N)), ``q_win`` ([n_inst, G, w, d], the newest
    queries) and ``q_dec`` ([n_inst, G, d], the queries of the decode step that
    follows the round), from the same distributions as ``make_round_inputs``
    (no sinks: those sit at the start of the trace).  The first three are the
    draws of ``refresh_buffer`` with the same ``step_seed``.
    """
    dt = cfg.torch_dtype
    n, B, d = n_inst, cfg.B, cfg.d
    g = _gen(device, 1_000_003 * (step_seed + 1) + cfg.seed)
    k_new = torch.randn((n, B, d), generator=g, device=device, dtype=torch.float32).to(dt)
    vv = torch.randn((n, B, d), generator=g, device=device, dtype=torch.float32)
    if cfg.out_p > 0:
        vv *= _outlier_scale((n, B, 1), cfg, g, device)
    v_new = vv.to(dt)
    del vv
    q_win = torch.empty((n, cfg.G, cfg.w, d), dtype=dt, device=device)
    _fill_normal(q_win, g, 256)
    q_dec = torch.empty((n, cfg.G, d), dtype=dt, device=device)
    _fill_normal(q_dec, g, 256)
    return {"k_new": k_new, "v_new": v_new, "q_win": q_win, "q_dec": q_dec}
