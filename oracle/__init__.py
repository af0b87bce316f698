"""CPU oracle for one VaSE-AttnV eviction round.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU-baseline
leg of the benchmark may import this package.  The product library never links,
loads or calls it, and the two share no source.

The arithmetic lives in ``vase_oracle.c`` (plain C, double precision, OpenMP over
independent head instances).  This module builds it with gcc, loads it with
ctypes and converts arrays: bf16/fp32 tensors are upcast exactly to float64
before they reach the C code.

Paper references (the paper is "Value-Aware Stochastic KV Cache Eviction for
Reasoning Models"):
  * ``score``   -- Eq. (2) over Eq. (1) rows, with average pooling (Sec. 2, footnote)
  * ``vrange``  -- Eq. (5), Range(v) (Sec. 3.1)
  * ``select``  -- VaSE-AttnV reservation + weighted sampling (Sec. 3.2)
  * ``compact`` -- periodic eviction restores the cache to K slots (Sec. 2)
  * ``decode``  -- Eq. (1)
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "vase_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libvase_oracle.so")
_lock = threading.Lock()
_lib = None

FLAG_DETERMINISTIC = 1

OK = 0
ERR_ARG = -1
ERR_NOMEM = -2
ERR_BUDGET = -3


def build(force: bool = True) -> str:
    """Compile libvase_oracle.so with gcc (IEEE fp32, no contraction)."""
    if not force and os.path.exists(_LIB_PATH) and \
            os.path.getmtime(_LIB_PATH) >= os.path.getmtime(_SRC):
        return _LIB_PATH
    tmp = _LIB_PATH + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared", "-Wall", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(_LIB_PATH) or \
                os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        i32, u32, u64, sz = ctypes.c_int, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_size_t
        lib.vo_philox4x32_10.argtypes = [P, P, P]
        lib.vo_philox4x32_10.restype = None
        lib.vo_uniform.argtypes = [u32]
        lib.vo_uniform.restype = ctypes.c_float
        lib.vo_neglog.argtypes = [ctypes.c_float]
        lib.vo_neglog.restype = ctypes.c_float
        lib.vo_neglog_n.argtypes = [P, P, ctypes.c_int64]
        lib.vo_neglog_n.restype = None
        lib.vo_noise.argtypes = [u64, u32, u32, u32, ctypes.c_int32]
        lib.vo_noise.restype = ctypes.c_float
        lib.vo_score.argtypes = [P, P, i32, i32, i32, i32, i32, i32, P, P]
        lib.vo_score.restype = i32
        lib.vo_vrange.argtypes = [P, i32, i32, i32, i32, P]
        lib.vo_vrange.restype = i32
        lib.vo_select.argtypes = [P, P, i32, u32, i32, i32, i32, u64, u32, u32, P, P]
        lib.vo_select.restype = i32
        lib.vo_compact.argtypes = [P, P, P, i32, i32, i32, sz]
        lib.vo_order_compact.argtypes = [P, P, i32, i32, i32, P, P]
        lib.vo_order_compact.restype = i32
        lib.vo_compact.restype = i32
        lib.vo_decode.argtypes = [P, P, P, i32, i32, i32, i32, i32, P]
        lib.vo_value_score.restype = i32
        lib.vo_value_score.argtypes = [P, i32, u32, i32, i32, i32, i32, u64, u32, P]
        lib.vo_cos2pi.restype = ctypes.c_float
        lib.vo_cos2pi.argtypes = [ctypes.c_float]
        lib.vo_dkv_gaussian.restype = None
        lib.vo_dkv_gaussian.argtypes = [u64, u32, u32, i32, i32, P]
        lib.vo_dkv_score_g.restype = i32
        lib.vo_dkv_score_g.argtypes = [P, P, P, i32, i32, i32, i32, i32, P]
        lib.vo_dkv_score.restype = i32
        lib.vo_dkv_score.argtypes = [P, P, i32, u32, i32, i32, i32, i32, u64, u32, P]
        lib.vo_decode.restype = i32
        lib.vo_decode_lse.argtypes = [P, P, i32, i32, i32, i32, i32, P]
        lib.vo_decode_lse.restype = i32
        lib.vo_score_lse.argtypes = [P, P, P, i32, i32, i32, i32, i32, i32, P]
        lib.vo_score_lse.restype = i32
        lib.vo_quantize.argtypes = [P, i32, i32, i32, i32, i32, i32, i32, P, P, P, P, P]
        lib.vo_quantize.restype = i32
        lib.vo_dequantize.argtypes = [P, P, P, P, i32, i32, i32, i32, i32, i32, i32, i32, P]
        lib.vo_dequantize.restype = i32
        _lib = lib
        return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _f64(x) -> np.ndarray:
    """Exact upcast of a torch tensor (bf16/fp16/fp32/fp64) or array to float64."""
    try:
        import torch
        if isinstance(x, torch.Tensor):
            return np.ascontiguousarray(x.detach().to("cpu", torch.float64).numpy())
    except ImportError:  # pragma: no cover
        pass
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _f32(x) -> np.ndarray:
    try:
        import torch
        if isinstance(x, torch.Tensor):
            assert x.dtype == torch.float32
            return np.ascontiguousarray(x.detach().cpu().numpy())
    except ImportError:  # pragma: no cover
        pass
    a = np.asarray(x)
    assert a.dtype == np.float32
    return np.ascontiguousarray(a)


def _check(rc: int, what: str):
    if rc != OK:
        raise RuntimeError("oracle %s failed with code %d" % (what, rc))


# --------------------------------------------------------------------------
# scalar building blocks
# --------------------------------------------------------------------------
def philox4x32_10(ctr, key) -> np.ndarray:
    lib = _load()
    c = np.asarray(ctr, dtype=np.uint32).copy()
    k = np.asarray(key, dtype=np.uint32).copy()
    out = np.zeros(4, dtype=np.uint32)
    lib.vo_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def uniform(x: int) -> float:
    return float(np.float32(_load().vo_uniform(int(x))))


def neglog(u: float) -> np.float32:
    return np.float32(_load().vo_neglog(float(np.float32(u))))


def neglog_array(u: np.ndarray) -> np.ndarray:
    uu = np.ascontiguousarray(u, dtype=np.float32)
    out = np.empty_like(uu)
    _load().vo_neglog_n(_ptr(uu), _ptr(out), uu.size)
    return out


def noise(seed: int, inst_id: int, rnd: int, slot: int, purpose: int = 0) -> np.float32:
    return np.float32(_load().vo_noise(seed, inst_id, rnd, purpose, slot))


# --------------------------------------------------------------------------
# the round's steps
# --------------------------------------------------------------------------
def score(q_win, k_cache, K: int, pool: int, return_abar: bool = False):
    """Pooled window-mean attention score.

    q_win: [n_inst, G, w, d] (or [n_inst, R, d]); k_cache: [n_inst, N, d].
    Returns attn [n_inst, K] float32 (and, if asked, the unpooled row mean
    over all N slots as float64 [n_inst, N]).
    """
    q = _f64(q_win)
    k = _f64(k_cache)
    n_inst, N, d = k.shape
    q = q.reshape(n_inst, -1, d)
    R = q.shape[1]
    attn = np.zeros((n_inst, K), dtype=np.float32)
    abar = np.zeros((n_inst, N), dtype=np.float64) if return_abar else None
    rc = _load().vo_score(_ptr(q), _ptr(k), n_inst, R, N, K, d, pool, _ptr(attn),
                          _ptr(abar) if abar is not None else None)
    _check(rc, "score")
    return (attn, abar) if return_abar else attn


def vrange(v_cache, K: int) -> np.ndarray:
    v = _f64(v_cache)
    n_inst, N, d = v.shape
    out = np.zeros((n_inst, K), dtype=np.float32)
    _check(_load().vo_vrange(_ptr(v), n_inst, N, K, d, _ptr(out)), "vrange")
    return out


VALUE_RANGE, VALUE_L2, VALUE_VAR, VALUE_RANDOM = 0, 1, 2, 3


def value_score(v_cache, K: int, kind: int, seed: int = 0, rnd: int = 0, inst_base: int = 0,
                n_inst: int = None) -> np.ndarray:
    """Value score of the K candidates: Range (Eq. 5), L2 or Var (Appendix A), or a
    Philox uniform per slot (random reservation, Appendix D) -> [n_inst, K] float32."""
    if kind == VALUE_RANDOM and v_cache is None:
        v, N, d = None, K, 1
    else:
        v = _f64(v_cache)
        n_inst, N, d = v.shape
    out = np.zeros((n_inst, K), dtype=np.float32)
    rc = _load().vo_value_score(_ptr(v) if v is not None else None, n_inst, inst_base & 0xFFFFFFFF,
                                N, K, d, kind, seed & 0xFFFFFFFFFFFFFFFF, rnd & 0xFFFFFFFF, _ptr(out))
    _check(rc, "value_score")
    return out


def select(attn, vr, K: int, B: int, Nv: int, seed: int, rnd: int, inst_base: int = 0,
           flags: int = 0, return_keys: bool = False):
    """Survivor map src [n_inst, K] int32 (and the selection keys if asked)."""
    a = _f32(attn)
    r = _f32(vr)
    n_inst = a.shape[0]
    assert a.shape == (n_inst, K) and r.shape == (n_inst, K)
    src = np.zeros((n_inst, K), dtype=np.int32)
    keys = np.zeros((n_inst, K), dtype=np.float32) if return_keys else None
    rc = _load().vo_select(_ptr(a), _ptr(r), n_inst, inst_base, K, B, Nv, seed, rnd, flags,
                           _ptr(src), _ptr(keys) if keys is not None else None)
    _check(rc, "select")
    return (src, keys) if return_keys else src


def compact(k_cache: np.ndarray, v_cache: np.ndarray, src: np.ndarray) -> None:
    """In-place stable compaction on host arrays of any dtype: [n_inst, N, d]."""
    assert k_cache.flags.c_contiguous and v_cache.flags.c_contiguous
    assert k_cache.shape == v_cache.shape and k_cache.dtype == v_cache.dtype
    n_inst, N, d = k_cache.shape
    s = np.ascontiguousarray(src, dtype=np.int32)
    K = s.shape[1]
    row_bytes = d * k_cache.itemsize
    rc = _load().vo_compact(_ptr(k_cache), _ptr(v_cache), _ptr(s), n_inst, N, K, row_bytes)
    _check(rc, "compact")


def order_compact(ord_map: np.ndarray, src: np.ndarray, B: int):
    """Compaction under an order map (ord_map[i][t] = slot of temporal rank t):
    returns (new order map [n_inst, K], moves [n_inst, B]) where buffer row K + b
    is copied to slot moves[i][b] and every survivor stays in its slot."""
    o = np.ascontiguousarray(ord_map, dtype=np.int32)
    s = np.ascontiguousarray(src, dtype=np.int32)
    n_inst, K = o.shape
    assert s.shape == (n_inst, K)
    o_new = np.empty_like(o)
    moves = np.empty((n_inst, B), np.int32)
    rc = _load().vo_order_compact(_ptr(o), _ptr(s), n_inst, K, B, _ptr(o_new), _ptr(moves))
    _check(rc, "order_compact")
    return o_new, moves


def apply_moves(k_cache: np.ndarray, v_cache: np.ndarray, moves: np.ndarray, K: int) -> None:
    """Copy buffer row K + b of each instance to slot moves[i][b], in place."""
    n_inst, B = moves.shape
    rows = np.arange(n_inst)[:, None]
    k_cache[rows, moves] = k_cache[:, K:K + B]
    v_cache[rows, moves] = v_cache[:, K:K + B]


def decode(q, k_cache, v_cache, n_valid: int) -> np.ndarray:
    """Decode attention output [n_inst, G, d] float64 over slots [0, n_valid)."""
    qq = _f64(q)
    k = _f64(k_cache)
    v = _f64(v_cache)
    n_inst, N, d = k.shape
    G = qq.shape[1]
    out = np.zeros((n_inst, G, d), dtype=np.float64)
    rc = _load().vo_decode(_ptr(qq), _ptr(k), _ptr(v), n_inst, N, n_valid, G, d, _ptr(out))
    _check(rc, "decode")
    return out


def decode_lse(q, k_cache, n_persist: int) -> np.ndarray:
    """ln sum_{i < n_persist} exp(q_g . k_i / sqrt(d)) -> [n_inst, G] float64: the
    persistent-slot part of Eq. (1)'s normaliser that a decode step hands the round."""
    qq = _f64(q)
    k = _f64(k_cache)
    n_inst, N, d = k.shape
    G = qq.shape[1]
    out = np.zeros((n_inst, G), dtype=np.float64)
    rc = _load().vo_decode_lse(_ptr(qq), _ptr(k), n_inst, N, n_persist, G, d, _ptr(out))
    _check(rc, "decode_lse")
    return out


def score_lse(q_win, k_cache, K: int, pool: int, lse_win) -> np.ndarray:
    """Pooled window score with each row's persistent normaliser supplied
    (lse_win [n_inst, G, w], natural log over slots [0, K)) -> [n_inst, K] float32."""
    q = _f64(q_win)
    k = _f64(k_cache)
    n_inst, N, d = k.shape
    q = np.ascontiguousarray(q.reshape(n_inst, -1, d))
    R = q.shape[1]
    lw = np.ascontiguousarray(_f64(lse_win).reshape(n_inst, R))
    out = np.zeros((n_inst, K), dtype=np.float32)
    rc = _load().vo_score_lse(_ptr(q), _ptr(k), _ptr(lw), n_inst, R, N, K, d, pool, _ptr(out))
    _check(rc, "score_lse")
    return out


def round_(q_win, k_cache, v_cache, K: int, B: int, Nv: int, pool: int, seed: int, rnd: int,
           inst_base: int = 0, flags: int = 0):
    """One full eviction round on host copies: returns (attn, vrange, src)."""
    attn = score(q_win, k_cache, K, pool)
    vr = vrange(v_cache, K)
    src = select(attn, vr, K, B, Nv, seed, rnd, inst_base=inst_base, flags=flags)
    return attn, vr, src


# --------------------------------------------------------------------------
# VaSE-DKV (Sec. 3.2, product score of Eq. 4)
# --------------------------------------------------------------------------
DKV_RANK = 20   # r of the Gaussian projection (Appendix B)


def cos2pi(u: float) -> np.float32:
    """cos(2 pi u) for u in (0, 1), fp32, fixed operation sequence."""
    return np.float32(_load().vo_cos2pi(ctypes.c_float(u)))


def dkv_gaussian(seed: int, inst_id: int, rnd: int, d: int, r: int = DKV_RANK) -> np.ndarray:
    """G_t of one instance, [d, r] float32, entries N(0, 1/r)."""
    g = np.zeros((d, r), dtype=np.float32)
    _load().vo_dkv_gaussian(seed & 0xFFFFFFFFFFFFFFFF, inst_id & 0xFFFFFFFF, rnd & 0xFFFFFFFF, d, r,
                            _ptr(g))
    return g


def dkv_score_g(k_cache, v_cache, g, K: int) -> np.ndarray:
    """s_i = ||g^T k_i||^2 ||g^T v_i||^2 for i < K; g [n_inst, d, r] float32 -> [n_inst, K]."""
    k = _f64(k_cache)
    v = _f64(v_cache)
    gg = np.ascontiguousarray(g, dtype=np.float32)
    n_inst, N, d = k.shape
    r = gg.shape[2]
    assert gg.shape == (n_inst, d, r)
    out = np.zeros((n_inst, K), dtype=np.float32)
    rc = _load().vo_dkv_score_g(_ptr(k), _ptr(v), _ptr(gg), n_inst, N, K, d, r, _ptr(out))
    _check(rc, "dkv_score_g")
    return out


def dkv_score(k_cache, v_cache, K: int, seed: int, rnd: int, inst_base: int = 0,
              r: int = DKV_RANK) -> np.ndarray:
    """The DKV score of one round (fresh G_t per instance) -> [n_inst, K] float32."""
    k = _f64(k_cache)
    v = _f64(v_cache)
    n_inst, N, d = k.shape
    out = np.zeros((n_inst, K), dtype=np.float32)
    rc = _load().vo_dkv_score(_ptr(k), _ptr(v), n_inst, inst_base & 0xFFFFFFFF, N, K, d, r,
                              seed & 0xFFFFFFFFFFFFFFFF, rnd & 0xFFFFFFFF, _ptr(out))
    _check(rc, "dkv_score")
    return out


def dkv_round(k_cache, v_cache, K: int, B: int, seed: int, rnd: int, inst_base: int = 0,
              r: int = DKV_RANK):
    """One VaSE-DKV round on host copies: (score, src); survivors are the K-B
    highest scores plus the buffer (deterministic selection, no reservation)."""
    s = dkv_score(k_cache, v_cache, K, seed, rnd, inst_base=inst_base, r=r)
    vr = np.zeros_like(s)
    src = select(s, vr, K, B, 0, seed, rnd, inst_base=inst_base, flags=FLAG_DETERMINISTIC)
    return s, src


# --------------------------------------------------------------------------
# Range-based per-token quantisation (Eq. 6) with a full-precision reserve
# --------------------------------------------------------------------------
def quantize(x_cache, K: int, bits: int, group: int, Nv: int = 0):
    """Quantise rows [0, K) of x_cache [n_inst, N, d] (bf16/fp32 values).

    Returns dict(codes [n_inst, K, d*bits/8] uint8, params [n_inst, K, d/group, 2]
    float32 (Delta, z), range [n_inst, K] float32, mse [n_inst, K] float32,
    hp_idx [n_inst, Nv] int32: the reserved rows, ascending)."""
    x = _f64(x_cache)
    n_inst, N, d = x.shape
    codes = np.zeros((n_inst, K, d * bits // 8), dtype=np.uint8)
    params = np.zeros((n_inst, K, d // group, 2), dtype=np.float32)
    rng = np.zeros((n_inst, K), dtype=np.float32)
    mse = np.zeros((n_inst, K), dtype=np.float32)
    hp = np.zeros((n_inst, max(Nv, 1)), dtype=np.int32)
    rc = _load().vo_quantize(_ptr(x), n_inst, N, K, d, bits, group, Nv, _ptr(codes), _ptr(params),
                             _ptr(rng), _ptr(mse), _ptr(hp) if Nv > 0 else None)
    _check(rc, "quantize")
    return dict(codes=codes, params=params, range=rng, mse=mse, hp_idx=hp[:, :Nv])


def dequantize(codes, params, N: int, bits: int, group: int, out_bf16: bool,
               hp_rows=None, hp_idx=None) -> np.ndarray:
    """Reconstruct rows [0, K) into a fresh [n_inst, N, d] array of raw output bits
    (uint16 for bf16, float32 otherwise); rows [K, N) are zero.  hp_rows: raw
    bits [n_inst, Nv, d] of the reserved rows, hp_idx [n_inst, Nv]."""
    c = np.ascontiguousarray(codes, dtype=np.uint8)
    p = np.ascontiguousarray(params, dtype=np.float32)
    n_inst, K, rb = c.shape
    d = rb * 8 // bits
    Nv = 0 if hp_idx is None else int(np.asarray(hp_idx).shape[1])
    out = np.zeros((n_inst, N, d), dtype=np.uint16 if out_bf16 else np.float32)
    hr = np.ascontiguousarray(hp_rows) if Nv > 0 else None
    hi = np.ascontiguousarray(hp_idx, dtype=np.int32) if Nv > 0 else None
    rc = _load().vo_dequantize(_ptr(c), _ptr(p), _ptr(hr) if hr is not None else None,
                               _ptr(hi) if hi is not None else None, n_inst, N, K, d, bits, group,
                               Nv, 1 if out_bf16 else 0, _ptr(out))
    _check(rc, "dequantize")
    return out
