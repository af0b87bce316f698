"""Python binding of libvase.so: the VaSE-AttnV eviction round on MI355X.

Argument marshalling only.  Tensors supply device pointers, the current HIP
stream supplies the stream, and every step of the round runs in the library's
HIP kernels.  There is no CPU fallback: if ``libvase.so`` is missing or a call
fails, a ``VaseError`` is raised.

Entry points (names as in ``include/vase.h``):
  * :func:`score`        -- pooled window-mean attention score + Range (Eq. 2, Eq. 5)
  * :func:`select`       -- reservation + weighted sampling -> survivor map (Sec. 3.2)
  * :func:`compact`      -- in-place stable compaction to K slots (Sec. 2)
  * :func:`decode_attn`  -- decode attention over the compacted cache (Eq. 1)
  * :func:`compact_decode` -- compaction and one decode step, the cache read once
  * :func:`dkv_projection`, :func:`dkv_score` -- VaSE-DKV scoring (Sec. 3.2)
  * :func:`order_scores`, :func:`compact_decode_map` -- the round on a cache whose
    temporal order is kept in an order map (``score(..., ord=...)`` scores it);
    compaction then moves only the B buffer rows
"""
from __future__ import annotations

import ctypes
import os
import re
import threading
from typing import Optional, Tuple

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libvase.so")
HEADER_PATH = os.path.join(os.path.dirname(_PKG), "include", "vase.h")

BF16 = 0
F32 = 1
DETERMINISTIC = 1
# device status word bits (vase.h VASE_STATUS_*)
STATUS_ROW_NORM, STATUS_VALUE_ROW, STATUS_SELECT_ATTN, STATUS_SELECT_VALUE = 1, 2, 4, 8
# the library's per-GPU scratch of vase_decode_step_noalloc (vase.h)
DECODE_SCRATCH_BYTES = 64 << 20
OP_SCORE, OP_SELECT, OP_COMPACT, OP_DECODE, OP_COMPACT_DECODE, OP_SCORE_MAP = 0, 1, 2, 3, 4, 5
MAX_K = 8192
DEC_LOGITS_LDS = 92160    # VASE_DEC_LOGITS_LDS
VALUE_RANGE, VALUE_L2, VALUE_VAR, VALUE_RANDOM, VALUE_SKIP = 0, 1, 2, 3, 4

OK = 0
ERR_INVALID_ARG = -1
ERR_DTYPE = -2
ERR_WORKSPACE = -3
ERR_HIP = -4
ERR_UNSUPPORTED = -5


class VaseError(RuntimeError):
    def __init__(self, what: str, status: int):
        super().__init__("%s failed: %s (%d)" % (what, status_str(status), status))
        self.status = status


_lock = threading.Lock()
_lib = None


def load() -> ctypes.CDLL:
    """Load libvase.so (raises if it has not been built)."""
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libvase.so is not built; run `python -m paper_2606_03928_amd.build` "
                               "(the eviction round has no CPU fallback)")
        lib = ctypes.CDLL(LIB_PATH)
        P, I, U32, U64, SZ = (ctypes.c_void_p, ctypes.c_int, ctypes.c_uint32, ctypes.c_uint64,
                              ctypes.c_size_t)
        lib.vase_version.argtypes = []
        lib.vase_version.restype = I
        lib.vase_status_str.argtypes = [I]
        lib.vase_status_str.restype = ctypes.c_char_p
        lib.vase_workspace_bytes.argtypes = [I, I, I, I, I, I, I, I]
        lib.vase_workspace_bytes.restype = SZ
        lib.vase_score.argtypes = [P, P, P, I, I, I, I, I, I, I, I, P, P, P, SZ, P, P]
        lib.vase_score.restype = I
        lib.vase_score_ex.argtypes = [P, P, P, I, I, I, I, I, I, I, I, I, U64, U32, U32, P, P, P,
                                      SZ, P, P]
        lib.vase_score_ex.restype = I
        lib.vase_select.argtypes = [P, P, I, U32, I, I, I, U64, U32, U32, P, P, P, P]
        lib.vase_select.restype = I
        lib.vase_compact.argtypes = [P, P, I, I, I, I, I, P, P, SZ, P]
        lib.vase_compact.restype = I
        lib.vase_decode_attn.argtypes = [P, P, P, I, I, I, I, I, I, I, P, P, SZ, P]
        lib.vase_decode_attn_lse.argtypes = [P, P, P, I, I, I, I, I, I, I, I, P, P, P, SZ, P]
        lib.vase_decode_attn_lse.restype = I
        lib.vase_decode_step.argtypes = [P, P, P, P, P, I, I, I, I, I, I, I, I, P, P, P, P, SZ, P]
        lib.vase_decode_step.restype = I
        lib.vase_decode_step_noalloc.argtypes = [P, P, P, P, P, I, I, I, I, I, I, I, I, P, P, P, P]
        lib.vase_decode_step_noalloc.restype = I
        lib.vase_score_lse.argtypes = [P, P, P, P, I, I, I, I, I, I, I, I, I, U64, U32, U32, P, P,
                                       P, SZ, P, P]
        lib.vase_score_lse.restype = I
        lib.vase_quantize.argtypes = [P, I, I, I, I, I, I, I, I, P, P, P, P, P, P, P]
        lib.vase_quantize.restype = I
        lib.vase_dequantize.argtypes = [P, P, P, P, I, I, I, I, I, I, I, I, P, P]
        lib.vase_dequantize.restype = I
        lib.vase_compact_decode.restype = I
        lib.vase_compact_decode.argtypes = [P, P, I, I, I, I, I, P, P, I, P, P, SZ, P]
        lib.vase_compact_decode_ex.argtypes = [P, P, I, I, I, I, I, P, P, I, P, I, P, P, SZ, P]
        lib.vase_compact_decode_ex.restype = I
        lib.vase_dkv_projection.restype = I
        lib.vase_dkv_projection.argtypes = [I, U32, I, I, U64, U32, P, P]
        lib.vase_dkv_score.restype = I
        lib.vase_dkv_score.argtypes = [P, P, P, I, I, I, I, I, I, P, P, I, P, P]
        lib.vase_decode_attn.restype = I
        lib.vase_score_map.argtypes = [P, P, P, P, P, I, I, I, I, I, I, I, I, I, U64, U32, U32, P,
                                       P, P, P, P, SZ, P, P]
        lib.vase_score_map.restype = I
        lib.vase_order_scores.argtypes = [P, P, P, I, I, I, P, P, P]
        lib.vase_order_scores.restype = I
        lib.vase_compact_decode_map.argtypes = [P, P, I, I, I, I, I, P, P, P, I, P, I, P, P, P, P]
        lib.vase_compact_decode_map.restype = I
        _lib = lib
        return lib


def header_functions() -> list:
    """Names of the functions ``include/vase.h`` declares."""
    with open(HEADER_PATH) as f:
        txt = f.read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(vase_\w+)\s*\(", txt, re.M)))


def status_str(status: int) -> str:
    try:
        return load().vase_status_str(status).decode()
    except Exception:  # library missing while formatting an error
        return "status"


def version() -> Tuple[int, int]:
    v = load().vase_version()
    return v >> 16, v & 0xFFFF


def _check(rc: int, what: str) -> None:
    if rc != OK:
        raise VaseError(what, rc)


def dtype_code(t: torch.dtype) -> int:
    if t == torch.bfloat16:
        return BF16
    if t == torch.float32:
        return F32
    raise VaseError("dtype %s" % t, ERR_DTYPE)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream_ptr(device: torch.device, stream: Optional[torch.cuda.Stream]):
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return ctypes.c_void_p(s.cuda_stream)


def _status_ptr(status: Optional[torch.Tensor], device):
    """Device pointer of a one-element int32 status word, or NULL."""
    if status is None:
        return None
    _require(status.dtype == torch.int32 and status.numel() >= 1 and status.device == device
             and status.is_contiguous(), "status must be a contiguous int32 tensor on the device")
    return _ptr(status)


def _require(cond: bool, msg: str) -> None:
    if not cond:
        raise ValueError(msg)


def _dev(t: torch.Tensor, name: str) -> None:
    _require(t.is_cuda, "%s must be a device tensor" % name)
    _require(t.is_contiguous(), "%s must be contiguous" % name)


def workspace_bytes(op: int, dtype: torch.dtype, n_inst: int, K: int, B: int, d: int,
                    G: int = 1, w: int = 1) -> int:
    return int(load().vase_workspace_bytes(op, dtype_code(dtype), n_inst, K, B, d, G, w))


def _workspace(ws: Optional[torch.Tensor], nbytes: int, device) -> Optional[torch.Tensor]:
    if nbytes == 0:
        return ws
    if ws is None:
        return torch.empty(nbytes, dtype=torch.uint8, device=device)
    _require(ws.numel() * ws.element_size() >= nbytes, "workspace too small")
    return ws


def _ws_args(ws: Optional[torch.Tensor]):
    if ws is None:
        return None, 0
    return _ptr(ws), ws.numel() * ws.element_size()


def score(k: torch.Tensor, v: torch.Tensor, q_win: torch.Tensor, K: int, B: int, pool: int,
          attn: Optional[torch.Tensor] = None, vrange: Optional[torch.Tensor] = None,
          ws: Optional[torch.Tensor] = None, stream=None, value_kind: int = VALUE_RANGE,
          seed: int = 0, round: int = 0, inst_base: int = 0,
          lse_win: Optional[torch.Tensor] = None, ord: Optional[torch.Tensor] = None,
          q_dec: Optional[torch.Tensor] = None, dec_logits: Optional[torch.Tensor] = None,
          status: Optional[torch.Tensor] = None):
    """Pooled window-mean attention score and value score of the K candidate slots.

    k, v: [n_inst, K+B, d]; q_win: [n_inst, G, w, d] (same dtype, bf16 or fp32).
    value_kind picks Range (default), L2, Var or random reservation (VALUE_*);
    seed, round and inst_base feed the random one only.  lse_win [n_inst, G, w]
    fp32 (as decode_step leaves it) switches to the one-pass score.  ord
    [n_inst, K] int32 (an order map) scores the cache read through it: the
    outputs are indexed by temporal rank (vase_score_map).  With ord, q_dec
    [n_inst, G, d] bf16 and dec_logits [n_inst, G, K+B] float32, the pass over the
    keys also writes the decode queries' logits q_dec . k per physical slot, for
    compact_decode_map(dec_logits=...).  status: an int32 device tensor of one
    element (or None) into which the call ORs the STATUS_* data-fault bits.
    Returns (attn, vrange), both [n_inst, K] float32 on the device.
    """
    for t, n in ((k, "k"), (v, "v"), (q_win, "q_win")):
        _dev(t, n)
    n_inst, N, d = k.shape
    _require(N == K + B and v.shape == k.shape, "cache must be [n_inst, K+B, d]")
    _require(q_win.dim() == 4 and q_win.shape[0] == n_inst and q_win.shape[3] == d,
             "q_win must be [n_inst, G, w, d]")
    _require(q_win.dtype == k.dtype == v.dtype, "k, v and q_win must share a dtype")
    G, w = int(q_win.shape[1]), int(q_win.shape[2])
    dev = k.device
    if attn is None:
        attn = torch.empty((n_inst, K), dtype=torch.float32, device=dev)
    if vrange is None and value_kind != VALUE_SKIP:
        vrange = torch.empty((n_inst, K), dtype=torch.float32, device=dev)
    _dev(attn, "attn")
    if vrange is not None:
        _dev(vrange, "vrange")
    _require(dec_logits is None or ord is not None, "dec_logits needs an order map")
    op = OP_SCORE if ord is None else OP_SCORE_MAP
    ws = _workspace(ws, workspace_bytes(op, k.dtype, n_inst, K, B, d, G, w), dev)
    wp, wn = _ws_args(ws)
    st = _stream_ptr(dev, stream)
    if lse_win is not None:
        _dev(lse_win, "lse_win")
        _require(lse_win.dtype == torch.float32 and tuple(lse_win.shape) == (n_inst, G, w),
                 "lse_win must be float32 [n_inst, G, w]")
    if ord is not None:
        _dev(ord, "ord")
        _require(ord.dtype == torch.int32 and tuple(ord.shape) == (n_inst, K),
                 "ord must be int32 [n_inst, K]")
        if dec_logits is not None:
            _require(q_dec is not None, "dec_logits needs q_dec")
            _dev(q_dec, "q_dec")
            _dev(dec_logits, "dec_logits")
            _require(q_dec.dtype == k.dtype and tuple(q_dec.shape) == (n_inst, G, d),
                     "q_dec must be [n_inst, G, d] of the cache dtype")
            _require(dec_logits.dtype == torch.float32 and tuple(dec_logits.shape) == (n_inst, G, N),
                     "dec_logits must be float32 [n_inst, G, K+B]")
        rc = load().vase_score_map(_ptr(k), _ptr(v), _ptr(q_win), _ptr(lse_win), _ptr(ord),
                                   dtype_code(k.dtype), n_inst, K, B, d, G, w, pool, value_kind,
                                   seed & 0xFFFFFFFFFFFFFFFF, round & 0xFFFFFFFF,
                                   inst_base & 0xFFFFFFFF, _ptr(attn), _ptr(vrange),
                                   _ptr(q_dec if dec_logits is not None else None),
                                   _ptr(dec_logits), wp, wn, _status_ptr(status, dev), st)
    elif lse_win is not None:
        rc = load().vase_score_lse(_ptr(k), _ptr(v), _ptr(q_win), _ptr(lse_win),
                                   dtype_code(k.dtype), n_inst, K, B, d, G, w, pool, value_kind,
                                   seed & 0xFFFFFFFFFFFFFFFF, round & 0xFFFFFFFF,
                                   inst_base & 0xFFFFFFFF, _ptr(attn), _ptr(vrange), wp, wn,
                                   _status_ptr(status, dev), st)
    elif value_kind == VALUE_RANGE:
        rc = load().vase_score(_ptr(k), _ptr(v), _ptr(q_win), dtype_code(k.dtype), n_inst, K, B,
                               d, G, w, pool, _ptr(attn), _ptr(vrange), wp, wn,
                               _status_ptr(status, dev), st)
    else:
        rc = load().vase_score_ex(_ptr(k), _ptr(v), _ptr(q_win), dtype_code(k.dtype), n_inst, K,
                                  B, d, G, w, pool, value_kind, seed & 0xFFFFFFFFFFFFFFFF,
                                  round & 0xFFFFFFFF, inst_base & 0xFFFFFFFF, _ptr(attn),
                                  _ptr(vrange), wp, wn, _status_ptr(status, dev), st)
    _check(rc, "vase_score")
    return attn, vrange


def select(attn: torch.Tensor, vrange: torch.Tensor, K: int, B: int, Nv: int, seed: int,
           round: int, inst_base: int = 0, flags: int = 0, src: Optional[torch.Tensor] = None,
           keys: Optional[torch.Tensor] = None, want_keys: bool = False, stream=None,
           status: Optional[torch.Tensor] = None):
    """Survivor map src [n_inst, K] int32 (and the selection keys if asked).  status as
    in score (STATUS_SELECT_* bits)."""
    _dev(attn, "attn")
    _dev(vrange, "vrange")
    _require(attn.dtype == torch.float32 and vrange.dtype == torch.float32, "scores must be fp32")
    n_inst = attn.shape[0]
    _require(tuple(attn.shape) == (n_inst, K) and tuple(vrange.shape) == (n_inst, K),
             "scores must be [n_inst, K]")
    dev = attn.device
    if src is None:
        src = torch.empty((n_inst, K), dtype=torch.int32, device=dev)
    _dev(src, "src")
    if want_keys and keys is None:
        keys = torch.empty((n_inst, K), dtype=torch.float32, device=dev)
    rc = load().vase_select(_ptr(attn), _ptr(vrange), n_inst, inst_base & 0xFFFFFFFF, K, B, Nv,
                            seed & 0xFFFFFFFFFFFFFFFF, round & 0xFFFFFFFF, flags, _ptr(src),
                            _ptr(keys), _status_ptr(status, dev), _stream_ptr(dev, stream))
    _check(rc, "vase_select")
    return (src, keys) if (want_keys or keys is not None) else src


def compact(k: torch.Tensor, v: torch.Tensor, src: torch.Tensor, K: int, B: int,
            ws: Optional[torch.Tensor] = None, stream=None) -> None:
    """In-place stable compaction: k[:, j] <- k[:, src[j]] (and v) for j < K."""
    _dev(k, "k")
    _dev(v, "v")
    _dev(src, "src")
    n_inst, N, d = k.shape
    _require(N == K + B and v.shape == k.shape and v.dtype == k.dtype, "cache shape mismatch")
    _require(src.dtype == torch.int32 and tuple(src.shape) == (n_inst, K), "src must be int32 [n_inst, K]")
    ws = _workspace(ws, workspace_bytes(OP_COMPACT, k.dtype, n_inst, K, B, d), k.device)
    wp, wn = _ws_args(ws)
    rc = load().vase_compact(_ptr(k), _ptr(v), dtype_code(k.dtype), n_inst, K, B, d, _ptr(src),
                             wp, wn, _stream_ptr(k.device, stream))
    _check(rc, "vase_compact")


def decode_attn(k: torch.Tensor, v: torch.Tensor, q: torch.Tensor, K: int, B: int, n_valid: int,
                out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                stream=None, n_persist: Optional[int] = None,
                lse: Optional[torch.Tensor] = None):
    """Decode attention of q [n_inst, G, d] over the first n_valid cache slots.

    With n_persist, also the natural-log LSE of each query's scores over slots
    [0, n_persist) into lse [n_inst, G] fp32; returns (out, lse) then.
    """
    for t, n in ((k, "k"), (v, "v"), (q, "q")):
        _dev(t, n)
    n_inst, N, d = k.shape
    _require(N == K + B and v.shape == k.shape, "cache must be [n_inst, K+B, d]")
    _require(q.dim() == 3 and q.shape[0] == n_inst and q.shape[2] == d, "q must be [n_inst, G, d]")
    _require(q.dtype == k.dtype == v.dtype, "k, v and q must share a dtype")
    G = int(q.shape[1])
    if out is None:
        out = torch.empty_like(q)
    _dev(out, "out")
    ws = _workspace(ws, workspace_bytes(OP_DECODE, k.dtype, n_inst, K, B, d, G), k.device)
    wp, wn = _ws_args(ws)
    if n_persist is None:
        rc = load().vase_decode_attn(_ptr(k), _ptr(v), _ptr(q), dtype_code(k.dtype), n_inst, K, B,
                                     d, G, n_valid, _ptr(out), wp, wn, _stream_ptr(k.device, stream))
        _check(rc, "vase_decode_attn")
        return out
    if lse is None:
        lse = torch.empty((n_inst, G), dtype=torch.float32, device=k.device)
    _dev(lse, "lse")
    _require(lse.dtype == torch.float32 and tuple(lse.shape) == (n_inst, G), "lse must be [n_inst, G]")
    rc = load().vase_decode_attn_lse(_ptr(k), _ptr(v), _ptr(q), dtype_code(k.dtype), n_inst, K, B,
                                     d, G, n_valid, n_persist, _ptr(out), _ptr(lse), wp, wn,
                                     _stream_ptr(k.device, stream))
    _check(rc, "vase_decode_attn_lse")
    return out, lse


def decode_step(k: torch.Tensor, v: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor,
                q: torch.Tensor, K: int, B: int, pos: int, q_win: torch.Tensor,
                lse_win: torch.Tensor, out: Optional[torch.Tensor] = None,
                ws: Optional[torch.Tensor] = None, stream=None,
                noalloc: bool = False) -> torch.Tensor:
    """Append (k_new, v_new) [n_inst, d] at slot K + pos, cache q [n_inst, G, d] in the
    window ring q_win [n_inst, G, w, d], attend over K + pos + 1 slots, and store the
    persistent-slot LSE in lse_win [n_inst, G, w] (ring slot pos % w).  noalloc: use
    vase_decode_step_noalloc (the library's own scratch; ws is ignored; `out` must
    be given so that nothing is allocated here either)."""
    for t, n in ((k, "k"), (v, "v"), (k_new, "k_new"), (v_new, "v_new"), (q, "q"),
                 (q_win, "q_win"), (lse_win, "lse_win")):
        _dev(t, n)
    n_inst, N, d = k.shape
    _require(N == K + B and v.shape == k.shape, "cache must be [n_inst, K+B, d]")
    _require(tuple(k_new.shape) == (n_inst, d) and k_new.shape == v_new.shape,
             "k_new, v_new must be [n_inst, d]")
    _require(q.dim() == 3 and q.shape[0] == n_inst and q.shape[2] == d, "q must be [n_inst, G, d]")
    G = int(q.shape[1])
    _require(q_win.dim() == 4 and tuple(q_win.shape[:2]) == (n_inst, G) and q_win.shape[3] == d,
             "q_win must be [n_inst, G, w, d]")
    w = int(q_win.shape[2])
    _require(lse_win.dtype == torch.float32 and tuple(lse_win.shape) == (n_inst, G, w),
             "lse_win must be float32 [n_inst, G, w]")
    _require(k.dtype == v.dtype == k_new.dtype == v_new.dtype == q.dtype == q_win.dtype,
             "cache, new rows and queries must share a dtype")
    if noalloc:
        _require(out is not None, "noalloc needs a caller-provided out")
        _dev(out, "out")
        rc = load().vase_decode_step_noalloc(_ptr(k), _ptr(v), _ptr(k_new), _ptr(v_new), _ptr(q),
                                             dtype_code(k.dtype), n_inst, K, B, d, G, w, pos,
                                             _ptr(q_win), _ptr(lse_win), _ptr(out),
                                             _stream_ptr(k.device, stream))
        _check(rc, "vase_decode_step_noalloc")
        return out
    if out is None:
        out = torch.empty_like(q)
    _dev(out, "out")
    ws = _workspace(ws, workspace_bytes(OP_DECODE, k.dtype, n_inst, K, B, d, G), k.device)
    wp, wn = _ws_args(ws)
    rc = load().vase_decode_step(_ptr(k), _ptr(v), _ptr(k_new), _ptr(v_new), _ptr(q),
                                 dtype_code(k.dtype), n_inst, K, B, d, G, w, pos, _ptr(q_win),
                                 _ptr(lse_win), _ptr(out), wp, wn, _stream_ptr(k.device, stream))
    _check(rc, "vase_decode_step")
    return out


def compact_decode(k: torch.Tensor, v: torch.Tensor, src: torch.Tensor, q: torch.Tensor, K: int,
                   B: int, out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                   stream=None, vrange_out: Optional[torch.Tensor] = None,
                   value_kind: int = VALUE_RANGE) -> torch.Tensor:
    """compact(k, v, src) followed by decode_attn(k, v, q, n_valid=K), fused.

    With vrange_out [n_inst, K] fp32, also the value score (value_kind) of every
    compacted row: the next round's candidate scores (score with VALUE_SKIP)."""
    for t, n in ((k, "k"), (v, "v"), (src, "src"), (q, "q")):
        _dev(t, n)
    n_inst, N, d = k.shape
    _require(N == K + B and v.shape == k.shape and v.dtype == k.dtype, "cache shape mismatch")
    _require(src.dtype == torch.int32 and tuple(src.shape) == (n_inst, K), "src must be int32 [n_inst, K]")
    _require(q.dim() == 3 and q.shape[0] == n_inst and q.shape[2] == d and q.dtype == k.dtype,
             "q must be [n_inst, G, d] of the cache dtype")
    G = int(q.shape[1])
    if out is None:
        out = torch.empty_like(q)
    _dev(out, "out")
    ws = _workspace(ws, workspace_bytes(OP_COMPACT_DECODE, k.dtype, n_inst, K, B, d, G), k.device)
    wp, wn = _ws_args(ws)
    if vrange_out is None:
        rc = load().vase_compact_decode(_ptr(k), _ptr(v), dtype_code(k.dtype), n_inst, K, B, d,
                                        _ptr(src), _ptr(q), G, _ptr(out), wp, wn,
                                        _stream_ptr(k.device, stream))
    else:
        _dev(vrange_out, "vrange_out")
        _require(vrange_out.dtype == torch.float32 and tuple(vrange_out.shape) == (n_inst, K),
                 "vrange_out must be float32 [n_inst, K]")
        rc = load().vase_compact_decode_ex(_ptr(k), _ptr(v), dtype_code(k.dtype), n_inst, K, B, d,
                                           _ptr(src), _ptr(q), G, _ptr(out), value_kind,
                                           _ptr(vrange_out), wp, wn, _stream_ptr(k.device, stream))
    _check(rc, "vase_compact_decode")
    return out


def identity_order(n_inst: int, K: int, device) -> torch.Tensor:
    """The order map of a cache whose slots are in temporal order (after a prefill)."""
    return torch.arange(K, dtype=torch.int32, device=device).repeat(n_inst, 1)


def order_scores(attn_phys: torch.Tensor, ord: torch.Tensor, pool: int,
                 vrange_phys: Optional[torch.Tensor] = None, attn: Optional[torch.Tensor] = None,
                 vrange: Optional[torch.Tensor] = None, stream=None):
    """Per-slot scores into temporal order through ord [n_inst, K] int32:
    attn[t] = P-wide box filter of attn_phys[ord[.]] around rank t, and
    vrange[t] = vrange_phys[ord[t]] (if given).  Returns (attn, vrange)."""
    _dev(attn_phys, "attn_phys")
    _dev(ord, "ord")
    n_inst, K = attn_phys.shape
    _require(ord.dtype == torch.int32 and tuple(ord.shape) == (n_inst, K), "ord must be int32 [n_inst, K]")
    if attn is None:
        attn = torch.empty_like(attn_phys)
    if vrange_phys is not None and vrange is None:
        vrange = torch.empty_like(vrange_phys)
    rc = load().vase_order_scores(_ptr(attn_phys), _ptr(vrange_phys), _ptr(ord), n_inst, K, pool,
                                  _ptr(attn), _ptr(vrange), _stream_ptr(attn_phys.device, stream))
    _check(rc, "vase_order_scores")
    return attn, vrange


def compact_decode_map(k: torch.Tensor, v: torch.Tensor, src: torch.Tensor, ord: torch.Tensor,
                       K: int, B: int, q: Optional[torch.Tensor] = None,
                       out: Optional[torch.Tensor] = None, stream=None,
                       vrange_out: Optional[torch.Tensor] = None,
                       value_kind: int = VALUE_RANGE,
                       vrange_in: Optional[torch.Tensor] = None,
                       dec_logits: Optional[torch.Tensor] = None) -> Optional[torch.Tensor]:
    """Compaction under the order map ord [n_inst, K] int32 (updated in place): the
    B buffer rows go into the slots of the evicted ranks, survivors stay.  With q
    [n_inst, G, d], also one decode step over the K slots (returned); with
    vrange_out, the value score of every rank's row (the next round's candidates).
    vrange_in (the scores the selection used; may be vrange_out) lets survivors
    keep theirs, so only the buffer rows are scored.  dec_logits [n_inst, G, K+B]
    float32 (written by score(..., q_dec=q, dec_logits=...) on this cache before
    compaction) replaces the q.k products, so no K row is read for the decode."""
    for t, n in ((k, "k"), (v, "v"), (src, "src"), (ord, "ord")):
        _dev(t, n)
    n_inst, N, d = k.shape
    _require(N == K + B and v.shape == k.shape and v.dtype == k.dtype, "cache shape mismatch")
    _require(src.dtype == torch.int32 and tuple(src.shape) == (n_inst, K), "src must be int32 [n_inst, K]")
    _require(ord.dtype == torch.int32 and tuple(ord.shape) == (n_inst, K), "ord must be int32 [n_inst, K]")
    G = 0
    if q is not None:
        _dev(q, "q")
        _require(q.dim() == 3 and q.shape[0] == n_inst and q.shape[2] == d and q.dtype == k.dtype,
                 "q must be [n_inst, G, d] of the cache dtype")
        G = int(q.shape[1])
        if out is None:
            out = torch.empty_like(q)
        _dev(out, "out")
    for t, n in ((vrange_out, "vrange_out"), (vrange_in, "vrange_in")):
        if t is not None:
            _dev(t, n)
            _require(t.dtype == torch.float32 and tuple(t.shape) == (n_inst, K),
                     "%s must be float32 [n_inst, K]" % n)
    if dec_logits is not None:
        _dev(dec_logits, "dec_logits")
        _require(dec_logits.dtype == torch.float32 and tuple(dec_logits.shape) == (n_inst, G, N),
                 "dec_logits must be float32 [n_inst, G, K+B]")
    rc = load().vase_compact_decode_map(_ptr(k), _ptr(v), dtype_code(k.dtype), n_inst, K, B, d,
                                        _ptr(src), _ptr(ord), _ptr(q), G, _ptr(out), value_kind,
                                        _ptr(vrange_in), _ptr(vrange_out), _ptr(dec_logits),
                                        _stream_ptr(k.device, stream))
    _check(rc, "vase_compact_decode_map")
    return out


DKV_RANK = 20


def dkv_projection(n_inst: int, d: int, seed: int, round: int, r: int = DKV_RANK,
                   inst_base: int = 0, out: Optional[torch.Tensor] = None, device="cuda",
                   stream=None) -> torch.Tensor:
    """Per-instance Gaussian projections G_t [n_inst, d, r] float32 (entries N(0, 1/r))."""
    if out is None:
        out = torch.empty((n_inst, d, r), dtype=torch.float32, device=device)
    _dev(out, "out")
    _require(tuple(out.shape) == (n_inst, d, r) and out.dtype == torch.float32,
             "out must be float32 [n_inst, d, r]")
    rc = load().vase_dkv_projection(n_inst, inst_base & 0xFFFFFFFF, d, r,
                                    seed & 0xFFFFFFFFFFFFFFFF, round & 0xFFFFFFFF, _ptr(out),
                                    _stream_ptr(out.device, stream))
    _check(rc, "vase_dkv_projection")
    return out


def dkv_score(k: torch.Tensor, v: torch.Tensor, g: torch.Tensor, K: int, B: int,
              out: Optional[torch.Tensor] = None, stream=None, q_dec: Optional[torch.Tensor] = None,
              dec_logits: Optional[torch.Tensor] = None) -> torch.Tensor:
    """s_i = ||G^T k_i||^2 ||G^T v_i||^2 for the K candidate slots -> [n_inst, K] float32.
    With q_dec [n_inst, G, d] bf16 and dec_logits [n_inst, G, K+B] float32, the same
    pass writes q_dec . k for every slot (for compact_decode_map(dec_logits=...))."""
    for t, n in ((k, "k"), (v, "v"), (g, "g")):
        _dev(t, n)
    n_inst, N, d = k.shape
    _require(N == K + B and v.shape == k.shape and v.dtype == k.dtype, "cache shape mismatch")
    _require(g.dim() == 3 and g.shape[0] == n_inst and g.shape[1] == d and g.dtype == torch.float32,
             "g must be float32 [n_inst, d, r]")
    r = int(g.shape[2])
    if out is None:
        out = torch.empty((n_inst, K), dtype=torch.float32, device=k.device)
    _dev(out, "out")
    Gd = 0
    if dec_logits is not None:
        _require(q_dec is not None, "dec_logits needs q_dec")
        _dev(q_dec, "q_dec")
        _dev(dec_logits, "dec_logits")
        Gd = int(q_dec.shape[1])
        _require(q_dec.dim() == 3 and q_dec.shape[0] == n_inst and q_dec.shape[2] == d
                 and q_dec.dtype == k.dtype, "q_dec must be [n_inst, G, d] of the cache dtype")
        _require(dec_logits.dtype == torch.float32 and tuple(dec_logits.shape) == (n_inst, Gd, N),
                 "dec_logits must be float32 [n_inst, G, K+B]")
    rc = load().vase_dkv_score(_ptr(k), _ptr(v), _ptr(g), dtype_code(k.dtype), n_inst, K, B, d, r,
                               _ptr(out), _ptr(q_dec if dec_logits is not None else None), Gd,
                               _ptr(dec_logits), _stream_ptr(k.device, stream))
    _check(rc, "vase_dkv_score")
    return out


def quantize(x: torch.Tensor, K: int, B: int, bits: int, group: int, Nv: int = 0,
             out: Optional[dict] = None, want_mse: bool = True, stream=None) -> dict:
    """Range-based per-token quantisation (Eq. 6) of rows [0, K) of x [n_inst, K+B, d].

    Returns dict(codes [n_inst, K, d*bits/8] uint8, params [n_inst, K, d/group, 2]
    fp32, range [n_inst, K] fp32, mse [n_inst, K] fp32 (or None), hp_rows
    [n_inst, Nv, d] x.dtype and hp_idx [n_inst, Nv] int32 when Nv > 0)."""
    _dev(x, "x")
    n_inst, N, d = x.shape
    _require(N == K + B, "cache must be [n_inst, K+B, d]")
    dev = x.device
    if out is None:
        out = dict(codes=torch.empty((n_inst, K, d * bits // 8), dtype=torch.uint8, device=dev),
                   params=torch.empty((n_inst, K, d // group, 2), dtype=torch.float32, device=dev),
                   range=torch.empty((n_inst, K), dtype=torch.float32, device=dev),
                   mse=torch.empty((n_inst, K), dtype=torch.float32, device=dev) if want_mse else None,
                   hp_rows=torch.empty((n_inst, Nv, d), dtype=x.dtype, device=dev) if Nv else None,
                   hp_idx=torch.empty((n_inst, Nv), dtype=torch.int32, device=dev) if Nv else None)
    rc = load().vase_quantize(_ptr(x), dtype_code(x.dtype), n_inst, K, B, d, bits, group, Nv,
                              _ptr(out["codes"]), _ptr(out["params"]), _ptr(out["range"]),
                              _ptr(out["mse"]), _ptr(out["hp_rows"]), _ptr(out["hp_idx"]),
                              _stream_ptr(dev, stream))
    _check(rc, "vase_quantize")
    return out


def dequantize(q: dict, K: int, B: int, bits: int, group: int, dtype: torch.dtype,
               out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Inverse of quantize: rows [0, K) of out [n_inst, K+B, d] (rows [K, N) untouched)."""
    codes, params = q["codes"], q["params"]
    n_inst, _, rb = codes.shape
    d = rb * 8 // bits
    Nv = 0 if q.get("hp_idx") is None else int(q["hp_idx"].shape[1])
    if out is None:
        out = torch.zeros((n_inst, K + B, d), dtype=dtype, device=codes.device)
    _dev(out, "out")
    rc = load().vase_dequantize(_ptr(codes), _ptr(params), _ptr(q.get("hp_rows")),
                                _ptr(q.get("hp_idx")), dtype_code(dtype), n_inst, K, B, d, bits,
                                group, Nv, _ptr(out), _stream_ptr(codes.device, stream))
    _check(rc, "vase_dequantize")
    return out


def dec_logits_fit(N: int, d: int, G: int) -> bool:
    """Whether the score pass keeps an instance's decode logits in LDS (the fast
    case; see VASE_DEC_LOGITS_LDS), judged with all N slots as one range."""
    return G * ((N + 3) // 4 * 4) * 4 + G * d * 2 <= DEC_LOGITS_LDS


class Round:
    """Buffers for repeated eviction rounds of one workload (no per-call allocation)."""

    def __init__(self, n_inst: int, K: int, B: int, d: int, G: int, w: int, dtype: torch.dtype,
                 device, layout: str = "stable", dec_logits: bool = True):
        """layout "stable": compaction keeps the slots in temporal order; "map": an
        order map (self.ord, the identity until the first round) keeps it, and
        compaction moves only the buffer rows.  Under the map, with bf16,
        G <= 8 and logits that fit the score's LDS (dec_logits_fit),
        dec_logits=True lets the score pass leave the decode queries' logits for
        the compaction's decode step, which then reads no K row."""
        _require(layout in ("stable", "map"), "layout must be 'stable' or 'map'")
        self.n_inst, self.K, self.B, self.d, self.G, self.w = n_inst, K, B, d, G, w
        self.dtype = dtype
        self.layout = layout
        dev = torch.device(device)
        self.ord = identity_order(n_inst, K, dev) if layout == "map" else None
        use_dl = (dec_logits and layout == "map" and dtype == torch.bfloat16 and G <= 8
                  and dec_logits_fit(K + B, d, G))
        self.dec_logits = (torch.empty((n_inst, G, K + B), dtype=torch.float32, device=dev)
                           if use_dl else None)
        self.attn = torch.empty((n_inst, K), dtype=torch.float32, device=dev)
        self.vrange = torch.empty((n_inst, K), dtype=torch.float32, device=dev)
        self.src = torch.empty((n_inst, K), dtype=torch.int32, device=dev)
        self.out = torch.empty((n_inst, G, d), dtype=dtype, device=dev)
        nb = max(workspace_bytes(op, dtype, n_inst, K, B, d, G, w)
                 for op in (OP_SCORE, OP_COMPACT, OP_DECODE, OP_COMPACT_DECODE, OP_SCORE_MAP))
        self.ws = torch.empty(max(nb, 256), dtype=torch.uint8, device=dev)
        self.carried_kind = None      # value kind whose scores of [0, K) self.vrange holds

    def run(self, k, v, q_win, q_dec, Nv: int, pool: int, seed: int, rnd: int,
            inst_base: int = 0, flags: int = 0, stream=None, value_kind: int = VALUE_RANGE,
            carry: bool = False, lse_win: Optional[torch.Tensor] = None) -> torch.Tensor:
        """score -> select -> compact + decode over the compacted cache (returned),
        or compaction alone when q_dec is None (returns None).

        With carry=True the compaction also leaves the value scores of the
        compacted rows in self.vrange, and the next carry=True round of the same
        cache skips computing them (the persistent rows do not change between
        rounds; the caller only appends to the buffer).  Results are identical
        either way.  The stable layout's compaction alone carries nothing.
        lse_win (from decode_step) makes the score one-pass."""
        K, B = self.K, self.B
        carried = carry and self.carried_kind == value_kind and value_kind != VALUE_RANDOM
        # the decode logits ride on the score's pass over every key (not in the
        # one-pass score, which reads only the buffer's keys)
        dl = self.dec_logits if (lse_win is None and q_dec is not None) else None
        score(k, v, q_win, K, B, pool, attn=self.attn, vrange=self.vrange, ws=self.ws, stream=stream,
              value_kind=VALUE_SKIP if carried else value_kind, seed=seed, round=rnd,
              inst_base=inst_base, lse_win=lse_win, ord=self.ord, q_dec=q_dec if dl is not None else None,
              dec_logits=dl)
        select(self.attn, self.vrange, K, B, Nv, seed, rnd, inst_base=inst_base, flags=flags,
               src=self.src, stream=stream)
        keep = carry and value_kind != VALUE_RANDOM
        if self.layout == "map":
            # the survivors keep the value scores this round's selection used
            compact_decode_map(k, v, self.src, self.ord, K, B, q=q_dec,
                               out=self.out if q_dec is not None else None,
                               stream=stream, vrange_out=self.vrange if keep else None,
                               vrange_in=self.vrange if keep else None, value_kind=value_kind,
                               dec_logits=dl)
        elif q_dec is not None:
            compact_decode(k, v, self.src, q_dec, K, B, out=self.out, ws=self.ws, stream=stream,
                           vrange_out=self.vrange if keep else None, value_kind=value_kind)
        else:
            compact(k, v, self.src, K, B, ws=self.ws, stream=stream)
            keep = False
        self.carried_kind = value_kind if keep else None
        return self.out if q_dec is not None else None

    def temporal(self, x: torch.Tensor) -> torch.Tensor:
        """A cache tensor [n_inst, K+B, d] in temporal order (a copy under the map
        layout; x itself under the stable one)."""
        if self.ord is None:
            return x
        idx = self.ord.long()[:, :, None].expand(-1, -1, x.shape[2])
        return torch.cat([torch.gather(x[:, :self.K], 1, idx), x[:, self.K:]], dim=1)
