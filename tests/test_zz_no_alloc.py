"""vase_decode_step_noalloc: the decode step without a caller workspace.

Its split partials live in a scratch array the library keeps on the GPU, so
the call allocates nothing.  Through the C ABI it must give exactly what
vase_decode_step gives with a workspace -- the appended rows, the window ring,
the persistent-slot LSE and the attention output, bit for bit -- on two calls
in a row, the second on a smaller input, whose partials then reuse the part of
the scratch the first call filled.  Shapes whose partials exceed the scratch
are rejected on the host.
"""
import ctypes

import pytest
import torch

from paper_2606_03928_amd import synth, vase

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def _lib():
    lib = vase.load()
    assert hasattr(lib, "vase_decode_step_noalloc")
    return lib


def _state(cfg, n, seed):
    x = synth.make_round_inputs(cfg, DEV, seed=seed, n_inst=n)
    g = torch.Generator(device=DEV)
    g.manual_seed(seed + 100)
    d, G, w = cfg.d, cfg.G, cfg.w
    st = {
        "k": x["k"], "v": x["v"],
        "k_new": torch.randn((n, d), generator=g, device=DEV).to(cfg.torch_dtype),
        "v_new": torch.randn((n, d), generator=g, device=DEV).to(cfg.torch_dtype),
        "q": torch.randn((n, G, d), generator=g, device=DEV).to(cfg.torch_dtype),
        "q_win": x["q_win"].clone(),
        "lse_win": torch.randn((n, G, w), generator=g, device=DEV),
        "out": torch.full((n, G, d), float("nan"), device=DEV).to(cfg.torch_dtype),
    }
    return st


def _clone(st):
    return {k_: t.clone() for k_, t in st.items()}


def _ptrs(st):
    return [ctypes.c_void_p(st[n].data_ptr()) for n in ("k", "v", "k_new", "v_new", "q")]


def _run_noalloc(lib, st, cfg, pos):
    n = st["k"].shape[0]
    return lib.vase_decode_step_noalloc(*_ptrs(st), 0, n, cfg.K, cfg.B, cfg.d, cfg.G, cfg.w, pos,
                                        ctypes.c_void_p(st["q_win"].data_ptr()),
                                        ctypes.c_void_p(st["lse_win"].data_ptr()),
                                        ctypes.c_void_p(st["out"].data_ptr()),
                                        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))


def _run_ws(lib, st, cfg, pos):
    n = st["k"].shape[0]
    nb = vase.workspace_bytes(vase.OP_DECODE, cfg.torch_dtype, n, cfg.K, cfg.B, cfg.d, cfg.G)
    ws = torch.empty(max(nb, 16), dtype=torch.uint8, device=DEV)
    rc = lib.vase_decode_step(*_ptrs(st), 0, n, cfg.K, cfg.B, cfg.d, cfg.G, cfg.w, pos,
                              ctypes.c_void_p(st["q_win"].data_ptr()),
                              ctypes.c_void_p(st["lse_win"].data_ptr()),
                              ctypes.c_void_p(st["out"].data_ptr()), ctypes.c_void_p(ws.data_ptr()),
                              ctypes.c_size_t(ws.numel()),
                              ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    return rc, nb


def test_noalloc_matches_workspace_step_twice():
    lib = _lib()
    cfg = synth.CONFIGS["qwen3-8b"]
    # the full Qwen3-8B shape (its partials fill 10 MB of the scratch), then a
    # smaller batch at another buffer position
    for n, pos, seed in ((cfg.n_inst, 0, 1), (96, 77, 2)):
        a = _state(cfg, n, seed)
        b = _clone(a)
        assert _run_noalloc(lib, a, cfg, pos) == vase.OK
        rc, nb = _run_ws(lib, b, cfg, pos)
        assert rc == vase.OK and 0 < nb <= vase.DECODE_SCRATCH_BYTES
        torch.cuda.synchronize()
        for name in ("k", "v", "q_win", "lse_win", "out"):
            assert torch.equal(a[name], b[name]), (n, pos, name)
        assert torch.isfinite(a["out"].float()).all()


def test_noalloc_rejects_partials_beyond_the_scratch():
    lib = _lib()
    # fp32 caches of the Qwen3-32B shape: 32768 instances, each with a split for
    # the persistent slots and one for the buffer rows, 277 MB of partials (bf16
    # decode folds the buffer rows into the last persistent split, and its
    # partials stay far below the scratch at every shape)
    cfg = synth.CONFIGS["qwen3-32b"]
    nb = vase.workspace_bytes(vase.OP_DECODE, torch.float32, cfg.n_inst, cfg.K, cfg.B, cfg.d,
                              cfg.G)
    assert nb > vase.DECODE_SCRATCH_BYTES
    fake = ctypes.c_void_p(1 << 20)            # validation rejects the call before any device work
    rc = lib.vase_decode_step_noalloc(fake, fake, fake, fake, fake, 1, cfg.n_inst, cfg.K, cfg.B,
                                      cfg.d, cfg.G, cfg.w, 5, fake, fake, fake, None)
    assert rc == vase.ERR_WORKSPACE
