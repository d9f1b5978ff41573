"""The C-ABI library loads and exports every entry point its headers declare,
and host-side argument checks work without a GPU (no kernels run here)."""

import ctypes as C
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2608_08086_amd", "_lib", "libarcher.so")


def _declared():
    names = set()
    for h in ("archer.h", "archer_ops.h"):
        text = open(os.path.join(ROOT, "include", h)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"\b(archer_[a-z_0-9]+)\s*\(", text))
    return names


def test_headers_declare_the_four_named_calls():
    d = _declared()
    for n in ("archer_init", "archer_step", "archer_refresh_prompt", "archer_decode"):
        assert n in d


def test_library_exports_every_declared_symbol():
    assert os.path.exists(LIB), "build the library first (python -m paper_2608_08086_amd.build)"
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True, check=True).stdout
    exported = {l.split()[-1] for l in out.splitlines() if " T " in l}
    missing = _declared() - exported
    assert not missing, missing
    lib = C.CDLL(LIB)
    for n in _declared():
        getattr(lib, n)


def test_binding_lists_every_declared_symbol():
    from paper_2608_08086_amd import archer
    assert set(archer.EXPORTED) == _declared()


def _cfg(archer, **kw):
    base = dict(n_layers=2, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64, d_ff=1024, vocab=1024,
                mask_id=1023, rms_eps=1e-5, rope_theta=10000.0, dtype=archer.FP32)
    base.update(kw)
    return archer.ModelCfg(**base)


def test_workspace_bytes_and_host_side_errors():
    from paper_2608_08086_amd import archer
    lim = archer.Limits(1, 64, 64, 32)
    n = archer.lib.archer_workspace_bytes(C.byref(_cfg(archer)), C.byref(lim))
    assert n > 0 and n % 256 == 0
    # fp16 gate/up operands are a bf16-model option (rejected above for fp32)
    assert archer.lib.archer_workspace_bytes(C.byref(_cfg(archer, dtype=archer.BF16, gateup_fp16=1)),
                                             C.byref(lim)) > 0
    # bigger limits need more workspace
    lim2 = archer.Limits(2, 128, 256, 32)
    assert archer.lib.archer_workspace_bytes(C.byref(_cfg(archer)), C.byref(lim2)) > n
    bad = [dict(head_dim=96), dict(n_kv_heads=3), dict(d_model=250), dict(mask_id=1024), dict(dtype=7),
           dict(gateup_fp16=1), dict(dtype=archer.FP16)]
    for kw in bad:
        assert archer.lib.archer_workspace_bytes(C.byref(_cfg(archer, **kw)), C.byref(lim)) == 0
        assert archer.lib.archer_last_error()
    for lim_bad in (archer.Limits(0, 64, 64, 32), archer.Limits(1, 64, 64, 30), archer.Limits(65, 64, 64, 32),
                    archer.Limits(1, 64, 32, 32)):
        assert archer.lib.archer_workspace_bytes(C.byref(_cfg(archer)), C.byref(lim_bad)) == 0
    # null arguments are rejected before any HIP call
    h = C.c_void_p()
    assert archer.lib.archer_init(None, None, None, None, 0, None, C.byref(h)) != 0
    assert archer.lib.archer_step(None, None, None, None) == archer.E_ARG
    assert archer.lib.archer_decode(None, 1, None, None, None, None, None) == archer.E_ARG
    assert archer.lib.archer_op_gemm(archer.BF16, 0, 64, 64, None, None, None, None, None) == archer.E_ARG
    # session, state-read and precision calls refuse a null context before any HIP call
    assert archer.lib.archer_session_begin(None, 1, None, None, None, None, None) == archer.E_ARG
    assert archer.lib.archer_session_advance(None, 1, 0, None) == archer.E_ARG
    assert archer.lib.archer_session_response(None, None) == archer.E_ARG
    assert archer.lib.archer_session_state_bytes(None) == 0
    assert archer.lib.archer_session_save(None, None, 0) == archer.E_ARG
    assert archer.lib.archer_session_restore(None, None, 0) == archer.E_ARG
    assert archer.lib.archer_read_state(None, 0, 0, 0, None, 0) == archer.E_ARG
    assert archer.lib.archer_set_single_term(None, 0) == archer.E_ARG
    # shape checks happen on the host before any launch (N not a multiple of 64)
    assert archer.lib.archer_op_gemm(archer.BF16, 8, 60, 64, C.c_void_p(16), None, C.c_void_p(16),
                                     C.c_void_p(16), None) == archer.E_SHAPE
    # weight packing: host-side checks before any launch
    pk = archer.lib.archer_pack_weight
    a0, a1 = C.c_void_p(1 << 20), C.c_void_p(1 << 30)
    assert pk(archer.FP32, 64, 64, a0, a1, None) == archer.E_UNSUPPORTED
    assert pk(archer.BF16, 64, 64, None, a1, None) == archer.E_ARG
    assert pk(archer.BF16, 64, 48, a0, a1, None) == archer.E_SHAPE
    assert pk(archer.BF16, 0, 64, a0, a1, None) == archer.E_SHAPE
    assert pk(archer.BF16, 64, 64, a0, C.c_void_p((1 << 20) + 4096), None) == archer.E_ARG   # overlap
    assert pk(archer.BF16, 64, 64, C.c_void_p((1 << 20) + 8), a1, None) == archer.E_ARG      # alignment
    # the k-block weight layout is refused for fp32 models, unknown layouts for any model
    cfg32 = _cfg(archer, dtype=archer.FP32)
    L = cfg32.n_layers
    per = (C.c_void_p * L)(*([16] * L))
    pp = C.cast(per, C.POINTER(C.c_void_p))
    for dt, layout, want in ((archer.FP32, archer.LAYOUT_KBLOCK, archer.E_UNSUPPORTED),
                             (archer.BF16, 7, archer.E_ARG)):
        w = archer.Weights(16, 16, 16, pp, pp, pp, pp, pp, pp, pp, layout)
        assert archer.lib.archer_init(C.byref(_cfg(archer, dtype=dt)), C.byref(w), C.byref(lim), None, 0, None,
                                      C.byref(h)) == want
