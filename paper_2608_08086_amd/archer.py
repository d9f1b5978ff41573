"""Python binding of libarcher.so (ctypes).  Argument marshalling only.

Every computation runs in the library's HIP kernels; this module turns torch
CUDA tensors into device pointers and the C structs of include/archer.h and
include/archer_ops.h.  torch provides device memory and the stream.  If the
shared library has not been built the import fails loudly -- there is no
fallback path.
"""

from __future__ import annotations

import ctypes as C
import math
import os

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "_lib", "libarcher.so")
if not os.path.exists(_LIB_PATH):
    raise ImportError(f"{_LIB_PATH} is missing: build it with `python -m paper_2608_08086_amd.build`")
lib = C.CDLL(_LIB_PATH)

OK, E_ARG, E_SHAPE, E_STATE, E_HIP, E_WORKSPACE, E_UNSUPPORTED = 0, -1, -2, -3, -4, -5, -6
BF16, FP32, FP16 = 0, 1, 2
HAMMING, AGE, ALWAYS = 0, 1, 2
LAYOUT_ROWMAJOR, LAYOUT_KBLOCK = 0, 1
NEVER = 2**31 - 1
K_EMBED, K_NORM, K_GEMM_QKV, K_ATTN, K_ATTN_FULL, K_GEMM_O, K_GEMM_GATEUP, K_GEMM_DOWN, K_GEMM_HEAD, K_DECIDE = range(10)
K_GEMM_QKV_FULL, K_GEMM_O_FULL, K_GEMM_GATEUP_FULL, K_GEMM_DOWN_FULL = range(10, 14)
K_COUNT = 14
K_NAMES = ["embed", "norm", "gemm_qkv", "attn", "attn_full", "gemm_o", "gemm_gateup", "gemm_down",
           "gemm_head", "decide", "gemm_qkv_full", "gemm_o_full", "gemm_gateup_full", "gemm_down_full"]

EXPORTED = [
    "archer_workspace_bytes", "archer_init", "archer_refresh_prompt", "archer_step", "archer_decide",
    "archer_decode", "archer_sync", "archer_destroy", "archer_last_error", "archer_op_gemm",
    "archer_op_attention_ws_bytes", "archer_op_attention", "archer_timing_begin", "archer_timing_end",
    "archer_pack_weight", "archer_session_begin", "archer_session_advance", "archer_session_response",
    "archer_session_state_bytes", "archer_session_save", "archer_session_restore", "archer_read_state",
    "archer_set_single_term", "archer_op_attention_noalloc",
]
FORWARD_CONTROLLER, FORWARD_REFRESH, FORWARD_CACHED = 0, 1, 2
READ_LOGITS, READ_HIDDEN, READ_RESIDUAL, READ_PROMPT_K, READ_PROMPT_V = range(5)
# projection classes that can take a single-term activation (archer_set_single_term)
SINGLE_TERM_CLASSES = {"qkv": K_GEMM_QKV, "o": K_GEMM_O, "gateup": K_GEMM_GATEUP, "down": K_GEMM_DOWN,
                       "head": K_GEMM_HEAD}


class ModelCfg(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("d_ff", C.c_int32),
                ("vocab", C.c_int32), ("mask_id", C.c_int32), ("rms_eps", C.c_float),
                ("rope_theta", C.c_float), ("dtype", C.c_int32), ("gateup_fp16", C.c_int32)]


class Weights(C.Structure):
    _fields_ = [("tok_emb", C.c_void_p), ("lm_head", C.c_void_p), ("final_norm", C.c_void_p),
                ("attn_norm", C.POINTER(C.c_void_p)), ("w_qkv", C.POINTER(C.c_void_p)),
                ("w_o", C.POINTER(C.c_void_p)), ("mlp_norm", C.POINTER(C.c_void_p)),
                ("w_gate", C.POINTER(C.c_void_p)), ("w_up", C.POINTER(C.c_void_p)),
                ("w_down", C.POINTER(C.c_void_p)), ("layout", C.c_int32)]


class Limits(C.Structure):
    _fields_ = [("max_batch", C.c_int32), ("max_prompt_len", C.c_int32),
                ("max_prompt_total", C.c_int32), ("resp_len", C.c_int32)]


class DecideCfg(C.Structure):
    _fields_ = [("unmask_per_step", C.c_int32), ("remask_threshold", C.c_float),
                ("max_remask", C.c_int32), ("final_step", C.c_int32)]


class DecodeCfg(C.Structure):
    _fields_ = [("policy", C.c_int32), ("K", C.c_int32), ("steps", C.c_int32),
                ("unmask_per_step", C.c_int32), ("remask_threshold", C.c_float),
                ("max_remask", C.c_int32), ("keep_logits", C.c_int32)]


class Trace(C.Structure):
    _fields_ = [("refreshed", C.c_void_p), ("dist", C.c_void_p), ("age", C.c_void_p),
                ("unmask_pos", C.c_void_p), ("unmask_tok", C.c_void_p), ("remask_pos", C.c_void_p)]


P = C.c_void_p
lib.archer_workspace_bytes.restype = C.c_size_t
lib.archer_workspace_bytes.argtypes = [C.POINTER(ModelCfg), C.POINTER(Limits)]
lib.archer_init.restype = C.c_int
lib.archer_init.argtypes = [C.POINTER(ModelCfg), C.POINTER(Weights), C.POINTER(Limits), P, C.c_size_t, P,
                            C.POINTER(P)]
lib.archer_refresh_prompt.restype = C.c_int
lib.archer_refresh_prompt.argtypes = [P, C.c_int32, P, C.POINTER(C.c_int32), P, P, P]
lib.archer_step.restype = C.c_int
lib.archer_step.argtypes = [P, P, P, P]
lib.archer_decide.restype = C.c_int
lib.archer_decide.argtypes = [P, P, P, P, C.POINTER(DecideCfg), P, P, P]
lib.archer_decode.restype = C.c_int
lib.archer_decode.argtypes = [P, C.c_int32, P, C.POINTER(C.c_int32), P, C.POINTER(DecodeCfg), C.POINTER(Trace)]
lib.archer_sync.restype = C.c_int
lib.archer_sync.argtypes = [P]
lib.archer_destroy.restype = None
lib.archer_destroy.argtypes = [P]
lib.archer_last_error.restype = C.c_char_p
lib.archer_last_error.argtypes = []
lib.archer_op_gemm.restype = C.c_int
lib.archer_op_gemm.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.c_int32, P, P, P, P, P]
lib.archer_op_attention_ws_bytes.restype = C.c_size_t
lib.archer_op_attention_ws_bytes.argtypes = [C.c_int32] * 5
lib.archer_op_attention.restype = C.c_int
lib.archer_op_attention.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_int32, P, P, P, C.c_int32,
                                    C.c_int32, P, P, C.c_int32, C.c_int32, P, P, C.c_size_t, P]
lib.archer_pack_weight.restype = C.c_int
lib.archer_pack_weight.argtypes = [C.c_int32, C.c_int32, C.c_int32, P, P, P]
lib.archer_session_begin.restype = C.c_int
lib.archer_session_begin.argtypes = [P, C.c_int32, P, C.POINTER(C.c_int32), P, C.POINTER(DecodeCfg),
                                     C.POINTER(Trace)]
lib.archer_session_advance.restype = C.c_int
lib.archer_session_advance.argtypes = [P, C.c_int32, C.c_int32, C.POINTER(C.c_int32)]
lib.archer_session_response.restype = C.c_int
lib.archer_session_response.argtypes = [P, P]
lib.archer_session_state_bytes.restype = C.c_size_t
lib.archer_session_state_bytes.argtypes = [P]
lib.archer_session_save.restype = C.c_int
lib.archer_session_save.argtypes = [P, P, C.c_size_t]
lib.archer_session_restore.restype = C.c_int
lib.archer_session_restore.argtypes = [P, P, C.c_size_t]
lib.archer_read_state.restype = C.c_int
lib.archer_read_state.argtypes = [P, C.c_int32, C.c_int32, C.c_int32, P, C.c_size_t]
lib.archer_set_single_term.restype = C.c_int
lib.archer_set_single_term.argtypes = [P, C.c_uint32]
lib.archer_op_attention_noalloc.restype = C.c_int
lib.archer_op_attention_noalloc.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_int32, P, P, P,
                                            C.c_int32, C.c_int32, P, P, C.c_int32, C.c_int32, P, P]
lib.archer_timing_begin.restype = C.c_int
lib.archer_timing_begin.argtypes = [P, C.c_uint32, C.c_int32]
lib.archer_timing_end.restype = C.c_int
lib.archer_timing_end.argtypes = [P, C.POINTER(C.c_int64), C.POINTER(C.c_double), C.POINTER(C.c_double),
                                  C.POINTER(C.c_double)]


class ArcherError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"archer status {status}: {msg}")
        self.status = status


def _check(status: int):
    if status != OK:
        raise ArcherError(status, lib.archer_last_error().decode())


def _ptr(t):
    if t is None:
        return None
    assert t.is_cuda and t.is_contiguous(), "device tensors must be contiguous CUDA tensors"
    return C.c_void_p(t.data_ptr())


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def torch_dtype(dtype: int):
    return torch.bfloat16 if dtype == BF16 else torch.float32


def qkv_dtype(dtype: int):
    """Element type of stored queries, keys and values (the prompt cache): fp16 for bf16 models."""
    return torch.float16 if dtype == BF16 else torch.float32


class Context:
    """One archer_ctx: a model's weights (device tensors), limits and workspace."""

    def __init__(self, shape, weights: dict, max_batch: int, max_prompt_len: int, max_prompt_total: int,
                 resp_len: int):
        self.shape = shape
        self.dtype = BF16 if shape.dtype == "bf16" else FP32
        gu16 = int(bool(getattr(shape, "gateup_fp16", False)))
        self.cfg = ModelCfg(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim,
                            shape.d_ff, shape.vocab, shape.mask_id, shape.rms_eps, shape.rope_theta, self.dtype,
                            gu16)
        want = torch.float16 if gu16 else torch_dtype(self.dtype)
        for L_ in weights["layers"]:
            for k in ("w_gate", "w_up"):
                if L_[k].dtype != want:
                    raise ArcherError(E_ARG, f"{k} must be {want} for this model (gateup_fp16={gu16})")
        self.lim = Limits(max_batch, max_prompt_len, max_prompt_total, resp_len)
        self.G = resp_len
        self.V = shape.vocab
        self.weights = weights  # keep device tensors alive
        L = shape.n_layers

        def arr(key):
            a = (C.c_void_p * L)(*[w[key].data_ptr() for w in weights["layers"]])
            return C.cast(a, C.POINTER(C.c_void_p)), a

        self._keep = []
        fields = {}
        for key in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate", "w_up", "w_down"):
            p, a = arr(key)
            self._keep.append(a)
            fields[key] = p
        self.cw = Weights(weights["tok_emb"].data_ptr(), weights["lm_head"].data_ptr(),
                          weights["final_norm"].data_ptr(), **fields,
                          layout=weights.get("layout", LAYOUT_ROWMAJOR))
        nbytes = lib.archer_workspace_bytes(C.byref(self.cfg), C.byref(self.lim))
        if nbytes == 0:
            raise ArcherError(E_ARG, lib.archer_last_error().decode())
        self.ws_bytes = nbytes
        self.workspace = torch.empty(nbytes + 256, dtype=torch.uint8, device="cuda")
        off = (-self.workspace.data_ptr()) % 256
        self._ws_ptr = self.workspace.data_ptr() + off
        h = C.c_void_p()
        _check(lib.archer_init(C.byref(self.cfg), C.byref(self.cw), C.byref(self.lim), C.c_void_p(self._ws_ptr),
                               nbytes, _stream(), C.byref(h)))
        self.h = h
        if getattr(shape, "single_term", ()):
            self.set_single_term(shape.single_term)

    def close(self):
        if getattr(self, "h", None):
            lib.archer_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- calls of archer.h -------------------------------------------------------------------
    def new_logits(self, batch):
        return torch.empty(batch, self.G, self.V, dtype=torch.float32, device="cuda")

    def refresh_prompt(self, prompt, prompt_len, response, seq_sel=None, logits=None):
        B = len(prompt_len)
        logits = self.new_logits(B) if logits is None else logits
        pl = (C.c_int32 * B)(*prompt_len)
        sel = None if seq_sel is None else (C.c_uint8 * B)(*[1 if s else 0 for s in seq_sel])
        _check(lib.archer_refresh_prompt(self.h, B, _ptr(prompt), pl, _ptr(response), sel, _ptr(logits)))
        return logits

    def step(self, response, seq_sel=None, logits=None):
        B = response.shape[0]
        logits = self.new_logits(B) if logits is None else logits
        sel = None if seq_sel is None else (C.c_uint8 * B)(*[1 if s else 0 for s in seq_sel])
        _check(lib.archer_step(self.h, _ptr(response), sel, _ptr(logits)))
        return logits

    def decide(self, logits, g_in, k=1, tau=0.1, max_remask=1, final=False):
        B = g_in.shape[0]
        g_out = torch.empty_like(g_in)
        dist = torch.empty(B, dtype=torch.int32, device="cuda")
        um = torch.empty(B, k, dtype=torch.int32, device="cuda")
        rm = torch.empty(B, dtype=torch.int32, device="cuda")
        dc = DecideCfg(k, tau, max_remask, 1 if final else 0)
        _check(lib.archer_decide(self.h, _ptr(logits), _ptr(g_in), _ptr(g_out), C.byref(dc), _ptr(dist),
                                 _ptr(um), _ptr(rm)))
        return g_out, dist, um, rm

    @staticmethod
    def _trace(steps, B, k):
        dev = dict(device="cuda", dtype=torch.int32)
        tens = dict(refreshed=torch.zeros(steps, B, **dev), dist=torch.zeros(steps, B, **dev),
                    age=torch.zeros(steps, B, **dev), unmask_pos=torch.full((steps, B, k), -1, **dev),
                    unmask_tok=torch.full((steps, B, k), -1, **dev),
                    remask_pos=torch.full((steps, B), -1, **dev))
        return tens, Trace(*[t.data_ptr() for t in tens.values()])

    def decode(self, prompt, prompt_len, response, *, policy, K, steps, k=1, tau=0.1, max_remask=1,
               trace=True, keep_logits=False):
        B = len(prompt_len)
        pl = (C.c_int32 * B)(*prompt_len)
        dc = DecodeCfg(policy, int(min(K, NEVER)), steps, k, tau, max_remask, 1 if keep_logits else 0)
        tens, tr = self._trace(steps, B, k) if trace else (None, None)
        _check(lib.archer_decode(self.h, B, _ptr(prompt), pl, _ptr(response), C.byref(dc),
                                 C.byref(tr) if tr is not None else None))
        return response, tens

    # -- the resumable session (Algorithm 1 a few decisions at a time) --------------------------
    def session_begin(self, prompt, prompt_len, response_init, *, policy, K, steps, k=1, tau=0.1,
                      max_remask=1, trace=True, keep_logits=False):
        """Start a session; returns the trace tensors (or None).  prompt and the trace tensors are
        kept alive by the context while the session may use them."""
        B = len(prompt_len)
        pl = (C.c_int32 * B)(*prompt_len)
        dc = DecodeCfg(policy, int(min(K, NEVER)), steps, k, tau, max_remask, 1 if keep_logits else 0)
        tens, tr = self._trace(steps, B, k) if trace else (None, None)
        self._session = (prompt, tens, tr)
        self.B = B
        _check(lib.archer_session_begin(self.h, B, _ptr(prompt), pl, _ptr(response_init), C.byref(dc),
                                        C.byref(tr) if tr is not None else None))
        return tens

    def session_advance(self, n, first_forward=FORWARD_CONTROLLER):
        t = C.c_int32(0)
        _check(lib.archer_session_advance(self.h, n, first_forward, C.byref(t)))
        return t.value

    def session_response(self):
        out = torch.empty(self.B, self.G, dtype=torch.int32, device="cuda")
        _check(lib.archer_session_response(self.h, _ptr(out)))
        return out

    def session_state_bytes(self):
        n = lib.archer_session_state_bytes(self.h)
        if n == 0:
            raise ArcherError(E_ARG, lib.archer_last_error().decode())
        return n

    def session_save(self):
        """Snapshot of the session's decoder state (a device tensor; 256-byte aligned view)."""
        n = self.session_state_bytes()
        buf = torch.empty(n + 256, dtype=torch.uint8, device="cuda")
        off = (-buf.data_ptr()) % 256
        snap = buf[off: off + n]
        _check(lib.archer_session_save(self.h, _ptr(snap), n))
        return snap

    def session_restore(self, snap):
        _check(lib.archer_session_restore(self.h, _ptr(snap), snap.numel()))

    # -- read-only state copies and the precision switch of archer_ops.h ------------------------
    def read_logits(self, batch):
        out = torch.empty(batch, self.G, self.V, dtype=torch.float32, device="cuda")
        _check(lib.archer_read_state(self.h, READ_LOGITS, 0, 0, _ptr(out), out.numel() * 4))
        return out

    def read_rows(self, what, n_seq):
        """Final normalised hidden (READ_HIDDEN) or final residual (READ_RESIDUAL) of the response
        rows of the last forward: fp32 [n_seq * G][d]."""
        out = torch.empty(n_seq * self.G, self.shape.d_model, dtype=torch.float32, device="cuda")
        _check(lib.archer_read_state(self.h, what, 0, 0, _ptr(out), out.numel() * 4))
        return out

    def read_prompt_kv(self, layer, seq, prompt_len):
        """Cached post-RoPE prompt K and prompt V of one layer and sequence: two [Hkv][P][hd] tensors."""
        m = self.shape
        shape = (m.n_kv_heads, prompt_len, m.head_dim)
        out = []
        for what in (READ_PROMPT_K, READ_PROMPT_V):
            t = torch.empty(shape, dtype=qkv_dtype(self.dtype), device="cuda")
            _check(lib.archer_read_state(self.h, what, layer, seq, _ptr(t), t.numel() * t.element_size()))
            out.append(t)
        return out[0], out[1]

    def set_single_term(self, classes):
        """classes: names from SINGLE_TERM_CLASSES whose activation operand is a single bf16 value."""
        mask = 0
        for c in classes:
            mask |= 1 << SINGLE_TERM_CLASSES[c]
        _check(lib.archer_set_single_term(self.h, mask))

    def sync(self):
        _check(lib.archer_sync(self.h))

    # -- timing of archer_ops.h ---------------------------------------------------------------
    def timing_begin(self, classes, every=1):
        """Record every `every`-th launch of each class in `classes` (1 = all)."""
        mask = 0
        for c in classes:
            mask |= 1 << c
        _check(lib.archer_timing_begin(self.h, mask, every))

    def timing_end(self):
        n = (C.c_int64 * K_COUNT)()
        ms = (C.c_double * K_COUNT)()
        by = (C.c_double * K_COUNT)()
        fl = (C.c_double * K_COUNT)()
        _check(lib.archer_timing_end(self.h, n, ms, by, fl))
        return {K_NAMES[i]: dict(launches=n[i], ms=ms[i], bytes=by[i], flops=fl[i]) for i in range(K_COUNT)}


def upload_weights(W: dict, dtype: str, gateup_fp16: bool = False) -> dict:
    """Host weights (synth layout: uint16 bf16 bits or float32) -> contiguous CUDA tensors.
    gateup_fp16 (bf16 models): w_gate and w_up are converted to fp16, the element type a
    model with gateup_fp16 takes for them."""
    def dev(a):
        if a.dtype.name == "uint16":
            t = torch.from_numpy(a.view("int16")).view(torch.bfloat16)
        else:
            t = torch.from_numpy(a)
        return t.to("cuda").contiguous()

    def dev_layer(k, v):
        t = dev(v)
        return t.to(torch.float16) if gateup_fp16 and dtype == "bf16" and k in ("w_gate", "w_up") else t

    out = {k: dev(W[k]) for k in ("tok_emb", "lm_head", "final_norm")}
    out["layers"] = [{k: dev_layer(k, v) for k, v in L.items()} for L in W["layers"]]
    return out


PROJECTIONS = ("w_qkv", "w_o", "w_gate", "w_up", "w_down")


def pack_weight(w):
    """Row-major bf16 or fp16 [rows][cols] CUDA tensor -> a new tensor in the k-block layout
    (archer_pack_weight)."""
    assert w.dtype in (torch.bfloat16, torch.float16) and w.dim() == 2
    out = torch.empty_like(w)
    dt = BF16 if w.dtype == torch.bfloat16 else FP16
    _check(lib.archer_pack_weight(dt, w.shape[0], w.shape[1], _ptr(w), _ptr(out), _stream()))
    return out


def pack_weights(weights: dict, drop_source: bool = False) -> dict:
    """Weights dict (row-major device tensors) -> the same model with every projection matrix
    (lm_head and the per-layer w_qkv, w_o, w_gate, w_up, w_down) in the k-block layout.
    drop_source releases each source matrix once it is packed (its dict entry is replaced)."""
    out = {k: v for k, v in weights.items() if k != "layers"}
    out["lm_head"] = pack_weight(weights["lm_head"])
    if drop_source:
        weights["lm_head"] = None
    out["layers"] = []
    for L in weights["layers"]:
        P = dict(L)
        for k in PROJECTIONS:
            P[k] = pack_weight(L[k])
            if drop_source:
                L[k] = None
        out["layers"].append(P)
    out["layout"] = LAYOUT_KBLOCK
    return out


# -- single-kernel hooks of archer_ops.h --------------------------------------------------------
def op_gemm(A, Wt, dtype=BF16, A_lo=None):
    M, K = A.shape
    N = Wt.shape[0]
    Y = torch.empty(M, N, dtype=torch.float32, device="cuda")
    _check(lib.archer_op_gemm(dtype, M, N, K, _ptr(A), _ptr(A_lo), _ptr(Wt), _ptr(Y), _stream()))
    return Y


def op_attention(Q, K1, Vt1, nk1, K2, Vt2, nk2, dtype=BF16):
    """Q [Hq][Mq][hd]; K1 [Hkv][ld1][hd], Vt1 [Hkv][hd][ld1]; same for segment 2 (fp16 for BF16,
    fp32 for FP32).  Returns O [Mq][Hq*hd] (bf16 for BF16, fp32 for FP32)."""
    Hq, Mq, hd = Q.shape
    Hkv, ld1, _ = K1.shape
    ld2 = K2.shape[1]
    for t in (Q, K1, Vt1, K2, Vt2):
        assert t.dtype == qkv_dtype(dtype), "queries, keys and values: fp16 for BF16, fp32 for FP32"
    O = torch.empty(Mq, Hq * hd, dtype=torch_dtype(dtype), device="cuda")
    nbytes = lib.archer_op_attention_ws_bytes(dtype, Mq, Hq, hd, ((nk1 + 63) // 64) * 64 + nk2)
    ws = torch.empty(max(nbytes, 1) + 256, dtype=torch.uint8, device="cuda")
    wp = ws.data_ptr() + ((-ws.data_ptr()) % 256)
    _check(lib.archer_op_attention(dtype, Mq, Hq, Hkv, hd, _ptr(Q), _ptr(K1), _ptr(Vt1), nk1, ld1, _ptr(K2),
                                   _ptr(Vt2), nk2, ld2, _ptr(O), C.c_void_p(wp), nbytes, _stream()))
    return O


def op_attention_noalloc(Q, K1, Vt1, nk1, K2, Vt2, nk2, dtype=BF16, O=None):
    """archer_op_attention_noalloc: as op_attention, with the split-KV partials in the library's
    fixed scratch array (no workspace).  O may be given (preallocated); returns it."""
    Hq, Mq, hd = Q.shape
    Hkv, ld1, _ = K1.shape
    ld2 = K2.shape[1]
    for t in (Q, K1, Vt1, K2, Vt2):
        assert t.dtype == qkv_dtype(dtype), "queries, keys and values: fp16 for BF16, fp32 for FP32"
    if O is None:
        O = torch.empty(Mq, Hq * hd, dtype=torch_dtype(dtype), device="cuda")
    _check(lib.archer_op_attention_noalloc(dtype, Mq, Hq, Hkv, hd, _ptr(Q), _ptr(K1), _ptr(Vt1), nk1, ld1,
                                           _ptr(K2), _ptr(Vt2), nk2, ld2, _ptr(O), _stream()))
    return O
