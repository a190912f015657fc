"""ctypes binding of libmg.so (include/mg.h, include/mg_ops.h).

Argument marshalling only: every step of the hot path runs in the library's HIP
kernels.  torch supplies device memory and the stream; tensors are passed as raw
device pointers.  load() raises when the library is missing: there is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmg.so")

MG_OK = 0
# repair actions (include/mg.h)
REPAIR_ON_MISMATCH, REPAIR_TOKEN_ONLY, REPAIR_COPY_ALWAYS = 0, 1, 2
KIND_FAST_GEMM, KIND_FAST_ATTN, KIND_CANON_GEMV, KIND_CANON_ATTN, KIND_GATE = range(5)
WPL = 12

_STATUS = {0: "ok", -1: "invalid argument", -2: "unsupported model shape", -3: "workspace or KV pool too small",
           -4: "HIP runtime error", -5: "invalid state"}


class MgError(RuntimeError):
    def __init__(self, call, status):
        super().__init__(f"{call} failed: {_STATUS.get(status, status)} ({status})")
        self.status = status


class MgModelCfg(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("n_layers", "d_model", "n_q_heads", "n_kv_heads", "head_dim", "d_ffn",
                                         "vocab", "qkv_bias")] + \
               [("rope_theta", C.c_float), ("rms_eps", C.c_float)] + \
               [(n, C.c_int32) for n in ("page_size", "max_batch", "max_pages_per_row", "n_pages", "max_prefill")]


# name -> (restype, argtypes); the set of C-ABI symbols the binding uses
P, I, F, I64, SZ = C.c_void_p, C.c_int, C.c_float, C.c_int64, C.c_size_t
SIGNATURES = {
    "mg_weight_count": (I, [P]),
    "mg_kv_pool_bytes": (SZ, [P]),
    "mg_kv_col_elems": (SZ, [P]),
    "mg_workspace_bytes": (SZ, [P]),
    "mg_status_string": (C.c_char_p, [I]),
    "mg_create": (I, [P, P, P, SZ, P, SZ, P]),
    "mg_destroy": (I, [P]),
    "mg_decode_step": (I, [P, I, P, P, P, P, P]),
    "mg_margin_gate": (I, [P, I, P, P, F, P, P, P, P, P, P, P]),
    "mg_margin_gate_noalloc": (I, [I, I, P, P, F, P, P, P, P, P, P]),
    "mg_verify_rows": (I, [P, I, P, P, P, P, P, P, P, P, P]),
    "mg_repair_kv_column": (I, [P, I, P, P, P, P, P, P, P, P, P, P]),
    "mg_repair_kv_column_action": (I, [P, I, P, P, P, P, P, P, P, P, P, I, P]),
    "mg_verify_rows_mfma": (I, [P, I, P, P, P, P, P, P, P, P]),
    "mg_prefill": (I, [P, I, P, P, P, P, P]),
    "mg_advance": (I, [P, I, P, P, P, P]),
    "mg_profile_begin": (I, [P, I, I]),
    "mg_profile_end": (I, [P, I, P, P, P, P]),
    "mg_op_copy": (I, [I64, P, P, P]),
    "mg_op_read_stream_sink_words": (I, []),
    "mg_op_read_stream": (I, [I64, P, P, P]),
    "mg_op_probe_bf16": (I, [I64, P, P, P]),
    "mg_op_probe_exp": (I, [I64, P, P, P]),
    "mg_op_probe_divsqrt": (I, [I64, P, P, P, P, P]),
    "mg_op_probe_mfma_fma": (I, [I, P, P, P, P, P]),
    "mg_op_probe_mfma4_fma": (I, [I, P, P, P, P, P]),
    "mg_op_linear_workspace_bytes": (SZ, [I, I, I]),
    "mg_op_linear": (I, [I, I, I, I, P, P, P, P, P, SZ, P]),
    "mg_op_fast_gemm_config": (I, [I, I, I, I, P, P]),
    "mg_op_canon_gemv_config": (I, [I, I, I, I, I, P, P, P, P, P]),
    "mg_op_rmsnorm": (I, [I, I, P, P, F, P, P]),
    "mg_op_decode_step_taps": (I, [P, I, P, P, P, P, P, P]),
}

_lib = None


def load():
    """Open libmg.so (built in-tree by build_lib.py).  Raises if it is not there."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2605_30218_amd.build_lib` "
                               "(or __graft_entry__.build()); there is no fallback path")
        lib = C.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(lib, name)
            f.restype = res
            f.argtypes = args
        _lib = lib
    return _lib


def host_count_slot():
    """A few int32 of coherent, mapped pinned host memory (hipHostMalloc), for a count that
    a kernel stores with system scope and the host polls.  Returns (device pointer, numpy
    view of the int32s).  The memory is held until the process ends."""
    hip = C.CDLL("libamdhip64.so")
    host = C.c_void_p()
    flags = 0x40000000 | 0x2  # hipHostMallocCoherent | hipHostMallocMapped
    if hip.hipHostMalloc(C.byref(host), C.c_size_t(64), C.c_uint(flags)) != 0 or not host.value:
        raise RuntimeError("hipHostMalloc of the gate count slot failed")
    dev = C.c_void_p()
    if hip.hipHostGetDevicePointer(C.byref(dev), host, C.c_uint(0)) != 0 or not dev.value:
        raise RuntimeError("hipHostGetDevicePointer of the gate count slot failed")
    view = np.ctypeslib.as_array((C.c_int32 * 16).from_address(host.value))
    return dev.value, view


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _check(call, rc):
    if rc != MG_OK:
        raise MgError(call, rc)


def make_cfg(shape, max_batch, max_pages_per_row, n_pages, max_prefill=0) -> MgModelCfg:
    return MgModelCfg(shape.n_layers, shape.d_model, shape.n_q_heads, shape.n_kv_heads, shape.head_dim,
                      shape.d_ffn, shape.vocab, int(shape.qkv_bias), float(shape.rope_theta), float(shape.rms_eps),
                      shape.page_size, max_batch, max_pages_per_row, n_pages, max_prefill)


class Engine:
    """A libmg context over caller-owned device memory: weights (list of int16 tensors holding bf16
    bits, None for absent biases), the paged KV pool and the workspace."""

    def __init__(self, shape, weights, max_batch, max_pages_per_row, n_pages, max_prefill=0, device="cuda"):
        self.lib = load()
        self.shape = shape
        self.cfg = make_cfg(shape, max_batch, max_pages_per_row, n_pages, max_prefill)
        self.device = torch.device(device)
        nw = self.lib.mg_weight_count(C.byref(self.cfg))
        assert len(weights) == nw, (len(weights), nw)
        self.weights = [None if w is None else w.to(self.device) for w in weights]
        self._wtab = (C.c_void_p * nw)(*[None if w is None else w.data_ptr() for w in self.weights])
        kv_bytes = self.lib.mg_kv_pool_bytes(C.byref(self.cfg))
        ws_bytes = self.lib.mg_workspace_bytes(C.byref(self.cfg))
        if ws_bytes == 0:
            raise MgError("mg_workspace_bytes", -2)
        self.kv_pool = torch.zeros(kv_bytes // 2, dtype=torch.int16, device=self.device)
        self.workspace = torch.zeros(ws_bytes, dtype=torch.uint8, device=self.device)
        self.col_elems = self.lib.mg_kv_col_elems(C.byref(self.cfg))
        ctx = C.c_void_p()
        _check("mg_create", self.lib.mg_create(C.byref(self.cfg), self._wtab, self.kv_pool.data_ptr(), kv_bytes,
                                               self.workspace.data_ptr(), ws_bytes, C.byref(ctx)))
        self.ctx = ctx

    def close(self):
        if getattr(self, "ctx", None):
            self.lib.mg_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def kv_view(self):
        s, c = self.shape, self.cfg
        return self.kv_pool.view(s.n_layers, c.n_pages, 2, s.n_kv_heads, s.page_size, s.head_dim)

    # the C-ABI calls, same names without the mg_ prefix
    def decode_step(self, B, tokens, positions, page_table, logits, stream=None):
        _check("mg_decode_step", self.lib.mg_decode_step(self.ctx, B, _ptr(tokens), _ptr(positions),
                                                         _ptr(page_table), _ptr(logits), _stream(stream)))

    def decode_step_taps(self, B, tokens, positions, page_table, logits, x_taps, stream=None):
        """mg_op_decode_step_taps: the fast step plus the residual stream at every layer boundary
        (x_taps int16 [(n_layers + 1), B, d_model] holding bf16 bits)."""
        _check("mg_op_decode_step_taps", self.lib.mg_op_decode_step_taps(
            self.ctx, B, _ptr(tokens), _ptr(positions), _ptr(page_table), _ptr(logits), _ptr(x_taps),
            _stream(stream)))

    def margin_gate(self, B, logits, protected_mask, tau, top1, margin, gate, gated_rows, n_gated,
                    n_gated_host=None, stream=None):
        """n_gated_host: optional pinned CPU int32 tensor that receives the count too."""
        _check("mg_margin_gate", self.lib.mg_margin_gate(self.ctx, B, _ptr(logits), _ptr(protected_mask), float(tau),
                                                         _ptr(top1), _ptr(margin), _ptr(gate), _ptr(gated_rows),
                                                         _ptr(n_gated), _ptr(n_gated_host), _stream(stream)))

    def verify_rows(self, n, rows, n_dev, tokens, positions, page_table, v_logits, v_tok, v_kvcol, stream=None):
        _check("mg_verify_rows", self.lib.mg_verify_rows(self.ctx, n, _ptr(rows), _ptr(n_dev), _ptr(tokens),
                                                         _ptr(positions), _ptr(page_table), _ptr(v_logits),
                                                         _ptr(v_tok), _ptr(v_kvcol), _stream(stream)))

    def repair_kv_column(self, n, rows, n_dev, positions, page_table, top1, v_tok, v_kvcol, emitted, n_repaired,
                         stream=None):
        _check("mg_repair_kv_column", self.lib.mg_repair_kv_column(
            self.ctx, n, _ptr(rows), _ptr(n_dev), _ptr(positions), _ptr(page_table), _ptr(top1), _ptr(v_tok),
            _ptr(v_kvcol), _ptr(emitted), _ptr(n_repaired), _stream(stream)))

    def verify_rows_mfma(self, n, rows, tokens, positions, page_table, v_logits, v_tok, v_kvcol, stream=None):
        _check("mg_verify_rows_mfma", self.lib.mg_verify_rows_mfma(
            self.ctx, n, _ptr(rows), _ptr(tokens), _ptr(positions), _ptr(page_table), _ptr(v_logits), _ptr(v_tok),
            _ptr(v_kvcol), _stream(stream)))

    def repair_kv_column_action(self, n, rows, n_dev, positions, page_table, top1, v_tok, v_kvcol, emitted,
                                n_repaired, action, stream=None):
        _check("mg_repair_kv_column_action", self.lib.mg_repair_kv_column_action(
            self.ctx, n, _ptr(rows), _ptr(n_dev), _ptr(positions), _ptr(page_table), _ptr(top1), _ptr(v_tok),
            _ptr(v_kvcol), _ptr(emitted), _ptr(n_repaired), int(action), _stream(stream)))

    def prefill(self, n_items, tokens, positions, item_rows, page_table, stream=None):
        _check("mg_prefill", self.lib.mg_prefill(self.ctx, n_items, _ptr(tokens), _ptr(positions), _ptr(item_rows),
                                                 _ptr(page_table), _stream(stream)))

    def advance(self, B, emitted, tokens, positions, stream=None):
        _check("mg_advance", self.lib.mg_advance(self.ctx, B, _ptr(emitted), _ptr(tokens), _ptr(positions),
                                                 _stream(stream)))

    def profile_begin(self, kind, max_launches):
        _check("mg_profile_begin", self.lib.mg_profile_begin(self.ctx, kind, max_launches))

    def profile_end(self, kind):
        n, ms, b, f = C.c_int(), C.c_double(), C.c_double(), C.c_double()
        _check("mg_profile_end", self.lib.mg_profile_end(self.ctx, kind, C.byref(n), C.byref(ms), C.byref(b),
                                                         C.byref(f)))
        return n.value, ms.value, b.value, f.value


def margin_gate_noalloc(B, V, logits, protected_mask, tau, top1, margin, gate, gated_rows, n_gated, stream=None):
    """mg_margin_gate_noalloc: the margin gate with no context and no allocation (its scratch is a
    static device array of the library)."""
    _check("mg_margin_gate_noalloc", load().mg_margin_gate_noalloc(
        int(B), int(V), _ptr(logits), _ptr(protected_mask), float(tau), _ptr(top1), _ptr(margin), _ptr(gate),
        _ptr(gated_rows), _ptr(n_gated), _stream(stream)))


# ---------------------------------------------------------------- op-level calls (tests)

def op_copy(src, dst):
    _check("mg_op_copy", load().mg_op_copy(src.numel() * src.element_size(), src.data_ptr(), dst.data_ptr(),
                                           _stream()))


def op_read_stream(src, sink):
    """mg_op_read_stream: read every byte of src once (the HBM read-rate reference)."""
    _check("mg_op_read_stream", load().mg_op_read_stream(src.numel() * src.element_size(), src.data_ptr(),
                                                         sink.data_ptr(), _stream()))


def read_stream_sink_words():
    return int(load().mg_op_read_stream_sink_words())


def op_probe_bf16(x):
    out = torch.empty(x.shape, dtype=torch.int16, device=x.device)
    _check("mg_op_probe_bf16", load().mg_op_probe_bf16(x.numel(), x.data_ptr(), out.data_ptr(), _stream()))
    return out


def op_probe_exp(x):
    out = torch.empty_like(x)
    _check("mg_op_probe_exp", load().mg_op_probe_exp(x.numel(), x.data_ptr(), out.data_ptr(), _stream()))
    return out


def op_probe_divsqrt(a, b):
    q, r = torch.empty_like(a), torch.empty_like(a)
    _check("mg_op_probe_divsqrt", load().mg_op_probe_divsqrt(a.numel(), a.data_ptr(), b.data_ptr(), q.data_ptr(),
                                                             r.data_ptr(), _stream()))
    return q, r


def op_probe_mfma_fma(a, b, c):
    d = torch.empty_like(c)
    _check("mg_op_probe_mfma_fma", load().mg_op_probe_mfma_fma(a.shape[0], a.data_ptr(), b.data_ptr(), c.data_ptr(),
                                                               d.data_ptr(), _stream()))
    return d


def op_probe_mfma4_fma(a, b, c):
    d = torch.empty_like(c)
    _check("mg_op_probe_mfma4_fma", load().mg_op_probe_mfma4_fma(a.shape[0], a.data_ptr(), b.data_ptr(), c.data_ptr(),
                                                                 d.data_ptr(), _stream()))
    return d


def op_linear(canon, X, W):
    n, K = X.shape
    N = W.shape[0]
    Y = torch.empty((n, N), dtype=torch.float32, device=X.device)
    lib = load()
    wsb = lib.mg_op_linear_workspace_bytes(n, N, K)
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=X.device)
    _check("mg_op_linear", lib.mg_op_linear(int(canon), n, N, K, X.data_ptr(), W.data_ptr(), None, Y.data_ptr(),
                                            ws.data_ptr(), wsb, _stream()))
    return Y


def fast_gemm_config(n, N, K, n_cu=256):
    """(split-K factor, waves per block) of the fast GEMM launch for n rows of an N x K
    projection on a device of n_cu compute units (host logic, no device call)."""
    S, w = C.c_int(0), C.c_int(0)
    _check("mg_op_fast_gemm_config", load().mg_op_fast_gemm_config(n, N, K, n_cu, C.byref(S), C.byref(w)))
    return S.value, w.value


def canon_gemv_config(n, N, K, swiglu=False, n_cu=256):
    """(kernel, rows per tile, 4-row quads, waves per feature group, ring depth) of the
    verifier's canonical GEMV for n rows of an N x K projection (kernel 2: the vector-fma
    kernel, the rest 0; 3: the matrix-core kernel) on a device of n_cu compute units (host
    logic, no device call)."""
    out = [C.c_int(0) for _ in range(5)]
    _check("mg_op_canon_gemv_config",
           load().mg_op_canon_gemv_config(n, N, K, int(bool(swiglu)), n_cu, *[C.byref(o) for o in out]))
    return tuple(o.value for o in out)


def op_rmsnorm(x, gamma, eps):
    n, d = x.shape
    y = torch.empty_like(x)
    _check("mg_op_rmsnorm", load().mg_op_rmsnorm(n, d, x.data_ptr(), gamma.data_ptr(), float(eps), y.data_ptr(),
                                                 _stream()))
    return y
