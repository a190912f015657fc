"""ctypes binding of the CPU oracle (liboracle_mg.so) plus the oracle's own gated decode loop.

TEST INFRASTRUCTURE ONLY.  Imported by tests/, by the smoke check and by the CPU
baseline leg of bench.py; never by the product package.  It imports nothing from the
GPU package: shapes arrive as any object with the model-shape attributes, weights
and state as numpy arrays.

The gated loop below follows the MarginGate decode step of arXiv 2605.30218:
Sec. 3.1 (margin trigger g < tau), Sec. 3.2 (fast commit / verified commit /
single-column repair) and Sec. 3.3 (r_verify, r_repair accounting).
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle_mg.so")

PLAIN = 0
CANON = 1
# repair actions of the commit (Sec. 3.2; the token-only ablation of Sec. 4)
REPAIR_ON_MISMATCH = 0
REPAIR_TOKEN_ONLY = 1
REPAIR_COPY_ALWAYS = 2
WPL = 12  # weight pointers per layer


class MgoCfg(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("n_layers", "d_model", "n_q_heads", "n_kv_heads", "head_dim",
                                         "d_ffn", "vocab", "qkv_bias")] + \
               [("rope_theta", C.c_float), ("rms_eps", C.c_float)] + \
               [(n, C.c_int32) for n in ("page_size", "max_batch", "max_pages_per_row", "n_pages")]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            import importlib.util
            spec = importlib.util.spec_from_file_location("build_oracle", os.path.join(HERE, "build_oracle.py"))
            mod = importlib.util.module_from_spec(spec)
            spec.loader.exec_module(mod)
            mod.build()
        _lib = C.CDLL(LIB_PATH)
        P = C.c_void_p
        i32, f32 = C.c_int, C.c_float
        _lib.mgo_bf16_from_f32.restype = C.c_uint16
        _lib.mgo_bf16_from_f32.argtypes = [f32]
        _lib.mgo_f32_from_bf16.restype = f32
        _lib.mgo_f32_from_bf16.argtypes = [C.c_uint16]
        _lib.mgo_exp.restype = f32
        _lib.mgo_exp.argtypes = [f32]
        _lib.mgo_bf16_round_many.argtypes = [C.c_int64, P, P]
        _lib.mgo_exp_many.argtypes = [C.c_int64, P, P]
        _lib.mgo_cdot.restype = f32
        _lib.mgo_cdot.argtypes = [i32, P, P]
        _lib.mgo_rmsnorm.argtypes = [i32, i32, P, P, f32, P]
        _lib.mgo_linear.argtypes = [i32, i32, i32, P, P, P, P, P]
        _lib.mgo_rope.argtypes = [i32, i32, C.c_double, i32, P]
        _lib.mgo_swiglu.argtypes = [i32, i32, P, P, P]
        _lib.mgo_attend.argtypes = [i32, i32, i32, P, P, P, P]
        _lib.mgo_top2.argtypes = [i32, P, P, P]
        for name, args in (
            ("mgo_decode_step", [P, P, i32, i32, P, P, P, P, P]),
            ("mgo_margin_gate", [i32, i32, P, P, f32, P, P, P, P, P]),
            ("mgo_verify_rows", [P, P, i32, i32, P, P, P, P, P, P, P, P]),
            ("mgo_repair_kv_column", [P, i32, P, P, P, P, P, P, P, P, P]),
            ("mgo_repair_kv_column_action", [P, i32, P, P, P, P, P, P, P, P, P, i32]),
            ("mgo_prefill", [P, P, i32, i32, P, P, P]),
            ("mgo_embed", [P, P, i32, P, P]),
            ("mgo_layer", [P, P, i32, i32, i32, P, P, P, P]),
            ("mgo_head", [P, P, i32, i32, P, P]),
        ):
            f = getattr(_lib, name)
            f.restype = C.c_int
            f.argtypes = args
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _chk(rc, what):
    if rc != 0:
        raise RuntimeError(f"oracle {what} failed with status {rc}")


# ------------------------------------------------------------------ scalar / op level

def bf16_from_f32(x) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, np.uint16)
    lib().mgo_bf16_round_many(x.size, _p(x), _p(out))
    return out


def f32_from_bf16(h) -> np.ndarray:
    h = np.ascontiguousarray(h, dtype=np.uint16)
    return (h.astype(np.uint32) << 16).view(np.float32)


def exp(x) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty_like(x)
    lib().mgo_exp_many(x.size, _p(x), _p(out))
    return out


def cdot(x, w) -> float:
    x = np.ascontiguousarray(x, np.float32)
    w = np.ascontiguousarray(w, np.float32)
    return float(lib().mgo_cdot(x.size, _p(x), _p(w)))


def rmsnorm(mode, x, gamma, eps) -> np.ndarray:
    x = np.ascontiguousarray(x, np.uint16)
    y = np.empty_like(x)
    lib().mgo_rmsnorm(mode, x.size, _p(x), _p(np.ascontiguousarray(gamma, np.uint16)), eps, _p(y))
    return y


def linear(mode, x, W, bias=None, fp32=False):
    x = np.ascontiguousarray(x, np.uint16)
    W = np.ascontiguousarray(W, np.uint16)
    N, K = W.shape
    assert x.size == K
    b = None if bias is None else np.ascontiguousarray(bias, np.uint16)
    if fp32:
        y = np.empty(N, np.float32)
        lib().mgo_linear(mode, N, K, _p(x), _p(W), _p(b), None, _p(y))
    else:
        y = np.empty(N, np.uint16)
        lib().mgo_linear(mode, N, K, _p(x), _p(W), _p(b), _p(y), None)
    return y


def rope(hd, pos, theta, v) -> np.ndarray:
    v = np.array(v, dtype=np.uint16, copy=True, order="C")
    lib().mgo_rope(hd, pos, theta, v.size // hd, _p(v))
    return v


def swiglu(mode, g, u) -> np.ndarray:
    g = np.ascontiguousarray(g, np.uint16)
    u = np.ascontiguousarray(u, np.uint16)
    a = np.empty_like(g)
    lib().mgo_swiglu(mode, g.size, _p(g), _p(u), _p(a))
    return a


def attend(mode, q, K, V) -> np.ndarray:
    q = np.ascontiguousarray(q, np.uint16)
    K = np.ascontiguousarray(K, np.uint16)
    V = np.ascontiguousarray(V, np.uint16)
    n, hd = K.shape
    out = np.empty(hd, np.uint16)
    lib().mgo_attend(mode, hd, n, _p(q), _p(K), _p(V), _p(out))
    return out


def top2(logits):
    logits = np.ascontiguousarray(logits, np.float32)
    t = np.zeros(1, np.int32)
    m = np.zeros(1, np.float32)
    lib().mgo_top2(logits.size, _p(logits), _p(t), _p(m))
    return int(t[0]), float(m[0])


# ------------------------------------------------------------------ model level

def make_cfg(shape, max_batch, max_pages_per_row, n_pages) -> MgoCfg:
    return MgoCfg(shape.n_layers, shape.d_model, shape.n_q_heads, shape.n_kv_heads, shape.head_dim,
                  shape.d_ffn, shape.vocab, int(shape.qkv_bias), float(shape.rope_theta), float(shape.rms_eps),
                  shape.page_size, max_batch, max_pages_per_row, n_pages)


class OracleModel:
    """Host-memory decoder state: weights (uint16 bf16 arrays, fixed order), KV pool, page table."""

    def __init__(self, shape, weights, max_batch, max_pages_per_row, n_pages):
        self.shape = shape
        self.cfg = make_cfg(shape, max_batch, max_pages_per_row, n_pages)
        self.weights = [None if w is None else np.ascontiguousarray(w, np.uint16) for w in weights]
        assert len(self.weights) == 3 + WPL * shape.n_layers
        self._wptr = (C.c_void_p * len(self.weights))(*[None if w is None else w.ctypes.data
                                                        for w in self.weights])
        self.kv_pool = np.zeros(self.kv_elems(), np.uint16)

    def kv_elems(self):
        s, c = self.shape, self.cfg
        return s.n_layers * c.n_pages * 2 * s.n_kv_heads * s.page_size * s.head_dim

    def col_elems(self):
        s = self.shape
        return s.n_layers * 2 * s.n_kv_heads * s.head_dim

    def kv_view(self):
        s, c = self.shape, self.cfg
        return self.kv_pool.reshape(s.n_layers, c.n_pages, 2, s.n_kv_heads, s.page_size, s.head_dim)

    def decode_step(self, mode, tokens, positions, page_table):
        tokens = np.ascontiguousarray(tokens, np.int32)
        positions = np.ascontiguousarray(positions, np.int32)
        page_table = np.ascontiguousarray(page_table, np.int32)
        B = tokens.size
        logits = np.empty((B, self.shape.vocab), np.float32)
        _chk(lib().mgo_decode_step(C.byref(self.cfg), self._wptr, mode, B, _p(tokens), _p(positions),
                                   _p(page_table), _p(self.kv_pool), _p(logits)), "decode_step")
        return logits

    # -------------------------------------------------------------- the step cut at layers

    def embed(self, tokens):
        """Residual stream entering layer 0: the embedding rows, bf16 [B][d]."""
        tokens = np.ascontiguousarray(tokens, np.int32)
        x = np.empty((tokens.size, self.shape.d_model), np.uint16)
        _chk(lib().mgo_embed(C.byref(self.cfg), self._wptr, tokens.size, _p(tokens), _p(x)), "embed")
        return x

    def layer(self, mode, layer, x, positions, page_table):
        """One decoder layer on the residual stream x [B][d] (returns the layer's output; the
        rows' K/V columns of that layer are appended to the cache)."""
        x = np.array(x, np.uint16, copy=True, order="C")
        positions = np.ascontiguousarray(positions, np.int32)
        page_table = np.ascontiguousarray(page_table, np.int32)
        _chk(lib().mgo_layer(C.byref(self.cfg), self._wptr, mode, layer, positions.size, _p(positions),
                             _p(page_table), _p(self.kv_pool), _p(x)), "layer")
        return x

    def head(self, mode, x):
        """Final RMSNorm and LM head: fp32 logits [B][V] from the residual stream x [B][d]."""
        x = np.ascontiguousarray(x, np.uint16)
        B = x.shape[0]
        logits = np.empty((B, self.shape.vocab), np.float32)
        _chk(lib().mgo_head(C.byref(self.cfg), self._wptr, mode, B, _p(x), _p(logits)), "head")
        return logits

    @staticmethod
    def margin_gate(logits, protected, tau):
        logits = np.ascontiguousarray(logits, np.float32)
        B, V = logits.shape
        prot = None if protected is None else np.ascontiguousarray(protected, np.uint8)
        top1 = np.empty(B, np.int32)
        margin = np.empty(B, np.float32)
        gate = np.empty(B, np.uint8)
        rows = np.empty(max(B, 1), np.int32)
        n = np.zeros(1, np.int32)
        _chk(lib().mgo_margin_gate(B, V, _p(logits), _p(prot), float(tau), _p(top1), _p(margin), _p(gate),
                                   _p(rows), _p(n)), "margin_gate")
        return top1, margin, gate, rows[: int(n[0])].copy()

    def verify_rows(self, rows, tokens, positions, page_table, mode=CANON, want_logits=True):
        rows = np.ascontiguousarray(rows, np.int32)
        tokens = np.ascontiguousarray(tokens, np.int32)
        positions = np.ascontiguousarray(positions, np.int32)
        page_table = np.ascontiguousarray(page_table, np.int32)
        n = rows.size
        v_logits = np.empty((n, self.shape.vocab), np.float32) if want_logits else None
        v_tok = np.empty(n, np.int32)
        v_kvcol = np.empty((n, self.col_elems()), np.uint16)
        _chk(lib().mgo_verify_rows(C.byref(self.cfg), self._wptr, mode, n, _p(rows), _p(tokens), _p(positions),
                                   _p(page_table), _p(self.kv_pool), _p(v_logits), _p(v_tok), _p(v_kvcol)),
             "verify_rows")
        return v_logits, v_tok, v_kvcol

    def repair(self, rows, positions, page_table, top1, v_tok, v_kvcol, emitted, action=REPAIR_ON_MISMATCH):
        """Commit (Sec. 3.2).  action: REPAIR_ON_MISMATCH (the method), REPAIR_TOKEN_ONLY (the
        repair-action ablation of Sec. 4), REPAIR_COPY_ALWAYS (copy on every verified row)."""
        rows = np.ascontiguousarray(rows, np.int32)
        emitted = np.array(emitted, np.int32, copy=True)
        nrep = np.zeros(1, np.int32)
        _chk(lib().mgo_repair_kv_column_action(C.byref(self.cfg), rows.size, _p(rows),
                                               _p(np.ascontiguousarray(positions, np.int32)),
                                               _p(np.ascontiguousarray(page_table, np.int32)),
                                               _p(np.ascontiguousarray(top1, np.int32)),
                                               _p(np.ascontiguousarray(v_tok, np.int32)),
                                               _p(np.ascontiguousarray(v_kvcol, np.uint16)), _p(self.kv_pool),
                                               _p(emitted), _p(nrep), int(action)), "repair")
        return emitted, int(nrep[0])

    def prefill(self, mode, tokens, page_table_row):
        tokens = np.ascontiguousarray(tokens, np.int32)
        ptr = np.ascontiguousarray(page_table_row, np.int32)
        _chk(lib().mgo_prefill(C.byref(self.cfg), self._wptr, mode, tokens.size, _p(tokens), _p(ptr),
                               _p(self.kv_pool)), "prefill")

    # -------------------------------------------------------------- the gated loop

    def gated_step(self, fast_mode, tokens, positions, page_table, protected, tau, verify="gated",
                   action=REPAIR_ON_MISMATCH):
        """One MarginGate step (Sec. 3.1-3.3).  verify in {"off", "gated", "always"}.
        Returns (emitted, record) where record holds logits, top1, margin, gate, rows, v_tok, n_repaired."""
        logits = self.decode_step(fast_mode, tokens, positions, page_table)
        top1, margin, gate, rows = self.margin_gate(logits, protected, tau)
        if verify == "off":
            rows = rows[:0]
        elif verify == "always":
            B = tokens.size
            prot = np.ones(B, np.uint8) if protected is None else np.asarray(protected, np.uint8)
            rows = np.nonzero(prot)[0].astype(np.int32)
        emitted = top1.copy()
        v_tok = np.empty(0, np.int32)
        nrep = 0
        if rows.size:
            _, v_tok, v_kvcol = self.verify_rows(rows, tokens, positions, page_table, want_logits=False)
            emitted, nrep = self.repair(rows, positions, page_table, top1, v_tok, v_kvcol, emitted, action)
        return emitted, dict(logits=logits, top1=top1, margin=margin, gate=gate, rows=rows, v_tok=v_tok,
                             n_repaired=nrep)
