"""The C-ABI library loads, exports every symbol include/*.h declares, and rejects bad
host arguments without touching a GPU (no compute calls here)."""
import ctypes as C
import os
import re

import pytest

from paper_2605_30218_amd import mg, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = set()
    for f in os.listdir(os.path.join(ROOT, "include")):
        if f.endswith(".h"):
            src = open(os.path.join(ROOT, "include", f)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names |= set(re.findall(r"\b(mg_[a-z0-9_]+)\s*\(", src))
    return sorted(names)


def test_every_declared_symbol_is_exported():
    lib = mg.load()
    names = declared_functions()
    assert len(names) >= 20
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_covers_every_declared_symbol():
    assert sorted(mg.SIGNATURES) == declared_functions()


def test_sizes_and_status_strings():
    lib = mg.load()
    cfg = mg.make_cfg(synth.TINY, 4, 4, 16)
    assert lib.mg_weight_count(C.byref(cfg)) == 3 + 12 * synth.TINY.n_layers
    s = synth.TINY
    assert lib.mg_kv_pool_bytes(C.byref(cfg)) == s.n_layers * 16 * 2 * s.n_kv_heads * 16 * s.head_dim * 2
    assert lib.mg_kv_col_elems(C.byref(cfg)) == s.kv_col_elems
    assert lib.mg_workspace_bytes(C.byref(cfg)) > 0
    assert lib.mg_status_string(-3) == b"workspace or KV pool too small"
    assert lib.mg_status_string(0) == b"ok"


@pytest.mark.parametrize("field,value", [("page_size", 8), ("head_dim", 96), ("max_batch", 0), ("max_batch", 300),
                                         ("n_kv_heads", 3), ("d_model", 200)])
def test_unsupported_shapes_have_no_workspace(field, value):
    lib = mg.load()
    cfg = mg.make_cfg(synth.TINY, 4, 4, 16)
    setattr(cfg, field, value)
    assert lib.mg_workspace_bytes(C.byref(cfg)) == 0


def test_null_arguments_are_rejected_before_any_work():
    lib = mg.load()
    cfg = mg.make_cfg(synth.TINY, 4, 4, 16)
    out = C.c_void_p()
    assert lib.mg_create(None, None, None, 0, None, 0, C.byref(out)) == -1
    assert lib.mg_create(C.byref(cfg), None, None, 0, None, 0, C.byref(out)) == -1
    assert lib.mg_decode_step(None, 1, None, None, None, None, None) == -1
    assert lib.mg_margin_gate(None, 1, None, None, 0.5, None, None, None, None, None, None, None) == -1
    assert lib.mg_verify_rows(None, 1, None, None, None, None, None, None, None, None, None) == -1
    assert lib.mg_repair_kv_column(None, 1, None, None, None, None, None, None, None, None, None, None) == -1
    assert lib.mg_prefill(None, 1, None, None, None, None, None) == -1
    assert lib.mg_advance(None, 1, None, None, None, None) == -1
    assert lib.mg_profile_begin(None, 0, 1) == -1
    assert lib.mg_destroy(None) == -1
    assert lib.mg_op_linear(1, 0, 16, 8, None, None, None, None, None, 0, None) == -1
    assert lib.mg_op_linear(1, 4, 15, 8, 1, 1, None, 1, None, 0, None) == -1   # N % 16
    assert lib.mg_op_linear(1, 4, 16, 12, 1, 1, None, 1, None, 0, None) == -1  # K % 8
    assert lib.mg_op_linear(4, 4, 16, 8, 1, 1, None, 1, None, 0, None) == -1   # no such kernel
    assert lib.mg_op_linear(-1, 4, 16, 8, 1, 1, None, 1, None, 0, None) == -1
    assert lib.mg_op_probe_exp(-1, None, None, None) == -1
    assert lib.mg_op_probe_mfma_fma(-1, None, None, None, None, None) == -1
    assert lib.mg_op_probe_mfma_fma(2, None, None, None, None, None) == -1
    assert lib.mg_op_probe_mfma4_fma(-1, None, None, None, None, None) == -1
    assert lib.mg_op_probe_mfma4_fma(2, None, None, None, None, None) == -1


def test_create_rejects_small_buffers_and_missing_weights():
    lib = mg.load()
    cfg = mg.make_cfg(synth.TINY, 4, 4, 16)
    nw = lib.mg_weight_count(C.byref(cfg))
    fake = (C.c_void_p * nw)(*([1] * nw))
    out = C.c_void_p()
    kvb = lib.mg_kv_pool_bytes(C.byref(cfg))
    wsb = lib.mg_workspace_bytes(C.byref(cfg))
    assert lib.mg_create(C.byref(cfg), fake, 1, kvb - 2, 1, wsb, C.byref(out)) == -3
    assert lib.mg_create(C.byref(cfg), fake, 1, kvb, 1, wsb - 1, C.byref(out)) == -3
    fake[2] = None  # layer 0 wq (entry 1 + 12*0 + 1)
    assert lib.mg_create(C.byref(cfg), fake, 1, kvb, 1, wsb, C.byref(out)) == -1


def test_load_raises_when_library_missing(monkeypatch, tmp_path):
    monkeypatch.setattr(mg, "_lib", None)
    monkeypatch.setattr(mg, "LIB_PATH", str(tmp_path / "libmg.so"))
    with pytest.raises(RuntimeError, match="no fallback"):
        mg.load()


def test_fast_gemm_launch_rule():
    """The fast GEMM's (split-K factor, waves per block) choice, host logic only: on the
    Llama-3.1-8B projections at 64 rows it takes the launches measured fastest per shape
    (every block resident at once with the least weight per CU, 4-wave blocks for the
    several-round LM head); splits stay within the partial-tile cap; the register operand
    path (K % 128 != 0, or more than 128 rows) keeps 8-wave blocks."""
    llama = {(6144, 4096): (4, 8), (4096, 4096): (4, 4), (28672, 4096): (1, 8), (4096, 14336): (8, 8),
             (128256, 4096): (1, 4)}
    for (N, K), want in llama.items():
        assert mg.fast_gemm_config(64, N, K) == want, (N, K)
    for n in (1, 9, 16, 20, 33, 64, 100, 128, 129, 256):
        for (N, K) in [(48, 688), (64, 1032), (256, 4096), (4096, 4096), (6144, 4096), (28672, 4096), (4096, 14336),
                       (128256, 4096), (3584, 18944), (152064, 5120)]:
            S, w = mg.fast_gemm_config(n, N, K)
            assert w in (4, 8) and 1 <= S <= 32
            assert S == 1 or S * max(n, 16) * 16 <= K  # partial tiles at most an eighth of the weight bytes
            if K % 128 or n > 128:
                assert w == 8
    # the exact-integer GPU cases cover both block sizes at 2, 4 and 8 row tiles
    assert [mg.fast_gemm_config(n, 16512, 512)[1] for n in (20, 64, 128)] == [8, 8, 8]
    assert [mg.fast_gemm_config(*c)[1] for c in [(9, 64, 512), (20, 128, 1024), (64, 256, 4096), (128, 96, 2048)]] \
        == [4, 4, 4, 4]
    with pytest.raises(Exception):
        mg.fast_gemm_config(0, 64, 512)


def test_canon_gemv_launch_rule():
    """The verifier's canonical GEMV launch, host logic only: the vector-fma kernel up to 8
    rows, the matrix-core kernel above; one 16-row tile up to 16 rows and from 25 to 48, a
    16-row tile plus one 4-row quad at 17..20 rows and two at 21..24, two 16-row tiles per
    block above 48; the 4-stage ring where the launch has at most one block per CU (else 2);
    16 waves with the stage parity on the waves only for such a launch over K >= 8192 with
    16-row tiles.  Llama-3.1-8B projections at 12 rows take the launches measured fastest."""
    assert [mg.canon_gemv_config(n, 4096, 4096)[0] for n in range(1, 10)] == [2] * 8 + [3]
    assert mg.canon_gemv_config(8, 4096, 4096) == (2, 0, 0, 0, 0)
    tiles = {9: (16, 0), 16: (16, 0), 17: (32, 1), 20: (32, 1), 21: (32, 2), 24: (32, 2), 25: (16, 0),
             48: (16, 0), 49: (32, 0), 64: (32, 0), 256: (32, 0)}
    for n, (tr, q) in tiles.items():
        assert mg.canon_gemv_config(n, 28672, 4096)[1:3] == (tr, q), n
    llama12 = {(6144, 4096, False): (3, 16, 0, 8, 2), (4096, 4096, False): (3, 16, 0, 8, 4),
               (14336, 4096, True): (3, 16, 0, 8, 2), (4096, 14336, False): (3, 16, 0, 16, 4),
               (128256, 4096, False): (3, 16, 0, 8, 2)}
    for (N, K, sw), want in llama12.items():
        assert mg.canon_gemv_config(12, N, K, sw) == want, (N, K, sw)
    # the deep ring needs every block resident at once: 256 feature groups on 256 CUs, not 257
    assert mg.canon_gemv_config(12, 4096, 4096, n_cu=256)[4] == 4
    assert mg.canon_gemv_config(12, 4112, 4096, n_cu=256)[4] == 2
    assert mg.canon_gemv_config(12, 4096, 4096, n_cu=128)[4] == 2
    # two 16-row tiles at 30 rows double the blocks; 32-row tiles keep 8 waves over a long K
    assert mg.canon_gemv_config(30, 2048, 14336) == (3, 16, 0, 16, 4)
    assert mg.canon_gemv_config(30, 4096, 14336) == (3, 16, 0, 8, 2)
    assert mg.canon_gemv_config(20, 4096, 14336) == (3, 32, 1, 8, 4)
    assert mg.canon_gemv_config(12, 4096, 8184)[3] == 8 and mg.canon_gemv_config(12, 4096, 8192)[3] == 16
    with pytest.raises(Exception):
        mg.canon_gemv_config(0, 4096, 4096)
    with pytest.raises(Exception):
        mg.canon_gemv_config(12, 4096, 4100)
