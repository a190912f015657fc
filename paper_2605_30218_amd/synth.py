"""Seeded synthetic inputs: model shapes, random-init bf16 weights, prompts, page tables.

This module holds none of the method's arithmetic.  It is the one piece of code that
both the GPU path (through its tests and benchmark) and the CPU oracle consume, so the
two sides read the same bytes.  The real models and datasets of arXiv 2605.30218
(Sec. 4.1: Llama-3.x, Qwen2.5, MATH500, GSM8K, ...) are not available; these inputs
stand in for them with the same shapes: weights N(0, 0.02) rounded to bf16, RMSNorm
gains 1, untied embedding and LM head, uniform random prompt token ids.
"""
from __future__ import annotations

import dataclasses

import numpy as np
import torch

WPL = 12  # weight tensors per layer, in the order listed by weight_specs()


@dataclasses.dataclass(frozen=True)
class ModelShape:
    name: str
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    d_ffn: int
    vocab: int
    qkv_bias: bool
    rope_theta: float
    rms_eps: float
    page_size: int = 16

    @property
    def kv_col_elems(self) -> int:
        """bf16 elements of one request's K/V column over all layers: [L][2][Hkv][hd]."""
        return self.n_layers * 2 * self.n_kv_heads * self.head_dim

    def n_params(self) -> int:
        return sum(int(np.prod(s)) for _, s in weight_specs(self) if s is not None)


TINY = ModelShape("tiny", 2, 256, 4, 2, 64, 688, 4096, False, 1e4, 1e-5)
LLAMA8B = ModelShape("llama3.1-8b", 32, 4096, 32, 8, 128, 14336, 128256, False, 5e5, 1e-5)
QWEN7B = ModelShape("qwen2.5-7b", 28, 3584, 28, 4, 128, 18944, 152064, True, 1e6, 1e-6)
QWEN14B = ModelShape("qwen2.5-14b", 48, 5120, 40, 8, 128, 13824, 152064, True, 1e6, 1e-6)
SHAPES = {s.name: s for s in (TINY, LLAMA8B, QWEN7B, QWEN14B)}


def weight_specs(s: ModelShape):
    """(name, shape or None) in the fixed pointer-table order shared by both libraries."""
    d, q, kv, F, V = s.d_model, s.n_q_heads * s.head_dim, s.n_kv_heads * s.head_dim, s.d_ffn, s.vocab
    specs = [("embed", (V, d))]
    for l in range(s.n_layers):
        specs += [
            (f"l{l}.attn_norm", (d,)), (f"l{l}.wq", (q, d)), (f"l{l}.wk", (kv, d)), (f"l{l}.wv", (kv, d)),
            (f"l{l}.bq", (q,) if s.qkv_bias else None), (f"l{l}.bk", (kv,) if s.qkv_bias else None),
            (f"l{l}.bv", (kv,) if s.qkv_bias else None),
            (f"l{l}.wo", (d, q)), (f"l{l}.ffn_norm", (d,)), (f"l{l}.w_gate", (F, d)), (f"l{l}.w_up", (F, d)),
            (f"l{l}.w_down", (d, F)),
        ]
    specs += [("final_norm", (d,)), ("lm_head", (V, d))]
    return specs


def make_weights(s: ModelShape, seed: int = 0, device="cpu", std: float = 0.02):
    """Random-init weights as int16 torch tensors holding bf16 bit patterns (None for absent biases).

    Tensors are drawn in weight_specs() order from one torch.Generator on `device`:
    fp32 N(0, std) rounded to bf16 by torch (round to nearest even).  Norm gains are 1.0.
    CPU and GPU generators give different streams, so a model is identified by
    (shape, seed, device)."""
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    out = []
    for name, shp in weight_specs(s):
        if shp is None:
            out.append(None)
        elif name.endswith("norm"):
            out.append(torch.ones(shp, dtype=torch.bfloat16, device=device).view(torch.int16))
        else:
            w = torch.randn(shp, generator=g, device=device, dtype=torch.float32)
            w.mul_(std)
            out.append(w.to(torch.bfloat16).view(torch.int16))
            del w
    return out


def weights_to_numpy(ws):
    return [None if w is None else w.cpu().numpy().view(np.uint16) for w in ws]


def make_prompts(n_rows: int, lengths, vocab: int, seed: int = 1):
    """Uniform random token ids, one int32 array per row (length lengths[i])."""
    g = torch.Generator()
    g.manual_seed(seed)
    return [torch.randint(0, vocab, (int(L),), generator=g, dtype=torch.int64).numpy().astype(np.int32)
            for L in lengths]


def make_lengths(n_rows: int, lo: int, hi: int, seed: int = 2):
    """Prompt lengths drawn uniformly from [lo, hi]."""
    g = torch.Generator()
    g.manual_seed(seed)
    return torch.randint(lo, hi + 1, (n_rows,), generator=g).numpy().astype(np.int32)


def make_page_table(max_ctx, page_size: int, max_pages_per_row: int, seed: int = 5, extra_pages: int = 0):
    """Give row i ceil(max_ctx[i] / page_size) distinct pages from a seeded permutation of the pool,
    so rows interleave in memory and the page indirection is exercised.  Unused entries are -1.
    Returns (page_table int32 [rows][max_pages_per_row], n_pages)."""
    need = [-(-int(c) // page_size) for c in max_ctx]
    assert max(need) <= max_pages_per_row
    n_pages = sum(need) + extra_pages
    g = torch.Generator()
    g.manual_seed(seed)
    perm = torch.randperm(n_pages, generator=g).numpy().astype(np.int32)
    pt = np.full((len(need), max_pages_per_row), -1, np.int32)
    o = 0
    for i, k in enumerate(need):
        pt[i, :k] = perm[o:o + k]
        o += k
    return pt, n_pages


def random_bf16(shape, seed: int, std: float = 1.0):
    """Seeded N(0, std) values rounded to bf16, as a uint16 numpy array (op-level test inputs)."""
    g = torch.Generator()
    g.manual_seed(seed)
    return (torch.randn(shape, generator=g) * std).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def small_int_bf16(shape, seed: int, lo: int = -3, hi: int = 3):
    """Seeded small integers stored as bf16 (every partial sum below 2^24 is exact in fp32)."""
    g = torch.Generator()
    g.manual_seed(seed)
    v = torch.randint(lo, hi + 1, shape, generator=g).to(torch.float32)
    return v.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def perturb_lm_head_tie_pairs(weights, shape: ModelShape, seed: int = 4, n_pairs: int = 8, boost: float = 8.0,
                              tau: float = 0.5):
    """The high-trigger regime of the Qwen2.5-7B-shaped workload: a seeded low-rank change of the
    LM head that makes about half of the steps have a top-1/top-2 margin below tau.

    P seeded pairs of distinct token ids (a_k, b_k) and directions u_k ~ N(0, 1/d) give
        W'_a = W_a + s u_k,    W'_b = c W_b + (1 - c) W_a + s u_k        (rank <= 2P).
    Both rows of a pair gain the same logit s u_k . h, so with s = 8 one pair usually holds the
    top two logits, and their gap becomes c (W_a - W_b) . h ~ N(0, 2 c^2 sigma^2), where
    sigma = 0.02 sqrt(d) is the logit scale of an RMS-normalised h (||h||^2 = d).  The margin
    is then |N(0, sqrt(2) c sigma)|, below tau with probability erf(tau / (2 c sigma));
    c = tau / (0.954 sigma) makes that 1/2.  Returns a new weight list with the LM head
    replaced (rows rounded to bf16); the other tensors are shared."""
    d, V = shape.d_model, shape.vocab
    sigma = 0.02 * float(np.sqrt(d))
    c = tau / (0.954 * sigma)
    g = torch.Generator()
    g.manual_seed(seed)
    ids = torch.randperm(V, generator=g)[: 2 * n_pairs]
    a_ids, b_ids = ids[:n_pairs], ids[n_pairs:]
    u = torch.randn((n_pairs, d), generator=g, dtype=torch.float32) / float(np.sqrt(d))
    lm = weights[-1]
    dev = lm.device
    W = lm.clone()
    wa = W[a_ids.to(dev)].view(torch.bfloat16).float()
    wb = W[b_ids.to(dev)].view(torch.bfloat16).float()
    su = (boost * u).to(dev)
    na = wa + su
    nb = c * wb + (1.0 - c) * wa + su
    W[a_ids.to(dev)] = na.to(torch.bfloat16).view(torch.int16)
    W[b_ids.to(dev)] = nb.to(torch.bfloat16).view(torch.int16)
    return list(weights[:-1]) + [W]


def fill_synthetic_kv(kv_view, pages, seed: int, std: float = 1.0):
    """Seeded N(0, std) bf16 values in every layer, K and V, of the given pages of a paged KV
    pool view [L][n_pages][2][Hkv][page][hd] (int16 tensor holding bf16 bits).  Stands in for
    the cache of a long prompt where a prefill would take minutes; the parity tests copy the
    cache to the oracle, so its contents need not come from a forward pass."""
    dev = kv_view.device
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    idx = torch.as_tensor(np.asarray(pages, np.int64), device=dev)
    shp = (idx.numel(),) + tuple(kv_view.shape[2:])
    for layer in range(kv_view.shape[0]):
        vals = torch.randn(shp, generator=g, device=dev, dtype=torch.float32)
        vals.mul_(std)
        kv_view[layer, idx] = vals.to(torch.bfloat16).view(torch.int16)
        del vals
