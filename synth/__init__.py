"""Seeded synthetic workloads for the batched speculative-Jacobi rollout.

This module only draws numbers: model shapes, random-init weights and
class-conditional token prefixes shaped like the paper's LlamaGen / ImageNet
setting (Sec. 5.1 "Rollout settings": W=16, H=24, CFG 2.0). It holds none of
the method's arithmetic, and both the oracle and the HIP path consume what it
returns. Trained weights and ImageNet prefixes are not available, so these
inputs stand in for them.

Weight blob order (fp32, one flat array), shared as an interface:
  tok_emb [V x d], cls_emb [(C+1) x d]   (row C is the null class used by CFG)
  per layer: g_attn [d], Wqkv [3d x d], Wo [d x d], g_ffn [d],
             W1 [f x d], W3 [f x d], W2 [d x f]
  g_out [d], W_lm [V x d], then b_lm [V] when the model has an lm_head bias.
Every matrix is stored out x in, row-major (y = x @ W.T).
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np


@dataclasses.dataclass(frozen=True)
class ModelShape:
    n_layers: int
    d_model: int
    n_heads: int
    mlp_hidden: int
    vocab: int
    n_classes: int
    grid: int
    has_lm_bias: bool = False
    rms_eps: float = 1e-5
    rope_base: float = 10000.0

    @property
    def T(self) -> int:
        return self.grid * self.grid

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_heads


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    model: ModelShape
    dtype: str                  # "f32" or "bf16": the arithmetic type of the GPU path
    batch: int
    window: int
    history: int
    top_k: int
    cfg_scale: float            # 0 = no classifier-free guidance
    weight_std: float = 0.02
    bias_std: float = 0.0       # std of b_lm when the model has one
    prefix: str = "uniform"     # "uniform" or "bimodal"
    prefix_lo: int = 0
    prefix_hi: int = 0
    temperature: str = "1.0"    # "1.0" or "alt0.3/1.5" (even image 0.3, odd 1.5)


def _shape_tiny() -> ModelShape:
    return ModelShape(2, 64, 4, 176, 256, 10, 8)


def _shape_b(grid: int = 16, bias: bool = False) -> ModelShape:
    return ModelShape(12, 768, 12, 2048, 16384, 1000, grid, has_lm_bias=bias)


def teacher_shape(student: ModelShape) -> ModelShape:
    """The teacher of the scoring step: the LlamaGen-L architecture (24 layers,
    d 1024, 16 heads, f 2816) on the student's grid, vocabulary and classes."""
    return ModelShape(24, 1024, 16, 2816, student.vocab, student.n_classes, student.grid)


WORKLOADS: Dict[str, Workload] = {
    # 2 layers, d 64, 8x8 grid, batch 4, prefix 0-16, W=4, fp32
    "tiny": Workload("tiny", _shape_tiny(), "f32", 4, 4, 24, 0, 0.0,
                     prefix_lo=0, prefix_hi=16),
    # LlamaGen-B shape, 16x16 grid, batch 32, prefix 0-128, W=16, top-k 2000
    "llamagen_b": Workload("llamagen_b", _shape_b(), "bf16", 32, 16, 24, 2000, 0.0,
                           prefix_lo=0, prefix_hi=128),
    # LlamaGen-L shape, 24x24 grid, batch 64, prefix 0-288, W=16
    "llamagen_l": Workload("llamagen_l", ModelShape(24, 1024, 16, 2816, 16384, 1000, 24),
                           "bf16", 64, 16, 24, 2000, 0.0, prefix_lo=0, prefix_hi=288),
    # LlamaGen-XL shape with CFG: 128 images -> 256 rows, W=32, top-k 1000
    "llamagen_xl_cfg": Workload("llamagen_xl_cfg",
                                ModelShape(36, 1280, 20, 3456, 16384, 1000, 16),
                                "bf16", 128, 32, 24, 1000, 2.0, prefix_lo=0, prefix_hi=128),
    # ragged / compaction stress on the B shape: 24x24, batch 256, W=24,
    # bimodal prefixes, lm_head bias N(0, 4^2), temperatures 0.3 / 1.5
    "stress_b": Workload("stress_b", _shape_b(grid=24, bias=True), "bf16", 256, 24, 24,
                         2000, 0.0, bias_std=4.0, prefix="bimodal",
                         temperature="alt0.3/1.5"),
}


def blob_layout(m: ModelShape) -> List[tuple]:
    """(name, shape, kind) in blob order; kind is 'w' (matrix/embedding),
    'g' (RMSNorm gain, set to 1.0) or 'b' (lm_head bias)."""
    d, f, V, C = m.d_model, m.mlp_hidden, m.vocab, m.n_classes
    out = [("tok_emb", (V, d), "w"), ("cls_emb", (C + 1, d), "w")]
    for layer in range(m.n_layers):
        out += [
            (f"l{layer}.g_attn", (d,), "g"),
            (f"l{layer}.wqkv", (3 * d, d), "w"),
            (f"l{layer}.wo", (d, d), "w"),
            (f"l{layer}.g_ffn", (d,), "g"),
            (f"l{layer}.w1", (f, d), "w"),
            (f"l{layer}.w3", (f, d), "w"),
            (f"l{layer}.w2", (d, f), "w"),
        ]
    out += [("g_out", (d,), "g"), ("w_lm", (V, d), "w")]
    if m.has_lm_bias:
        out.append(("b_lm", (V,), "b"))
    return out


def blob_size(m: ModelShape) -> int:
    return int(sum(int(np.prod(s)) for _, s, _ in blob_layout(m)))


def make_weights(m: ModelShape, seed: int = 0, std: float = 0.02,
                 bias_std: float = 4.0) -> np.ndarray:
    """One fp32 blob: N(0, std) matrices and embeddings, gains 1.0,
    lm_head bias N(0, bias_std^2), all drawn from numpy PCG64(seed) in blob order."""
    rng = np.random.Generator(np.random.PCG64(seed))
    n = blob_size(m)
    blob = rng.standard_normal(n, dtype=np.float32)
    off = 0
    for _, shape, kind in blob_layout(m):
        k = int(np.prod(shape))
        seg = blob[off:off + k]
        if kind == "w":
            seg *= np.float32(std)
        elif kind == "g":
            seg[:] = 1.0
        else:
            seg *= np.float32(bias_std)
        off += k
    return blob


def bf16_rounded_blob(m: ModelShape, blob: np.ndarray) -> np.ndarray:
    """The weights a bf16 workload uses: every matrix and embedding of the blob
    rounded to the nearest bf16 (ties to even) and returned as fp32; RMSNorm
    gains and the lm_head bias stay fp32. Both the GPU (which rounds the blob
    it is given the same way) and the fp32 oracle of a bf16 comparison see
    these values."""
    out = np.array(blob, dtype=np.float32, copy=True)
    chunk = 1 << 20                  # in place, a cache-sized piece at a time
    t = np.empty(chunk, dtype=np.uint32)
    off = 0
    for _, shape, kind in blob_layout(m):
        k = int(np.prod(shape))
        if kind == "w":
            u = out[off:off + k].view(np.uint32)
            for s in range(0, k, chunk):
                v = u[s:s + chunk]
                r = t[:v.size]
                np.right_shift(v, np.uint32(16), out=r)
                np.bitwise_and(r, np.uint32(1), out=r)
                np.add(r, np.uint32(0x7FFF), out=r)
                np.add(v, r, out=v)
                np.bitwise_and(v, np.uint32(0xFFFF0000), out=v)
        off += k
    return out


def split_blob(m: ModelShape, blob: np.ndarray) -> Dict[str, np.ndarray]:
    """Named views into a blob (no copies)."""
    out, off = {}, 0
    for name, shape, _ in blob_layout(m):
        k = int(np.prod(shape))
        out[name] = blob[off:off + k].reshape(shape)
        off += k
    assert off == blob.size
    return out


@dataclasses.dataclass
class Batch:
    prefix_tokens: np.ndarray   # int32 [B, T]; the first prefix_len[b] entries are the real prefix
    prefix_len: np.ndarray      # int32 [B]
    labels: np.ndarray          # int32 [B]
    temperature: np.ndarray     # float32 [B]


def make_batch(w: Workload, seed: int = 1, batch: Optional[int] = None) -> Batch:
    """Prefix lengths uniform over the workload's range (or bimodal), prefix tokens
    uniform over the vocabulary, labels uniform over the classes: PCG64(seed)."""
    m = w.model
    B = w.batch if batch is None else batch
    rng = np.random.Generator(np.random.PCG64(seed))
    T = m.T
    if w.prefix == "bimodal":
        half = B // 2
        lo = rng.integers(0, 32, size=half, endpoint=True)
        hi = rng.integers(448, 560, size=B - half, endpoint=True)
        plen = np.concatenate([lo, hi])
    else:
        plen = rng.integers(w.prefix_lo, w.prefix_hi, size=B, endpoint=True)
    plen = np.minimum(plen, T).astype(np.int32)
    toks = rng.integers(0, m.vocab, size=(B, T)).astype(np.int32)
    labels = rng.integers(0, m.n_classes, size=B).astype(np.int32)
    if w.temperature == "alt0.3/1.5":
        temp = np.where(np.arange(B) % 2 == 0, 0.3, 1.5).astype(np.float32)
    else:
        temp = np.full(B, float(w.temperature), dtype=np.float32)
    return Batch(toks, plen, labels, temp)


def small_shape(**kw) -> ModelShape:
    """A custom (usually tiny) shape for tests."""
    base = dict(n_layers=2, d_model=16, n_heads=2, mlp_hidden=32, vocab=4,
                n_classes=3, grid=2)
    base.update(kw)
    return ModelShape(**base)
