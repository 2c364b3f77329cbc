"""Helpers shared by the GPU tests: contexts for synthetic workloads and the
matching oracle models (same seeded weights; bf16-rounded for bf16 contexts)."""
from __future__ import annotations

import numpy as np

import oracle
import synth


def desc_of(shape: synth.ModelShape, dtype: str):
    import paper_2608_18183_amd as P
    return P.ModelDesc(shape.n_layers, shape.d_model, shape.n_heads, shape.mlp_hidden,
                       shape.vocab, shape.n_classes, shape.grid,
                       P.DTYPE_BF16 if dtype == "bf16" else P.DTYPE_F32,
                       bool(shape.has_lm_bias), shape.rms_eps, shape.rope_base)


def make_ctx(shape, dtype, blob, max_kv_bytes=0):
    import paper_2608_18183_amd as P
    ctx = P.Context(desc_of(shape, dtype), max_kv_bytes=max_kv_bytes)
    ctx.hbsjd_load_weights(blob)
    return ctx


def bf16_rounded_blob(shape, blob):
    """The blob as a bf16 context holds it (see synth.bf16_rounded_blob)."""
    return synth.bf16_rounded_blob(shape, blob)


def device_batch(batch):
    import torch
    return torch.from_numpy(np.ascontiguousarray(batch.prefix_tokens, dtype=np.int32)).cuda()
