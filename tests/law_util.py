"""Exact output law of token-by-token sampling (Sec. 3.1, Eq. 2) on a tiny
model, and a chi-square test of drawn suffixes against it. Shared by the GPU
law tests and the CPU test that shows the statistic's power on the oracle."""
from __future__ import annotations

import numpy as np
from scipy import stats

import oracle
import synth

# head_dim 64 and dimensions in multiples of 64, as a bf16 context needs.
# Small weights (std 0.1) keep the bf16 forward within a few 1e-3 of the
# oracle's logits. A large lm_head bias (std 3) fixes one top-3 set with a wide
# margin at every context, while the context still moves the law inside it.
LAW_SHAPE = dict(n_layers=2, d_model=64, n_heads=1, mlp_hidden=128, vocab=64, n_classes=3,
                 grid=2, has_lm_bias=True)
LAW_WEIGHT_SEED, LAW_WEIGHT_STD, LAW_BIAS_STD = 38, 0.1, 3.0

CASES = {
    # two free positions over the full vocabulary under guidance: 4096
    # suffixes, all in one window
    "full_vocab_cfg": dict(prefix=[7, 21], top_k=0, tau=1.5, cfg=2.0, W=2, H=1),
    # four free positions, top-3: 81 suffixes; windows of 3 end at position 3,
    # then one more
    "top3": dict(prefix=[], top_k=3, tau=1.0, cfg=0.0, W=3, H=2),
}


def law_model():
    shape = synth.small_shape(**LAW_SHAPE)
    blob = synth.make_weights(shape, LAW_WEIGHT_SEED, std=LAW_WEIGHT_STD,
                              bias_std=LAW_BIAS_STD)
    return shape, blob


def exact_law(om, shape, cls, prefix, top_k, tau, cfg):
    """Exact law of the suffix after `prefix` under token-by-token sampling:
    ({suffix: probability}, every (class, context) the walk evaluated, the
    smallest gap between the k-th and (k+1)-th guided logit at those contexts)."""
    law, contexts, gap = {}, [], [np.inf]

    def walk(seq, pr):
        t = len(seq)
        if t == shape.T:
            law[tuple(seq[len(prefix):])] = pr
            return
        contexts.append((cls, list(seq)))
        l = om.forward_seq(cls, seq)[t]
        if cfg:
            contexts.append((shape.n_classes, list(seq)))
            l = oracle.cfg_combine(l, om.forward_seq(shape.n_classes, seq)[t], cfg)
        if top_k:
            s = np.sort(l)[::-1]
            gap[0] = min(gap[0], float(s[top_k - 1] - s[top_k]))
        p = oracle.transform(l, tau, top_k).astype(np.float64)
        for x in np.flatnonzero(p):
            walk(seq + [int(x)], pr * p[x])

    walk(list(prefix), 1.0)
    return law, contexts, gap[0]


def chi2_against_law(tokens, k, law, V):
    """(p-value, cells with >= 5 expected draws) of the suffixes tokens[:, k:]
    against `law`; cells below 5 expected draws are pooled. Raises
    AssertionError on a suffix outside the law's support."""
    suffixes = list(law)
    code_of = {}
    for i, s in enumerate(suffixes):
        c = 0
        for x in s:
            c = c * V + x
        code_of[c] = i
    code = np.zeros(len(tokens), dtype=np.int64)
    for t in range(k, tokens.shape[1]):
        code = code * V + tokens[:, t]
    obs = np.zeros(len(suffixes))
    for c, n in zip(*np.unique(code, return_counts=True)):
        assert int(c) in code_of, f"drew a suffix outside the support (code {int(c)})"
        obs[code_of[int(c)]] = n
    exp = np.array([law[s] for s in suffixes]) * len(tokens)
    big = exp >= 5
    o = np.append(obs[big], obs[~big].sum())
    e = np.append(exp[big], exp[~big].sum())
    if e[-1] == 0:
        o, e = o[:-1], e[:-1]
    return stats.chisquare(o, e * o.sum() / e.sum()).pvalue, int(big.sum())


def waited(counts) -> bool:
    """Some image had a round with no commit before a round with one (it
    waited at a shared window boundary). counts: [rounds, B]."""
    c = np.asarray(counts)
    idle_before = np.cumsum(c == 0, axis=0) > 0
    return bool((idle_before[:-1] & (c[1:] > 0)).any())
