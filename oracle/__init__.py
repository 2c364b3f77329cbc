"""ctypes wrapper of the fp32 CPU oracle (hbsjd_oracle.c).

TEST INFRASTRUCTURE ONLY: imported by tests/, by the smoke check and by the
benchmark's CPU-baseline leg, never by the product path. It shares no code
with the HIP library and imports nothing from it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "hbsjd_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = False) -> str:
    """Compile the oracle with gcc: fp32, no contraction, no fast-math, OpenMP."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O3", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
                               "-std=c11", "-shared", "-fPIC", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class _Desc(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int), ("d", ctypes.c_int), ("n_heads", ctypes.c_int),
                ("f", ctypes.c_int), ("V", ctypes.c_int), ("C", ctypes.c_int),
                ("G", ctypes.c_int), ("has_bias", ctypes.c_int),
                ("eps", ctypes.c_float), ("rope_base", ctypes.c_float)]


_P = ctypes.c_void_p


class _Args(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int), ("prefix_tokens", _P), ("prefix_len", _P),
                ("labels", _P), ("temperature", _P), ("W", ctypes.c_int),
                ("H", ctypes.c_int), ("top_k", ctypes.c_int), ("cfg_scale", ctypes.c_float),
                ("seed", ctypes.c_uint64), ("greedy", ctypes.c_int),
                ("exec_mode", ctypes.c_int), ("gamma", ctypes.c_int),
                ("max_rounds", ctypes.c_int), ("sync", ctypes.c_int)]


class _Out(ctypes.Structure):
    _fields_ = [("tokens", _P), ("counts", _P), ("rounds", _P), ("active_hist", _P),
                ("mode_hist", _P), ("stats", _P), ("trace_drafts", _P), ("trace_q", _P)]


def lib():
    global _lib
    with _lock:
        if _lib is None:
            L = ctypes.CDLL(build())
            L.om_create.restype = _P
            L.om_create.argtypes = [ctypes.POINTER(_Desc), _P, ctypes.c_long]
            L.om_free.argtypes = [_P]
            L.om_forward_seq.argtypes = [_P, ctypes.c_int, _P, ctypes.c_int, _P]
            L.om_forward_batch.argtypes = [_P, ctypes.c_int] + [_P] * 6
            L.om_philox.argtypes = [ctypes.c_uint64, _P, _P]
            L.om_uniforms3.argtypes = [ctypes.c_uint64, ctypes.c_int, ctypes.c_int, _P]
            L.om_pinned_sum.restype = ctypes.c_float
            L.om_pinned_sum.argtypes = [_P, ctypes.c_int]
            L.om_inv_cdf.argtypes = [_P, ctypes.c_int, ctypes.c_float]
            L.om_transform.argtypes = [_P, ctypes.c_int, ctypes.c_float, ctypes.c_int, _P]
            L.om_cfg_combine.argtypes = [_P, _P, ctypes.c_int, ctypes.c_float, _P]
            L.om_argmax.argtypes = [_P, ctypes.c_int]
            L.om_verify_probs.argtypes = [ctypes.c_int] * 3 + [_P] * 7
            L.om_rollout.argtypes = [_P, ctypes.POINTER(_Args), ctypes.POINTER(_Out)]
            L.om_rollout_ar.argtypes = [_P, ctypes.POINTER(_Args), _P]
            L.om_rope.argtypes = [_P, _P, ctypes.c_int]
            L.om_set_debug.argtypes = [ctypes.c_int]
            _lib = L
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def set_debug(flags: int) -> None:
    """Plant a known mistake in the oracle (for the oracle's own power tests)."""
    lib().om_set_debug(int(flags))


DEBUG_RESIDUAL_DROPS_Q = 1
DEBUG_INVERTED_RATIO = 2
DEBUG_ROPE_SIGN = 4
DEBUG_HISTORY_SHIFT = 8
DEBUG_REUSE_SHIFT = 16


def round_bf16(x: np.ndarray) -> np.ndarray:
    """fp32 -> nearest bf16 (ties to even), returned as fp32."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + r) & np.uint32(0xFFFF0000)).view(np.float32)


class Model:
    """The decoder with weights from a blob (see synth.blob_layout)."""

    def __init__(self, shape, blob: np.ndarray):
        self.shape = shape
        self._blob = np.ascontiguousarray(blob, dtype=np.float32)
        d = _Desc(shape.n_layers, shape.d_model, shape.n_heads, shape.mlp_hidden, shape.vocab,
                  shape.n_classes, shape.grid, int(shape.has_lm_bias), shape.rms_eps,
                  shape.rope_base)
        self._h = lib().om_create(ctypes.byref(d), _ptr(self._blob), self._blob.size)
        if not self._h:
            raise ValueError("oracle rejected the model shape or blob size")
        self._blob = None

    def __del__(self):
        h = getattr(self, "_h", None)
        if h:
            lib().om_free(h)
            self._h = None

    @property
    def T(self) -> int:
        return self.shape.T

    def forward_seq(self, cls: int, tokens) -> np.ndarray:
        """Logits [(n+1), V] of the teacher-forced sequence [class, x_1..x_n]."""
        tok = np.ascontiguousarray(tokens, dtype=np.int32)
        out = np.empty((tok.size + 1, self.shape.vocab), dtype=np.float32)
        if lib().om_forward_seq(self._h, int(cls), _ptr(tok), tok.size, _ptr(out)) != 0:
            raise ValueError("bad sequence length")
        return out

    def forward_batch(self, classes, token_lists) -> list:
        """forward_seq for several sequences, in parallel over sequences."""
        n = len(token_lists)
        lens = np.array([len(t) for t in token_lists], dtype=np.int32)
        offs = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int32)
        toks = np.ascontiguousarray(np.concatenate([np.asarray(t, dtype=np.int32).ravel()
                                                    for t in token_lists] + [np.zeros(1, np.int32)]))
        row0 = np.concatenate([[0], np.cumsum(lens + 1)[:-1]]).astype(np.int64)
        cls = np.ascontiguousarray(classes, dtype=np.int32)
        out = np.empty((int(np.sum(lens + 1)), self.shape.vocab), dtype=np.float32)
        if lib().om_forward_batch(self._h, n, _ptr(cls), _ptr(toks), _ptr(offs), _ptr(lens),
                                  _ptr(row0), _ptr(out)) != 0:
            raise ValueError("bad sequence length")
        return [out[row0[i]:row0[i] + lens[i] + 1] for i in range(n)]

    def rope(self, u: np.ndarray, pos: int) -> np.ndarray:
        v = np.ascontiguousarray(u, dtype=np.float32).copy()
        lib().om_rope(self._h, _ptr(v), int(pos))
        return v

    def _args(self, batch, W, H, top_k, cfg_scale, seed, greedy, exec_mode, gamma, max_rounds,
              sync=False):
        self._keep = [np.ascontiguousarray(batch.prefix_tokens, dtype=np.int32),
                      np.ascontiguousarray(batch.prefix_len, dtype=np.int32),
                      np.ascontiguousarray(batch.labels, dtype=np.int32),
                      np.ascontiguousarray(batch.temperature, dtype=np.float32)]
        B = self._keep[1].size
        assert self._keep[0].shape == (B, self.T)
        return _Args(B, *[_ptr(a) for a in self._keep], int(W), int(H), int(top_k),
                     float(cfg_scale), int(seed), int(greedy), int(exec_mode), int(gamma),
                     int(max_rounds), int(bool(sync)))

    def rollout(self, batch, W: int, H: int = 24, top_k: int = 0, cfg_scale: float = 0.0,
                seed: int = 0, greedy: bool = False, exec_mode: int = 2, gamma: int = 0,
                max_rounds: Optional[int] = None, allow_partial: bool = False,
                sync: bool = False, trace: bool = False) -> dict:
        """Batched SJD rollout. exec_mode 0 Full, 1 Compact, 2 Auto (Full iff A > gamma).
        sync=True runs the Batch-Synchronous SJD ablation (shared window
        boundaries, Sec. 4.2 and Table 2) instead of independent progress.
        trace=True also returns the window after the prefill and after every
        round: 'trace_drafts' [rounds+1, B, W] (-1 past T or once complete) and
        'trace_q' [rounds+1, B, W], each draft's proposal probability q(z)
        (the reused row's p(z); 1 for a history draft and in greedy mode; 0
        where the draft is -1)."""
        B = len(batch.prefix_len)
        if max_rounds is None:
            max_rounds = int(self.T - np.min(batch.prefix_len)) + 1
        a = self._args(batch, W, H, top_k, cfg_scale, seed, greedy, exec_mode, gamma, max_rounds,
                       sync)
        tokens = np.zeros((B, self.T), dtype=np.int32)
        counts = np.zeros((max_rounds, B), dtype=np.int32)
        rounds = np.zeros(1, dtype=np.int32)
        ahist = np.zeros(max_rounds, dtype=np.int32)
        mhist = np.zeros(max_rounds, dtype=np.int32)
        stats = np.zeros(3, dtype=np.int64)
        tr_d = tr_q = None
        if trace:
            tr_d = np.full((max_rounds + 1, B, W), -1, dtype=np.int32)
            tr_q = np.zeros((max_rounds + 1, B, W), dtype=np.float32)
        o = _Out(_ptr(tokens), _ptr(counts), _ptr(rounds), _ptr(ahist), _ptr(mhist), _ptr(stats),
                 _ptr(tr_d) if trace else None, _ptr(tr_q) if trace else None)
        st = lib().om_rollout(self._h, ctypes.byref(a), ctypes.byref(o))
        if st != 0 and not (st == -2 and allow_partial):
            raise RuntimeError(f"oracle rollout failed with status {st}")
        r = int(rounds[0])
        res = dict(tokens=tokens, counts=counts[:r], rounds=r, active=ahist[:r],
                   mode=mhist[:r], verified=int(stats[0]), rejected=int(stats[1]),
                   image_rounds=int(stats[2]), complete=(st == 0))
        if trace:
            res["trace_drafts"] = tr_d[:r + 1]
            res["trace_q"] = tr_q[:r + 1]
        return res

    def rollout_ar(self, batch, top_k: int = 0, cfg_scale: float = 0.0, seed: int = 0,
                   greedy: bool = False) -> np.ndarray:
        """Token-by-token sampling with the same uniforms (u_draft at each position)."""
        B = len(batch.prefix_len)
        a = self._args(batch, 1, 1, top_k, cfg_scale, seed, greedy, 0, 0, 1)
        tokens = np.zeros((B, self.T), dtype=np.int32)
        lib().om_rollout_ar(self._h, ctypes.byref(a), _ptr(tokens))
        return tokens


def philox(seed: int, counter) -> np.ndarray:
    c = np.ascontiguousarray(counter, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().om_philox(int(seed), _ptr(c), _ptr(out))
    return out


def uniforms(seed: int, b: int, t: int) -> np.ndarray:
    """(u_draft, u_acc, u_res) for image b at position t."""
    out = np.zeros(3, dtype=np.float32)
    lib().om_uniforms3(int(seed), int(b), int(t), _ptr(out))
    return out


def pinned_sum(w: np.ndarray) -> np.float32:
    w = np.ascontiguousarray(w, dtype=np.float32)
    return np.float32(lib().om_pinned_sum(_ptr(w), w.size))


def inv_cdf(w: np.ndarray, u: float) -> int:
    w = np.ascontiguousarray(w, dtype=np.float32)
    return int(lib().om_inv_cdf(_ptr(w), w.size, float(np.float32(u))))


def transform(logits: np.ndarray, tau: float, top_k: int) -> np.ndarray:
    l = np.ascontiguousarray(logits, dtype=np.float32)
    p = np.empty_like(l)
    lib().om_transform(_ptr(l), l.size, float(np.float32(tau)), int(top_k), _ptr(p))
    return p


def cfg_combine(lc, lu, s: float) -> np.ndarray:
    lc = np.ascontiguousarray(lc, dtype=np.float32)
    lu = np.ascontiguousarray(lu, dtype=np.float32)
    out = np.empty_like(lc)
    lib().om_cfg_combine(_ptr(lc), _ptr(lu), lc.size, float(np.float32(s)), _ptr(out))
    return out


def argmax(l) -> int:
    l = np.ascontiguousarray(l, dtype=np.float32)
    return int(lib().om_argmax(_ptr(l), l.size))


def verify_probs(p: np.ndarray, q: np.ndarray, drafts: np.ndarray, u_acc: np.ndarray,
                 u_res: np.ndarray):
    """p, q [B, W, V] fp32 rows; drafts, u_acc [B, W]; u_res [B].
    Returns (counts [B], tokens [B, W] with -1 past each count)."""
    p = np.ascontiguousarray(p, dtype=np.float32)
    q = np.ascontiguousarray(q, dtype=np.float32)
    B, W, V = p.shape
    dr = np.ascontiguousarray(drafts, dtype=np.int32)
    ua = np.ascontiguousarray(u_acc, dtype=np.float32)
    ur = np.ascontiguousarray(u_res, dtype=np.float32)
    counts = np.zeros(B, dtype=np.int32)
    tokens = np.zeros((B, W), dtype=np.int32)
    lib().om_verify_probs(B, W, V, _ptr(p), _ptr(q), _ptr(dr), _ptr(ua), _ptr(ur),
                          _ptr(counts), _ptr(tokens))
    return counts, tokens


# ---------------------------------------------------------------- teacher scoring (Eq. 3)


def bikl(ls, lt) -> np.ndarray:
    """Bidirectional KL of Sec. 3.1, Eq. 3: D(p, q) = KL(p||q)/2 + KL(q||p)/2, where
    p and q are the softmax of the student and teacher logits rows (last axis).
    Computed in float64: log-probabilities through an explicit log-sum-exp."""
    ls = np.asarray(ls, dtype=np.float64)
    lt = np.asarray(lt, dtype=np.float64)

    def log_softmax(l):
        m = np.max(l, axis=-1, keepdims=True)
        return l - (m + np.log(np.sum(np.exp(l - m), axis=-1, keepdims=True)))

    lp, lq = log_softmax(ls), log_softmax(lt)
    p, q = np.exp(lp), np.exp(lq)
    kl_pq = np.sum(p * (lp - lq), axis=-1)
    kl_qp = np.sum(q * (lq - lp), axis=-1)
    return 0.5 * kl_pq + 0.5 * kl_qp


def score_bikl(student: Model, teacher: Model, tokens, prefix_len, labels):
    """The distillation loss of Eq. 3 for completed sequences (Sec. 3.1): both
    models see [class, x_1..x_{T-1}] teacher-forced; the logits row at position
    t-1 is each model's distribution of x_t; per image the biKL is averaged over
    the generated positions t = k_b+1..T. Returns (per_position [B][T] float64,
    entry t-1 for position t and 0 for t <= k_b; loss [B], 0 for k_b = T)."""
    tokens = np.asarray(tokens)
    B, T = tokens.shape
    per = np.zeros((B, T))
    loss = np.zeros(B)
    seqs = [tokens[b, :T - 1] for b in range(B)]
    ls = student.forward_batch(labels, seqs)
    lt = teacher.forward_batch(labels, seqs)
    for b in range(B):
        k = int(prefix_len[b])
        if k >= T:
            continue
        d = bikl(ls[b][k:T], lt[b][k:T])
        per[b, k:T] = d
        loss[b] = float(np.mean(d))
    return per, loss
