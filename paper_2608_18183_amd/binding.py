"""ctypes binding of libhbsjd.so (see include/hbsjd.h for the contract of each call).

Device buffers are torch CUDA (HIP) tensors; host buffers are numpy arrays.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import threading
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libhbsjd.so")
_lock = threading.Lock()
_lib = None

DTYPE_F32, DTYPE_BF16 = 0, 1
EXEC_AUTO, EXEC_FULL, EXEC_COMPACT = 0, 1, 2
VERIFY_PROB, VERIFY_GREEDY, VERIFY_AR, VERIFY_AR_GREEDY = 0, 1, 2, 3
PROGRESS_INDEPENDENT, PROGRESS_SYNC = 0, 1
KERNELS = ["setup", "embed", "qkv", "attn", "oproj", "norm", "w13", "w2", "lmhead",
           "transform", "verify", "bikl"]
_STATUS = {0: "OK", 1: "EINVAL", 2: "ENOMEM", 3: "EHIP", 4: "ESTATE", 5: "EINTERNAL"}

_P = ctypes.c_void_p
_I32 = ctypes.c_int32


class HbsjdError(RuntimeError):
    def __init__(self, status: int, where: str, message: str):
        self.status = status
        self.code = _STATUS.get(status, str(status))
        super().__init__(f"{where}: {self.code}: {message}")


class _ModelDesc(ctypes.Structure):
    _fields_ = [("n_layers", _I32), ("d_model", _I32), ("n_heads", _I32), ("mlp_hidden", _I32),
                ("vocab", _I32), ("n_classes", _I32), ("grid", _I32), ("dtype", _I32),
                ("has_lm_bias", _I32), ("rms_eps", ctypes.c_float), ("rope_base", ctypes.c_float)]


class _RolloutArgs(ctypes.Structure):
    _fields_ = [("batch", _I32), ("prefix_tokens", _P), ("prefix_len", _P), ("class_labels", _P),
                ("temperature", _P), ("window", _I32), ("history", _I32), ("top_k", _I32),
                ("cfg_scale", ctypes.c_float), ("seed", ctypes.c_uint64), ("verify_mode", _I32),
                ("exec_mode", _I32), ("gamma", _I32), ("max_rounds", _I32), ("progress", _I32)]


class _RolloutOut(ctypes.Structure):
    _fields_ = [("tokens", _P), ("counts", _P), ("rounds", _P), ("active_per_round", _P),
                ("mode_per_round", _P), ("stats", _P)]


_SIGS = {
    "hbsjd_create": (_I32, [ctypes.POINTER(_ModelDesc), ctypes.c_uint64, _P, ctypes.POINTER(_P)]),
    "hbsjd_load_weights": (_I32, [_P, _P, ctypes.c_size_t]),
    "hbsjd_rollout": (_I32, [_P, ctypes.POINTER(_RolloutArgs), ctypes.POINTER(_RolloutOut)]),
    "hbsjd_rollout_begin": (_I32, [_P, ctypes.POINTER(_RolloutArgs)]),
    "hbsjd_round": (_I32, [_P, _I32, _P, _P]),
    "hbsjd_get_state": (_I32, [_P, _P, _P, _P, _P]),
    "hbsjd_forward": (_I32, [_P, _I32, _P, _P, _P, _P]),
    "hbsjd_score_bikl": (_I32, [_P, _P, _I32, _P, _P, _P, _P, _P]),
    "hbsjd_bikl_rows": (_I32, [_P, _P, ctypes.c_int64, _I32, _P, _P]),
    "hbsjd_verify_probs": (_I32, [_I32, _I32, _I32, _P, _P, _P, _P, _P, _P, _P, _P]),
    "hbsjd_transform_rows": (_I32, [_I32, _I32, _P, _I32, ctypes.c_float, _P, _I32,
                                    ctypes.c_uint64, _P, _P, _P, _P, _P]),
    "hbsjd_transform_rows_noalloc": (_I32, [_I32, _I32, _P, _I32, ctypes.c_float, _P, _I32,
                                            ctypes.c_uint64, _P, _P, _P, _P, _P]),
    "hbsjd_philox": (_I32, [ctypes.c_uint64, _I32, _P, _P, _P]),
    "hbsjd_mfma_probe": (_I32, [_I32, _I32, _P, _P]),
    "hbsjd_calibrate_gamma": (_I32, [_P, _I32, _I32, _P]),
    "hbsjd_profile_start": (_I32, [_P, ctypes.c_uint32]),
    "hbsjd_profile_sample": (_I32, [_P, ctypes.c_int32]),
    "hbsjd_profile_read": (_I32, [_P, _P, _P]),
    "hbsjd_destroy": (None, [_P]),
    "hbsjd_last_error": (ctypes.c_char_p, []),
    "hbsjd_version": (ctypes.c_char_p, []),
}


def library_path() -> str:
    return _LIB_PATH


def load_library():
    """Load libhbsjd.so; raises if it has not been built (there is no fallback)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB_PATH):
                raise ImportError(f"{_LIB_PATH} is missing: build it with "
                                  "python paper_2608_18183_amd/build.py")
            L = ctypes.CDLL(_LIB_PATH)
            for name, (res, args) in _SIGS.items():
                fn = getattr(L, name)
                fn.restype = res
                fn.argtypes = args
            _lib = L
    return _lib


def _check(status: int, where: str):
    if status != 0:
        msg = load_library().hbsjd_last_error().decode(errors="replace")
        raise HbsjdError(status, where, msg)


def _np_ptr(a: np.ndarray):
    return a.ctypes.data_as(_P)


def _dev_ptr(t) -> int:
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda or not t.is_contiguous():
        raise ValueError("expected a contiguous device tensor")
    return t.data_ptr()


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        import torch
        if not torch.cuda.is_available():
            return 0
        return torch.cuda.current_stream().cuda_stream
    if hasattr(stream, "cuda_stream"):   # a torch.cuda.Stream
        return stream.cuda_stream
    return int(stream)


def hbsjd_version() -> str:
    return load_library().hbsjd_version().decode()


@dataclasses.dataclass
class ModelDesc:
    n_layers: int
    d_model: int
    n_heads: int
    mlp_hidden: int
    vocab: int
    n_classes: int
    grid: int
    dtype: int = DTYPE_BF16
    has_lm_bias: bool = False
    rms_eps: float = 1e-5
    rope_base: float = 10000.0

    @property
    def T(self) -> int:
        return self.grid * self.grid

    def _c(self) -> _ModelDesc:
        return _ModelDesc(self.n_layers, self.d_model, self.n_heads, self.mlp_hidden, self.vocab,
                          self.n_classes, self.grid, self.dtype, int(self.has_lm_bias),
                          self.rms_eps, self.rope_base)


class Context:
    """An hbsjd_ctx: one model on one GPU, bound to one stream."""

    def __init__(self, desc: ModelDesc, max_kv_bytes: int = 0, stream=None):
        self.desc = desc
        self._lib = load_library()
        h = _P()
        md = desc._c()
        _check(self._lib.hbsjd_create(ctypes.byref(md), int(max_kv_bytes),
                                      _P(_stream_handle(stream)), ctypes.byref(h)), "hbsjd_create")
        self._h = h
        self._keep = []
        self._B, self._W = 0, 0

    def close(self):
        if getattr(self, "_h", None):
            self._lib.hbsjd_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def hbsjd_load_weights(self, blob: np.ndarray):
        blob = np.ascontiguousarray(blob, dtype=np.float32)
        _check(self._lib.hbsjd_load_weights(self._h, _np_ptr(blob), blob.size),
               "hbsjd_load_weights")

    def _args(self, prefix_tokens, prefix_len, class_labels, temperature, window, history,
              top_k, cfg_scale, seed, verify_mode, exec_mode, gamma, max_rounds,
              progress=PROGRESS_INDEPENDENT):
        pl = np.ascontiguousarray(prefix_len, dtype=np.int32)
        lab = np.ascontiguousarray(class_labels, dtype=np.int32)
        tau = np.ascontiguousarray(temperature, dtype=np.float32)
        B = pl.size
        if max_rounds is None:
            max_rounds = int(self.desc.T - pl.min()) if B else 1
            max_rounds = max(max_rounds, 1)
        self._keep = [pl, lab, tau, prefix_tokens]
        a = _RolloutArgs(B, _P(_dev_ptr(prefix_tokens)), _np_ptr(pl), _np_ptr(lab), _np_ptr(tau),
                         int(window), int(history), int(top_k), float(cfg_scale), int(seed),
                         int(verify_mode), int(exec_mode), int(gamma), int(max_rounds),
                         int(progress))
        return a, B, max_rounds

    def hbsjd_rollout(self, prefix_tokens, prefix_len, class_labels, temperature, window: int,
                      history: int = 24, top_k: int = 0, cfg_scale: float = 0.0, seed: int = 0,
                      verify_mode: int = VERIFY_PROB, exec_mode: int = EXEC_AUTO,
                      gamma: int = -1, max_rounds: Optional[int] = None, out_tokens=None,
                      out_counts=None, progress: int = PROGRESS_INDEPENDENT) -> dict:
        import torch
        a, B, max_rounds = self._args(prefix_tokens, prefix_len, class_labels, temperature,
                                      window, history, top_k, cfg_scale, seed, verify_mode,
                                      exec_mode, gamma, max_rounds, progress)
        dev = prefix_tokens.device
        tokens = out_tokens if out_tokens is not None else torch.empty(
            (B, self.desc.T), dtype=torch.int32, device=dev)
        counts = out_counts if out_counts is not None else torch.empty(
            (max_rounds, B), dtype=torch.int32, device=dev)
        rounds = np.zeros(1, dtype=np.int32)
        ah = np.zeros(max_rounds, dtype=np.int32)
        mh = np.zeros(max_rounds, dtype=np.int32)
        stats = np.zeros(4, dtype=np.int64)
        o = _RolloutOut(_P(_dev_ptr(tokens)), _P(_dev_ptr(counts)), _np_ptr(rounds), _np_ptr(ah),
                        _np_ptr(mh), _np_ptr(stats))
        _check(self._lib.hbsjd_rollout(self._h, ctypes.byref(a), ctypes.byref(o)), "hbsjd_rollout")
        r = int(rounds[0])
        return dict(tokens=tokens, counts=counts[:r], rounds=r, active=ah[:r], mode=mh[:r],
                    verified=int(stats[0]), rejected=int(stats[1]), image_rounds=int(stats[2]),
                    rows=int(stats[3]))

    def hbsjd_rollout_begin(self, prefix_tokens, prefix_len, class_labels, temperature,
                            window: int, history: int = 24, top_k: int = 0,
                            cfg_scale: float = 0.0, seed: int = 0,
                            verify_mode: int = VERIFY_PROB, exec_mode: int = EXEC_AUTO,
                            gamma: int = -1, max_rounds: Optional[int] = None,
                            progress: int = PROGRESS_INDEPENDENT):
        a, B, _ = self._args(prefix_tokens, prefix_len, class_labels, temperature, window,
                             history, top_k, cfg_scale, seed, verify_mode, exec_mode, gamma,
                             max_rounds, progress)
        self._B, self._W = B, int(window)
        _check(self._lib.hbsjd_rollout_begin(self._h, ctypes.byref(a)), "hbsjd_rollout_begin")

    def hbsjd_round(self, exec_mode: int = EXEC_AUTO):
        counts = np.zeros(max(self._B, 1), dtype=np.int32)
        active = np.zeros(1, dtype=np.int32)
        _check(self._lib.hbsjd_round(self._h, int(exec_mode), _np_ptr(counts), _np_ptr(active)),
               "hbsjd_round")
        return counts, int(active[0])

    def hbsjd_get_state(self) -> dict:
        B, W, T = max(self._B, 1), max(self._W, 1), self.desc.T
        tokens = np.zeros((B, T), dtype=np.int32)
        cursors = np.zeros(B, dtype=np.int32)
        drafts = np.zeros((B, W), dtype=np.int32)
        q = np.zeros((B, W), dtype=np.float32)
        _check(self._lib.hbsjd_get_state(self._h, _np_ptr(tokens), _np_ptr(cursors),
                                         _np_ptr(drafts), _np_ptr(q)), "hbsjd_get_state")
        return dict(tokens=tokens, cursors=cursors, drafts=drafts, q_token_prob=q)

    def hbsjd_forward(self, tokens, lens, labels):
        """Teacher-forced logits [sum(len+1), V] (fp32 device tensor)."""
        import torch
        ln = np.ascontiguousarray(lens, dtype=np.int32)
        lab = np.ascontiguousarray(labels, dtype=np.int32)
        rows = int(np.sum(ln + 1))
        out = torch.empty((rows, self.desc.vocab), dtype=torch.float32, device=tokens.device)
        _check(self._lib.hbsjd_forward(self._h, ln.size, _P(_dev_ptr(tokens)), _np_ptr(ln),
                                       _np_ptr(lab), _P(_dev_ptr(out))), "hbsjd_forward")
        return out

    def hbsjd_score_bikl(self, teacher: "Context", tokens, prefix_len, class_labels):
        """Eq. 3 scoring of completed sequences with this context as the student.
        tokens: int32 device tensor [B, T]. Returns (per_position [B, T],
        loss [B]) fp32 device tensors."""
        import torch
        pl = np.ascontiguousarray(prefix_len, dtype=np.int32)
        lab = np.ascontiguousarray(class_labels, dtype=np.int32)
        B = pl.size
        per = torch.empty((B, self.desc.T), dtype=torch.float32, device=tokens.device)
        loss = torch.empty(B, dtype=torch.float32, device=tokens.device)
        _check(self._lib.hbsjd_score_bikl(self._h, teacher._h, B, _P(_dev_ptr(tokens)),
                                          _np_ptr(pl), _np_ptr(lab), _P(_dev_ptr(per)),
                                          _P(_dev_ptr(loss))), "hbsjd_score_bikl")
        return per, loss

    def hbsjd_profile_start(self, classes=()):
        mask = 0
        for k in classes:
            mask |= 1 << KERNELS.index(k)
        _check(self._lib.hbsjd_profile_start(self._h, mask), "hbsjd_profile_start")

    def hbsjd_profile_sample(self, every: int = 1):
        _check(self._lib.hbsjd_profile_sample(self._h, int(every)), "hbsjd_profile_sample")

    def hbsjd_profile_read(self) -> dict:
        ms = np.zeros(len(KERNELS), dtype=np.float64)
        n = np.zeros(len(KERNELS), dtype=np.int64)
        _check(self._lib.hbsjd_profile_read(self._h, _np_ptr(ms), _np_ptr(n)), "hbsjd_profile_read")
        return {k: (float(ms[i]), int(n[i])) for i, k in enumerate(KERNELS)}

    def hbsjd_calibrate_gamma(self, batch: int, window: int) -> int:
        g = np.zeros(1, dtype=np.int32)
        _check(self._lib.hbsjd_calibrate_gamma(self._h, int(batch), int(window), _np_ptr(g)),
               "hbsjd_calibrate_gamma")
        return int(g[0])


def hbsjd_verify_probs(p, q, drafts, u_acc, u_res, stream=None):
    """p, q: fp32 [B, W, V]; drafts int32 and u_acc fp32 [B, W]; u_res fp32 [B]
    (device tensors). Returns (counts [B], tokens [B, W]) device tensors."""
    import torch
    B, W, V = p.shape
    counts = torch.empty(B, dtype=torch.int32, device=p.device)
    tokens = torch.empty((B, W), dtype=torch.int32, device=p.device)
    L = load_library()
    _check(L.hbsjd_verify_probs(B, W, V, _P(_dev_ptr(p)), _P(_dev_ptr(q)), _P(_dev_ptr(drafts)),
                                _P(_dev_ptr(u_acc)), _P(_dev_ptr(u_res)), _P(_dev_ptr(counts)),
                                _P(_dev_ptr(tokens)), _P(_stream_handle(stream))),
           "hbsjd_verify_probs")
    return counts, tokens


def hbsjd_transform_rows(logits, temperature, position, top_k: int = 0, cfg_scale: float = 0.0,
                         seed: int = 0, stream=None, out=None, noalloc: bool = False):
    """logits: fp32 device tensor [rows, V] or, with guidance, [rows, 2, V]
    (conditional then unconditional row); temperature fp32 and position int32
    device tensors [rows]. Returns (p [rows, V], argmax [rows], draw [rows])
    device tensors, written into `out` when given. noalloc=True calls
    hbsjd_transform_rows_noalloc (no device allocation inside the library)."""
    import torch
    if logits.dim() == 2:
        rows, V = logits.shape
        cfg = 1
    else:
        rows, cfg, V = logits.shape
    if out is None:
        out = (torch.empty((rows, V), dtype=torch.float32, device=logits.device),
               torch.empty(rows, dtype=torch.int32, device=logits.device),
               torch.empty(rows, dtype=torch.int32, device=logits.device))
    p, amax, draw = out
    L = load_library()
    fn = L.hbsjd_transform_rows_noalloc if noalloc else L.hbsjd_transform_rows
    _check(fn(rows, V, _P(_dev_ptr(logits)), cfg, float(cfg_scale), _P(_dev_ptr(temperature)),
              int(top_k), int(seed), _P(_dev_ptr(position)), _P(_dev_ptr(p)),
              _P(_dev_ptr(amax)), _P(_dev_ptr(draw)), _P(_stream_handle(stream))),
           "hbsjd_transform_rows_noalloc" if noalloc else "hbsjd_transform_rows")
    return p, amax, draw


def hbsjd_bikl_rows(logits_s, logits_t, stream=None):
    """logits_s, logits_t: fp32 device tensors [rows, V]. Returns the per-row
    bidirectional KL of their softmaxes, fp32 device tensor [rows]."""
    import torch
    rows, V = logits_s.shape
    if tuple(logits_t.shape) != (rows, V):
        raise ValueError("logits_s and logits_t must have the same shape")
    out = torch.empty(rows, dtype=torch.float32, device=logits_s.device)
    L = load_library()
    _check(L.hbsjd_bikl_rows(_P(_dev_ptr(logits_s)), _P(_dev_ptr(logits_t)), rows, V,
                             _P(_dev_ptr(out)), _P(_stream_handle(stream))), "hbsjd_bikl_rows")
    return out


def hbsjd_mfma_probe(workgroups: int, iters: int, sink, stream=None):
    """The MFMA calibration kernel (asynchronous on `stream`); sink: a device
    tensor of at least 1 KB. One launch does workgroups x 4 x iters x 8 x 16384
    flops."""
    if sink.numel() * sink.element_size() < 1024:
        raise ValueError("sink must hold at least 1 KB")
    L = load_library()
    _check(L.hbsjd_mfma_probe(int(workgroups), int(iters), _P(_dev_ptr(sink)),
                              _P(_stream_handle(stream))), "hbsjd_mfma_probe")


def hbsjd_philox(seed: int, bt, stream=None):
    """bt: uint32-compatible int32 device tensor [n, 2] of (image, position);
    returns the four Philox words per pair as an int32 device tensor [n, 4]."""
    import torch
    n = bt.shape[0]
    out = torch.empty((n, 4), dtype=torch.int32, device=bt.device)
    L = load_library()
    _check(L.hbsjd_philox(int(seed), n, _P(_dev_ptr(bt)), _P(_dev_ptr(out)),
                          _P(_stream_handle(stream))), "hbsjd_philox")
    return out
