"""ctypes binding of libgmc.so (include/gmc.h), one call per C entry point.

The binding only marshals arguments: it checks dtype, device, shape and
contiguity of the torch tensors, passes their device pointers and the current
HIP stream, and raises GmcError on a non-OK status.  Every step of the path
runs in the library's HIP kernels; there is no fallback of any kind, and
importing this module fails loudly when libgmc.so has not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence, Tuple, Union

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgmc.so")

GMC_TOPK_GLOBAL, GMC_TOPK_SEGMENTED, GMC_RBGS, GMC_TOPK_APPROX = 0, 1, 2, 3
GMC_OK, GMC_EINVAL, GMC_ENOMEM, GMC_EDEVICE, GMC_ESTATE = 0, -1, -2, -3, -4
GMC_OPT_FORCE_FULL_SELECT, GMC_OPT_CAND_MARGIN, GMC_OPT_CAND_CAP_MULT, GMC_OPT_PROFILE = 1, 2, 3, 4
GMC_OPT_SAMPLE_STRATUM, GMC_OPT_SPARSE_MOMENTUM, GMC_OPT_CHANGE_LIST = 5, 6, 7
MAX_WORKERS = 64
STAGES = ("fused_vec", "fused_gen", "select", "emit", "aggregate", "apply")

COMPRESSORS = {"topk": GMC_TOPK_GLOBAL, "topk_seg": GMC_TOPK_SEGMENTED, "rbgs": GMC_RBGS,
               "approx": GMC_TOPK_APPROX}

# every entry point include/gmc.h declares
EXPORTS = ("gmc_init", "gmc_set_segments", "gmc_set_block", "gmc_set_stream", "gmc_message_len",
           "gmc_index_len", "gmc_step", "gmc_aggregate", "gmc_apply", "gmc_get_step", "gmc_set_step",
           "gmc_set_option", "gmc_stats", "gmc_profile_read", "gmc_last_error", "gmc_destroy",
           "gmc_calib_copy", "gmc_aggregate_apply", "gmc_set_rule", "gmc_set_eta", "gmc_set_lambda",
           "gmc_step_detach", "gmc_finish", "gmc_detach", "gmc_iteration", "gmc_calib_stream", "gmc_pair_stats",
           "gmc_count", "gmc_aggregate_static", "gmc_iteration_inplace")

RULES = {"gmc": 0, "server_momentum": 1, "lr_in_residual": 2}


class GmcError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__("gmc status %d: %s" % (status, msg))
        self.status = status


_lib = None


def load() -> ctypes.CDLL:
    """Load libgmc.so from the package directory (built by
    ``__graft_entry__.build()``); raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError("libgmc.so is not built: run __graft_entry__.build() "
                          "(hipcc --offload-arch=gfx950)")
    lib = ctypes.CDLL(LIB_PATH)
    P, i32, i64, u64, dbl = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_double
    lib.gmc_init.argtypes = [ctypes.POINTER(P), i64, i32, i32, dbl, dbl, dbl, u64]
    lib.gmc_set_segments.argtypes = [P, i32, P]
    lib.gmc_set_block.argtypes = [P, i32]
    lib.gmc_set_stream.argtypes = [P, P]
    lib.gmc_message_len.argtypes = [P]
    lib.gmc_message_len.restype = i64
    lib.gmc_index_len.argtypes = [P]
    lib.gmc_index_len.restype = i64
    lib.gmc_step.argtypes = [P, P, P, P, P, P, P, P]
    lib.gmc_aggregate.argtypes = [P, P, P, P, P]
    lib.gmc_apply.argtypes = [P, P, P, P]
    lib.gmc_get_step.argtypes = [P, ctypes.POINTER(i64)]
    lib.gmc_set_step.argtypes = [P, i64]
    lib.gmc_set_option.argtypes = [P, i32, i64]
    lib.gmc_stats.argtypes = [P, P, i32]
    lib.gmc_profile_read.argtypes = [P, P, P, i32]
    lib.gmc_last_error.argtypes = [P]
    lib.gmc_last_error.restype = ctypes.c_char_p
    lib.gmc_destroy.argtypes = [P]
    lib.gmc_destroy.restype = None
    lib.gmc_calib_copy.argtypes = [P, P, P, i64]
    lib.gmc_aggregate_apply.argtypes = [P, P, P, P, P, P, P]
    lib.gmc_set_rule.argtypes = [P, i32]
    lib.gmc_set_eta.argtypes = [P, dbl]
    lib.gmc_set_lambda.argtypes = [P, dbl]
    lib.gmc_step_detach.argtypes = [P, P, P, P, P, P, P, P, P]
    lib.gmc_finish.argtypes = [P, P, P, P, P, P, P, P, P, P]
    lib.gmc_detach.argtypes = [P, P, P, P]
    lib.gmc_iteration.argtypes = [P, P, P, P, P, P, P, P]
    lib.gmc_iteration_inplace.argtypes = [P, P, P, P, P, P, P, P]
    lib.gmc_calib_stream.argtypes = [P, P, P, i64, i32, i64]
    lib.gmc_pair_stats.argtypes = [P, P, P, i32, ctypes.POINTER(i32)]
    lib.gmc_aggregate_static.argtypes = [i64, i32, dbl, P, i64, P, i64, P, P, P]
    lib.gmc_aggregate_static.restype = ctypes.c_int
    lib.gmc_count.argtypes = [i64, dbl]
    lib.gmc_count.restype = i64
    for name in ("gmc_init", "gmc_set_segments", "gmc_set_block", "gmc_set_stream", "gmc_step",
                 "gmc_aggregate", "gmc_apply", "gmc_get_step", "gmc_set_step", "gmc_set_option",
                 "gmc_stats", "gmc_profile_read", "gmc_calib_copy", "gmc_aggregate_apply",
                 "gmc_set_rule", "gmc_set_eta", "gmc_set_lambda", "gmc_step_detach", "gmc_finish",
                 "gmc_detach", "gmc_iteration", "gmc_calib_stream", "gmc_pair_stats", "gmc_iteration_inplace"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _torch():
    import torch
    return torch


def _check(t, dtype, numel: Optional[int] = None, name: str = "tensor"):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if t.device.type != "cuda":
        raise ValueError("%s must be on a GPU device" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if numel is not None and t.numel() < numel:
        raise ValueError("%s needs at least %d elements, has %d" % (name, numel, t.numel()))
    return t.data_ptr()


def _rows(x, d: int, K: int, name: str) -> List[int]:
    """K device pointers from a [K, >=d] tensor (row stride may exceed d) or
    a sequence of K [d] tensors."""
    torch = _torch()
    if isinstance(x, torch.Tensor):
        if x.dim() != 2 or x.shape[0] != K or x.shape[1] < d:
            raise ValueError("%s must be [K, >=d]" % name)
        if x.dtype != torch.float32 or x.device.type != "cuda" or x.stride(1) != 1:
            raise ValueError("%s must be a float32 GPU tensor with unit inner stride" % name)
        return [x[k].data_ptr() for k in range(K)]
    if len(x) != K:
        raise ValueError("%s must hold K=%d tensors" % (name, K))
    return [_check(t, torch.float32, d, "%s[%d]" % (name, k)) for k, t in enumerate(x)]


def count(n: int, ratio: float) -> int:
    """Items a fraction ratio of n keeps (gmc_count: the top-s count of a
    segment of n, RBGS blocks of nb); host only."""
    k = int(load().gmc_count(int(n), float(ratio)))
    if k < 0:
        raise ValueError("count needs 1 <= n < 2^31 and 0 < ratio <= 1")
    return k


def aggregate_static(d: int, K: int, eta: float, idx, val, msg_len, update):
    """gmc_aggregate_static: the server's update of K top-s messages (idx
    int32 [K, index_len], val fp32 [K, message_len], msg_len int64 [K]) into
    update (fp32 [d]) with no context and no device allocation, on torch's
    current stream."""
    torch = _torch()
    lib = load()
    if idx.dim() != 2 or idx.shape[0] != K or val.dim() != 2 or val.shape[0] != K:
        raise ValueError("idx and val must be [K, row]")
    pi = _check(idx, torch.int32, None, "idx")
    pv = _check(val, torch.float32, None, "val")
    pl = _check(msg_len, torch.int64, K, "msg_len")
    pu = _check(update, torch.float32, d, "update")
    st = lib.gmc_aggregate_static(int(d), int(K), float(eta), pi, int(idx.shape[1]), pv, int(val.shape[1]), pl, pu,
                                  ctypes.c_void_p(torch.cuda.current_stream(update.device).cuda_stream))
    if st != GMC_OK:
        raise GmcError(st, lib.gmc_last_error(None).decode())


def calib_copy(dst, src):
    """Plain device copy dst[:] = src[:] (fp32), the reference kernel for
    memory-counter calibration."""
    torch = _torch()
    n = src.numel()
    pd = _check(dst, torch.float32, n, "dst")
    ps = _check(src, torch.float32, n, "src")
    lib = load()
    st = lib.gmc_calib_copy(ctypes.c_void_p(torch.cuda.current_stream(src.device).cuda_stream), pd, ps, n)
    if st != GMC_OK:
        raise GmcError(st, lib.gmc_last_error(None).decode())


def calib_stream(e, g):
    """e[k, :] += g[k, :] for two [K, d] fp32 views with the same row stride,
    in the fused worker pass's access pattern: the stream ceiling that pass
    is measured against."""
    torch = _torch()
    for name, t in (("e", e), ("g", g)):
        if not isinstance(t, torch.Tensor) or t.dim() != 2 or t.dtype != torch.float32 \
                or t.device.type != "cuda" or t.stride(1) != 1:
            raise ValueError("%s must be a [K, d] float32 GPU tensor with unit inner stride" % name)
    if e.shape != g.shape or e.stride(0) != g.stride(0):
        raise ValueError("e and g must have the same shape and row stride")
    K, d = e.shape
    lib = load()
    st = lib.gmc_calib_stream(ctypes.c_void_p(torch.cuda.current_stream(e.device).cuda_stream),
                              e.data_ptr(), g.data_ptr(), e.stride(0), K, d)
    if st != GMC_OK:
        raise GmcError(st, lib.gmc_last_error(None).decode())


class Gmc:
    """One GMC context: ``step`` (workers), ``aggregate`` (server), ``apply``.

    compressor: "topk" (global top-s), "topk_seg" (top-s per segment; pass
    ``segments`` as the n_seg+1 offsets), "rbgs" (``block`` elements per
    block) or "approx" (the sampled-threshold top-s, ``stratum`` components
    per sample stratum).  Calls run on torch's current stream of the tensors' device.
    """

    def __init__(self, d: int, K: int, compressor: str = "topk", ratio: float = 0.001,
                 beta: float = 0.9, eta: float = 0.1, seed: int = 0,
                 segments: Optional[Sequence[int]] = None, block: Optional[int] = None,
                 rule: str = "gmc", lam: float = 0.0, stratum: Optional[int] = None):
        self._lib = load()
        self.d, self.K, self.compressor = int(d), int(K), compressor
        if compressor not in COMPRESSORS:
            raise ValueError("compressor must be one of %s" % list(COMPRESSORS))
        ctx = ctypes.c_void_p()
        st = self._lib.gmc_init(ctypes.byref(ctx), self.d, self.K, COMPRESSORS[compressor],
                                float(ratio), float(beta), float(eta), int(seed) & (2 ** 64 - 1))
        if st != GMC_OK:
            raise GmcError(st, self._lib.gmc_last_error(None).decode())
        self._ctx = ctx
        if segments is not None:
            off = (ctypes.c_int64 * len(segments))(*[int(x) for x in segments])
            self._call(self._lib.gmc_set_segments(self._ctx, len(segments) - 1, off))
        if block is not None:
            self._call(self._lib.gmc_set_block(self._ctx, int(block)))
        if stratum is not None:
            self.set_option(GMC_OPT_SAMPLE_STRATUM, int(stratum))
        if rule not in RULES:
            raise ValueError("rule must be one of %s" % list(RULES))
        self.rule = rule
        if rule != "gmc":
            self._call(self._lib.gmc_set_rule(self._ctx, RULES[rule]))
        if lam:
            self.set_lambda(lam)

    def set_eta(self, eta: float):
        """Learning rate of the following iterations (a schedule)."""
        self._call(self._lib.gmc_set_eta(self._ctx, float(eta)))

    def set_lambda(self, lam: float):
        """GMC+'s detach coefficient (Algorithm 2)."""
        self._call(self._lib.gmc_set_lambda(self._ctx, float(lam)))

    # -- plumbing -------------------------------------------------------
    def _call(self, st: int):
        if st != GMC_OK:
            raise GmcError(st, self._lib.gmc_last_error(self._ctx).decode())

    def _stream(self, device):
        torch = _torch()
        s = torch.cuda.current_stream(device)
        self._call(self._lib.gmc_set_stream(self._ctx, ctypes.c_void_p(s.cuda_stream)))

    def close(self):
        if getattr(self, "_ctx", None):
            self._lib.gmc_destroy(self._ctx)
            self._ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- sizes ------------------------------------------------------------
    @property
    def message_len(self) -> int:
        return int(self._lib.gmc_message_len(self._ctx))

    @property
    def index_len(self) -> int:
        return int(self._lib.gmc_index_len(self._ctx))

    def alloc_messages(self, device="cuda"):
        """Fresh (idx int32 [K, index_len], val fp32 [K, message_len],
        msg_len int64 [K]) buffers."""
        torch = _torch()
        return (torch.zeros((self.K, self.index_len), dtype=torch.int32, device=device),
                torch.zeros((self.K, self.message_len), dtype=torch.float32, device=device),
                torch.zeros((self.K,), dtype=torch.int64, device=device))

    # -- the three calls of one iteration ---------------------------------
    def step(self, w_t, w_prev, grads, err, idx, val, msg_len, w_k=None):
        """Worker pass; with ``w_k`` ([K, >=d] or K tensors) also GMC+'s
        detached points where they are already final (gmc_step_detach;
        ``finish`` with the same ``w_k`` completes them).  ``w_prev`` may be
        None right after a server pass in place that kept its changes."""
        torch = _torch()
        d, K = self.d, self.K
        pw = _check(w_t, torch.float32, d, "w_t")
        pp = None if w_prev is None else _check(w_prev, torch.float32, d, "w_prev")
        gp = (ctypes.c_void_p * K)(*_rows(grads, d, K, "grads"))
        ep = (ctypes.c_void_p * K)(*_rows(err, d, K, "err"))
        pi = _check(idx, torch.int32, K * self.index_len, "idx")
        pv = _check(val, torch.float32, K * self.message_len, "val")
        pl = _check(msg_len, torch.int64, K, "msg_len")
        self._stream(w_t.device)
        if w_k is None:
            self._call(self._lib.gmc_step(self._ctx, pw, pp, gp, ep, pi, pv, pl))
        else:
            yp = (ctypes.c_void_p * K)(*_rows(w_k, d, K, "w_k"))
            self._call(self._lib.gmc_step_detach(self._ctx, pw, pp, gp, ep, yp, pi, pv, pl))

    def finish(self, idx, val, msg_len, w, w_out, w_prev=None, update=None, err=None, w_k=None):
        """Server pass under the context's rule: w_out = w_{t+1} (w_prev is
        needed by momentum on the server and may be w_out itself), optionally
        the update and the completion of GMC+'s detached points ``w_k``."""
        torch = _torch()
        K, d = self.K, self.d
        pi = _check(idx, torch.int32, K * self.index_len, "idx")
        pv = _check(val, torch.float32, K * self.message_len, "val")
        pl = _check(msg_len, torch.int64, K, "msg_len")
        pw = _check(w, torch.float32, d, "w")
        po = _check(w_out, torch.float32, d, "w_out")
        pp = None if w_prev is None else _check(w_prev, torch.float32, d, "w_prev")
        pu = None if update is None else _check(update, torch.float32, d, "update")
        ep = yp = None
        if w_k is not None:
            ep = (ctypes.c_void_p * K)(*_rows(err, d, K, "err"))
            yp = (ctypes.c_void_p * K)(*_rows(w_k, d, K, "w_k"))
        self._stream(w.device)
        self._call(self._lib.gmc_finish(self._ctx, pi, pv, pl, pw, pp, po, pu, ep, yp))

    def iteration(self, w_t, w_prev_io, grads, err, idx, val, msg_len):
        """One whole iteration: the worker pass, then w_{t+1} written over
        w_prev_io (swap the two buffers afterwards)."""
        torch = _torch()
        d, K = self.d, self.K
        pw = _check(w_t, torch.float32, d, "w_t")
        pp = _check(w_prev_io, torch.float32, d, "w_prev_io")
        gp = (ctypes.c_void_p * K)(*_rows(grads, d, K, "grads"))
        ep = (ctypes.c_void_p * K)(*_rows(err, d, K, "err"))
        pi = _check(idx, torch.int32, K * self.index_len, "idx")
        pv = _check(val, torch.float32, K * self.message_len, "val")
        pl = _check(msg_len, torch.int64, K, "msg_len")
        self._stream(w_t.device)
        self._call(self._lib.gmc_iteration(self._ctx, pw, pp, gp, ep, pi, pv, pl))

    def iteration_inplace(self, w, w_prev, grads, err, idx, val, msg_len):
        """One whole iteration with w updated in place; ``w_prev`` is w_{t-1}
        (``w`` itself at t = 0) or None after an in-place iteration (the
        context keeps w_{t+1} - w_t; GMC_OPT_SPARSE_MOMENTUM and
        GMC_OPT_CHANGE_LIST 3)."""
        torch = _torch()
        d, K = self.d, self.K
        pw = _check(w, torch.float32, d, "w")
        pp = None if w_prev is None else _check(w_prev, torch.float32, d, "w_prev")
        gp = (ctypes.c_void_p * K)(*_rows(grads, d, K, "grads"))
        ep = (ctypes.c_void_p * K)(*_rows(err, d, K, "err"))
        pi = _check(idx, torch.int32, K * self.index_len, "idx")
        pv = _check(val, torch.float32, K * self.message_len, "val")
        pl = _check(msg_len, torch.int64, K, "msg_len")
        self._stream(w.device)
        self._call(self._lib.gmc_iteration_inplace(self._ctx, pw, pp, gp, ep, pi, pv, pl))

    def detach(self, w, err, w_k):
        """GMC+'s detached points in one dense pass: w_k = w - (lambda eta) err."""
        torch = _torch()
        K, d = self.K, self.d
        pw = _check(w, torch.float32, d, "w")
        ep = (ctypes.c_void_p * K)(*_rows(err, d, K, "err"))
        yp = (ctypes.c_void_p * K)(*_rows(w_k, d, K, "w_k"))
        self._stream(w.device)
        self._call(self._lib.gmc_detach(self._ctx, pw, ep, yp))

    def aggregate(self, idx, val, msg_len, update):
        torch = _torch()
        pi = _check(idx, torch.int32, self.K * self.index_len, "idx")
        pv = _check(val, torch.float32, self.K * self.message_len, "val")
        pl = _check(msg_len, torch.int64, self.K, "msg_len")
        pu = _check(update, torch.float32, self.d, "update")
        self._stream(update.device)
        self._call(self._lib.gmc_aggregate(self._ctx, pi, pv, pl, pu))

    def aggregate_apply(self, idx, val, msg_len, w, w_out, update=None):
        """w_out = w + update (update = the server's dense update, written to
        `update` when given); w_out may be w itself."""
        torch = _torch()
        pi = _check(idx, torch.int32, self.K * self.index_len, "idx")
        pv = _check(val, torch.float32, self.K * self.message_len, "val")
        pl = _check(msg_len, torch.int64, self.K, "msg_len")
        pw = _check(w, torch.float32, self.d, "w")
        po = _check(w_out, torch.float32, self.d, "w_out")
        pu = None if update is None else _check(update, torch.float32, self.d, "update")
        self._stream(w.device)
        self._call(self._lib.gmc_aggregate_apply(self._ctx, pi, pv, pl, pw, po, pu))

    def apply(self, w, update, w_prev_out=None):
        torch = _torch()
        pw = _check(w, torch.float32, self.d, "w")
        pu = _check(update, torch.float32, self.d, "update")
        pp = None if w_prev_out is None else _check(w_prev_out, torch.float32, self.d, "w_prev_out")
        self._stream(w.device)
        self._call(self._lib.gmc_apply(self._ctx, pw, pp, pu))

    # -- state and diagnostics ---------------------------------------------
    @property
    def t(self) -> int:
        v = ctypes.c_int64()
        self._call(self._lib.gmc_get_step(self._ctx, ctypes.byref(v)))
        return v.value

    @t.setter
    def t(self, value: int):
        self._call(self._lib.gmc_set_step(self._ctx, int(value)))

    def set_option(self, option: int, value: int):
        self._call(self._lib.gmc_set_option(self._ctx, int(option), int(value)))

    def stats(self) -> dict:
        out = (ctypes.c_int64 * 8)()
        self._call(self._lib.gmc_stats(self._ctx, out, 8))
        keys = ("steps", "from_candidates", "full_data", "candidates", "count_errors", "sparse_momentum_steps",
                "sparse_applies")
        return {k: int(out[i]) for i, k in enumerate(keys)}

    def pair_stats(self):
        """(mode, cand) per (worker, segment) pair of the last step, as [K, n_seg]
        int arrays: mode 0 = resolved from the speculative candidates, 1 =
        full-data path; cand = candidates the worker pass collected."""
        import numpy as np
        np_ = ctypes.c_int32(0)
        self._call(self._lib.gmc_pair_stats(self._ctx, None, None, 0, ctypes.byref(np_)))
        n = np_.value
        mode = np.zeros(n, np.int32)
        cand = np.zeros(n, np.int64)
        self._call(self._lib.gmc_pair_stats(self._ctx, mode.ctypes.data, cand.ctypes.data, n, ctypes.byref(np_)))
        return mode.reshape(self.K, -1), cand.reshape(self.K, -1)

    def profile(self, stages=None):
        """Time the given stage names (None: all; []: off) with HIP events."""
        if stages is None:
            mask = (1 << len(STAGES)) - 1
        else:
            mask = 0
            for name in stages:
                mask |= 1 << STAGES.index(name)
        self.set_option(GMC_OPT_PROFILE, mask)

    def profile_read(self) -> dict:
        ms = (ctypes.c_double * len(STAGES))()
        n = (ctypes.c_int64 * len(STAGES))()
        self._call(self._lib.gmc_profile_read(self._ctx, ms, n, len(STAGES)))
        return {name: (ms[i], int(n[i])) for i, name in enumerate(STAGES)}
