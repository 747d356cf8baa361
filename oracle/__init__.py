"""GMC oracle: a plain, slow, single-threaded CPU implementation of one GMC
iteration (Algorithm 1), of GMC+'s RBGS compressor and detached point
(Algorithm 2), of the two alternative update rules of the appendix
(momentum on the server; learning rate inside the residual), and of the
sampled-threshold top-s the experiments use (Section 5.1).

TEST INFRASTRUCTURE.  Only the test suite, ``__graft_entry__.smoke()`` and the
bench's ``cpu_baseline`` leg may import this package.  The device library does
not depend on it and must never fall back to it.

The C source (``gmc_oracle.c``) is built with gcc ``-O2 -ffp-contract=off``
(no fast-math, SSE2 scalar binary32).  This module only marshals numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import List, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gmc_oracle.c")
LIB_PATH = os.path.join(_HERE, "liboracle.so")

CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math",
          "-msse2", "-mfpmath=sse", "-fno-builtin"]

_lib = None


def build(force: bool = False, src: str = _SRC, out: str = LIB_PATH) -> str:
    """Compile the oracle with gcc.  Returns the library path."""
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(src):
        tmp = out + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", *CFLAGS, src, "-o", tmp, "-lm"])
        os.replace(tmp, out)
    return out


def _bind(lib):
    c_i64, c_f, c_vp = ctypes.c_int64, ctypes.c_float, ctypes.c_void_p
    lib.orc_count.argtypes = [c_i64, ctypes.c_double]
    lib.orc_count.restype = c_i64
    lib.orc_constants.argtypes = [ctypes.c_double, ctypes.c_double, ctypes.c_int,
                                  ctypes.POINTER(c_f), ctypes.POINTER(c_f)]
    lib.orc_constants.restype = None
    lib.orc_precompress.argtypes = [c_i64, c_f, c_vp, c_vp, c_vp, c_vp, c_vp]
    lib.orc_precompress.restype = None
    lib.orc_topk.argtypes = [c_i64, c_vp, c_i64, c_vp]
    lib.orc_topk.restype = ctypes.c_int
    lib.orc_compress_topk.argtypes = [c_vp, c_i64, c_vp, ctypes.c_double, c_vp, c_vp]
    lib.orc_compress_topk.restype = c_i64
    lib.orc_splitmix64_mix.argtypes = [ctypes.c_uint64]
    lib.orc_splitmix64_mix.restype = ctypes.c_uint64
    lib.orc_rbgs_draw.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64]
    lib.orc_rbgs_draw.restype = ctypes.c_uint64
    lib.orc_rbgs_blocks.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int32,
                                    ctypes.c_int32, c_vp]
    lib.orc_rbgs_blocks.restype = None
    lib.orc_compress_rbgs.argtypes = [c_vp, c_i64, c_i64, c_vp, ctypes.c_int32, c_vp]
    lib.orc_compress_rbgs.restype = c_i64
    lib.orc_aggregate.argtypes = [c_i64, ctypes.c_int, c_f, c_vp, c_vp, c_vp, c_vp]
    lib.orc_aggregate.restype = ctypes.c_int
    lib.orc_apply.argtypes = [c_i64, c_vp, c_vp]
    lib.orc_apply.restype = None
    lib.orc_detach_constant.argtypes = [ctypes.c_double, ctypes.c_double]
    lib.orc_detach_constant.restype = c_f
    lib.orc_detach.argtypes = [c_i64, c_f, c_vp, c_vp, c_vp]
    lib.orc_detach.restype = None
    lib.orc_variant_constants.argtypes = [ctypes.c_int, ctypes.c_double, ctypes.c_double, ctypes.c_int,
                                          ctypes.POINTER(c_f), ctypes.POINTER(c_f), ctypes.POINTER(c_f)]
    lib.orc_variant_constants.restype = None
    lib.orc_precompress_plain.argtypes = [c_i64, c_vp, c_vp, c_vp]
    lib.orc_precompress_plain.restype = None
    lib.orc_precompress_lr.argtypes = [c_i64, c_f, c_f, c_vp, c_vp, c_vp, c_vp, c_vp]
    lib.orc_precompress_lr.restype = None
    lib.orc_apply_server_momentum.argtypes = [c_i64, c_f, c_vp, c_vp, c_vp, c_vp]
    lib.orc_apply_server_momentum.restype = None
    u64 = ctypes.c_uint64
    lib.orc_sample_draw.argtypes = [u64, u64, u64, u64]
    lib.orc_sample_draw.restype = u64
    lib.orc_sample_positions.argtypes = [u64, u64, u64, c_i64, c_i64, c_vp]
    lib.orc_sample_positions.restype = c_i64
    lib.orc_compress_approx.argtypes = [c_vp, c_i64, u64, u64, u64, c_i64, ctypes.c_double, c_vp, c_vp]
    lib.orc_compress_approx.restype = c_i64
    return lib


def load(path: Optional[str] = None):
    """Load (building first if absent) the oracle library.  ``path`` loads a
    different build of the same interface (used by the mutation tests)."""
    global _lib
    if path is not None:
        return _bind(ctypes.CDLL(path))
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        _lib = _bind(ctypes.CDLL(LIB_PATH))
    return _lib


def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32)


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


# ---------------------------------------------------------------------------
# per-operation wrappers
# ---------------------------------------------------------------------------

def count(n: int, ratio: float, lib=None) -> int:
    return int((lib or load()).orc_count(n, ratio))


def constants(beta: float, eta: float, K: int, lib=None) -> Tuple[np.float32, np.float32]:
    c, s = ctypes.c_float(), ctypes.c_float()
    (lib or load()).orc_constants(beta, eta, K, ctypes.byref(c), ctypes.byref(s))
    return np.float32(c.value), np.float32(s.value)


def precompress(c, w_t, w_prev, g, e, lib=None) -> np.ndarray:
    w_t, w_prev, g, e = map(_f32, (w_t, w_prev, g, e))
    u = np.empty_like(w_t)
    (lib or load()).orc_precompress(w_t.size, ctypes.c_float(float(c)), _ptr(w_t), _ptr(w_prev),
                                    _ptr(g), _ptr(e), _ptr(u))
    return u


def topk(u, k: int, lib=None) -> np.ndarray:
    u = _f32(u)
    out = np.empty(max(k, 1), dtype=np.int64)
    rc = (lib or load()).orc_topk(u.size, _ptr(u), k, _ptr(out))
    if rc != 0:
        raise MemoryError("oracle top-k allocation failed")
    return out[:k]


def compress_topk(u: np.ndarray, seg_off, ratio: float, lib=None) -> Tuple[np.ndarray, np.ndarray]:
    """Top-k per segment.  ``u`` (fp32, contiguous) is overwritten with the
    residual; returns (idx int32, val fp32)."""
    assert u.dtype == np.float32 and u.flags.c_contiguous
    seg = np.ascontiguousarray(seg_off, dtype=np.int64)
    lib = lib or load()
    cap = sum(count(int(seg[i + 1] - seg[i]), ratio, lib) for i in range(len(seg) - 1))
    idx = np.empty(max(cap, 1), dtype=np.int32)
    val = np.empty(max(cap, 1), dtype=np.float32)
    m = lib.orc_compress_topk(_ptr(u), len(seg) - 1, _ptr(seg), ratio, _ptr(idx), _ptr(val))
    if m < 0:
        raise MemoryError("oracle compress allocation failed")
    return idx[:m], val[:m]


def splitmix64_mix(z: int, lib=None) -> int:
    return int((lib or load()).orc_splitmix64_mix(z))


def rbgs_draw(seed: int, t: int, i: int, lib=None) -> int:
    return int((lib or load()).orc_rbgs_draw(seed, t, i))


def rbgs_blocks(seed: int, t: int, nb: int, n_sel: int, lib=None) -> np.ndarray:
    out = np.empty(n_sel, dtype=np.int32)
    (lib or load()).orc_rbgs_blocks(seed, t, nb, n_sel, _ptr(out))
    return out


def compress_rbgs(u: np.ndarray, B: int, blocks: np.ndarray, lib=None) -> np.ndarray:
    assert u.dtype == np.float32 and u.flags.c_contiguous
    blocks = np.ascontiguousarray(blocks, dtype=np.int32)
    val = np.empty(max(1, len(blocks) * B), dtype=np.float32)
    m = (lib or load()).orc_compress_rbgs(_ptr(u), u.size, B, _ptr(blocks), len(blocks), _ptr(val))
    return val[:m]


def aggregate(d: int, s, idx_list: Sequence[np.ndarray], val_list: Sequence[np.ndarray],
              lib=None) -> np.ndarray:
    K = len(idx_list)
    idx_list = [np.ascontiguousarray(a, dtype=np.int32) for a in idx_list]
    val_list = [_f32(a) for a in val_list]
    ip = (ctypes.c_void_p * K)(*[_ptr(a) for a in idx_list])
    vp = (ctypes.c_void_p * K)(*[_ptr(a) for a in val_list])
    ln = np.array([a.size for a in idx_list], dtype=np.int64)
    delta = np.empty(d, dtype=np.float32)
    rc = (lib or load()).orc_aggregate(d, K, ctypes.c_float(float(s)), ctypes.cast(ip, ctypes.c_void_p),
                                       ctypes.cast(vp, ctypes.c_void_p), _ptr(ln), _ptr(delta))
    if rc != 0:
        raise MemoryError("oracle aggregate allocation failed")
    return delta


def apply(w: np.ndarray, delta, lib=None) -> None:
    assert w.dtype == np.float32 and w.flags.c_contiguous
    delta = _f32(delta)
    (lib or load()).orc_apply(w.size, _ptr(w), _ptr(delta))


def detach_constant(lam: float, eta: float, lib=None) -> np.float32:
    return np.float32((lib or load()).orc_detach_constant(lam, eta))


def detach(q, w_next, e_next, lib=None) -> np.ndarray:
    """w_{t+1,k} = w_{t+1} - q e_{t+1,k} (Algorithm 2), q = fl32(lambda eta)."""
    w_next, e_next = _f32(w_next), _f32(e_next)
    out = np.empty_like(w_next)
    (lib or load()).orc_detach(w_next.size, ctypes.c_float(float(q)), _ptr(w_next), _ptr(e_next), _ptr(out))
    return out


def sample_positions(seed: int, t: int, k: int, n: int, L: int, lib=None) -> np.ndarray:
    """The approximate top-s sample: one position per stratum of L."""
    out = np.empty(max(1, (n + L - 1) // L), dtype=np.int64)
    m = (lib or load()).orc_sample_positions(seed, t, k, n, L, _ptr(out))
    return out[:m]


def compress_approx(u: np.ndarray, seed: int, t: int, k: int, L: int, ratio: float,
                    lib=None) -> Tuple[np.ndarray, np.ndarray]:
    """Approximate top-s of Section 5.1; ``u`` becomes the residual."""
    assert u.dtype == np.float32 and u.flags.c_contiguous
    idx = np.empty(max(1, u.size), dtype=np.int32)
    val = np.empty(max(1, u.size), dtype=np.float32)
    m = (lib or load()).orc_compress_approx(_ptr(u), u.size, seed, t, k, L, ratio, _ptr(idx), _ptr(val))
    if m < 0:
        raise MemoryError("oracle approximate top-s allocation failed")
    return idx[:m], val[:m]


VARIANTS = {"gmc": 0, "server_momentum": 1, "lr_in_residual": 2}


def variant_constants(variant: str, beta: float, eta: float, K: int, lib=None):
    """(c, s, h) of an update rule: see ``orc_variant_constants``."""
    c, s, h = ctypes.c_float(), ctypes.c_float(), ctypes.c_float()
    (lib or load()).orc_variant_constants(VARIANTS[variant], beta, eta, K, ctypes.byref(c), ctypes.byref(s),
                                          ctypes.byref(h))
    return np.float32(c.value), np.float32(s.value), np.float32(h.value)


def precompress_plain(g, e, lib=None) -> np.ndarray:
    g, e = _f32(g), _f32(e)
    u = np.empty_like(g)
    (lib or load()).orc_precompress_plain(g.size, _ptr(g), _ptr(e), _ptr(u))
    return u


def precompress_lr(h, b, w_t, w_prev, g, e, lib=None) -> np.ndarray:
    w_t, w_prev, g, e = map(_f32, (w_t, w_prev, g, e))
    u = np.empty_like(w_t)
    (lib or load()).orc_precompress_lr(w_t.size, ctypes.c_float(float(h)), ctypes.c_float(float(b)), _ptr(w_t),
                                       _ptr(w_prev), _ptr(g), _ptr(e), _ptr(u))
    return u


def apply_server_momentum(b, w_t, w_prev, delta, lib=None) -> np.ndarray:
    w_t, w_prev, delta = map(_f32, (w_t, w_prev, delta))
    out = np.empty_like(w_t)
    (lib or load()).orc_apply_server_momentum(w_t.size, ctypes.c_float(float(b)), _ptr(w_t), _ptr(w_prev),
                                              _ptr(delta), _ptr(out))
    return out


# ---------------------------------------------------------------------------
# one GMC iteration for K workers, in the message layout of the device ABI
# ---------------------------------------------------------------------------

class GmcOracle:
    """Algorithm 1 for K simulated workers.

    ``step`` returns the messages in the layout the device library uses:
    ``idx`` int32 [K, index_len] (top-k: element indices; RBGS: block ids),
    ``val`` fp32 [K, message_len], ``msg_len`` int64 [K].  ``err`` ([K, d]) is
    updated in place to e_{t+1,k}.  The step counter t advances by one.
    """

    def __init__(self, d: int, K: int, compressor: str, ratio: float, beta: float, eta: float,
                 seed: int = 0, seg_off=None, block: int = 4096, lib=None, variant: str = "gmc",
                 lam: float = 0.0, stratum: int = 100):
        self.lib = lib or load()
        self.d, self.K, self.compressor = d, K, compressor
        self.ratio = ratio
        self.variant, self.beta, self.lam = variant, beta, lam
        self.set_eta(eta)
        self.seed, self.block, self.t = seed, block, 0
        if seg_off is None:
            seg_off = [0, d]
        self.seg_off = np.ascontiguousarray(seg_off, dtype=np.int64)
        self.stratum = stratum
        if compressor == "rbgs":
            self.nb = (d + block - 1) // block
            self.n_sel = count(self.nb, ratio, self.lib)
            self.index_len = self.n_sel
            self.message_len = self.n_sel * block
        elif compressor == "approx":
            self.index_len = self.message_len = d
        else:
            ks = [count(int(self.seg_off[i + 1] - self.seg_off[i]), ratio, self.lib)
                  for i in range(len(self.seg_off) - 1)]
            self.seg_k = np.array(ks, dtype=np.int64)
            self.index_len = self.message_len = int(sum(ks))

    def set_eta(self, eta: float) -> None:
        """The learning rate of the following iterations (a schedule)."""
        self.eta = eta
        self.c, self.s, self.h = variant_constants(self.variant, self.beta, eta, self.K, self.lib)
        self.q = detach_constant(self.lam, eta, self.lib)

    def precompress(self, w_t, w_prev, g, e) -> np.ndarray:
        if self.variant == "server_momentum":
            return precompress_plain(g, e, self.lib)
        if self.variant == "lr_in_residual":
            return precompress_lr(self.h, self.c, w_t, w_prev, g, e, self.lib)
        return precompress(self.c, w_t, w_prev, g, e, self.lib)

    def step(self, w_t, w_prev, grads, err):
        K, d = self.K, self.d
        idx = np.zeros((K, self.index_len), dtype=np.int32)
        val = np.zeros((K, self.message_len), dtype=np.float32)
        msg_len = np.zeros(K, dtype=np.int64)
        blocks = None
        if self.compressor == "rbgs":
            blocks = rbgs_blocks(self.seed, self.t, self.nb, self.n_sel, self.lib)
        for k in range(K):
            u = self.precompress(w_t, w_prev, grads[k], err[k])
            if self.compressor == "rbgs":
                v = compress_rbgs(u, self.block, blocks, self.lib)
                idx[k, :] = blocks
                val[k, :v.size] = v
                msg_len[k] = v.size
            elif self.compressor == "approx":
                i_k, v_k = compress_approx(u, self.seed, self.t, k, self.stratum, self.ratio, self.lib)
                idx[k, :i_k.size] = i_k
                val[k, :v_k.size] = v_k
                msg_len[k] = v_k.size
            else:
                i_k, v_k = compress_topk(u, self.seg_off, self.ratio, self.lib)
                idx[k, :] = i_k
                val[k, :] = v_k
                msg_len[k] = v_k.size
            err[k, :] = u
        self.t += 1
        return idx, val, msg_len

    def element_indices(self, idx_row: np.ndarray, length: int) -> np.ndarray:
        """Element indices a message row covers (RBGS: expand block ids)."""
        if self.compressor != "rbgs":
            return idx_row[:length].astype(np.int32)
        B = self.block
        parts = [np.arange(b * B, min((b + 1) * B, self.d), dtype=np.int32) for b in np.asarray(idx_row).tolist()]
        return np.concatenate(parts)[:length]

    def aggregate(self, idx, val, msg_len) -> np.ndarray:
        il = [self.element_indices(idx[k], int(msg_len[k])) for k in range(self.K)]
        vl = [val[k, :int(msg_len[k])] for k in range(self.K)]
        return aggregate(self.d, self.s, il, vl, self.lib)

    def apply(self, w: np.ndarray, delta) -> None:
        apply(w, delta, self.lib)

    def next_params(self, w_t, w_prev, delta) -> np.ndarray:
        """w_{t+1} from the server's sum: w_t + delta, or with momentum on
        the server (w_t + delta) + beta (w_t - w_{t-1})."""
        if self.variant == "server_momentum":
            return apply_server_momentum(self.c, w_t, w_prev, delta, self.lib)
        w = _f32(w_t).copy()
        apply(w, delta, self.lib)
        return w

    def detach(self, w_next, err) -> np.ndarray:
        """GMC+'s detached points w_{t+1,k} = w_{t+1} - (lambda eta) e_{t+1,k},
        [K, d] (Algorithm 2)."""
        return np.stack([detach(self.q, w_next, err[k], self.lib) for k in range(self.K)])
