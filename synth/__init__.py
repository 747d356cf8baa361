"""Seeded synthetic inputs for the GMC hot path.

This package is shared by the device path's tests, the bench and the CPU
oracle's tests: it produces the parameter vector w_0 and the per-worker
stochastic gradients g_{t,k} that stand in for the CIFAR/ImageNet/text
training runs of the paper (Section 5).  It contains none of the method's
arithmetic: no momentum term, no residual, no compressor, no aggregation.

Workloads (flat fp32 parameter vectors shaped like real models):

* ``tiny``      d = 2^20, K = 4, N(0,1) gradients, global top-k 1 %.
* ``resnet18``  d = 11,173,962 in 62 tensors, K = 8, non-IID Gaussian
                gradients with per-tensor log-uniform scales, global top-k 1 %.
* ``resnet50``  d = 25,557,032 in 161 tensors, K = 16, Student-t(3)
                gradients with per-tensor log-uniform scales, global top-k 0.1 %.
* ``rbgs``      d = 25,557,032, K = 8, N(0, 0.01^2) gradients, RBGS over
                4096-element blocks, 1 % of blocks per step.
* ``gpt2``      d = 124,439,808 in 148 tensors, K = 8, Student-t(4)
                gradients, per-tensor top-k 0.1 %.
* ``resnet50_approx``  the ``resnet50`` inputs with the sampled-threshold
                top-s of the experiments (|S| = d/100, rank |S|/1024).

Each workload can be shrunk (``shrink=f``) for oracle-sized parity tests: every
tensor keeps its place in the layout and is divided by ``f`` (at least one
element), which keeps the mix of tensor sizes, the ragged tails and the
distribution while cutting d.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
from dataclasses import dataclass, field, replace
from typing import List, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None

# stream purposes (upper bits of the stream id)
_P_W0, _P_GRAD, _P_SHIFT, _P_SCALE = 1, 2, 3, 4


def build(force: bool = False) -> str:
    """Compile libsynth.so with gcc (OpenMP).  Returns the library path."""
    src = os.path.join(_HERE, "synth.c")
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(src):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", src, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        lib.synth_fill_f32.argtypes = [
            ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int, ctypes.c_int,
            ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
            ctypes.c_double, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]
        lib.synth_fill_f32.restype = None
        lib.synth_uniform_f64.argtypes = [
            ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p]
        lib.synth_uniform_f64.restype = None
        lib.synth_max_threads.argtypes = []
        lib.synth_max_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def _threads() -> int:
    n = os.environ.get("OMP_NUM_THREADS")
    if n and n.isdigit():
        return max(1, int(n))
    return max(1, min(16, os.cpu_count() or 1))


# ----------------------------------------------------------------------------
# model-shaped tensor tables (shape arithmetic of the named architectures)
# ----------------------------------------------------------------------------

def resnet18_cifar_sizes() -> List[int]:
    """CIFAR ResNet-18: 3x3 stem, 4 stages x 2 BasicBlocks, 1x1 projection in
    the first block of stages 2-4, BN weight+bias after each conv, 10-way fc."""
    s = [3 * 3 * 3 * 64, 64, 64]
    cin = 64
    for stage, w in enumerate([64, 128, 256, 512]):
        for b in range(2):
            s += [9 * cin * w, w, w, 9 * w * w, w, w]
            if b == 0 and stage > 0:
                s += [cin * w, w, w]
            cin = w
    s += [512 * 10, 10]
    return s


def resnet50_sizes() -> List[int]:
    """ImageNet ResNet-50: 7x7 stem, bottlenecks [3,4,6,3], downsample in each
    stage's first block, 1000-way fc."""
    s = [7 * 7 * 3 * 64, 64, 64]
    cin = 64
    for nblocks, w in zip([3, 4, 6, 3], [64, 128, 256, 512]):
        for b in range(nblocks):
            s += [cin * w, w, w, 9 * w * w, w, w, w * 4 * w, 4 * w, 4 * w]
            if b == 0:
                s += [cin * 4 * w, 4 * w, 4 * w]
            cin = 4 * w
    s += [2048 * 1000, 1000]
    return s


def gpt2_small_sizes() -> List[int]:
    """12-layer, 768-wide decoder, vocabulary 50257, 1024 positions."""
    h, v, p = 768, 50257, 1024
    s = [v * h, p * h]
    for _ in range(12):
        s += [h, h, h * 3 * h, 3 * h, h * h, h, h, h, h * 4 * h, 4 * h, 4 * h * h, h]
    s += [h, h]
    return s


@dataclass
class Workload:
    name: str
    sizes: List[int]            # tensor sizes, contiguous in the flat vector
    K: int
    ratio: float                # top-k fraction per segment, or RBGS block fraction
    beta: float
    eta: float
    steps: int
    compressor: str             # "topk" | "topk_seg" | "rbgs"
    dist: str                   # "normal" | "student_t"
    nu: int = 0
    scale_lo: float = 1.0       # per-tensor log-uniform scale range
    scale_hi: float = 1.0
    grad_std: float = 1.0       # global std multiplier (rbgs: 1e-2)
    shift_frac: float = 0.0     # non-IID fixed per-worker mean shift, std = frac*scale
    w0_std: float = 0.01
    block: int = 4096
    seed: int = 0
    shrink: int = 1

    @property
    def d(self) -> int:
        return int(sum(self.sizes))

    def seg_off(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(np.asarray(self.sizes, dtype=np.int64))]).astype(np.int64)

    def topk_segments(self) -> np.ndarray:
        """Segment table the compressor works on: the whole vector for global
        top-k and RBGS, one segment per tensor for per-tensor top-k."""
        if self.compressor == "topk_seg":
            return self.seg_off()
        return np.array([0, self.d], dtype=np.int64)

    def shrunk(self, f: int, steps: Optional[int] = None, K: Optional[int] = None) -> "Workload":
        sizes = [max(1, int(math.ceil(x / f))) for x in self.sizes]
        return replace(self, sizes=sizes, shrink=self.shrink * f,
                       steps=self.steps if steps is None else steps,
                       K=self.K if K is None else K)

    # -------------------------------------------------------------- tensors
    def scales(self) -> np.ndarray:
        """Per-tensor gradient scale, log-uniform in [scale_lo, scale_hi],
        drawn once (independent of t and k)."""
        n = len(self.sizes)
        if self.scale_lo == self.scale_hi:
            return np.full(n, self.scale_lo * self.grad_std, dtype=np.float64)
        u = np.empty(n, dtype=np.float64)
        _load().synth_uniform_f64(self.seed, _P_SCALE << 48, 0, n, u.ctypes.data)
        lo, hi = math.log(self.scale_lo), math.log(self.scale_hi)
        return np.exp(lo + u * (hi - lo)) * self.grad_std

    def w0(self) -> np.ndarray:
        out = np.empty(self.d, dtype=np.float32)
        off = np.array([0, self.d], dtype=np.int64)
        sc = np.array([self.w0_std], dtype=np.float64)
        _load().synth_fill_f32(self.seed, _P_W0 << 48, 0, 0, self.d, 1, off.ctypes.data,
                               sc.ctypes.data, 0.0, None, out.ctypes.data, _threads())
        return out

    def _shift(self, k: int, scales: np.ndarray) -> Optional[np.ndarray]:
        if self.shift_frac == 0.0:
            return None
        out = np.empty(self.d, dtype=np.float32)
        off = self.seg_off()
        sc = np.ascontiguousarray(scales * self.shift_frac)
        _load().synth_fill_f32(self.seed, (_P_SHIFT << 48) | k, 0, 0, self.d, len(self.sizes),
                               off.ctypes.data, sc.ctypes.data, 0.0, None, out.ctypes.data, _threads())
        return out

    def grad(self, t: int, k: int, out: Optional[np.ndarray] = None) -> np.ndarray:
        """g_{t,k} as fp32 [d]: scale_i * X (+ the worker's fixed shift)."""
        if out is None:
            out = np.empty(self.d, dtype=np.float32)
        scales = self.scales()
        shift = self._shift(k, scales)
        off = self.seg_off()
        dist = 1 if self.dist == "student_t" else 0
        _load().synth_fill_f32(self.seed, (_P_GRAD << 48) | (t << 16) | k, dist, self.nu,
                               self.d, len(self.sizes), off.ctypes.data,
                               np.ascontiguousarray(scales).ctypes.data, 0.0,
                               None if shift is None else shift.ctypes.data,
                               out.ctypes.data, _threads())
        return out

    def grads(self, t: int) -> np.ndarray:
        """All K gradients of step t as fp32 [K, d]."""
        out = np.empty((self.K, self.d), dtype=np.float32)
        for k in range(self.K):
            self.grad(t, k, out=out[k])
        return out


WORKLOADS = {
    "tiny": Workload("tiny", [1 << 20], K=4, ratio=0.01, beta=0.9, eta=0.1, steps=5,
                     compressor="topk", dist="normal"),
    "resnet18": Workload("resnet18", resnet18_cifar_sizes(), K=8, ratio=0.01, beta=0.9,
                         eta=0.1, steps=20, compressor="topk", dist="normal",
                         scale_lo=1e-4, scale_hi=1e-1, shift_frac=0.1),
    "resnet50": Workload("resnet50", resnet50_sizes(), K=16, ratio=0.001, beta=0.9,
                         eta=0.1, steps=20, compressor="topk", dist="student_t", nu=3,
                         scale_lo=1e-5, scale_hi=1e-1),
    "rbgs": Workload("rbgs", resnet50_sizes(), K=8, ratio=0.01, beta=0.9, eta=0.1,
                     steps=20, compressor="rbgs", dist="normal", grad_std=1e-2, block=4096),
    "gpt2": Workload("gpt2", gpt2_small_sizes(), K=8, ratio=0.001, beta=0.9, eta=0.05,
                     steps=10, compressor="topk_seg", dist="student_t", nu=4,
                     scale_lo=1e-5, scale_hi=1e-2),
    # the ResNet-50-sized step with the experiments' sampled-threshold top-s
    # (|S| = d/100, threshold at rank |S|/1024)
    "resnet50_approx": Workload("resnet50_approx", resnet50_sizes(), K=16, ratio=1 / 1024, beta=0.9,
                                eta=0.1, steps=20, compressor="approx", dist="student_t", nu=3,
                                scale_lo=1e-5, scale_hi=1e-1),
}

EXPECTED_D = {"tiny": 1048576, "resnet18": 11173962, "resnet50": 25557032,
              "rbgs": 25557032, "gpt2": 124439808, "resnet50_approx": 25557032}


def workload(name: str) -> Workload:
    return WORKLOADS[name]
