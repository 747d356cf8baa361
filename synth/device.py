"""Device-side generation of the workloads' gradients for the bench.

Same recipe as the host generator (per-tensor log-uniform scales drawn by the
host generator, Gaussian or Student-t built from nu+1 normals, fixed
per-worker mean shifts for the non-IID workload), drawn with torch's seeded
GPU generator so that gigabytes of fresh gradients cost milliseconds.  The
values are not bit-identical to the host generator's: parity tests use the
host generator; the bench only needs the shapes and distributions.
"""
from __future__ import annotations

import torch

from . import Workload


def _scale_vector(wl: Workload, device) -> torch.Tensor:
    scales = torch.tensor(wl.scales(), dtype=torch.float64)
    sizes = torch.tensor(wl.sizes, dtype=torch.int64)
    return torch.repeat_interleave(scales, sizes).to(device=device, dtype=torch.float32)


def _draw(wl: Workload, shape, gen) -> torch.Tensor:
    dev = gen.device
    if wl.dist == "student_t":
        z0 = torch.randn(shape, generator=gen, device=dev, dtype=torch.float32)
        chi = torch.zeros(shape, device=dev, dtype=torch.float32)
        for _ in range(wl.nu):
            z = torch.randn(shape, generator=gen, device=dev, dtype=torch.float32)
            chi.addcmul_(z, z)
        return z0.div_(chi.div_(float(wl.nu)).sqrt_())
    return torch.randn(shape, generator=gen, device=dev, dtype=torch.float32)


ROW_ALIGN = 32   # floats: 128 bytes, one cache line


def rows(K: int, d: int, device, zero: bool = False) -> torch.Tensor:
    """A [K, d] fp32 view whose rows start on 128-byte boundaries (row pitch
    rounded up to a multiple of 32 floats), the layout of K per-worker
    buffers packed into one allocation."""
    pitch = (d + ROW_ALIGN - 1) // ROW_ALIGN * ROW_ALIGN
    buf = (torch.zeros if zero else torch.empty)((K, pitch), dtype=torch.float32, device=device)
    return buf[:, :d]


def grads(wl: Workload, t: int, device, out: torch.Tensor = None) -> torch.Tensor:
    """g_{t,k} for all K workers as fp32 [K, d] on `device` (by default in
    the line-aligned row layout of `rows`)."""
    device = torch.device(device)
    gen = torch.Generator(device=device)
    gen.manual_seed((wl.seed * 1_000_003 + 7919 * (t + 1)) & 0x7FFFFFFFFFFFFFFF)
    if out is None:
        out = rows(wl.K, wl.d, device)
    scale = _scale_vector(wl, device)
    for k in range(wl.K):
        x = _draw(wl, (wl.d,), gen)
        x.mul_(scale)
        if wl.shift_frac:
            sg = torch.Generator(device=device)
            sg.manual_seed((wl.seed * 1_000_003 + 104729 * (k + 1)) & 0x7FFFFFFFFFFFFFFF)
            x.add_(torch.randn((wl.d,), generator=sg, device=device, dtype=torch.float32)
                   .mul_(scale * wl.shift_frac))
        out[k].copy_(x)
    return out


def w0(wl: Workload, device) -> torch.Tensor:
    gen = torch.Generator(device=torch.device(device))
    gen.manual_seed((wl.seed * 1_000_003 + 1) & 0x7FFFFFFFFFFFFFFF)
    return torch.randn((wl.d,), generator=gen, device=device, dtype=torch.float32).mul_(wl.w0_std)
