"""Lock-step runner: the device library (through the C ABI) and the CPU
oracle take the same seeded inputs, step by step, and every output is
compared element by element."""
from __future__ import annotations

import sys
from dataclasses import dataclass
from typing import Callable, Optional

import numpy as np

import oracle
import synth


def bits(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


def assert_same_f32(got: np.ndarray, want: np.ndarray, what: str, rel=1e-6, abs_=1e-7):
    """Bit-for-bit equality expected by construction (same binary32
    operations in the same order on both sides); on a mismatch the message
    also says whether the looser 1e-6 relative / 1e-7 absolute bound holds."""
    g, w = bits(got).reshape(-1).copy(), bits(want).reshape(-1).copy()
    # a NaN result compares equal to any NaN (payloads are not specified)
    nan_g = (g & 0x7FFFFFFF) > 0x7F800000
    nan_w = (w & 0x7FFFFFFF) > 0x7F800000
    both = nan_g & nan_w
    g[both] = w[both]
    if np.array_equal(g, w):
        return
    bad = np.nonzero(g != w)[0]
    gf, wf = got.reshape(-1)[bad], want.reshape(-1)[bad]
    within = np.all(np.abs(gf - wf) <= abs_ + rel * np.abs(wf))
    raise AssertionError("%s: %d of %d elements differ (first at %d: got %r want %r); within 1e-6/1e-7: %s"
                         % (what, bad.size, g.size, bad[0], gf[0], wf[0], within))


@dataclass
class Case:
    wl: synth.Workload
    steps: int
    options: tuple = ()           # (option, value) pairs for gmc_set_option
    row_pad: int = 0              # extra floats between worker rows (misaligned rows)
    grad_hook: Optional[Callable] = None   # (t, grads) -> grads, host side
    label: str = ""
    fused_apply: bool = False     # gmc_aggregate_apply out of place, buffers swapped
    write_update: bool = True     # with fused_apply / finish: also materialise the update
    rule: str = "gmc"             # update rule (gmc, server_momentum, lr_in_residual)
    lam: float = 0.0              # GMC+ detach coefficient
    detach: str = ""              # "fused": gmc_step_detach + gmc_finish; "dense": gmc_detach
    eta_fn: Optional[Callable] = None      # t -> eta_t (a schedule)
    finish: bool = False          # server pass through gmc_finish (implied by rule / detach)
    stratum: int = 100            # sampled-threshold top-s: components per sample stratum
    sparse_w: bool = False        # GMC_OPT_SPARSE_MOMENTUM
    w0_hook: Optional[Callable] = None     # w0 -> w0, host side
    iteration: bool = False       # gmc_iteration (worker and server pass in one call, buffers swapped)
    # one parameter buffer updated in place: "iteration" (gmc_iteration_inplace)
    # or "apply" (gmc_step, then gmc_aggregate_apply with w_out = w); w_prev is
    # w itself at t = 0 and NULL after
    inplace: str = ""


def run_lockstep(case: Case, device="cuda:0", check_every=1, verbose=True):
    import torch
    from paper_1905_12948_amd import Gmc

    wl = case.wl
    d, K = wl.d, wl.K
    comp = wl.compressor
    seg = wl.topk_segments() if comp == "topk_seg" else None
    if verbose:
        print("lockstep %s: d=%d K=%d %s ratio=%g steps=%d opts=%s pad=%d rule=%s lam=%g detach=%s"
              % (case.label or wl.name, d, K, comp, wl.ratio, case.steps, case.options, case.row_pad,
                 case.rule, case.lam, case.detach or "-"), flush=True)
    g = Gmc(d, K, comp, wl.ratio, wl.beta, wl.eta, seed=wl.seed,
            segments=None if seg is None else seg.tolist(),
            block=wl.block if comp == "rbgs" else None, rule=case.rule, lam=case.lam,
            stratum=case.stratum if comp == "approx" else None)
    for opt, val in case.options:
        g.set_option(opt, val)
    if case.sparse_w:
        from paper_1905_12948_amd import GMC_OPT_SPARSE_MOMENTUM
        g.set_option(GMC_OPT_SPARSE_MOMENTUM, 1)
    orc = oracle.GmcOracle(d, K, comp if comp in ("rbgs", "approx") else "topk", wl.ratio, wl.beta, wl.eta,
                           seed=wl.seed, seg_off=seg, block=wl.block, variant=case.rule, lam=case.lam,
                           stratum=case.stratum)
    use_finish = case.finish or case.rule != "gmc" or bool(case.detach)
    assert g.message_len == orc.message_len and g.index_len == orc.index_len

    dev = torch.device(device)
    w0 = wl.w0()
    if case.w0_hook is not None:
        w0 = case.w0_hook(w0)
    w_h, wp_h = w0.copy(), w0.copy()
    e_h = np.zeros((K, d), np.float32)
    stride = d + case.row_pad
    w = torch.from_numpy(w0).to(dev)
    wp = w.clone()
    e_store = torch.zeros(K * stride + 1, dtype=torch.float32, device=dev)
    g_store = torch.zeros(K * stride + 1, dtype=torch.float32, device=dev)
    off = 1 if case.row_pad else 0       # odd start: 4-byte but not 16-byte aligned rows
    e_rows = [e_store[off + k * stride: off + k * stride + d] for k in range(K)]
    g_rows = [g_store[off + k * stride: off + k * stride + d] for k in range(K)]
    wk_rows = None
    if case.detach:
        y_store = torch.full((K * stride + 1,), float("nan"), dtype=torch.float32, device=dev)
        wk_rows = [y_store[off + k * stride: off + k * stride + d] for k in range(K)]
    idx, val, ln = g.alloc_messages(dev)
    upd = torch.empty(d, dtype=torch.float32, device=dev)
    for t in range(case.steps):
        gr = wl.grads(t)
        if case.grad_hook is not None:
            gr = case.grad_hook(t, gr)
        for k in range(K):
            g_rows[k].copy_(torch.from_numpy(gr[k]))
        if case.eta_fn is not None:
            eta_t = case.eta_fn(t)
            g.set_eta(eta_t)
            orc.set_eta(eta_t)
        fused_detach = case.detach == "fused"
        if case.inplace:
            w_prev_arg = w if t == 0 else None   # w_{-1} = w_0, then the context's record
            if case.inplace == "iteration":
                g.iteration_inplace(w, w_prev_arg, g_rows, e_rows, idx, val, ln)
            else:
                g.step(w, w_prev_arg, g_rows, e_rows, idx, val, ln)
                g.aggregate_apply(idx, val, ln, w, w, update=upd if case.write_update else None)
        elif case.iteration:
            g.iteration(w, wp, g_rows, e_rows, idx, val, ln)
            w, wp = wp, w
        else:
            g.step(w, wp, g_rows, e_rows, idx, val, ln, w_k=wk_rows if fused_detach else None)
        if case.iteration or case.inplace:
            pass
        elif use_finish:
            g.finish(idx, val, ln, w, wp, w_prev=wp, update=upd if case.write_update else None,
                     err=e_rows if fused_detach else None, w_k=wk_rows if fused_detach else None)
            w, wp = wp, w
            if case.detach == "dense":
                g.detach(w, e_rows, wk_rows)
        elif case.fused_apply:
            g.aggregate_apply(idx, val, ln, w, wp, update=upd if case.write_update else None)
            w, wp = wp, w
        else:
            g.aggregate(idx, val, ln, upd)
            g.apply(w, upd, w_prev_out=wp)

        oi, ov, ol = orc.step(w_h, wp_h, gr, e_h)
        od = orc.aggregate(oi, ov, ol)
        wn = orc.next_params(w_h, wp_h, od)
        wp_h, w_h = w_h, wn
        wk_h = orc.detach(w_h, e_h) if case.detach else None
        if (t + 1) % check_every and t != case.steps - 1:
            continue
        torch.cuda.synchronize()
        tag = "%s step %d" % (case.label or wl.name, t)
        assert np.array_equal(ln.cpu().numpy(), ol), tag + ": message lengths"
        gi = idx.cpu().numpy()
        if comp == "approx":  # variable-length rows: compare the written part
            gi = np.where(np.arange(gi.shape[1])[None, :] < ol[:, None], gi, 0)
            oi = np.where(np.arange(oi.shape[1])[None, :] < ol[:, None], oi, 0)
        if not np.array_equal(gi, oi):
            bad = np.argwhere(gi != oi)
            raise AssertionError("%s: indices differ at %d places, first %s (got %d want %d)"
                                 % (tag, len(bad), bad[0], gi[tuple(bad[0])], oi[tuple(bad[0])]))
        gv = val.cpu().numpy()
        for k in range(K):
            m = int(ol[k])
            assert_same_f32(gv[k, :m], ov[k, :m], tag + ": values of worker %d" % k)
            assert_same_f32(e_rows[k].cpu().numpy(), e_h[k], tag + ": residual of worker %d" % k)
        if not case.iteration and case.inplace != "iteration" and \
                (case.write_update or not (case.fused_apply or use_finish or case.inplace)):
            assert_same_f32(upd.cpu().numpy(), od, tag + ": update")
        assert_same_f32(w.cpu().numpy(), w_h, tag + ": w")
        if not case.inplace:  # in place there is no second buffer
            assert_same_f32(wp.cpu().numpy(), wp_h, tag + ": w_prev")
        if case.detach:
            for k in range(K):
                assert_same_f32(wk_rows[k].cpu().numpy(), wk_h[k], tag + ": detached point of worker %d" % k)
        if verbose:
            print("  %s ok" % tag, flush=True)
    st = g.stats()
    g.close()
    assert st["count_errors"] == 0, st
    return st
