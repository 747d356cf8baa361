"""The workloads at their full sizes, in the launch configuration the bench
times (gmc_iteration with the sparse momentum term: the worker pass, then the
server pass writing w_{t+1} over w_{t-1}'s buffer, the two parameter buffers
swapping roles; GMC+ takes gmc_step_detach then gmc_finish), checked against
the oracle's per-element functions and the defining property of exact top-k
(a full CPU sort of every worker's vector would take minutes).  One case
keeps the dense path (gmc_step, then gmc_aggregate_apply writing the update
vector too).

For each step and two of the K workers (the first and the last):
  * u (recomputed by the oracle from the step's inputs) equals e_{t+1} off
    the sent components bit for bit, the sent values bit for bit, and the
    residual there is u - u;
  * per segment the message holds exactly k components, ascending, whose
    keys are the k largest with ties broken towards the lower index (the
    sampled-threshold top-s: exactly the oracle's selection on the same u);
w_{t+1} (and the update vector, where written) is compared with the oracle's
aggregation of all K messages and its apply, for every component.  Step 0
takes the full-data selection path and the dense parameter path, later steps
the candidate path and, with the sparse momentum term, read and write the
parameters only where they change.  With lambda > 0 the two workers'
detached points are compared with the oracle's too."""
import numpy as np
import pytest

import oracle
import synth
from gpu_harness import assert_same_f32

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def keys_of(a: np.ndarray) -> np.ndarray:
    return a.view(np.uint32) & np.uint32(0x7FFFFFFF)


def check_topk_segment(u: np.ndarray, sel: np.ndarray, k: int, tag: str):
    """sel (ascending, global-to-segment offsets) is the top-k of u by key,
    lowest index first among equal keys."""
    assert sel.size == k, tag + ": count"
    assert np.all(np.diff(sel) > 0), tag + ": not ascending"
    assert sel[0] >= 0 and sel[-1] < u.size, tag + ": out of range"
    key = keys_of(u)
    ks = key[sel]
    T = ks.min()
    mask = np.zeros(u.size, bool)
    mask[sel] = True
    rest = key[~mask]
    assert rest.size == 0 or rest.max() <= T, tag + ": an unsent component outranks the threshold"
    tie_sel = sel[ks == T]
    tie_rest = np.nonzero((~mask) & (key == T))[0]
    if tie_rest.size and tie_sel.size:
        assert tie_sel.max() < tie_rest.min(), tag + ": ties not broken towards the lower index"


@pytest.mark.parametrize("name,steps,lam,dense", [
    ("tiny", 3, 0.0, False), ("resnet18", 3, 0.0, False), ("resnet50", 3, 0.0, False), ("rbgs", 3, 0.0, False),
    ("gpt2", 3, 0.0, False), ("rbgs", 3, 0.5, False), ("resnet50", 2, 0.5, False),
    ("resnet50_approx", 3, 0.0, False), ("resnet50", 2, 0.0, True)])
def test_full_size_workload(name, steps, lam, dense):
    import torch
    import synth.device as sdev
    from paper_1905_12948_amd import Gmc, GMC_OPT_SPARSE_MOMENTUM

    wl = synth.workload(name)
    d, K = wl.d, wl.K
    dev = torch.device("cuda:0")
    rbgs = wl.compressor == "rbgs"
    approx = wl.compressor == "approx"
    seg = wl.topk_segments()
    g = Gmc(d, K, wl.compressor, wl.ratio, wl.beta, wl.eta, seed=wl.seed,
            segments=seg.tolist() if wl.compressor == "topk_seg" else None,
            block=wl.block if rbgs else None, lam=lam)
    orc = oracle.GmcOracle(d, K, wl.compressor if (rbgs or approx) else "topk", wl.ratio, wl.beta, wl.eta,
                           seed=wl.seed, seg_off=seg, block=wl.block, lam=lam)
    if not dense:
        g.set_option(GMC_OPT_SPARSE_MOMENTUM, 1)
    print("full size %s: d=%d K=%d %s lambda=%g %s" % (name, d, K, wl.compressor, lam,
                                                    "dense" if dense else "sparse momentum"), flush=True)
    bufs = [sdev.w0(wl, dev), None]
    bufs[1] = bufs[0].clone()
    err = sdev.rows(K, d, dev, zero=True)
    idx, val, ln = g.alloc_messages(dev)
    wk = sdev.rows(K, d, dev) if lam else None
    upd = torch.empty(d, dtype=torch.float32, device=dev)
    check = [0, K - 1]
    for t in range(steps):
        grads = sdev.grads(wl, t, dev)
        cur, prev = bufs[t % 2], bufs[(t + 1) % 2]
        w_h, wp_h = cur.cpu().numpy(), prev.cpu().numpy()
        e_before = {k: err[k].cpu().numpy() for k in check}
        if lam:
            g.step(cur, prev, grads, err, idx, val, ln, w_k=wk)
            g.finish(idx, val, ln, cur, prev, err=err, w_k=wk)
        elif dense:
            g.step(cur, prev, grads, err, idx, val, ln)
            g.aggregate_apply(idx, val, ln, cur, prev, update=upd)
        else:
            g.iteration(cur, prev, grads, err, idx, val, ln)
        torch.cuda.synchronize()
        gi, gv, gl = idx.cpu().numpy(), val.cpu().numpy(), ln.cpu().numpy()
        if rbgs:
            blocks = oracle.rbgs_blocks(wl.seed, t, orc.nb, orc.n_sel)
            assert all(np.array_equal(gi[k], blocks) for k in range(K)), "RBGS blocks"
            m = sum(min((b + 1) * wl.block, d) - b * wl.block for b in blocks)
            assert np.all(gl == m), "message lengths"
        elif not approx:
            assert np.all(gl == orc.message_len), "message lengths"
        for k in check:
            tag = "%s step %d worker %d" % (name, t, k)
            u = orc.precompress(w_h, wp_h, grads[k].cpu().numpy(), e_before[k])
            e_after = err[k].cpu().numpy()
            sent = orc.element_indices(gi[k], int(gl[k]))
            assert_same_f32(gv[k, :int(gl[k])], u[sent], tag + ": sent values")
            assert_same_f32(e_after[sent], u[sent] - u[sent], tag + ": residual at sent components")
            rest = np.ones(d, bool)
            rest[sent] = False
            assert_same_f32(e_after[rest], u[rest], tag + ": residual elsewhere")
            if approx:  # the sampled threshold: the oracle's selection on the same u
                oi_k, ov_k = oracle.compress_approx(u.copy(), wl.seed, t, k, orc.stratum, wl.ratio)
                assert np.array_equal(sent.astype(np.int64), oi_k.astype(np.int64)), tag + ": kept set"
                assert_same_f32(gv[k, :int(gl[k])], ov_k, tag + ": kept values")
            elif not rbgs:
                for s_i in range(len(orc.seg_off) - 1):
                    a, b = int(orc.seg_off[s_i]), int(orc.seg_off[s_i + 1])
                    sel = sent[(sent >= a) & (sent < b)] - a
                    check_topk_segment(u[a:b], sel, int(orc.seg_k[s_i]), tag + " segment %d" % s_i)
        delta = orc.aggregate(gi, gv, gl)
        if dense:
            assert_same_f32(upd.cpu().numpy(), delta, "%s step %d: update" % (name, t))
        w_next = w_h.copy()
        orc.apply(w_next, delta)
        assert_same_f32(prev.cpu().numpy(), w_next, "%s step %d: w_{t+1}" % (name, t))
        if lam:
            for k in check:
                want = oracle.detach(orc.q, w_next, err[k].cpu().numpy())
                assert_same_f32(wk[k].cpu().numpy(), want, "%s step %d: detached point of worker %d" % (name, t, k))
        print("  step %d ok (%s)" % (t, g.stats()), flush=True)
        del grads
    st = g.stats()
    g.close()
    if not dense:  # every step after the first moved the parameters only where they change
        assert st["sparse_momentum_steps"] == steps - 1 and st["sparse_applies"] == steps - 1, st
