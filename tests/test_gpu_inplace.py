"""Parameters updated in place (one buffer instead of two): the server pass
writes w_{t+1} over w_t and keeps w_{t+1} - w_t as its change list, from
which the next worker pass takes the momentum term of Algorithm 1 with
w_prev = NULL.  Every output against the oracle, step by step: global,
per-tensor (partial chunks, element-wise path) and sampled-threshold top-s,
the learning-rate-in-residual rule, misaligned rows (the element-wise
kernel), non-finite parameters, ranges whose every component changes; and
the call-order errors of the mode."""
import numpy as np
import pytest

import synth
from gpu_harness import Case, run_lockstep

pytestmark = pytest.mark.gpu

OPT_SPARSE, OPT_LIST = 6, 7
GMC_EINVAL, GMC_ESTATE = -1, -4
FULL_LIST = ((OPT_LIST, 3),)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def W(name):
    return synth.workload(name)


@pytest.mark.parametrize("name,shrink,K,extra", [
    ("resnet18", 16, 4, {}), ("resnet50", 32, 16, {}), ("gpt2", 64, 3, {}), ("resnet50_approx", 64, 4, {}),
    ("tiny", 4, 4, {}), ("resnet18", 16, 4, {"rule": "lr_in_residual"}), ("resnet18", 16, 8, {})])
@pytest.mark.parametrize("mode", ["iteration", "apply"])
def test_inplace_matches_the_oracle(name, shrink, K, extra, mode):
    st = run_lockstep(Case(W(name).shrunk(shrink, K=K), steps=5, inplace=mode, sparse_w=True, options=FULL_LIST,
                           label="in place (%s)/%s" % (mode, name), **extra))
    # every worker pass after the first takes the list, every server pass
    # after the first writes only the sent words
    assert st["sparse_momentum_steps"] == 4 and st["sparse_applies"] == 4, st


def test_inplace_misaligned_rows_and_ragged_segments():
    # rows one float off 16-byte alignment (the element-wise kernel, one
    # wavefront per chunk) and segments that start mid-chunk
    wl = synth.Workload("odd", [5000, 3, 77777, 2048 * 3 + 1], K=3, ratio=0.01, beta=0.9, eta=0.1,
                        steps=4, compressor="topk_seg", dist="normal")
    st = run_lockstep(Case(wl, steps=4, row_pad=1, inplace="iteration", sparse_w=True, options=FULL_LIST,
                           label="in place, misaligned"))
    assert st["sparse_momentum_steps"] == 3, st
    st = run_lockstep(Case(wl, steps=4, inplace="apply", sparse_w=True, options=FULL_LIST,
                           label="in place, ragged segments"))
    assert st["sparse_momentum_steps"] == 3, st


def test_inplace_non_finite_parameters():
    """Non-finite parameters from the start and from an infinite gradient at
    step 1: once a pass writes a non-finite w the in-place passes also visit
    the previous marks, so the non-finite components stay listed (with the
    NaN momentum term the two vectors would give)."""
    def poison(w0):
        w0 = w0.copy()
        w0[[5, 777, 4096, 9000]] = [np.inf, -np.inf, np.nan, np.inf]
        return w0

    def inject(t, g):
        if t == 1:
            g = g.copy()
            g[0, [33, 5000]] = np.inf
            g[1, 17] = -np.inf
        return g
    run_lockstep(Case(W("resnet18").shrunk(32, K=3), steps=5, inplace="iteration", sparse_w=True,
                      options=FULL_LIST, w0_hook=poison, label="in place, non-finite w"))
    run_lockstep(Case(W("resnet18").shrunk(32, K=3), steps=5, inplace="apply", sparse_w=True,
                      options=FULL_LIST, grad_hook=inject, label="in place, infinite gradient"))


def test_inplace_whole_ranges_change():
    """Clustered messages: the first three 4096-component ranges hold every
    worker's whole message, so every component of those ranges changes and
    their lists are full."""
    wl = synth.Workload("clustered", [1 << 22], K=4, ratio=0.002, beta=0.9, eta=0.1, steps=4,
                        compressor="topk", dist="normal")

    def cluster(t, g):
        g = g.copy()
        g[:, :12288] *= np.float32(1000.0)
        return g
    st = run_lockstep(Case(wl, steps=4, grad_hook=cluster, inplace="iteration", sparse_w=True, options=FULL_LIST,
                           label="in place, clustered"))
    assert st["sparse_applies"] == 3, st


def test_inplace_call_order():
    import torch
    from paper_1905_12948_amd import Gmc, GmcError
    wl = W("resnet18").shrunk(32, K=3)
    d, K = wl.d, wl.K
    dev = torch.device("cuda:0")
    grads = [torch.from_numpy(wl.grads(t)).to(dev) for t in range(3)]

    def expect(status, call):
        with pytest.raises(GmcError) as ei:
            call()
        assert ei.value.status == status, ei.value

    g = Gmc(d, K, "topk", wl.ratio, wl.beta, wl.eta, seed=wl.seed)
    w = torch.from_numpy(wl.w0()).to(dev)
    err = torch.zeros((K, d), device=dev)
    idx, val, ln = g.alloc_messages(dev)
    # the in-place iteration needs the sparse momentum term and whole-range lists
    expect(GMC_EINVAL, lambda: g.iteration_inplace(w, w, grads[0], err, idx, val, ln))
    g.set_option(OPT_SPARSE, 1)
    expect(GMC_EINVAL, lambda: g.iteration_inplace(w, w, grads[0], err, idx, val, ln))
    g.set_option(OPT_LIST, 3)
    # no record yet: w_prev = NULL is out of order
    expect(GMC_ESTATE, lambda: g.step(w, None, grads[0], err, idx, val, ln))
    expect(GMC_ESTATE, lambda: g.iteration_inplace(w, None, grads[0], err, idx, val, ln))
    assert g.t == 0
    g.iteration_inplace(w, w, grads[0], err, idx, val, ln)
    g.iteration_inplace(w, None, grads[1], err, idx, val, ln)
    # the whole-range list is fixed once stepping has started
    expect(GMC_ESTATE, lambda: g.set_option(OPT_LIST, 1))
    # dropping the record (setting the option again): w_prev = NULL is out of
    # order until the next in-place pass
    g.set_option(OPT_SPARSE, 1)
    expect(GMC_ESTATE, lambda: g.iteration_inplace(w, None, grads[2], err, idx, val, ln))
    assert g.t == 2
    torch.cuda.synchronize()
    g.close()
    # RBGS has no in-place mode
    gr = Gmc(10000, 2, "rbgs", 0.01, 0.9, 0.1, block=1000)
    gr.set_option(OPT_SPARSE, 1)
    expect(GMC_ESTATE, lambda: gr.set_option(OPT_LIST, 3) or gr.step(
        torch.zeros(10000, device=dev), None, torch.zeros((2, 10000), device=dev), torch.zeros((2, 10000), device=dev),
        *gr.alloc_messages(dev)))
    gr.close()


def test_inplace_checkpoint_resume():
    """The save/resume procedure of the in-place mode: the last iteration
    before the save runs its server pass out of place (gmc_step with w_prev =
    NULL, gmc_aggregate_apply into a second buffer), so the caller holds
    w_{t-1} and w_t; a fresh context restored with gmc_set_step continues in
    place from them.  Eight iterations so equal eight uninterrupted in-place
    iterations bit for bit, and the oracle's."""
    import torch
    from paper_1905_12948_amd import Gmc
    from gpu_harness import assert_same_f32
    import oracle
    wl = W("gpt2").shrunk(64, K=3)
    d, K = wl.d, wl.K
    seg = wl.topk_segments()
    dev = torch.device("cuda:0")
    grads = [torch.from_numpy(wl.grads(t)).to(dev) for t in range(8)]

    def ctx():
        g = Gmc(d, K, "topk_seg", wl.ratio, wl.beta, wl.eta, seed=wl.seed, segments=seg.tolist())
        g.set_option(OPT_SPARSE, 1)
        g.set_option(OPT_LIST, 3)
        return g

    # uninterrupted
    ga = ctx()
    wa = torch.from_numpy(wl.w0()).to(dev)
    ea = torch.zeros((K, d), device=dev)
    ia, va, la = ga.alloc_messages(dev)
    for t in range(8):
        ga.iteration_inplace(wa, wa if t == 0 else None, grads[t], ea, ia, va, la)
    torch.cuda.synchronize()
    # four in place, the fifth with its server pass out of place, save
    gb = ctx()
    wb = torch.from_numpy(wl.w0()).to(dev)
    eb = torch.zeros((K, d), device=dev)
    ib, vb, lb = gb.alloc_messages(dev)
    for t in range(4):
        gb.iteration_inplace(wb, wb if t == 0 else None, grads[t], eb, ib, vb, lb)
    w_next = torch.empty_like(wb)
    gb.step(wb, None, grads[4], eb, ib, vb, lb)
    gb.aggregate_apply(ib, vb, lb, wb, w_next)
    torch.cuda.synchronize()
    saved = dict(t=gb.t, w_prev=wb.cpu().clone(), w=w_next.cpu().clone(), e=eb.cpu().clone())
    gb.close()
    assert saved["t"] == 5
    # resume in a fresh context, in place
    gc = ctx()
    gc.t = saved["t"]
    wc = saved["w"].to(dev)
    wpc = saved["w_prev"].to(dev)
    ec = saved["e"].to(dev)
    ic, vc, lc = gc.alloc_messages(dev)
    for t in range(5, 8):
        gc.iteration_inplace(wc, wpc if t == 5 else None, grads[t], ec, ic, vc, lc)
    torch.cuda.synchronize()
    assert_same_f32(wc.cpu().numpy(), wa.cpu().numpy(), "resumed in place: w")
    assert_same_f32(ec.cpu().numpy(), ea.cpu().numpy(), "resumed in place: residuals")
    assert torch.equal(ic, ia) and torch.equal(lc, la)
    # and the oracle's
    orc = oracle.GmcOracle(d, K, "topk", wl.ratio, wl.beta, wl.eta, seed=wl.seed, seg_off=seg)
    w_h, wp_h = wl.w0(), wl.w0()
    e_h = np.zeros((K, d), np.float32)
    for t in range(8):
        oi, ov, ol = orc.step(w_h, wp_h, wl.grads(t), e_h)
        wn = orc.next_params(w_h, wp_h, orc.aggregate(oi, ov, ol))
        wp_h, w_h = w_h, wn
    assert_same_f32(wa.cpu().numpy(), w_h, "in place: w_8 against the oracle")
    assert_same_f32(ea.cpu().numpy(), e_h, "in place: e_8 against the oracle")
    for g in (ga, gc):
        assert g.stats()["count_errors"] == 0
        g.close()


@pytest.mark.parametrize("sizes,K,ratio", [([1], 3, 0.5), ([3], 2, 0.5), ([2, 1, 5], 2, 0.3), ([2048], 1, 1e-6),
                                           ([2049], 2, 0.999), ([4096 * 3 + 5, 1, 4093], 3, 0.05)])
def test_inplace_degenerate_sizes(sizes, K, ratio):
    # one-component segments, d = 1, a chunk's last partial range, ranges
    # that a segment boundary splits; every worker sends nearly every
    # component in the 0.999 case, so whole ranges change
    wl = synth.Workload("small", sizes, K=K, ratio=ratio, beta=0.9, eta=0.1, steps=4,
                        compressor="topk_seg", dist="normal")
    run_lockstep(Case(wl, steps=4, inplace="iteration", sparse_w=True, options=FULL_LIST,
                      label="in place small%s" % sizes))
