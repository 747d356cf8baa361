"""The same run twice gives the same bits: two fresh contexts take the same
workload at its full size from the same inputs over several iterations, and
every output (messages, message lengths, residuals, both parameter buffers)
is compared bit for bit on the device after each one.  The selection uses
device-scope atomics (candidate counts, histogram merges, last-workgroup
hand-offs) whose order varies from run to run; none of it may reach a
result.  Also with the parameters updated in place, and RBGS with GMC+'s
detached points."""
import pytest

import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _bits(x):
    import torch
    return x.contiguous().view(torch.int32) if x.dtype == torch.float32 else x


def _run(wl, steps, inplace):
    import torch
    import synth.device as sdev
    from paper_1905_12948_amd import Gmc, GMC_OPT_SPARSE_MOMENTUM, GMC_OPT_CHANGE_LIST
    dev = torch.device("cuda:0")
    d, K = wl.d, wl.K
    seg = wl.topk_segments().tolist() if wl.compressor == "topk_seg" else None
    lam = 0.5 if wl.compressor == "rbgs" else 0.0
    g = Gmc(d, K, wl.compressor, wl.ratio, wl.beta, wl.eta, seed=wl.seed, segments=seg,
            block=wl.block if wl.compressor == "rbgs" else None, lam=lam)
    g.set_option(GMC_OPT_SPARSE_MOMENTUM, 1)
    if inplace:
        g.set_option(GMC_OPT_CHANGE_LIST, 3)
    w = sdev.w0(wl, dev)
    wp = w.clone()
    err = sdev.rows(K, d, dev, zero=True)
    wk = sdev.rows(K, d, dev) if lam else None
    idx, val, ln = g.alloc_messages(dev)
    snaps = []
    for t in range(steps):
        gr = sdev.grads(wl, t, dev)
        if inplace:
            g.iteration_inplace(w, w if t == 0 else None, gr, err, idx, val, ln)
        elif lam:
            g.step(w, wp, gr, err, idx, val, ln, w_k=wk)
            g.finish(idx, val, ln, w, wp, err=err, w_k=wk)
            w, wp = wp, w
        else:
            g.iteration(w, wp, gr, err, idx, val, ln)
            w, wp = wp, w
        torch.cuda.synchronize()
        # a digest per step keeps the memory small: the sums of the bit
        # patterns of every output, in int64, plus the full message
        snap = {"ln": ln.clone(), "idx": idx.clone(), "val": _bits(val).clone()}
        for name, x in (("e", err), ("w", w), ("wp", wp)) + ((("wk", wk),) if wk is not None else ()):
            b = _bits(x).to(torch.int64)
            snap[name] = torch.stack([b.sum(), (b * (torch.arange(b.numel(), device=dev).view(b.shape) % 9973 + 1)).sum()])
        snaps.append(snap)
    st = g.stats()
    g.close()
    assert st["count_errors"] == 0, st
    return snaps


@pytest.mark.parametrize("name,steps,inplace", [("resnet50", 4, False), ("resnet18", 4, False), ("gpt2", 3, False),
                                                ("gpt2", 3, True), ("resnet50_approx", 3, False), ("rbgs", 4, False)])
def test_same_run_twice(name, steps, inplace):
    import torch
    wl = synth.workload(name)
    print("determinism %s: d=%d K=%d steps=%d in place=%s" % (name, wl.d, wl.K, steps, inplace), flush=True)
    a = _run(wl, steps, inplace)
    b = _run(wl, steps, inplace)
    for t, (x, y) in enumerate(zip(a, b)):
        for key in x:
            assert torch.equal(x[key], y[key]), "%s step %d: %s differs between two runs" % (name, t, key)
