"""gmc_aggregate_static, the entry point that allocates nothing, against
gmc_aggregate through the C ABI: the same top-s messages (from a worker pass
of a context) give the same update bit for bit, on two calls in a row, the
second with a smaller problem (fewer components and workers), so the second
call reads row pointers the first call's larger layout left in the static
scratch only where it wrote them itself."""
import numpy as np
import pytest

import synth
from gpu_harness import assert_same_f32

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _messages(wl, steps=2):
    """A context's messages after `steps` worker passes, and the context."""
    import torch
    from paper_1905_12948_amd import Gmc
    dev = torch.device("cuda:0")
    seg = wl.topk_segments()
    g = Gmc(wl.d, wl.K, wl.compressor, wl.ratio, wl.beta, wl.eta, seed=wl.seed,
            segments=seg.tolist() if wl.compressor == "topk_seg" else None)
    w = torch.from_numpy(wl.w0()).to(dev)
    wp = w.clone()
    err = torch.zeros((wl.K, wl.d), device=dev)
    idx, val, ln = g.alloc_messages(dev)
    for t in range(steps):
        g.step(w, wp, torch.from_numpy(wl.grads(t)).to(dev), err, idx, val, ln)
    return g, idx, val, ln


def test_static_aggregate_matches_the_context_aggregate():
    import torch
    from paper_1905_12948_amd.gmc import aggregate_static
    dev = torch.device("cuda:0")
    cases = [synth.workload("gpt2").shrunk(16, K=6),        # per-tensor top-s, many ranges
             synth.workload("resnet18").shrunk(64, K=3),    # smaller d, fewer workers
             synth.workload("resnet50_approx").shrunk(128, K=2)]  # messages of varying length
    for wl in cases:
        g, idx, val, ln = _messages(wl)
        want = torch.empty(wl.d, dtype=torch.float32, device=dev)
        got = torch.full((wl.d,), float("nan"), dtype=torch.float32, device=dev)
        g.aggregate(idx, val, ln, want)
        aggregate_static(wl.d, wl.K, wl.eta, idx, val, ln, got)
        torch.cuda.synchronize()
        print("static aggregate %s: d=%d K=%d" % (wl.name, wl.d, wl.K), flush=True)
        assert_same_f32(got.cpu().numpy(), want.cpu().numpy(), "static aggregate, %s d=%d K=%d" % (wl.name, wl.d, wl.K))
        # a second call on the same messages, into a fresh buffer
        got2 = torch.full((wl.d,), float("nan"), dtype=torch.float32, device=dev)
        aggregate_static(wl.d, wl.K, wl.eta, idx, val, ln, got2)
        torch.cuda.synchronize()
        assert_same_f32(got2.cpu().numpy(), want.cpu().numpy(), "static aggregate again, %s" % wl.name)
        g.close()
