"""Seeded random shapes against the oracle, every output bit for bit over
three steps: global, per-tensor (random tensor splits, ragged sizes),
sampled-threshold top-s and RBGS (random block lengths), random K, ratios from
1e-4 to 1, random beta and eta, normal or heavy-tailed gradients, quantised
gradients (ties), misaligned rows, and each call pattern (gmc_step with
gmc_aggregate and gmc_apply, gmc_aggregate_apply and gmc_iteration with the
sparse momentum term, the in-place iteration).  Case i is reproducible from
its seed alone."""
import os

import numpy as np
import pytest

import synth
from gpu_harness import Case, run_lockstep

pytestmark = pytest.mark.gpu

COMPRESSORS = ("topk", "topk_seg", "approx", "rbgs")
# GMC_RANDOM_CASES widens the sweep for a longer run
N_CASES = int(os.environ.get("GMC_RANDOM_CASES", "96"))
FIRST_CASE = int(os.environ.get("GMC_RANDOM_FIRST", "0"))  # a later block of the same sequence
OPT_LIST = 7


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def random_case(i: int) -> Case:
    rng = np.random.default_rng(7919 * (i + 1))
    comp = COMPRESSORS[i % len(COMPRESSORS)]
    big = rng.random() < 0.3   # several compaction groups and selection slices per pair
    if comp == "topk_seg":
        sizes = [int(x) for x in rng.integers(1, 400000 if big else 40000, size=int(rng.integers(1, 12)))]
    else:
        sizes = [int(rng.integers(1, 3000000 if big else 300000))]
    K = int(rng.integers(1, 10))
    ratio = float(rng.choice([1.0, 0.999, 0.5, 0.1, 0.03, 0.01, 0.003, 0.001, 1e-4]))
    dist = str(rng.choice(["normal", "student_t"]))
    wl = synth.Workload("rand%d" % i, sizes, K=K, ratio=ratio, beta=float(rng.uniform(0.0, 0.95)),
                        eta=float(10 ** rng.uniform(-3, 0)), steps=3, compressor=comp, dist=dist,
                        nu=3 if dist == "student_t" else 0, block=int(rng.choice([1, 7, 64, 1000, 4096])),
                        seed=i)
    if comp == "rbgs":
        # a block is at most d long; the oracle draws its blocks with a plain
        # quadratic membership test: keep the drawn blocks to at most 20,000
        wl.block = min(wl.block, wl.d)
        while wl.ratio * -(-wl.d // wl.block) > 20000 and wl.block < wl.d:
            wl.block = min(wl.block * 8, wl.d)
    kw = {}
    pattern = int(rng.integers(0, 4))
    if pattern == 1:
        kw.update(fused_apply=True, sparse_w=True)
    elif pattern == 2:
        kw.update(iteration=True, sparse_w=True)
    elif pattern == 3 and comp != "rbgs":
        kw.update(inplace="iteration", sparse_w=True, options=((OPT_LIST, 3),))
    if rng.random() < 0.25:
        kw["row_pad"] = 1
    if rng.random() < 0.25:
        kw["grad_hook"] = lambda t, g: np.round(g * 2.0).astype(np.float32)   # heavy ties and zeros
    return Case(wl, steps=3, label="random %d (%s, d=%d, K=%d, ratio=%g, pattern %d)"
                % (i, comp, wl.d, K, ratio, pattern), **kw)


@pytest.mark.parametrize("i", range(FIRST_CASE, FIRST_CASE + N_CASES))
def test_random_shape(i):
    run_lockstep(random_case(i), verbose=False)
