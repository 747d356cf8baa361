"""Device library vs the CPU oracle, element by element, on the same seeded
inputs: every workload shape (shrunk so the oracle finishes in seconds while
still spanning many chunks, items and ragged tails), both selection paths,
misaligned rows and the degenerate cases of the method."""
import dataclasses
import math

import numpy as np
import pytest

import oracle
import synth
from gpu_harness import Case, run_lockstep

pytestmark = pytest.mark.gpu

OPT_FULL, OPT_MARGIN, OPT_CAP = 1, 2, 3
OPT_LIST = 7     # GMC_OPT_CHANGE_LIST


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def W(name):
    return synth.workload(name)


def test_tiny_full_size():
    st = run_lockstep(Case(W("tiny"), steps=5, label="tiny"))
    # step 0 takes its thresholds from a sample of u, later steps from the
    # previous selection: every selection resolves from candidates
    assert st["full_data"] == 0 and st["from_candidates"] == 5 * 4, st


def test_sampled_first_threshold_falls_back_on_ties():
    # every gradient of the first step equal: the sample puts the threshold at
    # the floor of their key's bin, every component is a candidate, more than
    # the capacity holds, and the first step takes the full-data path
    def flat_first(t, g):
        return np.ones_like(g) if t == 0 else g
    st = run_lockstep(Case(W("resnet18").shrunk(16, K=4), steps=3, grad_hook=flat_first, label="flat first step"))
    assert st["full_data"] >= 4, st


def test_resnet18_shape_shrunk():
    run_lockstep(Case(W("resnet18").shrunk(16), steps=4, label="resnet18/16"))


def test_resnet50_shape_shrunk():
    run_lockstep(Case(W("resnet50").shrunk(32), steps=4, label="resnet50/32"))


def test_rbgs_shrunk():
    run_lockstep(Case(W("rbgs").shrunk(16), steps=5, label="rbgs/16"))


def test_gpt2_per_tensor_shrunk():
    run_lockstep(Case(W("gpt2").shrunk(64), steps=3, label="gpt2/64"))


def test_forced_full_data_path():
    st = run_lockstep(Case(W("resnet50").shrunk(32, K=6), steps=3, options=((OPT_FULL, 1),),
                           label="full-data"))
    assert st["from_candidates"] == 0


def test_candidate_overflow_takes_full_data_path():
    st = run_lockstep(Case(W("resnet18").shrunk(16, K=4), steps=4,
                           options=((OPT_CAP, 1), (OPT_MARGIN, 256)), label="overflow"))
    assert st["full_data"] > 0


def test_long_candidate_lists_stride_the_copy_launch():
    # margin 16 k: the candidate lists run to several times the 8 k + 2048 the
    # copy and selection launches are sized for (within the 64 k capacity),
    # so the copy workgroups stride over the extra tiles and the slices run long
    wl = W("resnet18").shrunk(16, K=4)
    k = oracle.count(wl.d, wl.ratio)
    st = run_lockstep(Case(wl, steps=4, options=((OPT_MARGIN, 64),), label="long lists"))
    assert st["from_candidates"] >= 2 * wl.K
    assert st["candidates"] / st["from_candidates"] > 8 * k + 2048


def test_misaligned_rows():
    wl = synth.Workload("odd", [5000, 3, 77777, 2048 * 3 + 1], K=3, ratio=0.01, beta=0.9, eta=0.1,
                        steps=3, compressor="topk_seg", dist="normal")
    run_lockstep(Case(wl, steps=3, row_pad=1, label="misaligned"))


def test_no_compression_is_momentum_sgd():
    wl = synth.Workload("dense", [1000, 24], K=1, ratio=1.0, beta=0.9, eta=0.1, steps=3,
                        compressor="topk", dist="normal")
    run_lockstep(Case(wl, steps=3, label="ratio=1,K=1"))
    wl = synth.Workload("dense4", [4099], K=4, ratio=1.0, beta=0.5, eta=0.3, steps=3,
                        compressor="topk", dist="normal")
    run_lockstep(Case(wl, steps=3, label="ratio=1,K=4"))


@pytest.mark.parametrize("sizes,K,ratio", [([1], 3, 0.5), ([3], 2, 0.5), ([2, 1, 5], 2, 0.3),
                                           ([2048], 1, 1e-6), ([2049], 2, 0.999)])
def test_degenerate_sizes(sizes, K, ratio):
    wl = synth.Workload("small", sizes, K=K, ratio=ratio, beta=0.9, eta=0.1, steps=3,
                        compressor="topk_seg", dist="normal")
    run_lockstep(Case(wl, steps=3, label="small%s" % sizes))


def test_heavy_ties_lowest_index_wins():
    def quantise(t, g):
        return np.sign(np.round(g)).astype(np.float32)          # values in {-1, 0, 1}
    wl = W("tiny").shrunk(8)
    run_lockstep(Case(wl, steps=4, grad_hook=quantise, label="ties"))


def test_all_zero_gradients():
    wl = W("tiny").shrunk(32, K=2)
    run_lockstep(Case(wl, steps=2, grad_hook=lambda t, g: np.zeros_like(g), label="zeros"))


def test_infinities_rank_first():
    def inject(t, g):
        if t == 1:
            g = g.copy()
            g[0, [5, 900]] = np.inf
            g[1, 17] = -np.inf
        return g
    wl = W("tiny").shrunk(64, K=2)
    run_lockstep(Case(wl, steps=2, grad_hook=inject, label="inf"))


def test_rbgs_partial_last_block_and_small_blocks():
    wl = synth.Workload("rb", [10000 + 1234], K=3, ratio=0.5, beta=0.9, eta=0.1, steps=6,
                        compressor="rbgs", dist="normal", block=1000)
    run_lockstep(Case(wl, steps=6, label="rbgs-partial"))
    wl = synth.Workload("rb7", [999], K=2, ratio=0.3, beta=0.9, eta=0.1, steps=3,
                        compressor="rbgs", dist="normal", block=7)
    run_lockstep(Case(wl, steps=3, label="rbgs-block7"))


def test_rbgs_more_blocks_than_the_lds_bitmap():
    # 275,000 blocks of 4: the block draw keeps its bitmap in global memory
    # (the workgroup's LDS holds 262,144 blocks)
    wl = synth.Workload("rb4", [1_100_000], K=2, ratio=0.01, beta=0.9, eta=0.1, steps=3,
                        compressor="rbgs", dist="normal", block=4)
    st = run_lockstep(Case(wl, steps=3, fused_apply=True, sparse_w=True, label="rbgs 275k blocks"))
    assert st["sparse_applies"] == 2, st


def test_sparse_messages_with_one_dense_range():
    # 200 one-component tensors (k = 1 each) fill the first range, ten large
    # tensors follow: on average 15 message entries per range, so the server
    # pass stages few entries per range, while the first range holds more
    # than 600 and is summed worker after worker from the messages
    wl = synth.Workload("dense-first", [1] * 200 + [100_000] * 10, K=3, ratio=0.001, beta=0.9, eta=0.1, steps=3,
                        compressor="topk_seg", dist="normal")
    run_lockstep(Case(wl, steps=3, label="one dense range"))
    st = run_lockstep(Case(wl, steps=3, iteration=True, sparse_w=True, label="one dense range, iteration"))
    assert st["sparse_applies"] == 2, st


def test_many_workers_and_a_margin_beyond_the_capacity():
    # K = 64, the most workers a context takes; a margin of 200 k puts the
    # speculative threshold so low that the candidates overflow the 64 k
    # capacity and the pairs take the full-data path
    wl = W("resnet50").shrunk(256, K=64)
    run_lockstep(Case(wl, steps=3, options=((OPT_MARGIN, 800),), label="K=64"))


@pytest.mark.parametrize("name,shrink,steps", [("resnet50", 32, 4), ("rbgs", 16, 4), ("gpt2", 64, 3)])
def test_fused_aggregate_apply_swapping_buffers(name, shrink, steps):
    run_lockstep(Case(W(name).shrunk(shrink), steps=steps, fused_apply=True, label="fused/" + name))


def test_fused_aggregate_apply_without_update():
    run_lockstep(Case(W("resnet18").shrunk(16, K=4), steps=3, fused_apply=True, write_update=False,
                      label="fused-no-update"))


# ---------------------------------------------------------------------------
# GMC+ detached points (Algorithm 2), the appendix's update rules, eta schedule
# ---------------------------------------------------------------------------

def _cosine(eta, T):
    return lambda t: eta * 0.5 * (1 + math.cos(math.pi * t / T))


@pytest.mark.parametrize("name,shrink,K", [("rbgs", 16, 8), ("resnet18", 16, 4), ("gpt2", 64, 3)])
def test_gmcplus_fused_detach(name, shrink, K):
    run_lockstep(Case(W(name).shrunk(shrink, K=K), steps=4, lam=0.5, detach="fused",
                      label="gmc+ fused/" + name))


def test_gmcplus_fused_detach_misaligned_rows():
    run_lockstep(Case(W("resnet18").shrunk(32, K=3), steps=3, lam=0.3, detach="fused", row_pad=1,
                      label="gmc+ fused misaligned"))


def test_gmcplus_fused_detach_full_data_path():
    run_lockstep(Case(W("resnet50").shrunk(64, K=4), steps=3, lam=1.0, detach="fused",
                      options=((OPT_FULL, 1),), label="gmc+ fused full-data"))


@pytest.mark.parametrize("rule", ["gmc", "server_momentum", "lr_in_residual"])
def test_dense_detach(rule):
    run_lockstep(Case(W("rbgs").shrunk(16, K=4), steps=3, lam=0.5, detach="dense", rule=rule,
                      label="dense detach/" + rule))


@pytest.mark.parametrize("name,shrink", [("resnet18", 16), ("rbgs", 16), ("gpt2", 64)])
def test_server_momentum_rule(name, shrink):
    run_lockstep(Case(W(name).shrunk(shrink, K=4), steps=4, rule="server_momentum",
                      label="server momentum/" + name))


@pytest.mark.parametrize("name,shrink", [("resnet50", 32), ("rbgs", 16)])
def test_lr_in_residual_rule(name, shrink):
    run_lockstep(Case(W(name).shrunk(shrink, K=6), steps=4, rule="lr_in_residual",
                      label="lr in residual/" + name))


def test_lr_in_residual_with_fused_detach():
    run_lockstep(Case(W("resnet18").shrunk(16, K=4), steps=3, rule="lr_in_residual", lam=0.5,
                      detach="fused", label="lr in residual + detach"))


@pytest.mark.parametrize("name,shrink,rule", [("resnet18", 16, "gmc"), ("rbgs", 16, "gmc"),
                                              ("resnet18", 16, "lr_in_residual")])
def test_eta_schedule(name, shrink, rule):
    wl = W(name).shrunk(shrink, K=4)
    run_lockstep(Case(wl, steps=5, rule=rule, eta_fn=_cosine(wl.eta, 6), label="cosine eta/" + name))


# ---------------------------------------------------------------------------
# the experiments' sampled-threshold top-s (Section 5.1)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("shrink,K,stratum", [(16, 4, 100), (64, 6, 7), (256, 3, 1)])
def test_sampled_threshold_topk(shrink, K, stratum):
    st = run_lockstep(Case(W("resnet50_approx").shrunk(shrink, K=K), steps=5, stratum=stratum,
                           label="approx/%d" % stratum))
    assert st["from_candidates"] > 0, st


def test_sampled_threshold_full_data_path():
    run_lockstep(Case(W("resnet50_approx").shrunk(32, K=4), steps=3, options=((OPT_FULL, 1),),
                      label="approx full-data"))


def test_sampled_threshold_ties_and_zeros():
    wl = dataclasses.replace(W("resnet50_approx").shrunk(64, K=3), ratio=0.01)
    quantise = lambda t, g: (np.round(g * 4) / 4).astype(np.float32)
    run_lockstep(Case(wl, steps=3, grad_hook=quantise, stratum=10, label="approx ties"))
    run_lockstep(Case(wl, steps=2, grad_hook=lambda t, g: np.zeros_like(g), label="approx zeros"))


def test_sampled_threshold_gmcplus_and_rules():
    wl = W("resnet50_approx").shrunk(64, K=4)
    run_lockstep(Case(wl, steps=3, lam=0.5, detach="fused", label="approx gmc+"))
    run_lockstep(Case(wl, steps=3, rule="server_momentum", label="approx server momentum"))


# ---------------------------------------------------------------------------
# argument and call-order errors answered before any kernel runs
# ---------------------------------------------------------------------------

def test_rule_and_compressor_errors():
    import torch
    from paper_1905_12948_amd import Gmc, GmcError, GMC_OPT_SAMPLE_STRATUM
    dev = torch.device("cuda:0")
    d, K = 4096, 2
    w = torch.zeros(d, device=dev)
    rows = torch.zeros((K, d), device=dev)
    g = Gmc(d, K, "topk", 0.01, 0.9, 0.1, rule="server_momentum")
    idx, val, ln = g.alloc_messages(dev)
    with pytest.raises(GmcError):
        g.step(w, w.clone(), rows, rows.clone(), idx, val, ln, w_k=rows.clone())   # detach needs w_{t+1} = w_t
    with pytest.raises(GmcError):
        g.aggregate_apply(idx, val, ln, w, w.clone())                              # needs w_{t-1}
    with pytest.raises(GmcError):
        g.apply(w, w.clone())
    with pytest.raises(GmcError):
        g.finish(idx, val, ln, w, w.clone())                                       # w_prev missing
    with pytest.raises(GmcError):
        g.set_option(GMC_OPT_SAMPLE_STRATUM, 10)                                   # not the sampled threshold
    with pytest.raises(GmcError):
        g.set_lambda(1.5)
    with pytest.raises(GmcError):
        g.set_eta(0.0)
    g.close()
    a = Gmc(d, K, "approx", 1 / 1024, 0.9, 0.1)
    with pytest.raises(GmcError):
        a._call(a._lib.gmc_set_segments(a._ctx, 2, (__import__("ctypes").c_int64 * 3)(0, 10, d)))
    with pytest.raises(GmcError):
        a.set_option(GMC_OPT_SAMPLE_STRATUM, 0)
    assert a.message_len == d and a.index_len == d
    a.close()



# ---------------------------------------------------------------------------
# GMC_OPT_SPARSE_MOMENTUM: w read only where the last server pass changed it
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name,shrink,K,extra", [
    ("resnet18", 16, 4, {}), ("resnet50", 32, 16, {}), ("rbgs", 16, 8, {}), ("gpt2", 64, 3, {}),
    ("resnet50_approx", 64, 4, {}), ("rbgs", 16, 4, {"lam": 0.5, "detach": "fused"}),
    ("resnet18", 16, 4, {"lam": 0.5, "detach": "fused"}), ("resnet18", 16, 4, {"rule": "lr_in_residual"}),
    ("resnet18", 32, 3, {"row_pad": 1}), ("resnet18", 16, 4, {"rule": "server_momentum"}),
    # 8 workers sending 1% each: the changed components are dense enough that
    # the worker pass puts each chunk's workers on one XCD
    ("resnet18", 16, 8, {}), ("tiny", 4, 8, {"rule": "lr_in_residual"})])
def test_sparse_momentum_is_bitwise_the_dense_path(name, shrink, K, extra):
    st = run_lockstep(Case(W(name).shrunk(shrink, K=K), steps=5, fused_apply=True, sparse_w=True,
                           label="sparse momentum/" + name, **extra))
    if extra.get("rule") != "server_momentum":
        assert st["sparse_momentum_steps"] == 4, st   # every step after the first
        assert st["sparse_applies"] == 4, st          # and its server pass


@pytest.mark.parametrize("name,shrink", [("resnet18", 32), ("rbgs", 16)])
def test_sparse_momentum_with_non_finite_parameters(name, shrink):
    # non-finite parameters outside the sent components stay marked; the RBGS
    # server pass then visits every range instead of the drawn blocks' ranges
    def poison(w0):
        w0 = w0.copy()
        w0[[5, 777, 4096, 9000]] = [np.inf, -np.inf, np.nan, np.inf]
        return w0
    st = run_lockstep(Case(W(name).shrunk(shrink, K=3), steps=4, fused_apply=True, sparse_w=True,
                           w0_hook=poison, label="sparse momentum, non-finite w/" + name))
    assert st["sparse_momentum_steps"] == 3, st
    assert st["sparse_applies"] == 3, st


def test_rbgs_sparse_apply_with_partial_and_small_blocks():
    # the RBGS server pass visits only the ranges of this step's and the last
    # step's blocks: blocks of 1000 (several per range, a partial last one)
    # and of 7 components, half and a third of them drawn
    for wl in (synth.Workload("rb", [10000 + 1234], K=3, ratio=0.5, beta=0.9, eta=0.1, steps=5,
                              compressor="rbgs", dist="normal", block=1000),
               synth.Workload("rb7", [999], K=2, ratio=0.3, beta=0.9, eta=0.1, steps=5,
                              compressor="rbgs", dist="normal", block=7)):
        st = run_lockstep(Case(wl, steps=5, fused_apply=True, sparse_w=True, label="rbgs sparse/" + wl.name))
        assert st["sparse_applies"] == 4, st


def test_sparse_momentum_falls_back_when_the_buffers_change():
    st = run_lockstep(Case(W("resnet18").shrunk(32, K=3), steps=4, sparse_w=True, label="sparse momentum, apply"))
    assert st["sparse_momentum_steps"] == 0, st   # gmc_aggregate + gmc_apply: no bitmap
    assert st["sparse_applies"] == 0, st



# ---------------------------------------------------------------------------
# gmc_iteration: the whole iteration in one call, the dense copy of the apply
# overlapped with the selection under the sparse momentum term
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name,shrink,K,extra", [
    ("resnet18", 16, 4, {"sparse_w": True}), ("resnet50", 32, 16, {"sparse_w": True}),
    ("gpt2", 64, 3, {"sparse_w": True}), ("resnet50_approx", 64, 4, {"sparse_w": True}),
    ("resnet18", 16, 4, {"sparse_w": True, "rule": "lr_in_residual"}),
    ("resnet18", 32, 3, {"sparse_w": True, "row_pad": 1}), ("rbgs", 16, 4, {"sparse_w": True}),
    ("resnet18", 16, 4, {}), ("resnet18", 16, 4, {"rule": "server_momentum", "sparse_w": True}),
    ("resnet18", 16, 8, {"sparse_w": True})])
def test_iteration_matches_the_oracle(name, shrink, K, extra):
    st = run_lockstep(Case(W(name).shrunk(shrink, K=K), steps=5, iteration=True, label="iteration/" + name, **extra))
    if extra.get("sparse_w") and extra.get("rule") != "server_momentum":
        assert st["sparse_momentum_steps"] == 4, st
        assert st["sparse_applies"] == 4, st


def test_iteration_with_non_finite_parameters():
    def poison(w0):
        w0 = w0.copy()
        w0[[5, 777, 4096, 9000]] = [np.inf, -np.inf, np.nan, np.inf]
        return w0
    st = run_lockstep(Case(W("resnet18").shrunk(32, K=3), steps=4, iteration=True, sparse_w=True, w0_hook=poison,
                           label="iteration, non-finite w"))
    assert st["sparse_applies"] == 3, st


@pytest.mark.parametrize("iteration", [True, False])
def test_server_pass_ranges_beyond_the_wave_stage(iteration):
    """Sparse messages on average, but clustered: the largest gradients all
    sit in the first 12288 components, so the first three 4096-component
    ranges hold every worker's whole message (thousands of entries, more
    than the one-wavefront server pass stages) while the other ranges hold
    none.  Those ranges take the block kernel after the one-wavefront pass;
    every output against the oracle."""
    wl = synth.Workload("clustered", [1 << 22], K=4, ratio=0.002, beta=0.9, eta=0.1, steps=4,
                        compressor="topk", dist="normal")

    def cluster(t, g):
        g = g.copy()
        g[:, :12288] *= np.float32(1000.0)
        return g
    run_lockstep(Case(wl, steps=4, grad_hook=cluster, iteration=iteration, fused_apply=not iteration,
                      sparse_w=True, label="clustered messages"))


@pytest.mark.parametrize("name,shrink,K,extra", [
    ("resnet18", 16, 4, {}), ("resnet50", 32, 16, {}), ("gpt2", 64, 3, {}), ("resnet50_approx", 64, 4, {}),
    ("resnet18", 16, 4, {"rule": "lr_in_residual"}), ("resnet18", 32, 3, {"row_pad": 1}),
    ("resnet18", 16, 8, {})])
def test_change_list_is_bitwise_the_dense_path(name, shrink, K, extra):
    """The worker pass's momentum term from the server pass's change list
    (forced on at these sizes), with gmc_iteration and with
    gmc_aggregate_apply: every output against the oracle."""
    for iteration in (True, False):
        st = run_lockstep(Case(W(name).shrunk(shrink, K=K), steps=5, iteration=iteration, fused_apply=not iteration,
                               sparse_w=True, options=((OPT_LIST, 1),), label="change list/" + name, **extra))
        assert st["sparse_momentum_steps"] == 4 and st["sparse_applies"] == 4, st


def test_change_list_overflow_and_non_finite():
    """Change lists that overflow (the clustered ranges send every component)
    and non-finite parameters (listed with w_t - w_t = NaN): the worker pass
    takes the marks and the parameter vectors for those ranges."""
    wl = synth.Workload("clustered", [1 << 22], K=4, ratio=0.002, beta=0.9, eta=0.1, steps=4,
                        compressor="topk", dist="normal")

    def cluster(t, g):
        g = g.copy()
        g[:, :12288] *= np.float32(1000.0)
        return g

    def poison(w0):
        w0 = w0.copy()
        w0[[5, 777, 4096, 9000, 3 << 20]] = [np.inf, -np.inf, np.nan, np.inf, np.nan]
        return w0
    run_lockstep(Case(wl, steps=4, grad_hook=cluster, iteration=True, sparse_w=True, w0_hook=poison,
                      options=((OPT_LIST, 1),), label="change list, clustered + non-finite"))
