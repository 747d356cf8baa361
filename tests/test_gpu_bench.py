"""bench.py end to end on the GPU, in this process: one JSON line with the
contract's fields for small runs of the tiny, per-tensor, RBGS and
sampled-threshold workloads (the ResNet-50-sized line is the bench's own
default run)."""
import json
import sys

import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.empty_cache()  # the later full-size tests need most of the device memory


@pytest.mark.parametrize("workload,extra", [("tiny", []), ("gpt2", []), ("rbgs", []), ("resnet50_approx", []),
                                            ("gpt2", ["--in-place"])])
def test_bench_line(workload, extra, capsys, monkeypatch):
    import bench
    import synth

    monkeypatch.setattr(sys, "argv", ["bench.py", "--workload", workload, "--steps", "3", "--warmup", "2",
                                      "--no-cpu-baseline"] + extra)
    print("bench line: %s" % workload, file=sys.stderr, flush=True)
    bench.main()
    lines = [ln for ln in capsys.readouterr().out.splitlines() if ln.startswith("{")]
    assert len(lines) == 1, lines
    j = json.loads(lines[0])
    wl = synth.workload(workload)
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "first_step",
                "selection", "hbm_peak_frac"):
        assert key in j, key
    assert j["n_gpus"] == 1 and j["steps"] == 3 and j["warmup"] == 2
    assert j["higher_is_better"] is True and j["dtype"] == "f32" and j["data"] == "synthetic"
    assert j["config"]["d"] == wl.d and j["config"]["K"] == wl.K and "workload" in j["config"]
    # the value is K d worker-elements per step over the host clock's time per step
    assert j["value"] == pytest.approx(wl.K * wl.d / (j["ms_per_step"] * 1e-3) / 1e9, rel=1e-3)
    r = j["roofline"]
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    assert 0.0 < r["frac"] <= 1.0 and r["frac"] == pytest.approx(r["achieved"] / r["peak"], abs=1e-3)
    assert r["kernel"] == ("rbgs_vec_kernel" if wl.compressor == "rbgs" else "topk_fused_vec_kernel")
    if wl.compressor != "rbgs":
        # the plain stream of the pass's pattern: the pass runs at about its
        # speed (cache-resident and launch-bound at the tiny size, where the
        # candidate staging weighs more)
        low = 0.25 if workload == "tiny" else 0.85
        assert low < r["stream_ceiling"]["kernel_time_frac"] <= 1.2, r["stream_ceiling"]
    # iteration 0: thresholds from a sample of u, every global top-s selection
    # resolved from its candidates; the full-data path measured on its own
    first = j["first_step"]
    assert first["ms"] > 0.0
    if wl.compressor == "topk":
        assert first["full_data_selections"] == 0
        assert j["full_data_step"]["full_data_selections"] == wl.K and j["full_data_step"]["ms"] > 0.0
    # the timed steps: sparse momentum term on every step, and the selections
    # resolved from candidates where the workload allows it
    sel = j["selection"]
    assert sel["count_errors"] == 0
    assert j["config"]["in_place"] == ("--in-place" in extra)
    # relative communication cost: messages plus the update's support, over
    # 2 K d; the support is at most the union of the K messages
    c = j["config"]
    assert 0 < c["update_support"] <= wl.K * c["message_len"] + wl.K
    assert c["rcc"] == pytest.approx((wl.K * c["message_len"] + wl.K * c["update_support"]) / (2 * wl.K * wl.d),
                                     rel=0.05)
    assert sel["sparse_momentum_steps"] == 3 and sel["sparse_applies"] == 3
    # the headline fraction takes the dense byte definition; the sparse one beside it
    assert j["alg_bytes_per_step"] == bench.survey_bytes(wl, j["config"]["message_len"], j["config"]["lambda"] > 0)
    assert "alg_bytes_per_step" in j["sparse_accounting"]
    if wl.compressor == "topk":
        assert sel["from_candidates"] == 3 * wl.K and sel["full_data"] == 0
