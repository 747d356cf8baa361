"""The C-ABI library loads and exports every entry point include/gmc.h
declares; argument checks answer before any device work (no GPU needed)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gmc.h")


def declared():
    with open(HEADER) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gmc_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    from paper_1905_12948_amd import gmc
    if not os.path.exists(gmc.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return gmc.load()


def test_header_lists_the_binding_exports():
    from paper_1905_12948_amd import EXPORTS
    assert declared() == sorted(EXPORTS)


def test_every_declared_symbol_is_exported(lib):
    for name in declared():
        assert hasattr(lib, name), name


@pytest.mark.parametrize("args,needle", [
    ((0, 4, 0, 0.01, 0.9, 0.1), "d must"),
    ((1 << 31, 4, 0, 0.01, 0.9, 0.1), "d must"),
    ((100, 0, 0, 0.01, 0.9, 0.1), "K must"),
    ((100, 65, 0, 0.01, 0.9, 0.1), "K must"),
    ((100, 4, 7, 0.01, 0.9, 0.1), "compressor"),
    ((100, 4, 0, 0.0, 0.9, 0.1), "ratio"),
    ((100, 4, 0, 1.5, 0.9, 0.1), "ratio"),
    ((100, 4, 0, float("nan"), 0.9, 0.1), "ratio"),
    ((100, 4, 0, 0.01, 1.0, 0.1), "beta"),
    ((100, 4, 0, 0.01, -0.1, 0.1), "beta"),
    ((100, 4, 0, 0.01, 0.9, 0.0), "eta"),
    ((100, 4, 0, 0.01, 0.9, float("inf")), "eta"),
])
def test_init_rejects_bad_arguments(lib, args, needle):
    ctx = ctypes.c_void_p(1234)
    st = lib.gmc_init(ctypes.byref(ctx), *args, 0)
    assert st == -1
    assert ctx.value is None
    assert needle in lib.gmc_last_error(None).decode()


def test_null_handles(lib):
    assert lib.gmc_init(None, 100, 4, 0, 0.01, 0.9, 0.1, 0) == -1
    assert lib.gmc_message_len(None) == -1
    assert lib.gmc_index_len(None) == -1
    assert lib.gmc_step(None, None, None, None, None, None, None, None) == -1
    assert lib.gmc_aggregate(None, None, None, None, None) == -1
    assert lib.gmc_apply(None, None, None, None) == -1
    assert lib.gmc_set_segments(None, 1, None) == -1
    assert lib.gmc_set_block(None, 4) == -1
    assert lib.gmc_set_option(None, 1, 1) == -1
    assert lib.gmc_set_rule(None, 0) == -1
    assert lib.gmc_set_eta(None, 0.1) == -1
    assert lib.gmc_set_lambda(None, 0.5) == -1
    assert lib.gmc_step_detach(None, None, None, None, None, None, None, None, None) == -1
    assert lib.gmc_finish(None, None, None, None, None, None, None, None, None, None) == -1
    assert lib.gmc_detach(None, None, None, None) == -1
    assert lib.gmc_iteration(None, None, None, None, None, None, None, None) == -1
    assert isinstance(lib.gmc_last_error(None), bytes)
    lib.gmc_destroy(None)


def test_binding_rejects_wrong_tensors_before_device_work():
    torch = pytest.importorskip("torch")
    from paper_1905_12948_amd.gmc import _check
    with pytest.raises(TypeError):
        _check(torch.zeros(4, dtype=torch.float64), torch.float32)
    with pytest.raises(ValueError):
        _check(torch.zeros(4, dtype=torch.float32), torch.float32)   # not on a GPU


def test_count_rule_matches_the_oracle(lib):
    """gmc_count (the library's host count rule) against the oracle's
    orc_count: the workloads' counts, products that binary64 lands just
    above an integer (7% of 100 and 300), power-of-two and decimal ratios,
    a ratio no small fraction gives, and the clamps."""
    import numpy as np
    import oracle
    from paper_1905_12948_amd import count
    assert count(100, 0.07) == 7 and count(300, 0.07) == 21
    rng = np.random.default_rng(3)
    ratios = [0.07, 0.01, 0.001, 1 / 1024, 0.5, 1.0, 0.3, 0.123, 1e-9, 0.1234567891, 3 / 7, 0.0005, 2.0 ** -30]
    ns = [1, 2, 7, 100, 300, 768, 6240, 1 << 20, 11173962, 25557032, 38597376, 2**31 - 1]
    ns += [int(x) for x in rng.integers(1, 1 << 31, 20)]
    for r in ratios:
        for n in ns:
            assert lib.gmc_count(n, r) == oracle.count(n, r), (n, r)
    assert lib.gmc_count(0, 0.5) == -1 and lib.gmc_count(1 << 31, 0.5) == -1
    assert lib.gmc_count(10, 0.0) == -1 and lib.gmc_count(10, 1.5) == -1
    assert lib.gmc_count(10, float("nan")) == -1


def test_static_aggregate_refuses_before_device_work(lib):
    """gmc_aggregate_static checks its arguments and its scratch bound on the
    host: 64 workers at d = 2^31 - 1 need 128 MiB of row pointers, beyond the
    8 MiB static array (the pointers are never dereferenced)."""
    import ctypes
    p = ctypes.c_void_p(256)
    assert lib.gmc_aggregate_static(2**31 - 1, 64, 0.1, p, 1, p, 1, p, p, None) == -1
    assert "static scratch" in lib.gmc_last_error(None).decode()
    assert lib.gmc_aggregate_static(0, 4, 0.1, p, 1, p, 1, p, p, None) == -1
    assert lib.gmc_aggregate_static(100, 0, 0.1, p, 1, p, 1, p, p, None) == -1
    assert lib.gmc_aggregate_static(100, 4, 0.0, p, 1, p, 1, p, p, None) == -1
    assert lib.gmc_aggregate_static(100, 4, 0.1, p, 5, p, 4, p, p, None) == -1   # message shorter than index row
    assert lib.gmc_aggregate_static(100, 4, 0.1, None, 1, p, 1, p, p, None) == -1
