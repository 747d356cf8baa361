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
