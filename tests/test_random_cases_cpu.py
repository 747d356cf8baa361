"""The seeded random-shape sweep draws only valid cases: positive sizes, 1-9
workers, an RBGS block within [1, d] and at most 20,000 drawn blocks unless
the block spans d (the oracle's block draw is quadratic).  CPU only."""
import math

import test_gpu_random_parity as rp


def test_random_cases_are_valid():
    for i in range(3000):
        wl = rp.random_case(i).wl
        assert wl.d >= 1 and all(n >= 1 for n in wl.sizes), i
        assert 1 <= wl.K <= 9, i
        assert 0.0 < wl.ratio <= 1.0, i
        if wl.compressor == "rbgs":
            assert 1 <= wl.block <= wl.d, (i, wl.block, wl.d)
            draws = math.ceil(wl.ratio * math.ceil(wl.d / wl.block))
            assert draws <= 20000 or wl.block == wl.d, (i, draws)
