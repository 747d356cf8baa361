"""Plants plausible mistakes in copies of the oracle (CPU only) and checks
that the pins catch every one: a dropped term, a wrong sign, a swapped
operand, a wrong index, a reversed order.  The oracle source itself is never
changed; each mutant is a text substitution compiled into a temporary
library."""
import os
import tempfile

import pytest

import oracle
from oracle_pins import ALL_PINS

MUTANTS = {
    "momentum_sign": ("u[j] = acc - mom;", "u[j] = acc + mom;"),
    "momentum_dropped": ("u[j] = acc - mom;", "u[j] = acc;"),
    "diff_swapped": ("float diff = w_t[j] - w_prev[j];", "float diff = w_prev[j] - w_t[j];"),
    "error_feedback_dropped": ("float acc = e[j] + g[j];", "float acc = g[j];"),
    "gradient_dropped": ("float acc = e[j] + g[j];", "float acc = e[j];"),
    "momentum_coeff_beta": ("*c = (float)(beta / eta);", "*c = (float)beta;"),
    "server_scale_dropped": ("delta[j] = -(s * acc[j]);", "delta[j] = -acc[j];"),
    "server_sign": ("delta[j] = -(s * acc[j]);", "delta[j] = s * acc[j];"),
    "server_scale_no_K": ("*s = (float)(eta / (double)K);", "*s = (float)eta;"),
    "server_worker_index": ("acc[idx[k][i]] = acc[idx[k][i]] + val[k][i];",
                            "acc[idx[k][i]] = acc[idx[k][i]] + val[0][i];"),
    "residual_not_cleared": ("u[idx[i]] = u[idx[i]] - sent;", "u[idx[i]] = u[idx[i]];"),
    "topk_smallest": ("if (x->key != y->key) return x->key > y->key ? -1 : 1;",
                      "if (x->key != y->key) return x->key < y->key ? -1 : 1;"),
    "topk_tie_high_index": ("if (x->pos != y->pos) return x->pos < y->pos ? -1 : 1;",
                            "if (x->pos != y->pos) return x->pos > y->pos ? -1 : 1;"),
    "topk_signed_key": ("return b & 0x7fffffffu;", "return b;"),
    "count_floor": ("k = (n * p + q - 1) / q;", "k = (n * p) / q;"),
    "count_binary64_product": ("k = (n * p + q - 1) / q;", "k = (int64_t)ceil(ratio * (double)n);"),
    "count_fraction_ignored": ("if (p / (double)q == ratio) {", "if (0) {"),
    "count_binary_value_floor": ("k = (int64_t)((num + ((one << sh) - 1)) >> sh);", "k = (int64_t)(num >> sh);"),
    "agg_reverse_worker_order": ("for (int k = 0; k < K; ++k)\n        for (int64_t i = 0; i < len[k]; ++i)",
                                 "for (int k = K - 1; k >= 0; --k)\n        for (int64_t i = 0; i < len[k]; ++i)"),
    "agg_start_from_first_value": ("for (int64_t j = 0; j < d; ++j) acc[j] = 0.0f;",
                                   "for (int64_t j = 0; j < d; ++j) acc[j] = -0.0f;"),
    "apply_sign": ("w[j] = w[j] + delta[j];", "w[j] = w[j] - delta[j];"),
    "floyd_no_dedup": ("blocks[have++] = dup ? (int32_t)J : r;", "blocks[have++] = r;"),
    "rbgs_short_block": ("int64_t lo = (int64_t)blocks[q] * B, hi = lo + B;",
                         "int64_t lo = (int64_t)blocks[q] * B, hi = lo + B - 1;"),
    "splitmix_shift": ("z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;",
                       "z = (z ^ (z >> 28)) * 0x94d049bb133111ebULL;"),
    "detach_sign": ("w_k[j] = w_next[j] - r;", "w_k[j] = w_next[j] + r;"),
    "detach_lambda_over_eta": ("return (float)(lambda * eta);", "return (float)(lambda / eta);"),
    "detach_eta_dropped": ("return (float)(lambda * eta);", "return (float)lambda;"),
    "plain_feedback_dropped": ("u[j] = e[j] + g[j];", "u[j] = g[j];"),
    "lr_gradient_unscaled": ("float sg = h * g[j];", "float sg = g[j];"),
    "lr_momentum_sign": ("u[j] = sum - pull;", "u[j] = sum + pull;"),
    "lr_coeff_over_eta": ("*c = (float)beta;", "*c = c_gmc;"),
    "lr_server_scale": ("*s = (float)(1.0 / (double)K);", "*s = s_gmc;"),
    "server_momentum_sign": ("w_next[j] = moved + push;", "w_next[j] = moved - push;"),
    "server_momentum_dropped": ("w_next[j] = moved + push;", "w_next[j] = moved;"),
    "server_coeff_over_eta": ("*c = b;", "*c = c_gmc;"),
    "approx_rank_off_by_one": ("uint32_t theta = keys[r - 1];", "uint32_t theta = keys[r];"),
    "approx_strict_threshold": ("if (key_of(u[j]) >= theta) {", "if (key_of(u[j]) > theta) {"),
    "approx_residual_kept": ("u[j] = kept - kept;", "u[j] = kept;"),
    "sample_stratum_overrun": ("pos[i] = lo + (int64_t)(((x >> 32) * (uint64_t)len) >> 32);",
                               "pos[i] = lo + (int64_t)(((x >> 32) * (uint64_t)L) >> 32);"),
    "sample_same_for_workers": ("^ orc_splitmix64_mix((k + 1) << 32);", ";"),
}


@pytest.fixture(scope="module")
def source():
    with open(os.path.join(os.path.dirname(oracle.__file__), "gmc_oracle.c")) as f:
        return f.read()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, source):
    old, new = MUTANTS[name]
    assert source.count(old) == 1, "mutation anchor not found: " + old
    with tempfile.TemporaryDirectory() as tmp:
        src = os.path.join(tmp, "m.c")
        with open(src, "w") as f:
            f.write(source.replace(old, new))
        lib = oracle.load(oracle.build(force=True, src=src, out=os.path.join(tmp, "m.so")))
        caught = []
        for pin in ALL_PINS:
            try:
                pin(lib)
            except (AssertionError, ValueError, IndexError, KeyError):
                caught.append(pin.__name__)
        assert caught, "no pin caught mutant " + name
