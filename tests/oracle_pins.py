"""Checks that pin the CPU oracle to what the paper and mathematics fix.

Each ``pin_*`` function takes an oracle library handle and raises
AssertionError when the oracle disagrees with:

* closed forms the paper states: GMC without compression is momentum SGD
  (Section 2.3, eq. 3); the update-rule rewrite (eq. 8); the auxiliary
  sequence z_t of Lemma 1; the toy quadratic of Section 3.2, whose
  uncompressed run has a closed form;
* properties of the compressors: top-s equals a brute-force sort; the
  delta-approximation bound of Assumption 1; the error-feedback identity
  C(u) + e_{t+1} = u; RBGS blocks that are distinct, sorted, reproducible,
  shared by the workers and uniform; the RBGS communication cost of
  Section 5.2;
* published test vectors (SplitMix64).

They are plain functions so that the mutation tests can run them against
deliberately broken builds of the oracle and check that each planted mistake
is caught by at least one of them.
"""
from __future__ import annotations

import itertools
import math
import os
from fractions import Fraction

import numpy as np

import oracle
import synth

EPS32 = 2.0 ** -24
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _bits(a: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


def _keys(a: np.ndarray) -> np.ndarray:
    return _bits(a) & np.uint32(0x7FFFFFFF)


def brute_topk(u: np.ndarray, k: int) -> np.ndarray:
    """Independent top-k: Python's sort of (-|u| bits, index) tuples."""
    keys = _keys(u).tolist()
    order = sorted(range(len(keys)), key=lambda j: (-keys[j], j))
    return np.array(sorted(order[:k]), dtype=np.int64)


def _run(lib, wl: synth.Workload, ratio: float, steps: int, grad_fn=None, w0=None):
    """Drive the oracle for `steps` iterations; returns per-step records."""
    orc = oracle.GmcOracle(wl.d, wl.K, "topk", ratio, wl.beta, wl.eta,
                           seg_off=[0, wl.d], lib=lib)
    w = (wl.w0() if w0 is None else np.asarray(w0, np.float32)).copy()
    w_prev = w.copy()
    err = np.zeros((wl.K, wl.d), np.float32)
    recs = []
    for t in range(steps):
        g = wl.grads(t) if grad_fn is None else grad_fn(t, w)
        e_before = err.copy()
        us = np.stack([orc.precompress(w, w_prev, g[k], err[k]) for k in range(wl.K)])
        idx, val, ln = orc.step(w, w_prev, g, err)
        delta = orc.aggregate(idx, val, ln)
        w_next = w.copy()
        orc.apply(w_next, delta)
        recs.append(dict(w_prev=w_prev, w=w, w_next=w_next, g=g, e=e_before, e_next=err.copy(),
                         u=us, idx=idx, val=val, ln=ln, delta=delta))
        w_prev, w = w, w_next
    return recs


def _run_rule(lib, wl: synth.Workload, ratio: float, steps: int, variant: str = "gmc", lam: float = 0.0,
              eta_fn=None, compressor: str = "topk", block: int = 4096):
    """Like ``_run`` for any of the update rules, an eta schedule and GMC+'s
    detached points (``wk``: w_{t+1,k} after each step)."""
    orc = oracle.GmcOracle(wl.d, wl.K, compressor, ratio, wl.beta, wl.eta, seg_off=[0, wl.d], lib=lib,
                           variant=variant, lam=lam, block=block)
    w = wl.w0().copy()
    w_prev = w.copy()
    err = np.zeros((wl.K, wl.d), np.float32)
    recs = []
    for t in range(steps):
        eta = wl.eta if eta_fn is None else eta_fn(t)
        orc.set_eta(eta)
        g = wl.grads(t)
        e_before = err.copy()
        us = np.stack([orc.precompress(w, w_prev, g[k], err[k]) for k in range(wl.K)])
        idx, val, ln = orc.step(w, w_prev, g, err)
        delta = orc.aggregate(idx, val, ln)
        w_next = orc.next_params(w, w_prev, delta)
        recs.append(dict(w_prev=w_prev, w=w, w_next=w_next, g=g, e=e_before, e_next=err.copy(), u=us,
                         idx=idx, val=val, ln=ln, delta=delta, eta=eta, wk=orc.detach(w_next, err)))
        w_prev, w = w, w_next
    return recs


# ---------------------------------------------------------------------------
# counts and constants
# ---------------------------------------------------------------------------

def _want_count(n: int, r: Fraction) -> int:
    return max(1, min(n, -((-n * r.numerator) // r.denominator)))


def pin_count_rule(lib):
    """k = ceil(n p / q), clamped to [1, n], with the ratio read as the
    fraction p/q it stands for: checked with Python's exact rationals parsed
    from decimal strings (an independent reading of the same numbers), on
    products that land just above an integer in binary64."""
    # s = d/1024 (Section 5.1) exactly when 1024 divides d
    for d in (1024, 1 << 20, 25557032):
        assert oracle.count(d, 1 / 1024, lib) == -(-d // 1024)
    # the workloads' stated per-worker counts
    assert oracle.count(1 << 20, 0.01, lib) == 10486
    assert oracle.count(25557032, 0.001, lib) == 25558
    assert oracle.count(11173962, 0.01, lib) == 111740
    assert oracle.count(6240, 0.01, lib) == 63
    # binary64 gives 0.07 * 100 = 7.000000000000001 and 0.07 * 300 = 21.000000000000004:
    # 7% keeps 7 and 21
    assert oracle.count(100, 0.07, lib) == 7
    assert oracle.count(300, 0.07, lib) == 21
    # clamps: at least one, at most all
    assert oracle.count(768, 0.001, lib) == 1
    assert oracle.count(5, 1.0, lib) == 5
    assert oracle.count(1, 1e-9, lib) == 1
    rng = np.random.default_rng(77)
    texts = ["0.07", "0.001", "0.01", "0.1", "0.3", "0.123", "0.0005", "0.035", "0.9", "0.99", "0.015",
             "0.0001", "0.25", "0.2", "0.6", "0.7", "0.17", "0.029"]
    fracs = [Fraction(t) for t in texts] + [Fraction(1, 1024), Fraction(3, 7), Fraction(1, 3),
                                            Fraction(999, 1000000), Fraction(1, 1 << 20)]
    for r in fracs:
        ns = [1, 2, 3, 7, 100, 300, 768, 1000, 4096] + [int(x) for x in rng.integers(1, 1 << 31, 8)]
        for n in ns:
            assert oracle.count(n, float(r), lib) == _want_count(n, r), (n, r)
    # a ratio that no fraction of denominator <= 2^20 rounds to: its exact binary value
    for x in (0.1234567891, 1e-7, 0.3333333333, 2.0 ** -30 * 3):
        assert float(Fraction(x).limit_denominator(1 << 20)) != x
        for n in (1, 10, 10**6, 2**31 - 1, 987654321):
            assert oracle.count(n, x, lib) == _want_count(n, Fraction(x)), (n, x)


def pin_constants(lib):
    c, s = oracle.constants(0.9, 0.1, 16, lib)
    assert c == np.float32(9.0)
    assert s == np.float32(0.1 / 16)
    c, s = oracle.constants(0.9, 0.05, 8, lib)
    assert c == np.float32(18.0) and s == np.float32(0.05 / 8)


# ---------------------------------------------------------------------------
# top-s against brute force, delta-approximation, error feedback
# ---------------------------------------------------------------------------

def _adversarial_vectors():
    rng = np.random.default_rng(1234)
    vecs = []
    vecs.append(rng.standard_normal(1000).astype(np.float32))
    vecs.append(rng.choice(np.array([0, 1, -1, 2, -2], np.float32), 777))          # heavy ties
    z = rng.choice(np.array([0.0, -0.0, 1e-45, -1e-45, 3e-40, 1.0], np.float32), 300)
    vecs.append(z)                                                                  # +-0, denormals
    x = rng.standard_normal(200).astype(np.float32)
    x[[3, 50, 51]] = [np.inf, -np.inf, np.nan]
    vecs.append(x)                                                                  # non-finite
    vecs.append(np.full(129, -3.5, np.float32))                                     # all equal
    return vecs


def pin_topk_bruteforce(lib):
    for u in _adversarial_vectors():
        n = u.size
        for k in sorted({1, 2, 7, n // 3, n - 1, n}):
            if k < 1:
                continue
            got = oracle.topk(u, k, lib)
            want = brute_topk(u, k)
            assert np.array_equal(got, want), (n, k)


def pin_delta_approximation(lib):
    """Assumption 1: top-k is a delta-approximate compressor with
    delta = k/n: ||C(u) - u||^2 <= (1 - k/n) ||u||^2 for every u."""
    rng = np.random.default_rng(7)
    for n, k in [(1000, 10), (4096, 41), (333, 333), (500, 1)]:
        u = (rng.standard_t(3, n) * rng.uniform(0.1, 10)).astype(np.float32)
        u0 = u.copy()
        idx, val = oracle.compress_topk(u, [0, n], k / n, lib)
        assert idx.size == k
        lhs = float(np.sum(u.astype(np.float64) ** 2))        # ||u - C(u)||^2: the residual
        rhs = (1 - k / n) * float(np.sum(u0.astype(np.float64) ** 2))
        assert lhs <= rhs * (1 + 1e-12) + 1e-300


def pin_error_feedback_identity(lib):
    """e_{t+1} = u - C(u): the kept components are sent unchanged and leave
    u - u = +0 behind; every other component keeps u bit for bit."""
    rng = np.random.default_rng(11)
    for u0 in [rng.standard_normal(5000).astype(np.float32)] + _adversarial_vectors()[:3]:
        n = u0.size
        seg = [0, n // 3, n // 3 + 1, n] if n > 10 else [0, n]
        u = u0.copy()
        idx, val = oracle.compress_topk(u, seg, 0.05, lib)
        assert np.all(np.diff(idx) > 0)
        assert np.array_equal(_bits(val), _bits(u0[idx]))
        assert np.all(_bits(u[idx]) == 0)
        mask = np.ones(n, bool)
        mask[idx] = False
        assert np.array_equal(_bits(u[mask]), _bits(u0[mask]))
        # per segment the kept set is that segment's own top-k
        for a, b in zip(seg[:-1], seg[1:]):
            sel = idx[(idx >= a) & (idx < b)] - a
            k = oracle.count(b - a, 0.05, lib)
            assert np.array_equal(sel, brute_topk(u0[a:b], k))


# ---------------------------------------------------------------------------
# multi-step closed forms (Section 2.3, eq. 8, Lemma 1)
# ---------------------------------------------------------------------------

def pin_msgd_reduction(lib):
    """Without compression (s = d) GMC is serial momentum SGD on the average
    gradient: m_{t+1} = beta m_t + eta gbar_t, w_{t+1} = w_t - m_{t+1}
    (Section 2.3), and the residual stays zero."""
    for K in (1, 4):
        wl = synth.Workload("msgd", [3000, 17], K=K, ratio=1.0, beta=0.9, eta=0.1, steps=25,
                            compressor="topk", dist="normal")
        recs = _run(lib, wl, 1.0, wl.steps)
        m = np.zeros(wl.d)
        w = recs[0]["w"].astype(np.float64)
        for r in recs:
            gbar = r["g"].astype(np.float64).mean(axis=0)
            m = wl.beta * m + wl.eta * gbar
            w = w - m
            assert np.all(_bits(r["e_next"]) == 0)
            got = r["w_next"].astype(np.float64)
            assert np.max(np.abs(got - w)) <= 2e-5 * (1 + np.max(np.abs(w))), K


def _eq8_terms(r, wl):
    f = lambda a: np.asarray(a, np.float64)
    gbar = f(r["g"]).mean(0)
    ebar, ebar1 = f(r["e"]).mean(0), f(r["e_next"]).mean(0)
    return gbar, ebar, ebar1


def pin_update_rule_eq8(lib):
    """eq. 8: w_{t+1} = w_t - eta gbar_t - eta ebar_t + eta ebar_{t+1}
    + beta (w_t - w_{t-1}), for any compressor; checked within the
    binary32 rounding bound of the operations involved."""
    wl = synth.Workload("eq8", [2500, 1500, 96], K=4, ratio=0.02, beta=0.9, eta=0.1, steps=12,
                        compressor="topk", dist="normal", scale_lo=1e-2, scale_hi=1.0)
    for r in _run(lib, wl, wl.ratio, wl.steps):
        f = lambda a: np.asarray(a, np.float64)
        gbar, ebar, ebar1 = _eq8_terms(r, wl)
        w, wp, wn = f(r["w"]), f(r["w_prev"]), f(r["w_next"])
        rhs = w - wl.eta * gbar - wl.eta * ebar + wl.eta * ebar1 + wl.beta * (w - wp)
        scale = (np.abs(w) + np.abs(wn) + wl.beta * np.abs(w - wp)
                 + wl.eta * (np.abs(f(r["g"])).mean(0) + np.abs(f(r["e"])).mean(0)
                             + wl.K * np.abs(f(r["u"])).mean(0)))
        assert np.all(np.abs(wn - rhs) <= 16 * EPS32 * scale + 1e-30)


def pin_lemma1(lib):
    """Lemma 1: z_t = w_t + beta/(1-beta)(w_t - w_{t-1}) - eta/(1-beta) ebar_t
    satisfies z_{t+1} = z_t - eta/(1-beta) gbar_t."""
    wl = synth.Workload("lemma1", [4000, 95], K=3, ratio=0.05, beta=0.9, eta=0.1, steps=10,
                        compressor="topk", dist="student_t", nu=3, scale_lo=1e-3, scale_hi=1.0)
    recs = _run(lib, wl, wl.ratio, wl.steps)
    b, eta = wl.beta, wl.eta
    f = lambda a: np.asarray(a, np.float64)
    for r in recs:
        gbar, ebar, ebar1 = _eq8_terms(r, wl)
        w, wp, wn = f(r["w"]), f(r["w_prev"]), f(r["w_next"])
        z = w + b / (1 - b) * (w - wp) - eta / (1 - b) * ebar
        z1 = wn + b / (1 - b) * (wn - w) - eta / (1 - b) * ebar1
        scale = (np.abs(w) + np.abs(wn) + np.abs(wp)
                 + eta * (np.abs(f(r["g"])).mean(0) + np.abs(f(r["e"])).mean(0)
                          + wl.K * np.abs(f(r["u"])).mean(0)))
        assert np.all(np.abs(z1 - (z - eta / (1 - b) * gbar)) <= 64 / (1 - b) * EPS32 * scale + 1e-30)


# ---------------------------------------------------------------------------
# aggregation and apply
# ---------------------------------------------------------------------------

def pin_aggregate_single_worker(lib):
    """K = 1: delta = -(eta) C(u): -(s*v) at the sent indices, -0 elsewhere,
    bit for bit, and w + delta = w - s*C(u)."""
    rng = np.random.default_rng(5)
    d = 1000
    idx = np.sort(rng.choice(d, 37, replace=False)).astype(np.int32)
    val = rng.standard_normal(37).astype(np.float32)
    s = np.float32(0.1)
    delta = oracle.aggregate(d, s, [idx], [val], lib)
    want = np.full(d, -0.0, np.float32)
    want[idx] = -(s * val)
    assert np.array_equal(_bits(delta), _bits(want))
    w = rng.standard_normal(d).astype(np.float32)
    w1 = w.copy()
    oracle.apply(w1, delta, lib)
    c = np.zeros(d, np.float32)
    c[idx] = val
    assert np.array_equal(_bits(w1), _bits(w - s * c))


def pin_aggregate_sum(lib):
    """The server's sum over workers is the plain sum of the sparse vectors:
    checked against an fp64 sum within K rounding errors, and on integer
    values (exact in binary32) bit for bit."""
    rng = np.random.default_rng(6)
    d, K = 5000, 6
    idx = [np.sort(rng.choice(d, 400, replace=False)).astype(np.int32) for _ in range(K)]
    val = [rng.integers(-50, 50, 400).astype(np.float32) for _ in range(K)]
    s = np.float32(0.25)
    delta = oracle.aggregate(d, s, idx, val, lib)
    dense = np.zeros((K, d))
    for k in range(K):
        dense[k, idx[k]] = val[k]
    want = -(0.25 * dense.sum(0))
    assert np.array_equal(delta.astype(np.float64), want)
    val = [rng.standard_normal(400).astype(np.float32) for _ in range(K)]
    delta = oracle.aggregate(d, np.float32(0.1 / K), idx, val, lib)
    for k in range(K):
        dense[k] = 0
        dense[k, idx[k]] = val[k]
    want = -(np.float32(0.1 / K) * dense.sum(0))
    bound = (K + 1) * EPS32 * (0.1 / K) * np.abs(dense).sum(0)
    assert np.all(np.abs(delta - want) <= bound + 1e-30)


def pin_aggregate_worker_order(lib):
    """The server adds the messages in worker order 0..K-1 starting from
    +0.0f (the order is this build's reading; Algorithm 1's server only
    receives from all workers).  Binary32 makes the order visible:
    2^24 + 1 rounds back to 2^24 (ties to even), so three workers sending
    2^24, 1, -2^24 at one index sum to +0, and -2^24, 1, 2^24 sum to 1.
    All-negative-zero sends sum to +0 from a +0 start (-0 from the first
    value), so the update there is -(s * +0) = -0."""
    big = np.float32(2.0 ** 24)
    one = np.float32(1.0)
    idx = [np.array([1, 2, 3], np.int32)] * 3
    val = [np.array([big, -big, -0.0], np.float32), np.array([one, one, -0.0], np.float32),
           np.array([-big, big, -0.0], np.float32)]
    delta = oracle.aggregate(5, np.float32(0.5), idx, val, lib)
    want = np.array([-0.0, -0.0, -0.5, -0.0, -0.0], np.float32)
    assert np.array_equal(_bits(delta), _bits(want)), delta


# ---------------------------------------------------------------------------
# RBGS
# ---------------------------------------------------------------------------

def pin_splitmix64_vectors(lib):
    with open(os.path.join(GOLDEN, "splitmix64_seed0.txt")) as f:
        want = [int(ln, 16) for ln in f.read().splitlines() if ln.startswith("0x")]
    gamma = 0x9E3779B97F4A7C15
    got = [oracle.splitmix64_mix((i * gamma) % (1 << 64), lib) for i in range(1, len(want) + 1)]
    assert got == want


def pin_rbgs_blocks(lib):
    for nb, n_sel in [(6240, 63), (10, 10), (7, 1), (1000, 999)]:
        for t in range(6):
            b = oracle.rbgs_blocks(42, t, nb, n_sel, lib)
            assert b.size == n_sel
            assert np.all(np.diff(b) > 0) and b[0] >= 0 and b[-1] < nb
            assert np.array_equal(b, oracle.rbgs_blocks(42, t, nb, n_sel, lib))
    a = [tuple(oracle.rbgs_blocks(1, t, 6240, 63, lib)) for t in range(20)]
    assert len(set(a)) == 20
    # uniform over subsets: every 3-subset of 8 blocks equally likely
    from scipy.stats import chisquare
    T = 28000
    counts = {c: 0 for c in itertools.combinations(range(8), 3)}
    for t in range(T):
        counts[tuple(int(x) for x in oracle.rbgs_blocks(9, t, 8, 3, lib))] += 1
    obs = np.array(list(counts.values()), dtype=float)
    assert chisquare(obs).pvalue > 1e-4


def pin_rbgs_step_and_cost(lib):
    """GMC with RBGS: the blocks are the same on every worker, so the
    aggregated update is nonzero exactly on those m components, and the
    relative communication cost (values only, Section 5.2) is m/d."""
    d, K, B = 50000, 3, 4096
    orc = oracle.GmcOracle(d, K, "rbgs", 0.1, 0.9, 0.1, seed=3, block=B, lib=lib)
    rng = np.random.default_rng(2)
    w = rng.standard_normal(d).astype(np.float32)
    wp = w.copy()
    err = np.zeros((K, d), np.float32)
    for t in range(4):
        g = rng.standard_normal((K, d)).astype(np.float32)
        us = [orc.precompress(w, wp, g[k], err[k]) for k in range(K)]
        idx, val, ln = orc.step(w, wp, g, err)
        blocks = oracle.rbgs_blocks(3, t, orc.nb, orc.n_sel, lib)
        assert all(np.array_equal(idx[k], blocks) for k in range(K))
        ei = orc.element_indices(idx[0], int(ln[0]))
        m = sum(min((b + 1) * B, d) - b * B for b in blocks)
        assert np.all(ln == m) and ei.size == m
        for k in range(K):
            assert np.array_equal(_bits(val[k, :m]), _bits(us[k][ei]))
            assert np.all(_bits(err[k][ei]) == 0)
            rest = np.ones(d, bool)
            rest[ei] = False
            assert np.array_equal(_bits(err[k][rest]), _bits(us[k][rest]))
        delta = orc.aggregate(idx, val, ln)
        nnz = int(np.count_nonzero(delta))
        assert nnz == m
        rcc = (K * nnz + int(ln.sum())) / (2 * d * K)
        assert abs(rcc - m / d) < 1e-15
        w_next = w.copy()
        orc.apply(w_next, delta)
        wp, w = w, w_next


# ---------------------------------------------------------------------------
# the toy quadratic of Section 3.2
# ---------------------------------------------------------------------------

def _toy_grads(d):
    i = np.arange(d, dtype=np.float32)
    coef = np.float32(2.0) * (np.float32(d) - i)
    shift = i + np.float32(1.0)

    def fn(t, w):
        return np.stack([coef * (w - shift), coef * (w + shift)]).astype(np.float32)
    return fn


def pin_toy_quadratic_closed_form(lib):
    """F(w) = sum_i (d-i)(w_i^2 + (i+1)^2) with K = 2 workers holding
    F_0, F_1.  With s = d GMC is momentum SGD on F, whose iterates solve
    w_{t+1} = (1 + beta - 2 eta (d-i)) w_t - beta w_{t-1}, w_{-1} = w_0."""
    beta, eta = 0.9, 0.005
    for d, w0 in [(2, [-1.0, 2.0]), (20, list(np.linspace(-3, 3, 20)))]:
        wl = synth.Workload("toy", [d], K=2, ratio=1.0, beta=beta, eta=eta, steps=300,
                            compressor="topk", dist="normal")
        recs = _run(lib, wl, 1.0, wl.steps, grad_fn=_toy_grads(d), w0=w0)
        w0 = np.asarray(w0, np.float64)
        a = 2 * eta * (d - np.arange(d))
        tr = 1 + beta - a
        disc = np.sqrt((tr ** 2 - 4 * beta).astype(complex))
        l1, l2 = (tr + disc) / 2, (tr - disc) / 2
        w1 = (1 - a) * w0
        B_ = (w1 - l1 * w0) / (l2 - l1)
        A_ = w0 - B_
        for t, r in enumerate(recs, start=1):
            want = np.real(A_ * l1 ** t + B_ * l2 ** t)
            got = r["w_next"].astype(np.float64)
            assert np.max(np.abs(got - want)) <= 1e-4 * (1 + np.max(np.abs(w0))), (d, t)


def pin_toy_quadratic_sparse_converges(lib):
    """Section 3.2: with top-s sparsification GMC still approaches the
    optimum w* = 0 from (-1, 2) (d = 2, s = d/2)."""
    d = 2
    wl = synth.Workload("toy", [d], K=2, ratio=0.5, beta=0.9, eta=0.005, steps=3000,
                        compressor="topk", dist="normal")
    recs = _run(lib, wl, 0.5, wl.steps, grad_fn=_toy_grads(d), w0=[-1.0, 2.0])
    dist = [float(np.linalg.norm(r["w_next"])) for r in recs]
    assert dist[-1] < 0.1 * math.sqrt(5.0)
    assert max(dist[-200:]) < 0.2 * math.sqrt(5.0)


# ---------------------------------------------------------------------------
# GMC+ (Algorithm 2): the detached point
# ---------------------------------------------------------------------------

def pin_detach_lambda_zero(lib):
    """lambda = 0: every worker's point is w_{t+1} itself, bit for bit, so
    GMC+ is GMC (Section 4)."""
    rng = np.random.default_rng(21)
    w = rng.standard_normal(3000).astype(np.float32)
    e = (rng.standard_normal(3000) * 10.0 ** rng.integers(-40, 3, 3000)).astype(np.float32)
    e[:4] = [0.0, -0.0, 1e-45, -3e-42]
    for eta in (0.1, 0.05, 1.0):
        q = oracle.detach_constant(0.0, eta, lib)
        assert np.array_equal(_bits(oracle.detach(q, w, e, lib)), _bits(w))


def _bar(recs, key):
    return [np.asarray(r[key], np.float64).mean(0) for r in recs]


def pin_gmcplus_average_rule(lib):
    """Section 4: with wbar_t the mean of the detached points and ebar_t that
    of the residuals, wbar_{t+1} = wbar_t + beta (wbar_t - wbar_{t-1})
    + eta (1 - lambda)(ebar_{t+1} - ebar_t) + beta lambda eta (ebar_t - ebar_{t-1})
    - eta gbar_t, for top-s and RBGS, checked within the binary32 rounding of
    the operations involved."""
    for comp, lam, ratio in [("topk", 0.5, 0.03), ("rbgs", 0.3, 0.25), ("topk", 1.0, 0.01)]:
        wl = synth.Workload("gmcplus", [3000, 1096], K=3, ratio=ratio, beta=0.9, eta=0.1, steps=8,
                            compressor=comp, dist="normal", scale_lo=1e-2, scale_hi=1.0)
        recs = _run_rule(lib, wl, ratio, wl.steps, lam=lam, compressor=comp, block=512)
        b, eta = wl.beta, wl.eta
        f = lambda a: np.asarray(a, np.float64)
        wbar = [f(recs[0]["w"])] + [f(r["wk"]).mean(0) for r in recs]      # wbar_0 = w_0
        ebar = [np.zeros(wl.d)] + [f(r["e_next"]).mean(0) for r in recs]  # ebar_0 = 0
        for t in range(1, len(recs)):
            r = recs[t]
            gbar = f(r["g"]).mean(0)
            rhs = (wbar[t] + b * (wbar[t] - wbar[t - 1]) + eta * (1 - lam) * (ebar[t + 1] - ebar[t])
                   + b * lam * eta * (ebar[t] - ebar[t - 1]) - eta * gbar)
            scale = (np.abs(f(r["w_next"])) + np.abs(f(r["w"])) + np.abs(f(r["w_prev"]))
                     + eta * (np.abs(f(r["g"])).mean(0) + np.abs(f(r["e"])).mean(0)
                              + np.abs(f(r["e_next"])).mean(0) + wl.K * np.abs(f(r["u"])).mean(0)))
            assert np.all(np.abs(wbar[t + 1] - rhs) <= 64 * EPS32 * scale + 1e-30), (comp, lam, t)


def pin_gmcplus_lemma(lib):
    """The auxiliary sequence of GMC+ (Section 4):
    zbar_t = wbar_t + beta/(1-beta)(wbar_t - wbar_{t-1})
             - [(1-lambda) eta ebar_t + beta lambda eta ebar_{t-1}]/(1-beta)
    moves by -eta/(1-beta) gbar_t per iteration."""
    lam = 0.5
    wl = synth.Workload("gmcplus", [2048, 77], K=4, ratio=0.05, beta=0.9, eta=0.1, steps=8,
                        compressor="topk", dist="student_t", nu=3, scale_lo=1e-3, scale_hi=1.0)
    recs = _run_rule(lib, wl, wl.ratio, wl.steps, lam=lam)
    b, eta = wl.beta, wl.eta
    f = lambda a: np.asarray(a, np.float64)
    wbar = [f(recs[0]["w"]), f(recs[0]["w"])] + [f(r["wk"]).mean(0) for r in recs]  # wbar_{-1}, wbar_0, ...
    ebar = [np.zeros(wl.d), np.zeros(wl.d)] + [f(r["e_next"]).mean(0) for r in recs]

    def z(i):  # i = t + 1 in the lists above
        return (wbar[i] + b / (1 - b) * (wbar[i] - wbar[i - 1])
                - ((1 - lam) * eta * ebar[i] + b * lam * eta * ebar[i - 1]) / (1 - b))
    for t, r in enumerate(recs):
        gbar = f(r["g"]).mean(0)
        scale = (np.abs(f(r["w_next"])) + np.abs(f(r["w"])) + np.abs(f(r["w_prev"]))
                 + eta * (np.abs(f(r["g"])).mean(0) + np.abs(f(r["e"])).mean(0)
                          + np.abs(f(r["e_next"])).mean(0) + wl.K * np.abs(f(r["u"])).mean(0)))
        assert np.all(np.abs(z(t + 2) - (z(t + 1) - eta / (1 - b) * gbar))
                      <= 256 / (1 - b) * EPS32 * scale + 1e-30), t


# ---------------------------------------------------------------------------
# the appendix's other update rules, and a learning-rate schedule
# ---------------------------------------------------------------------------

def _eq8_check(recs, wl, bound_mult=16):
    f = lambda a: np.asarray(a, np.float64)
    for r in recs:
        eta = r["eta"]
        gbar, ebar, ebar1 = _eq8_terms(r, wl)
        w, wp, wn = f(r["w"]), f(r["w_prev"]), f(r["w_next"])
        rhs = w - eta * gbar - eta * ebar + eta * ebar1 + wl.beta * (w - wp)
        scale = (np.abs(w) + np.abs(wn) + wl.beta * np.abs(w - wp)
                 + eta * (np.abs(f(r["g"])).mean(0) + np.abs(f(r["e"])).mean(0)
                          + wl.K * np.abs(f(r["u"])).mean(0)) + np.abs(f(r["e"])).mean(0))
        assert np.all(np.abs(wn - rhs) <= bound_mult * EPS32 * scale + 1e-30)


def pin_server_momentum_rule(lib):
    """Momentum on the server (appendix): without compression it is momentum
    SGD, and with it eq. 8 still holds (the appendix derives the same update
    rule once C is eliminated)."""
    wl = synth.Workload("srv", [3000, 17], K=3, ratio=1.0, beta=0.9, eta=0.1, steps=12,
                        compressor="topk", dist="normal")
    recs = _run_rule(lib, wl, 1.0, wl.steps, variant="server_momentum")
    m = np.zeros(wl.d)
    w = np.asarray(recs[0]["w"], np.float64)
    for r in recs:
        m = wl.beta * m + wl.eta * np.asarray(r["g"], np.float64).mean(0)
        w = w - m
        assert np.all(_bits(r["e_next"]) == 0)
        assert np.max(np.abs(np.asarray(r["w_next"], np.float64) - w)) <= 2e-5 * (1 + np.max(np.abs(w)))
    wl = synth.Workload("srv", [2500, 1500, 96], K=4, ratio=0.02, beta=0.9, eta=0.1, steps=12,
                        compressor="topk", dist="normal", scale_lo=1e-2, scale_hi=1.0)
    _eq8_check(_run_rule(lib, wl, wl.ratio, wl.steps, variant="server_momentum"), wl)


def pin_lr_in_residual_equals_gmc(lib):
    """Learning rate inside the residual (appendix) is GMC when eta is
    constant.  With eta a power of two every scaling by eta is exact in
    binary32, so the residuals and messages are exactly eta times GMC's and
    the parameters are identical, bit for bit."""
    eta = 0.125
    wl = synth.Workload("lr", [3000, 1096], K=3, ratio=0.03, beta=0.9, eta=eta, steps=6,
                        compressor="topk", dist="normal", scale_lo=1e-2, scale_hi=1.0)
    a = _run_rule(lib, wl, wl.ratio, wl.steps)
    b = _run_rule(lib, wl, wl.ratio, wl.steps, variant="lr_in_residual")
    e = np.float32(eta)
    for ra, rb in zip(a, b):
        assert np.array_equal(ra["idx"], rb["idx"])
        assert np.array_equal(_bits(ra["val"] * e), _bits(rb["val"]))
        assert np.array_equal(_bits(ra["e_next"] * e), _bits(rb["e_next"]))
        assert np.array_equal(_bits(ra["w_next"]), _bits(rb["w_next"]))


def pin_eta_schedule_eq8(lib):
    """Under the cosine schedule of Section 5.1 (eta_t = eta (1 + cos(pi t/T))/2),
    GMC's iterates satisfy eq. 8 with eta_t in every term, which holds only if
    the momentum coefficient of iteration t is beta/eta_t and the server's
    scale eta_t/K."""
    wl = synth.Workload("cos", [2500, 1500, 96], K=4, ratio=0.02, beta=0.9, eta=0.1, steps=12,
                        compressor="topk", dist="normal", scale_lo=1e-2, scale_hi=1.0)
    T = 16
    sched = lambda t: wl.eta * 0.5 * (1 + math.cos(math.pi * t / T))
    _eq8_check(_run_rule(lib, wl, wl.ratio, wl.steps, eta_fn=sched), wl)


# ---------------------------------------------------------------------------
# the experiments' approximate top-s (Section 5.1)
# ---------------------------------------------------------------------------

def pin_approx_sample(lib):
    """One position per stratum of L (|S| = ceil(n/L)), inside its stratum,
    reproducible, different across workers and steps, and uniform within a
    stratum."""
    for n, L in [(1000, 100), (1001, 100), (17, 5), (5, 100), (64, 1)]:
        pos = oracle.sample_positions(3, 2, 1, n, L, lib)
        m = (n + L - 1) // L
        assert pos.size == m
        lo = np.arange(m) * L
        assert np.all(pos >= lo) and np.all(pos < np.minimum(lo + L, n))
        assert np.array_equal(pos, oracle.sample_positions(3, 2, 1, n, L, lib))
    a = oracle.sample_positions(3, 2, 0, 100000, 100, lib)
    assert not np.array_equal(a, oracle.sample_positions(3, 2, 1, 100000, 100, lib))
    assert not np.array_equal(a, oracle.sample_positions(3, 3, 0, 100000, 100, lib))
    from scipy.stats import chisquare
    off = oracle.sample_positions(11, 0, 5, 8 * 40000, 8, lib) % 8
    assert chisquare(np.bincount(off, minlength=8)).pvalue > 1e-4


def pin_approx_threshold_bruteforce(lib):
    """C(u) keeps every component whose magnitude key reaches theta, the
    r-th largest key of the sample (r = count(|S|, ratio)), ties included;
    the residual is u - C(u)."""
    rng = np.random.default_rng(31)
    vecs = [rng.standard_normal(20000).astype(np.float32),
            rng.choice(np.array([0, 1, -1, 2, -2, 3], np.float32), 5000),
            (rng.standard_t(3, 30001) * 1e-3).astype(np.float32)]
    for u0 in vecs:
        for L, ratio in [(100, 1 / 1024), (10, 0.01), (3, 0.2)]:
            n = u0.size
            pos = oracle.sample_positions(7, 4, 2, n, L, lib)
            keys = sorted(_keys(u0[pos]).tolist(), reverse=True)
            theta = keys[oracle.count(len(keys), ratio, lib) - 1]
            want = np.nonzero(_keys(u0) >= theta)[0]
            u = u0.copy()
            idx, val = oracle.compress_approx(u, 7, 4, 2, L, ratio, lib)
            assert np.array_equal(idx.astype(np.int64), want)
            assert np.array_equal(_bits(val), _bits(u0[want]))
            rest = np.ones(n, bool)
            rest[want] = False
            assert np.array_equal(_bits(u[rest]), _bits(u0[rest]))
            assert np.all(_bits(u[want]) == 0)


def pin_approx_full_sample_is_topk(lib):
    """With L = 1 the sample is all of u, so theta is the k-th largest key and
    on tie-free data C(u) is exactly top-k."""
    rng = np.random.default_rng(41)
    for n, ratio in [(5000, 0.01), (777, 0.05), (64, 1 / 1024)]:
        u0 = rng.standard_normal(n).astype(np.float32)
        assert np.unique(_keys(u0)).size == n
        idx, _ = oracle.compress_approx(u0.copy(), 1, 0, 0, 1, ratio, lib)
        assert np.array_equal(idx.astype(np.int64), brute_topk(u0, oracle.count(n, ratio, lib)))


def pin_approx_count_near_target(lib):
    """Section 5.1: the number kept is approximately n/1024 (Gaussian u,
    |S| = n/100): within a factor 1.5 on each seed and within 10 % on
    average over seeds."""
    rng = np.random.default_rng(51)
    n = 1 << 20
    counts = []
    for seed in range(12):
        u = rng.standard_normal(n).astype(np.float32)
        idx, _ = oracle.compress_approx(u, seed, 0, 0, 100, 1 / 1024, lib)
        counts.append(idx.size)
        assert n / 1024 / 1.5 <= idx.size <= n / 1024 * 1.5, idx.size
    assert abs(np.mean(counts) / (n / 1024) - 1) < 0.1, counts


ALL_PINS = [pin_count_rule, pin_constants, pin_topk_bruteforce, pin_delta_approximation,
            pin_error_feedback_identity, pin_msgd_reduction, pin_update_rule_eq8, pin_lemma1,
            pin_aggregate_single_worker, pin_aggregate_sum, pin_aggregate_worker_order, pin_splitmix64_vectors,
            pin_rbgs_blocks, pin_rbgs_step_and_cost, pin_toy_quadratic_closed_form,
            pin_toy_quadratic_sparse_converges, pin_detach_lambda_zero, pin_gmcplus_average_rule,
            pin_gmcplus_lemma, pin_server_momentum_rule, pin_lr_in_residual_equals_gmc,
            pin_eta_schedule_eq8, pin_approx_sample, pin_approx_threshold_bruteforce,
            pin_approx_full_sample_is_topk, pin_approx_count_near_target]
