"""Pins of the oracle's rank allocation (Sec. 4.3, Eqs. 5-7) against facts that
do not come from the oracle itself: exhaustive search of Eq. 6 on small
problems, closed forms of Eq. 5, the greedy's structure (equal spectra share
ranks round-robin), and invariances.  Planted mistakes in a copy of the oracle
must fail at least one pin."""
import inspect
import itertools
import math

import numpy as np
import pytest

import oracle


def _spectra(rng, n_sv, distinct=True):
    """Random non-increasing spectra; distinct values across all blocks if asked."""
    total = int(sum(n_sv))
    vals = rng.permutation(total) + 1.0 if distinct else rng.integers(1, 4, total).astype(float)
    vals = vals * rng.uniform(0.5, 2.0)
    out, k = [], 0
    for n in n_sv:
        out.append(np.sort(vals[k:k + n])[::-1].copy())
        k += n
    return out


def _exhaustive(sig, r_total, r_min, r_max, eps):
    """Eq. 6 by enumeration: every feasible rank vector, keep the maximisers."""
    rng_per = [range(min(r_min, len(s)), min(r_max, len(s)) + 1) for s in sig]
    best, arg = -1.0, []
    for r in itertools.product(*rng_per):
        if sum(r) > r_total:
            continue
        h = sum(math.log1p(float(x) ** 2 / eps ** 2) for s, ri in zip(sig, r) for x in s[:ri])
        if h > best + 1e-9:
            best, arg = h, [r]
        elif abs(h - best) <= 1e-9:
            arg.append(r)
    return best, arg


def pin_exhaustive(alloc, info):
    rng = np.random.default_rng(1)
    for _ in range(60):
        n = int(rng.integers(1, 4))
        n_sv = [int(x) for x in rng.integers(1, 6, n)]
        r_min = int(rng.integers(0, 3))
        r_max = int(rng.integers(r_min, 6))
        floor = sum(min(r_min, m) for m in n_sv)
        r_total = floor + int(rng.integers(0, 8))
        sig = _spectra(rng, n_sv)
        eps = float(rng.choice([0.1, 1.0, 7.0]))
        _, arg = _exhaustive(sig, r_total, r_min, r_max, eps)
        got = tuple(int(x) for x in alloc(sig, r_total, r_min, r_max, eps))
        assert len(arg) == 1 and got == arg[0], (n_sv, r_total, r_min, r_max, got, arg)


def pin_information_closed_form(alloc, info):
    eps = 0.3
    s = np.full(7, eps * math.sqrt(math.e - 1.0))   # every term of Eq. 5 is log(e) = 1
    for r in range(8):
        assert abs(info(s, r, eps) - r) < 1e-12
    assert info(np.zeros(5), 5, eps) == 0.0


def pin_equal_spectra_round_robin(alloc, info):
    # equal spectra, strictly decreasing: the greedy hands out units block by
    # block in index order, so the first e blocks hold one more unit
    s = np.linspace(5.0, 1.0, 12)
    for n, m, e in [(4, 3, 1), (5, 0, 4), (3, 2, 0), (6, 5, 3)]:
        r = alloc([s] * n, n * (2 + m) + e, 2, 12, 0.5)
        assert list(r) == [2 + m + (1 if b < e else 0) for b in range(n)]


def pin_budget_edges(alloc, info):
    rng = np.random.default_rng(2)
    n_sv = [3, 9, 1, 6]
    sig = _spectra(rng, n_sv)
    floors = [min(4, m) for m in n_sv]
    caps = [min(7, m) for m in n_sv]
    assert list(alloc(sig, sum(floors), 4, 7, 1.0)) == floors
    assert list(alloc(sig, sum(caps), 4, 7, 1.0)) == caps
    assert list(alloc(sig, 10 ** 6, 4, 7, 1.0)) == caps          # the budget is not reached
    with pytest.raises(ValueError):
        alloc(sig, sum(floors) - 1, 4, 7, 1.0)


def pin_eps_independence(alloc, info):
    # log(1 + x^2/eps^2) is increasing in x for every eps > 0, so the greedy's
    # choices (and the allocation) do not depend on eps
    rng = np.random.default_rng(3)
    sig = _spectra(rng, [40, 17, 33, 25, 8])
    ref = list(alloc(sig, 70, 5, 30, 1.0))
    for eps in (1e-3, 0.05, 3.0, 1e4):
        assert list(alloc(sig, 70, 5, 30, eps)) == ref


def pin_unit_increments(alloc, info):
    # one more unit of budget raises exactly one block by one (until every block is capped)
    rng = np.random.default_rng(4)
    sig = _spectra(rng, [12, 5, 9], distinct=False)
    prev = alloc(sig, 6, 2, 10, 1.0)
    for R in range(7, 30):
        cur = alloc(sig, R, 2, 10, 1.0)
        d = np.asarray(cur) - np.asarray(prev)
        if sum(prev) == sum(min(10, len(s)) for s in sig):
            assert not d.any()
        else:
            assert sorted(d.tolist()) == [0, 0, 1]
        prev = cur


def pin_zero_spectra_last(alloc, info):
    # zero singular values add no information: positive ones go first, then the
    # zero-gain units in block order
    sig = [np.zeros(4), np.array([3.0, 2.0, 0.0, 0.0]), np.array([1.0, 0.5, 0.0])]
    assert list(alloc(sig, 3, 0, 4, 1.0)) == [0, 2, 1]
    assert list(alloc(sig, 4, 0, 4, 1.0)) == [0, 2, 2]
    assert list(alloc(sig, 6, 0, 4, 1.0)) == [2, 2, 2]     # ties at zero: lowest index first
    assert list(alloc(sig, 9, 0, 4, 1.0)) == [4, 3, 2]
    assert list(alloc(sig, 11, 0, 4, 1.0)) == [4, 4, 3]


def pin_rejects_unsorted(alloc, info):
    for bad in ([np.array([1.0, 2.0])], [np.array([1.0, -0.5])], [np.array([np.nan])]):
        with pytest.raises(ValueError):
            alloc(bad, 1, 0, 2, 1.0)


PINS = [pin_exhaustive, pin_information_closed_form, pin_equal_spectra_round_robin, pin_budget_edges,
        pin_eps_independence, pin_unit_increments, pin_zero_spectra_last, pin_rejects_unsorted]


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin(oracle.allocate_ranks, oracle.spectral_information)


MUTATIONS = [
    ("argmin instead of argmax", "i = int(np.argmax(nxt))", "i = int(np.argmin(np.where(nxt == -np.inf, np.inf, nxt)))"),
    ("ties to the highest index", "i = int(np.argmax(nxt))", "i = n - 1 - int(np.argmax(nxt[::-1]))"),
    ("gain of the wrong singular value", "x = sig[i][r[i]]\n", "x = sig[i][min(r[i] + 1, len(sig[i]) - 1)]\n"),
    ("cap ignores the block size", "cap = np.array([min(r_max, len(s))", "cap = np.array([r_max"),
    ("floor above the block size", "r = np.array([min(r_min, len(s))", "r = np.array([max(r_min, 0)"),
    ("two units per step", "left -= 1", "left -= 2"),
    ("stops one unit early", "while left > 0:", "while left > 1:"),
    ("information: eps squared dropped", "np.log1p(s * s / (eps * eps))", "np.log1p(s / eps)"),
    ("information: one value too many", "dtype=np.float64)[:r]", "dtype=np.float64)[:r + 1]"),
]


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_is_caught(name, old, new):
    src = inspect.getsource(oracle)
    assert src.count(old) == 1, f"mutation anchor not unique: {old!r}"
    ns = {"__name__": "oracle_mutant"}
    exec(compile(src.replace(old, new), "oracle_mutant", "exec"), ns)
    failed = []
    for pin in PINS:
        try:
            pin(ns["allocate_ranks"], ns["spectral_information"])
        except Exception:
            failed.append(pin.__name__)
    assert failed, f"planted mistake '{name}' passed every pin"


def test_workload_spectra_are_valid():
    import synth
    sp = synth.gen_spectra("tiny")
    for b, n in enumerate(sp.n_sv):
        row = sp.sigma[b, :n]
        assert np.all(row >= 0) and np.all(np.diff(row) <= 0)
    r = oracle.allocate_ranks([sp.sigma[b, :n] for b, n in enumerate(sp.n_sv)], sp.r_total, sp.r_min,
                              sp.r_max)
    assert r.sum() == sp.r_total and r.min() >= sp.r_min and r.max() <= sp.r_max


def test_exhaustive_search_hypothesis():
    # random small problems drawn by hypothesis, with equal values allowed: the
    # greedy reaches the exhaustive optimum of Eq. 6 (several maximisers may tie)
    hyp = pytest.importorskip("hypothesis")
    st = pytest.importorskip("hypothesis.strategies")

    @hyp.settings(max_examples=150, deadline=None, derandomize=True)
    @hyp.given(st.lists(st.lists(st.integers(0, 6), min_size=0, max_size=5), min_size=1, max_size=3),
               st.integers(0, 3), st.integers(0, 5), st.integers(0, 9))
    def check(rows, r_min, r_span, extra):
        sig = [np.array(sorted(r, reverse=True), dtype=np.float64) for r in rows]
        r_max = r_min + r_span
        floor = sum(min(r_min, len(s)) for s in sig)
        best, arg = _exhaustive(sig, floor + extra, r_min, r_max, 1.0)
        got = oracle.allocate_ranks(sig, floor + extra, r_min, r_max, 1.0)
        h = sum(oracle.spectral_information(s, int(r), 1.0) for s, r in zip(sig, got))
        assert abs(h - best) <= 1e-9 and tuple(int(x) for x in got) in arg

    check()
