"""Pins of the PSA-Search oracle (oracle/search.py): selections worked by hand from
Algorithm 3 and the dual interface, closed-form losses, and invariants of the rules."""
import numpy as np
import pytest

import oracle
from oracle import search as osearch

# (loss, sparsity) of six candidates of one head.  Sorted by loss (stable):
# 1 (0.004, .30), 3 (0.006, .60), 5 (0.006, .40), 0 (0.010, .50), 2 (0.020, .70), 4 (0.030, .90).
RESULTS = [(0.010, 0.50), (0.004, 0.30), (0.020, 0.70), (0.006, 0.60), (0.030, 0.90), (0.006, 0.40)]


@pytest.mark.parametrize("alpha,expect", [
    (0.015, 3),    # start at 1; 3 is sparser and qualifies; 5 and 0 are not sparser; 2 and 4 fail alpha
    (0.025, 2),    # as above, then 2 (loss 0.020 <= alpha, sparsity .70 > .60)
    (0.030, 4),    # the bound is inclusive: 4 qualifies with loss exactly alpha
    (0.001, 1),    # nothing qualifies: the lowest-loss mask stays
    (1.000, 4),
])
def test_hand_worked_alpha_selection(alpha, expect):
    assert osearch.select_alpha(RESULTS, alpha) == expect


def test_equal_sparsity_keeps_the_lower_loss():
    # Strictly higher sparsity is needed to replace the current choice.
    assert osearch.select_alpha([(0.02, 0.5), (0.01, 0.5)], 1.0) == 1
    assert osearch.select_alpha([(0.01, 0.5), (0.01, 0.5)], 1.0) == 0     # stable sort: first


@pytest.mark.parametrize("target,expect", [
    (0.55, 3),     # candidates 3 (.006), 2 (.020), 4 (.030) reach .55: the lowest loss is 3
    (0.80, 4),
    (0.00, 1),     # every candidate qualifies: the lowest loss overall
    (0.95, 4),     # none reaches .95: the sparsest candidate
])
def test_hand_worked_target_selection(target, expect):
    assert osearch.select_target(RESULTS, target) == expect


def test_selection_invariants_on_random_results():
    rng = np.random.default_rng(0)
    for _ in range(200):
        res = [(float(rng.uniform(0, 0.05)), float(rng.choice(np.linspace(0, 0.95, 20)))) for _ in range(30)]
        last = -1.0
        for alpha in np.linspace(0, 0.06, 13):
            i = osearch.select_alpha(res, alpha)
            qualified = [j for j, (l, _) in enumerate(res) if l <= alpha]
            if qualified:
                assert res[i][0] <= alpha
                assert res[i][1] == max(res[j][1] for j in qualified)
            else:
                assert res[i][0] == min(l for l, _ in res)
            assert res[i][1] >= last - 1e-12 or not qualified    # sparsity never drops as alpha grows
            last = res[i][1] if qualified else last
        for target in np.linspace(0, 1, 11):
            i = osearch.select_target(res, target)
            ok = [j for j, (_, s) in enumerate(res) if s >= target]
            if ok:
                assert res[i][1] >= target and res[i][0] == min(res[j][0] for j in ok)


def test_l2_loss_closed_forms():
    x = np.random.default_rng(1).standard_normal((40, 8))
    assert osearch.l2_loss(x, x) == 0.0
    assert osearch.l2_loss(np.zeros_like(x), x) == pytest.approx(1.0)
    assert osearch.l2_loss(2 * x, x) == pytest.approx(1.0)
    assert osearch.l2_loss(1.01 * x, x) == pytest.approx(0.01)
    y = x + 0.1 * np.random.default_rng(2).standard_normal(x.shape)
    assert osearch.l2_loss(3.0 * y, 3.0 * x) == pytest.approx(osearch.l2_loss(y, x))


def test_head_results_closed_forms():
    rng = np.random.default_rng(3)
    n, d, block = 96, 8, 16
    nb = n // block
    q = np.zeros((n, d))
    k = rng.standard_normal((n, d))
    v = rng.standard_normal((n, d))
    full = np.ones((nb, nb), np.uint8)
    ident = np.eye(nb, dtype=np.uint8)
    res = osearch.head_results(q, k, v, [full, ident], block, 0.5)
    assert res[0] == (0.0, 0.0)
    # Q = 0: every weight is equal, so O_full is the mean of all V rows and O_ident of row i is
    # the mean of V over the block of i.
    o_full = np.tile(v.mean(0), (n, 1))
    o_id = np.repeat(v.reshape(nb, block, d).mean(1), block, axis=0)
    expect = np.sqrt(((o_id - o_full) ** 2).sum() / (o_full ** 2).sum())
    assert res[1][0] == pytest.approx(expect, rel=1e-12) and res[1][1] == pytest.approx(1 - 1 / nb)
    # constant values: every mask returns the same output, loss 0
    res = osearch.head_results(rng.standard_normal((n, d)), k, np.ones((n, d)), [ident], block, 0.5)
    assert res[0][0] == pytest.approx(0.0, abs=1e-14)


def _pins_pass():
    try:
        for alpha, expect in [(0.015, 3), (0.025, 2), (0.030, 4), (0.001, 1)]:
            test_hand_worked_alpha_selection(alpha, expect)
        test_equal_sparsity_keeps_the_lower_loss()
        for target, expect in [(0.55, 3), (0.95, 4)]:
            test_hand_worked_target_selection(target, expect)
    except AssertionError:
        return False
    return True


def test_mutant_non_strict_sparsity_is_caught(monkeypatch):
    def mutant(results, alpha):
        order = sorted(range(len(results)), key=lambda i: results[i][0])
        best = order[0]
        for i in order:
            if results[i][0] <= alpha and results[i][1] >= results[best][1]:
                best = i
        return best
    monkeypatch.setattr(osearch, "select_alpha", mutant)
    assert not _pins_pass()


def test_mutant_exclusive_alpha_is_caught(monkeypatch):
    def mutant(results, alpha):
        order = sorted(range(len(results)), key=lambda i: results[i][0])
        best = order[0]
        for i in order:
            if results[i][0] < alpha and results[i][1] > results[best][1]:
                best = i
        return best
    monkeypatch.setattr(osearch, "select_alpha", mutant)
    assert not _pins_pass()


def test_mutant_first_candidate_start_is_caught(monkeypatch):
    def mutant(results, alpha):
        best = 0
        for i in sorted(range(len(results)), key=lambda i: results[i][0]):
            if results[i][0] <= alpha and results[i][1] > results[best][1]:
                best = i
        return best
    monkeypatch.setattr(osearch, "select_alpha", mutant)
    assert not _pins_pass()
