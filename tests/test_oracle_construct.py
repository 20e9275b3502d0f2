"""Pins of ``oracle.construct`` (offline construction, Alg. 1).

The greedy selection is pinned by what defines it rather than by re-running
it: for radius-prioritised de-duplication the appended sequence is the one
and only sequence in which (a) candidates appear by decreasing radius (ties:
lower index), (b) no appended entry lies strictly inside the ball of an
entry present before it, and (c) every eligible candidate that was passed
over either lies inside such a ball or found its class full (or the total
budget was used).  K-center is pinned by the farthest-first property checked
by brute force, and the priority strategy by an independent sort.  Hand
cases fix strictness, ties, budgets and eligibility; planted mutants must
break a pin.
"""
import inspect

import numpy as np
import pytest

import oracle
from oracle import lipcache_oracle as base


def line(xs, d=32):
    z = np.zeros((len(xs), d), np.float32)
    z[:, 0] = xs
    return z


def fresh(d=32, cap=1000, store="f32"):
    return oracle.CacheState(d=d, capacity=cap, store=store)


def mixture(n=600, d=32, C=5, seed=0):
    rng = np.random.default_rng(seed)
    mu = 3.0 * rng.standard_normal((C, d))
    lab = rng.integers(0, C, n).astype(np.int32)
    z = (mu[lab] + rng.standard_normal((n, d))).astype(np.float32)
    r = rng.uniform(0.5, 5.0, n).astype(np.float32)
    r[rng.random(n) < 0.05] = 0.0
    return z, lab, r


def check_dedup_definition(st0_z, st0_r, z, lab, r, sel, budget, per_class, guard=None):
    """(a), (b), (c) of the module docstring, by brute force."""
    z64 = z.astype(np.float64)
    elig = r > 0
    if guard is not None:
        elig &= guard == lab
    idx = np.flatnonzero(elig)
    order = idx[np.lexsort((idx, -r[idx].astype(np.float64)))]
    pos = {int(i): k for k, i in enumerate(order)}
    assert all(pos[int(a)] < pos[int(b)] for a, b in zip(sel[:-1], sel[1:])), "(a) order"
    centres = [(c, float(rad)) for c, rad in zip(st0_z.astype(np.float64), st0_r) if rad > 0]
    chosen = set()
    counts = {}
    k = 0
    for i in order:
        if k < sel.size and int(sel[k]) == int(i):
            inside = any(np.sum((z64[i] - c) ** 2) < rad * rad for c, rad in centres)
            assert not inside, "(b) an appended entry lies inside an earlier ball"
            centres.append((z64[i], float(r[i])))
            chosen.add(int(i))
            counts[int(lab[i])] = counts.get(int(lab[i]), 0) + 1
            k += 1
            continue
        if len(chosen) >= budget:
            break
        full = per_class > 0 and counts.get(int(lab[i]), 0) >= per_class
        inside = any(np.sum((z64[i] - c) ** 2) < rad * rad for c, rad in centres)
        assert full or inside, f"(c) candidate {i} was passed over without a reason"
    assert k == sel.size


def test_hand_case_line():
    z = line([0, 1, 1.5, 3, 10])
    r = np.array([2, 1, 0.4, 1.5, 1], np.float32)
    st = fresh()
    sel = oracle.construct(st, z, np.zeros(5, np.int32), r)
    assert sel.tolist() == [0, 3, 4]
    assert st.n == 3 and st.r.tolist() == [2, 1.5, 1]


def test_strict_ball_and_ties():
    # candidate 1 sits exactly on the boundary of candidate 0's ball: not a duplicate
    z = line([0, 2, 0.5, 0.5])
    r = np.array([2, 1, 1, 1], np.float32)
    sel = oracle.construct(fresh(), z, np.zeros(4, np.int32), r)
    assert sel.tolist() == [0, 1]
    # equal radii: the lower index goes first
    z = line([0, 5, 10])
    sel = oracle.construct(fresh(), z, np.zeros(3, np.int32), np.array([1, 1, 1], np.float32),
                           strategy="priority", priority=np.array([1, 1, 1], np.float32), budget_total=2)
    assert sel.tolist() == [0, 1]


def test_budgets_eligibility_and_existing_entries():
    z = line([0, 10, 20, 30, 40, 50])
    lab = np.array([0, 0, 1, 1, 0, 2], np.int32)
    r = np.array([6, 5, 4, 3, 2, 0], np.float32)
    assert oracle.construct(fresh(), z, lab, r, budget_per_class=1).tolist() == [0, 2]
    assert oracle.construct(fresh(), z, lab, r, budget_total=3).tolist() == [0, 1, 2]
    guard = np.array([0, 1, 1, 1, 0, 2], np.int32)          # candidate 1 is label-inconsistent
    assert oracle.construct(fresh(), z, lab, r, guard_label=guard).tolist() == [0, 2, 3, 4]
    st = fresh()
    oracle.insert(st, line([21]), np.array([7], np.int32), np.array([2], np.float32))
    assert oracle.construct(st, z, lab, r).tolist() == [0, 1, 3, 4]   # 20 lies in the ball at 21
    with pytest.raises(oracle.CapacityError):
        oracle.construct(fresh(cap=2), z, lab, r, budget_total=3)


@pytest.mark.parametrize("per_class,budget,guarded", [(0, 10 ** 5, False), (20, 10 ** 5, False), (0, 37, False),
                                                      (15, 50, True)])
def test_dedup_definition_on_mixture(per_class, budget, guarded):
    z, lab, r = mixture()
    guard = None
    if guarded:
        guard = lab.copy()
        guard[::7] = (guard[::7] + 1) % 5
    st = fresh(cap=10 ** 6)
    oracle.insert(st, z[:3] + 0.25, lab[:3], np.full(3, 2.0, np.float32))   # a few pre-existing entries
    z0, r0 = st.z.copy(), st.r.copy()
    sel = oracle.construct(st, z, lab, r, budget_total=budget, budget_per_class=per_class, guard_label=guard)
    assert 10 < sel.size < 600
    check_dedup_definition(z0, r0, z, lab, r, sel, budget, per_class, guard)
    if per_class:
        assert np.bincount(lab[sel]).max() <= per_class


def test_priority_strategy_is_a_sorted_take():
    z, lab, r = mixture(seed=3)
    pri = np.random.default_rng(9).random(z.shape[0]).astype(np.float32)
    sel = oracle.construct(fresh(cap=10 ** 6), z, lab, r, strategy="priority", priority=pri, budget_per_class=12,
                           budget_total=40)
    want, counts = [], np.zeros(5, int)
    for i in sorted(np.flatnonzero(r > 0), key=lambda i: (-float(pri[i]), i)):
        if len(want) == 40:
            break
        if counts[lab[i]] < 12:
            want.append(int(i))
            counts[lab[i]] += 1
    assert sel.tolist() == want


@pytest.mark.parametrize("per_class", [0, 8])
def test_kcenter_farthest_first(per_class):
    z, lab, r = mixture(n=300, seed=5)
    sel = oracle.construct(fresh(cap=10 ** 6), z, lab, r, strategy="kcenter", budget_per_class=per_class,
                           budget_total=30)
    assert sel.size == 30
    z64 = z.astype(np.float64)
    elig = r > 0
    groups = [sel] if per_class == 0 else [sel[lab[sel] == c] for c in sorted(set(lab[sel].tolist()))]
    if per_class:
        assert [int(lab[g[0]]) for g in groups] == sorted(int(lab[g[0]]) for g in groups)
        assert all(g.size <= per_class for g in groups)
    for g in groups:
        pool = np.flatnonzero(elig) if per_class == 0 else np.flatnonzero(elig & (lab == lab[g[0]]))
        first = pool[np.lexsort((pool, -r[pool].astype(np.float64)))[0]]
        assert g[0] == first
        for k in range(1, g.size):
            d2 = np.min(((z64[pool][:, None, :] - z64[g[:k]][None, :, :]) ** 2).sum(-1), axis=1)
            d2[np.isin(pool, g[:k])] = -1.0
            best = np.flatnonzero(d2 == d2.max())
            assert g[k] == pool[best[0]], f"pick {k} is not the (lowest-index) farthest candidate"


def test_bf16_store_uses_rounded_values():
    z = line([0.0, 1.0 + 2 ** -9])           # rounds to 1.0 in bfloat16
    st = fresh(store="bf16")
    sel = oracle.construct(st, z, np.zeros(2, np.int32), np.array([1.0, 0.5], np.float32))
    assert sel.tolist() == [0, 1]            # exactly on the boundary after rounding: not a duplicate
    assert st.z[1, 0] == 1.0


def _mutated(old, new):
    src = inspect.getsource(base.construct)
    assert old in src
    ns = dict(vars(base))
    exec(compile(src.replace(old, new), "<mutant>", "exec"), ns)
    return ns["construct"]


MUTANTS = {
    "non-strict ball": ("d2 < cr2", "d2 <= cr2"),
    "existing entries ignored": ("cz = state.z.astype(np.float64)\n        cr2 = state.r.astype(np.float64) ** 2\n"
                                 "        clive = state.r > 0",
                                 "cz = state.z[:0].astype(np.float64)\n        cr2 = state.r[:0].astype(np.float64) ** 2\n"
                                 "        clive = state.r[:0] > 0"),
    "ties to the higher index": ("order = idx[np.lexsort((idx, -key[idx].astype(np.float64)))]",
                                 "order = idx[np.lexsort((-idx, -key[idx].astype(np.float64)))]"),
    "class budget ignored": ("if not class_open(c):", "if False:"),
    "ascending radius": ("-key[idx].astype(np.float64)", "key[idx].astype(np.float64)"),
    "k-center nearest-first": ("j = int(np.flatnonzero(cand == cand.max())[0])",
                               "j = int(np.flatnonzero(cand == np.where(taken, np.inf, mind).min())[0])"),
}


def _all_pins(fn, monkeypatch):
    monkeypatch.setattr(oracle, "construct", fn)
    test_hand_case_line()
    test_strict_ball_and_ties()
    test_budgets_eligibility_and_existing_entries()
    for args in [(0, 10 ** 5, False), (20, 10 ** 5, False), (15, 50, True)]:
        test_dedup_definition_on_mixture(*args)
    test_priority_strategy_is_a_sorted_take()
    test_kcenter_farthest_first(0)
    test_bf16_store_uses_rounded_values()


@pytest.mark.parametrize("name", list(MUTANTS))
def test_construct_mutants_are_caught(name, monkeypatch):
    fn = _mutated(*MUTANTS[name])
    with pytest.raises(AssertionError):
        _all_pins(fn, monkeypatch)
