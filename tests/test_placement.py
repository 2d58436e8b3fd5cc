"""Expert placement and router-aided dynamic loading (host side): pinned to
the paper's Table tab:vars executed-expert expectations, its router-aided
loading example (Sec. "Load balancing strategies") and busy full loading,
and checked against brute force."""
import itertools
import math
import random

import pytest

from paper_2506_23635_amd import perf_model as pm
from paper_2506_23635_amd import placement as pl


def test_two_nodes_reproduce_table_tab_vars():
    # E[#exec. experts / node / layer] = 2.65 for 2 nodes (Table tab:vars):
    # the busiest of two 8-expert nodes under uniform top-4 routing
    e = pl.expected_busiest_load(pl.contiguous(16, 2), 4)
    assert round(e, 2) == 2.65


def test_four_nodes_with_pairwise_replicas_reproduce_table_tab_vars():
    # 4 nodes: 1.57 with overlapping experts (Sec. "Scalability").  The
    # paper does not print the placement; two pairs of nodes that each hold
    # one half of the experts (every expert on 2 nodes) gives the printed
    # value, the non-overlapping split does not
    pairs = pl.replicated(16, 4, copies=2, shift=2)
    assert pairs.experts_per_gpu() == [8, 8, 8, 8]
    assert pairs.local(0) == pairs.local(2) and pairs.local(1) == pairs.local(3)
    assert round(pl.expected_busiest_load(pairs, 4), 2) == 1.57
    assert round(pl.expected_busiest_load(pl.contiguous(16, 4), 4), 2) != 1.57


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 8, 16])
def test_contiguous_expectation_matches_count_enumeration(n):
    # two independent computations: the planner's exact assignment and the
    # performance model's per-node selected counts
    a = pl.expected_busiest_load(pl.contiguous(16, n), 4)
    b = pm.expected_busiest_node_experts(n)
    assert a == pytest.approx(b, abs=1e-12)


def test_busy_full_loading_runs_every_held_expert():
    # L_B on 2 nodes: 8 experts per node per layer (Sec. "Load balancing
    # strategies"), against 2.65 on average with L_R
    assert pl.busy_full_loads(pl.contiguous(16, 2)) == [8, 8]


def test_router_aided_example_fills_from_lru():
    # The paper's example: node 1 selects three experts, node 2 one, so node
    # 2 adds two least recently used experts and both execute three
    lr = pl.LRPlanner(pl.contiguous(16, 2))
    p = lr.plan([0, 1, 2, 9])
    assert p["max_load"] == 3
    assert p["executed"][0] == [0, 1, 2] and p["filled"][0] == []
    assert p["filled"][1] == [8, 10]          # never used; lower ids first
    assert p["executed"][1] == [8, 9, 10]
    # next layer: 8, 9, 10 were just used, so the fill takes the others
    p = lr.plan([3, 4, 5, 12])
    assert p["filled"][1] == [11, 13]
    assert p["executed"][1] == [11, 12, 13]
    # once every expert has run, the least recently used wins: step 2 fills
    # 15 (never used) and 8, step 3 fills 9 and 10 (step 0), so step 4 takes
    # 12 and 13 (last used at step 1)
    assert lr.plan([0, 1, 2, 14])["filled"][1] == [8, 15]
    assert lr.plan([0, 1, 2, 15])["filled"][1] == [9, 10]
    p = lr.plan([0, 1, 2, 11])
    assert p["filled"][1] == [12, 13]


def test_router_aided_without_fill_runs_only_selected():
    lr = pl.LRPlanner(pl.contiguous(16, 2), fill=False)
    p = lr.plan([0, 1, 2, 9])
    assert p["executed"] == [[0, 1, 2], [9]] and p["filled"] == [[], []]


def test_every_node_executes_the_layer_max_with_fill():
    rng = random.Random(7)
    for n in (2, 3, 4):
        lr = pl.LRPlanner(pl.contiguous(16, n))
        for _ in range(50):
            sel = rng.sample(range(16), 4)
            p = lr.plan(sel)
            assert all(len(x) == p["max_load"] for x in p["executed"])
            for g, ex in enumerate(p["executed"]):
                assert set(ex) <= set(lr.placement.local(g))
            assert sorted(e for e, _ in p["assign"].items()) == sorted(sel)


def _brute_best(sel, P):
    best = None
    for choice in itertools.product(*[P.holders[e] for e in sel]):
        m = max([choice.count(g) for g in range(P.n_gpus)])
        best = m if best is None else min(best, m)
    return best


def test_assignment_is_optimal_against_brute_force():
    rng = random.Random(3)
    for _ in range(300):
        E, G = rng.randint(2, 8), rng.randint(1, 4)
        holders = tuple(tuple(sorted(rng.sample(range(G), rng.randint(1, G)))) for _ in range(E))
        P = pl.Placement(G, holders)
        sel = rng.sample(range(E), rng.randint(1, E))
        where = pl.assign(sel, P)
        assert sorted(where) == sorted(sel)
        assert all(g in P.holders[e] for e, g in where.items())
        assert max(pl.loads(where, G)) == _brute_best(sel, P)


def test_assignment_depends_on_the_set_only():
    P = pl.replicated(16, 4, copies=2)
    rng = random.Random(11)
    for _ in range(100):
        sel = rng.sample(range(16), 6)
        assert pl.assign(sel, P) == pl.assign(list(reversed(sel)), P)
        assert pl.assign(sel + sel, P) == pl.assign(sel, P)


def test_full_replication_balances_perfectly():
    P = pl.replicated(16, 8, copies=8)
    for k in range(1, 17):
        for sel in itertools.islice(itertools.combinations(range(16), k), 200):
            assert max(pl.loads(pl.assign(sel, P), 8)) == math.ceil(k / 8)


def test_replication_never_raises_the_expected_busiest_load():
    for n in (2, 4, 8):
        prev = None
        for copies in range(1, n + 1):
            p = pl.contiguous(16, n) if copies == 1 else pl.replicated(16, n, copies)
            e = pl.expected_busiest_load(p, 4)
            assert prev is None or e <= prev + 1e-12
            prev = e
        assert prev == pytest.approx(math.ceil(4 / n))


def test_mi355x_memory_fit():
    # one MI355X holds every DBRX expert of all 40 layers (254 GB) and the
    # attention weights (7 GB) in 288 GB
    assert pl.fits_mi355x(pl.contiguous(16, 1))
    assert pl.DBRX_EXPERT_ALL_LAYERS * 16 == 253_671_505_920
    rows = pl.mi355x_placements(gpus=(2, 4))
    assert {(r["gpus"], r["copies"]) for r in rows} == {(2, 1), (2, 2), (4, 1), (4, 2), (4, 3), (4, 4)}


def test_bad_inputs():
    with pytest.raises(ValueError):
        pl.Placement(2, ((0,), (2,)))
    with pytest.raises(ValueError):
        pl.Placement(2, ((1, 0),))
    with pytest.raises(ValueError):
        pl.assign([16], pl.contiguous(16, 2))
    with pytest.raises(ValueError):
        pl.replicated(16, 4, copies=2, shift=4)
    assert pl.assign([], pl.contiguous(16, 2)) == {}


def test_placement_predictions_follow_eq_pm():
    rows = pl.mi355x_placement_predictions(6500.0, 1000.0, gpus=(2, 4))
    model, hw = pm.dbrx_exact(), pm.mi355x_hardware(6500.0, 1000.0, 20e-6, 150.0)
    for r in rows:
        est = pm.estimate(r["exec_experts"], model, hw, n_nodes=r["gpus"])
        assert r["ms_per_token"] == pytest.approx(est.time * 1e3)
    # more copies never predict a slower token on the same GPU count
    for n in (2, 4):
        t = [r["ms_per_token"] for r in rows if r["gpus"] == n]
        assert all(b <= a + 1e-12 for a, b in zip(t, t[1:]))
