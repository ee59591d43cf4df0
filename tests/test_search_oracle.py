"""Pins of the search-step oracle (oracle/nsga2.py, oracle.genome_mask) against
what the definitions fix: brute-force front peeling, closed-form crowding
distances, hand replays of the tournaments, and the invariants of messy
crossover.  CPU only."""
import itertools
import math
import random

import numpy as np
import pytest

import oracle
from oracle import nsga2 as ns


def _brute_fronts(objs):
    """Front index by repeatedly removing the points no remaining point dominates."""
    remaining = set(range(len(objs)))
    rank, r = [None] * len(objs), 0
    while remaining:
        front = [p for p in remaining if not any(ns.dominates(objs[q], objs[p]) for q in remaining)]
        for p in front:
            rank[p] = r
        remaining -= set(front)
        r += 1
    return rank


@pytest.mark.parametrize("seed,n,m,levels", [(1, 12, 2, 5), (2, 30, 2, 4), (3, 25, 3, 3), (4, 40, 2, 1000),
                                             (5, 1, 2, 3), (6, 9, 1, 4)])
def test_nondominated_sort_matches_brute_force_peeling(seed, n, m, levels):
    rng = random.Random(seed)
    objs = [tuple(rng.randrange(levels) for _ in range(m)) for _ in range(n)]
    rank = ns.nondominated_sort(objs)
    assert rank == _brute_fronts(objs)
    for a, b in itertools.permutations(range(n), 2):
        if rank[a] == rank[b]:
            assert not ns.dominates(objs[a], objs[b])          # a front is mutually non-dominated
    for p in range(n):
        if rank[p] > 0:                                          # dominated by the front above
            assert any(ns.dominates(objs[q], objs[p]) for q in range(n) if rank[q] == rank[p] - 1)


def test_dominance_definition_edge_cases():
    assert ns.dominates((1, 2), (1, 3)) and ns.dominates((0, 0), (1, 1))
    assert not ns.dominates((1, 2), (1, 2))                      # equal points do not dominate
    assert not ns.dominates((1, 3), (2, 2)) and not ns.dominates((2, 2), (1, 3))


@pytest.mark.parametrize("n", [3, 5, 11])
def test_crowding_distance_of_an_evenly_spaced_front(n):
    """Points (i, n-1-i) form one front; an interior point's neighbours are 2
    apart in each objective whose range is n-1: distance 2 * 2/(n-1)."""
    objs = [(float(i), float(n - 1 - i)) for i in range(n)]
    rank = ns.nondominated_sort(objs)
    assert set(rank) == {0}
    d = ns.crowding_distance(objs, rank)
    assert d[0] == math.inf and d[-1] == math.inf
    for i in range(1, n - 1):
        assert d[i] == 2.0 / (n - 1) + 2.0 / (n - 1)


def test_crowding_distance_closed_form_and_constant_objective():
    objs = [(0.0, 5.0, 1.0), (1.0, 3.0, 1.0), (4.0, 1.0, 1.0), (10.0, 0.0, 1.0)]
    rank = ns.nondominated_sort(objs)
    assert rank == [0, 0, 0, 0]
    d = ns.crowding_distance(objs, rank)
    # interior point 1: (4-0)/10 + (5-1)/5 ; point 2: (10-1)/10 + (3-0)/5 ; objective 3 is constant
    assert d[1] == 4.0 / 10.0 + 4.0 / 5.0 and d[2] == 9.0 / 10.0 + 3.0 / 5.0
    assert d[0] == math.inf and d[3] == math.inf
    # two-point and one-point fronts are all boundary
    assert ns.crowding_distance([(0, 1), (1, 0)], [0, 0]) == [math.inf, math.inf]
    assert ns.crowding_distance([(3, 3)], [0]) == [math.inf]


@pytest.mark.parametrize("seed", [7, 8])
def test_selection_elites_and_tournaments_by_hand(seed):
    rng = random.Random(seed)
    objs = [(rng.random(), rng.random()) for _ in range(20)]
    rank = ns.nondominated_sort(objs)
    dist = ns.crowding_distance(objs, rank)
    out = ns.select(rank, dist, 5, 20, seed, 3)
    assert len(out) == 20
    elites = out[:5]
    for a, b in zip(elites, elites[1:]):
        assert ns.crowded_better(a, b, rank, dist)
    for p in range(20):                                        # nobody outside is better than the last elite
        if p not in elites:
            assert not ns.crowded_better(p, elites[-1], rank, dist)
    for j, w in enumerate(out[5:]):
        r = oracle.philox((j, 3, 0, 7), (seed, 0))
        a, b = (int(r[0]) * 20) >> 32, (int(r[1]) * 20) >> 32
        expect = a if (rank[a], -dist[a], a) <= (rank[b], -dist[b], b) else b
        assert w == expect


def test_initial_population_has_three_edits_in_range():
    pop = ns.initial(50, 11, 0.4)
    kinds = set()
    for i, ind in enumerate(pop):
        assert [e[1] for e in ind] == [3 * i, 3 * i + 1, 3 * i + 2]
        for kind, _, value in ind:
            kinds.add(kind)
            if kind == ns.LR_EDIT:
                f = float(np.uint32(value).view(np.float32))
                assert 0.5 <= f <= 2.0
            else:
                assert int(0.4 * 2**24) - 1 <= value <= 2**24
    assert kinds == {ns.LR_EDIT, ns.PRUNE_EDIT}


def test_messy_crossover_keeps_the_edits_of_both_parents():
    pop = ns.initial(8, 12, 0.5)
    pop[3] = pop[3] + pop[5]                                   # unequal lengths
    kids = ns.breed(pop, 12, 1, cxpb=1.0, mutpb=0.0, rho_lo=0.5, id_base=1000, max_edits=64)
    for i in range(0, 8, 2):
        assert sorted(kids[i] + kids[i + 1]) == sorted(pop[i] + pop[i + 1])
    same = ns.breed(pop, 12, 1, cxpb=0.0, mutpb=0.0, rho_lo=0.5, id_base=1000, max_edits=64)
    assert same == pop
    cut = ns.breed(pop, 12, 1, cxpb=1.0, mutpb=0.0, rho_lo=0.5, id_base=1000, max_edits=2)
    assert all(len(k) <= 2 for k in cut)


def test_mutation_appends_one_edit_with_the_childs_id():
    pop = ns.initial(6, 13, 0.5)
    kids = ns.breed(pop, 13, 2, cxpb=0.0, mutpb=1.0, rho_lo=0.5, id_base=500, max_edits=64)
    for i in range(6):
        assert kids[i][:-1] == pop[i] and kids[i][-1][1] == 500 + i
    full = ns.breed(pop, 13, 2, cxpb=0.0, mutpb=1.0, rho_lo=0.5, id_base=500, max_edits=3)
    assert full == pop                                         # no room: no mutation


def test_apply_multiplies_rates_and_collects_prunes():
    half = int(np.float32(0.5).view(np.uint32))
    four = int(np.float32(4.0).view(np.uint32))
    edits = [(ns.LR_EDIT, 1, half), (ns.PRUNE_EDIT, 2, 2**23), (ns.LR_EDIT, 3, four), (ns.PRUNE_EDIT, 4, 2**22)]
    lr, ids, th, dens = ns.apply(edits, 0.01)
    assert lr == float(np.float32(np.float32(np.float32(0.01) * np.float32(0.5)) * np.float32(4.0)))
    assert ids == [2, 4] and th == [2**23, 2**22] and dens == 0.5 * 0.25
    assert ns.apply([], 0.05)[1:] == ([], [], 1.0)


def test_genome_mask_extends_the_initial_masks():
    dims = [40, 24, 6]
    for v in (0, 5):
        _, _, th = oracle.variant_hparams(21, v, (1e-3, 0.3), (0.4, 1.0))
        _, m = oracle.variant_init(21, v, dims, th)
        assert np.array_equal(oracle.genome_mask(21, dims, [v], [th]), m)   # one edit = variant v's mask
    a = oracle.genome_mask(21, dims, [7], [2**23])
    b = oracle.genome_mask(21, dims, [9], [3 * 2**22])
    both = oracle.genome_mask(21, dims, [7, 9], [2**23, 3 * 2**22])
    assert np.array_equal(both, a & b)                         # edits combine by logical and
    assert np.array_equal(oracle.genome_mask(21, dims, [9, 7], [3 * 2**22, 2**23]), both)
    assert oracle.genome_mask(21, dims, [], []).all()          # no edit keeps everything
    n = both.size                                              # kept fraction near 1/2 * 3/4
    assert abs(both.mean() - 0.375) < 5 * math.sqrt(0.375 * 0.625 / n)


def _narrow(params, dims, widths):
    """Parameters of the network whose hidden layers keep their first widths[l] units."""
    out, off = [], 0
    for l in range(1, len(dims)):
        din, dout = dims[l - 1], dims[l]
        W = params[off:off + din * dout].reshape(din, dout)
        b = params[off + din * dout:off + din * dout + dout]
        out += [W[:widths[l - 1], :widths[l]].ravel(), b[:widths[l]]]
        off += din * dout + dout
    return np.concatenate(out)


@pytest.mark.parametrize("mode", ["f64", "f32", "bf16"])
def test_a_narrowed_net_computes_what_the_narrow_net_computes(mode):
    """Structural width edits clear the weights into and out of the removed
    units and their biases; training the wide net then equals training the
    narrow net exactly (the removed units contribute exact zeros)."""
    dims = [20, 12, 9, 4]
    widths = [20, 7, 5, 4]
    rng = np.random.default_rng(8)
    params = rng.normal(0, 0.4, oracle.param_count(dims))
    prune = (rng.random(oracle.weight_count(dims)) < 0.8).astype(np.uint8)
    mask, bmask = oracle.structure_masks(dims, widths, [1, 1, 1], prune)
    bias_off = 0
    for l in range(1, len(dims)):                               # the wide net starts masked
        off = sum(dims[j - 1] * dims[j] + dims[j] for j in range(1, l))
        moff = sum(dims[j - 1] * dims[j] for j in range(1, l))
        n = dims[l - 1] * dims[l]
        params[off:off + n] *= mask[moff:moff + n]
        params[off + n:off + n + dims[l]] *= bmask[bias_off:bias_off + dims[l]]
        bias_off += dims[l]
    X = rng.random((64, 20), dtype=np.float32)
    y = rng.integers(0, 4, 64).astype(np.int32)
    perm = np.arange(64, dtype=np.uint32)
    wide = params.copy()
    narrow = _narrow(params, dims, widths)
    nmask = _narrow(np.concatenate([np.concatenate([mask[sum(dims[j - 1] * dims[j] for j in range(1, l)):][:dims[l - 1] * dims[l]],
                                                    np.ones(dims[l])]) for l in range(1, len(dims))]).astype(np.float64),
                    dims, widths)
    nmask = np.concatenate([nmask[sum(widths[j - 1] * widths[j] + widths[j] for j in range(1, l)):][:widths[l - 1] * widths[l]]
                            for l in range(1, len(dims))]).astype(np.uint8)
    rw = oracle.train_steps(mode, dims, wide, mask, 0.1, X, y, perm, 16, 0, 4, bmask=bmask)
    rn = oracle.train_steps(mode, widths, narrow, nmask, 0.1, X, y, perm, 16, 0, 4)
    assert rw == rn
    assert np.array_equal(_narrow(wide, dims, widths), narrow)


def test_removed_biases_stay_zero_and_the_rest_trains():
    dims = [10, 6, 3]
    rng = np.random.default_rng(9)
    params = rng.normal(0, 0.4, oracle.param_count(dims))
    mask, bmask = oracle.structure_masks(dims, dims, [0, 1])
    params[60:66] = 0.0                                         # layer-1 biases removed from the start
    X = rng.random((32, 10), dtype=np.float32)
    y = rng.integers(0, 3, 32).astype(np.int32)
    before = params.copy()
    oracle.train_steps("f64", dims, params, mask, 0.2, X, y, np.arange(32, dtype=np.uint32), 8, 0, 4, bmask=bmask)
    assert np.all(params[60:66] == 0.0) and not np.array_equal(params[84:87], before[84:87])
    assert list(bmask) == [0] * 6 + [1] * 3


def test_structure_and_density_of_edit_lists():
    dims = [100, 40, 20, 10]
    edits = [(ns.WIDTH_EDIT, 1, 30), (ns.PRUNE_EDIT, 5, 2**23), (ns.WIDTH_EDIT, 1, 35), (ns.BIAS_EDIT, 3, 0),
             (ns.WIDTH_EDIT, 2, 25)]
    widths, keep = ns.structure(edits, dims)
    assert widths == [100, 30, 20, 10] and keep == [1, 1, 0]
    total = 100 * 40 + 40 * 20 + 20 * 10
    assert ns.density(edits, dims) == 0.5 * ((100 * 30 + 30 * 20 + 20 * 10) / total)
