"""The search step's host code in libgevo (NSGA-II ranking and selection,
initial population, breeding) against the oracle, bit for bit, through the
C-ABI.  These entry points run on the host, so the tests run on the CPU."""
import ctypes
import math
import random

import numpy as np
import pytest

from oracle import nsga2 as ns

g = pytest.importorskip("paper_2310_10211_amd")


def _lib():
    try:
        return g.lib()
    except ImportError as e:            # the library is built by __graft_entry__.build()
        pytest.skip(str(e))


@pytest.mark.parametrize("seed,n,m,kind", [(1, 40, 2, "int"), (2, 64, 2, "float"), (3, 50, 3, "int"),
                                           (4, 17, 1, "int"), (5, 1, 2, "float"), (6, 256, 2, "float")])
def test_rank_and_crowding_match_the_oracle(seed, n, m, kind):
    _lib()
    rng = random.Random(seed)
    if kind == "int":
        objs = [tuple(float(rng.randrange(6)) for _ in range(m)) for _ in range(n)]
    else:
        objs = [tuple(rng.random() for _ in range(m)) for _ in range(n)]
    rank, crowd = g.nsga2_rank(objs)
    ro = ns.nondominated_sort(objs)
    co = ns.crowding_distance(objs, ro)
    assert [int(r) for r in rank] == ro
    assert all((a == b) or (math.isinf(a) and math.isinf(b)) for a, b in zip(crowd, co))


@pytest.mark.parametrize("seed,n,n_elite,n_select,gen", [(7, 40, 16, 40, 1), (8, 20, 0, 20, 3), (9, 64, 16, 64, 5),
                                                        (10, 5, 5, 5, 2), (11, 30, 4, 12, 9)])
def test_selection_matches_the_oracle(seed, n, n_elite, n_select, gen):
    _lib()
    rng = random.Random(seed)
    objs = [(float(rng.randrange(5)), rng.random()) for _ in range(n)]
    rank, crowd = g.nsga2_rank(objs)
    ro = ns.nondominated_sort(objs)
    co = ns.crowding_distance(objs, ro)
    assert g.nsga2_select(rank, crowd, n_elite, n_select, seed, gen) == ns.select(ro, co, n_elite, n_select, seed, gen)


@pytest.mark.parametrize("n,seed,rho_lo,n_mut", [(64, 3, 0.3, 3), (7, 4, 0.5, 1), (100, 5, 0.0, 5)])
def test_initial_population_matches_the_oracle(n, seed, rho_lo, n_mut):
    _lib()
    assert g.genomes_initial(n, seed, rho_lo, n_mut, id_base=11) == ns.initial(n, seed, rho_lo, n_mut, id_base=11)


@pytest.mark.parametrize("n,seed,gen,cxpb,mutpb,max_edits", [(48, 3, 1, 0.8, 0.5, 16), (7, 4, 2, 1.0, 1.0, 6),
                                                             (32, 5, 7, 0.0, 0.0, 16), (21, 6, 3, 0.5, 0.3, 3)])
def test_breeding_matches_the_oracle(n, seed, gen, cxpb, mutpb, max_edits):
    _lib()
    parents = ns.initial(n, seed + 100, 0.4)
    for i in range(0, n, 5):                               # unequal lengths, some empty
        parents[i] = parents[i] + parents[(i + 1) % n] if i % 2 else []
    got = g.genomes_breed(parents, seed, gen, cxpb, mutpb, 0.4, 1000, max_edits)
    assert got == ns.breed(parents, seed, gen, cxpb, mutpb, 0.4, 1000, max_edits)


def test_search_entry_points_reject_bad_arguments():
    L = _lib()
    nan = np.array([[0.0, float("nan")]], np.float64)
    rank = np.zeros(1, np.uint32)
    crowd = np.zeros(1, np.float64)
    u32p = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32))
    f64p = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
    assert L.gevo_nsga2_rank(1, 2, f64p(nan), u32p(rank), f64p(crowd)) == -1
    assert L.gevo_nsga2_rank(1, 0, f64p(nan), u32p(rank), f64p(crowd)) == -1
    out = np.zeros(4, np.uint32)
    assert L.gevo_nsga2_select(1, u32p(rank), f64p(crowd), 2, 4, 1, 1, u32p(out)) == -1     # n_elite > n
    assert L.gevo_nsga2_select(4, u32p(out), f64p(np.zeros(4)), 3, 2, 1, 1, u32p(out)) == -1  # n_elite > n_select
    with pytest.raises(g.GevoError):
        g.genomes_breed([[(0, 1, 0x3F800000)]], 1, 0, 0.5, 0.5, 0.4, 0, 8)                   # generation 0
    with pytest.raises(g.GevoError):
        g.genomes_breed([[(0, 1, 0x3F800000)]], 1, 1, 1.5, 0.5, 0.4, 0, 8)                   # cxpb > 1
    with pytest.raises(g.GevoError):
        g.genomes_initial(3, 1, 1.5)                                                         # rho_lo > 1
    off = np.array([0, 2, 1], np.uint32)                                                     # decreasing offsets
    edits = (g.GevoEdit * 2)()
    oo = np.zeros(3, np.uint32)
    assert L.gevo_genomes_breed(2, u32p(off), edits, 1, 1, 0.5, 0.5, 0.4, 0, 8, 0.0, 0, None, u32p(oo), edits,
                                8) == -1
    good = np.array([0, 1, 2], np.uint32)
    assert L.gevo_genomes_breed(2, u32p(good), edits, 1, 1, 0.5, 0.5, 0.4, 0, 8, 0.0, 0, None, u32p(oo), edits,
                                3) == -1                                              # capacity below n + edits
    with pytest.raises(g.GevoError):
        g.genomes_initial(3, 1, 0.4, struct_p=0.5)                                   # structural draws need dims


@pytest.mark.parametrize("dims,struct_p,seed", [([784, 256, 10], 0.3, 21), ([200, 96, 64, 10], 0.5, 22),
                                                ([50, 10], 1.0, 23)])
def test_structural_draws_match_the_oracle(dims, struct_p, seed):
    _lib()
    init = g.genomes_initial(40, seed, 0.4, 3, 0, struct_p, dims)
    assert init == ns.initial(40, seed, 0.4, 3, 0, struct_p, dims)
    kinds = {e[0] for ind in init for e in ind}
    assert ns.BIAS_EDIT in kinds
    if len(dims) > 2:
        assert ns.WIDTH_EDIT in kinds
        for ind in init:
            for kind, l, w in ind:
                if kind == ns.WIDTH_EDIT:
                    assert 1 <= l <= len(dims) - 2 and 1 <= w <= dims[l]
    kids = g.genomes_breed(init, seed, 2, 0.8, 1.0, 0.4, 500, 16, struct_p, dims)
    assert kids == ns.breed(init, seed, 2, 0.8, 1.0, 0.4, 500, 16, struct_p, dims)
