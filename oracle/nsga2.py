"""Oracle of the GEVO-ML search step: NSGA-II selection and breeding of
patch-list genomes.

TEST INFRASTRUCTURE ONLY.  Plain Python loops, written from the definitions,
for small populations.  Only the test-suite may import it.  It shares no code
with the product package; its random draws use the oracle's own Philox4x32-10
(``oracle.philox``, pinned by the published known-answer vectors).

Definitions:
  * non-dominated sorting, crowding distance and the crowded comparison follow
    Deb, Pratap, Agarwal and Meyarivan, "A fast and elitist multiobjective
    genetic algorithm: NSGA-II", IEEE Trans. Evol. Comput. 6(2), 2002
    (all objectives are minimised);
  * GEVO-ML (paper section 4): an individual is a list of edits to the
    original program (patch representation, section 4.2); each initial
    individual gets three random mutations (section 4); crossover is one-point
    messy crossover: concatenate two parents' edit lists, shuffle, cut at a
    random point (section 4.2); the best 16 individuals are copied unchanged
    to the next generation and the rest is chosen by tournament selection
    (section 4.4).
  * Edits here are the effects the paper attributes to its evolved edits: a
    changed learning rate (section 6.2) and pruned weights (abstract), and the
    structural ones of its MobileNet analysis and repair: removed biases
    (section 6.1) and shrunk tensors (section 4.1).  Edit (kind 0, id, value):
    multiply the learning rate by the binary32 factor whose bits are
    ``value``; (kind 1, id, value): keep a weight only when the top 24 bits of
    its mask draw under edit ``id`` fall below ``value``; (kind 2, l, w): keep
    the first w units of hidden layer l; (kind 3, l, 0): remove the biases of
    layer l.

Counter layout of the draws (key = seed), word w of Philox((c0, c1, c2, stream)):
  tournament j of generation g:     (j, g, 0, 7), words 0 and 1 = contestants
  crossover of pair i, generation g: (0, g, i, 8) word 0 = decision, word 1 = cut;
                                    (1 + t // 4, g, i, 8) word t % 4 = shuffle draw for position t
  mutation of child i, generation g >= 1: (0, g, i, 9) word 0 = decision;
                                    the new edit from words 1 (kind) and 2 (value) of (1, g, i, 9)
  edit j of initial individual i:   words 1 (kind) and 2 (value) of (j, 0, i, 9)
  a drawn edit is structural when word 1's u24 < struct_p: word 3 picks bias
  removal (u24 < 1/2, or no hidden layer) or a width, word 0 the layer, word 2
  the width (1 + multiply-shift onto [0, d_l)); otherwise a learning-rate edit
  when u24 < struct_p + (1 - struct_p) / 2, else pruning
Objectives must not be NaN (a NaN compares false and would never be dominated).

Parity status:
  nondominated_sort   pinned by brute-force peeling of non-dominated sets and by
                      the front invariants
  crowding_distance   pinned by closed forms (evenly spaced fronts, boundary
                      points, constant objective)
  select              pinned by the crowded-comparison order of the elites and
                      by replaying each tournament by hand
  breed, initial      pinned by the multiset and length invariants of messy
                      crossover and by the edit ranges
"""
from __future__ import annotations

import math

import numpy as np

from . import philox

STREAM_SELECT, STREAM_CROSS, STREAM_MUT = 7, 8, 9
LR_EDIT, PRUNE_EDIT, WIDTH_EDIT, BIAS_EDIT, LAYER_EDIT = 0, 1, 2, 3, 4
INF = float("inf")


def _draw(seed, c0, c1, c2, stream):
    return [int(w) for w in philox((c0, c1, c2, stream), (seed & 0xFFFFFFFF, seed >> 32))]


def _u24(r):
    return (r >> 8) * (1.0 / 16777216.0)


def _below(r, n):
    """Integer in [0, n) from a 32-bit draw (multiply-shift)."""
    return (r * n) >> 32


def _f32(x):
    return float(np.float32(x))


def _f32_bits(x):
    return int(np.float32(x).view(np.uint32))


def _bits_f32(b):
    return float(np.uint32(b).view(np.float32))


def dominates(a, b):
    return all(x <= y for x, y in zip(a, b)) and any(x < y for x, y in zip(a, b))


def nondominated_sort(objs):
    """Front index (0 = non-dominated) of every point, by Deb et al.'s fast
    non-dominated sort: count who dominates each point, peel the fronts."""
    n = len(objs)
    dominated_by_me = [[] for _ in range(n)]
    n_dominating = [0] * n
    for p in range(n):
        for q in range(n):
            if dominates(objs[p], objs[q]):
                dominated_by_me[p].append(q)
            elif dominates(objs[q], objs[p]):
                n_dominating[p] += 1
    rank = [None] * n
    front = [p for p in range(n) if n_dominating[p] == 0]
    r = 0
    while front:
        nxt = []
        for p in front:
            rank[p] = r
            for q in dominated_by_me[p]:
                n_dominating[q] -= 1
                if n_dominating[q] == 0:
                    nxt.append(q)
        front = nxt
        r += 1
    return rank


def crowding_distance(objs, rank):
    """Per point: the sum over objectives of the normalised gap between its two
    neighbours in its front (neighbours by objective value, then index); the
    extreme points of every objective get infinity."""
    n = len(objs)
    m = len(objs[0]) if n else 0
    dist = [0.0] * n
    for r in sorted(set(rank)):
        front = [i for i in range(n) if rank[i] == r]
        for k in range(m):
            order = sorted(front, key=lambda i: (objs[i][k], i))
            lo, hi = objs[order[0]][k], objs[order[-1]][k]
            dist[order[0]] = INF
            dist[order[-1]] = INF
            if hi > lo:
                for j in range(1, len(order) - 1):
                    i = order[j]
                    dist[i] = dist[i] + (objs[order[j + 1]][k] - objs[order[j - 1]][k]) / (hi - lo)
    return dist


def crowded_better(a, b, rank, dist):
    """Deb et al.'s crowded comparison (lower front, then larger distance), ties to the lower index."""
    if rank[a] != rank[b]:
        return rank[a] < rank[b]
    if dist[a] != dist[b]:
        return dist[a] > dist[b]
    return a < b


def select(rank, dist, n_elite, n_select, seed, gen):
    """The n_elite best by crowded comparison, in that order, then
    n_select - n_elite binary-tournament winners."""
    n = len(rank)
    order = sorted(range(n), key=lambda i: (rank[i], -dist[i], i))
    out = order[:n_elite]
    for j in range(n_select - n_elite):
        w = _draw(seed, j, gen, 0, STREAM_SELECT)
        a, b = _below(w[0], n), _below(w[1], n)
        out.append(a if (a == b or crowded_better(a, b, rank, dist)) else b)
    return out


def random_edit(seed, gen, i, j, edit_id, rho_lo, struct_p=0.0, dims=None):
    """The edit drawn from (j, gen, i, 9): with probability struct_p a
    structural edit (bias removal; for nets with hidden layers, with equal
    odds bias removal, a hidden width or a removed hidden layer), otherwise
    with equal odds a learning-rate factor log-uniform on [1/2, 2] or
    pruning at a density uniform on [rho_lo, 1]."""
    w = _draw(seed, j, gen, i, STREAM_MUT)
    u = _u24(w[2])
    uk = _u24(w[1])
    if uk < struct_p:
        L = len(dims) - 1
        us = _u24(w[3])
        if us < 1.0 / 3.0 or L < 2:
            return (BIAS_EDIT, 1 + _below(w[0], L), 0)
        layer = 1 + _below(w[0], L - 1)
        if us < 2.0 / 3.0:
            return (WIDTH_EDIT, layer, 1 + _below(w[2], int(dims[layer])))
        return (LAYER_EDIT, layer, 0)
    if uk < struct_p + (1.0 - struct_p) * 0.5:
        factor = _f32(math.exp(math.log(0.5) + u * math.log(4.0)))
        return (LR_EDIT, edit_id, _f32_bits(factor))
    rho = rho_lo + u * (1.0 - rho_lo)
    return (PRUNE_EDIT, edit_id, int(round(rho * 16777216.0)))


def initial(n, seed, rho_lo, n_mut=3, id_base=0, struct_p=0.0, dims=None):
    """Initial population: n individuals, each with n_mut random edits
    (edit ids id_base + n_mut * i + j)."""
    return [[random_edit(seed, 0, i, j, id_base + n_mut * i + j, rho_lo, struct_p, dims) for j in range(n_mut)]
            for i in range(n)]


def breed(parents, seed, gen, cxpb, mutpb, rho_lo, id_base, max_edits, struct_p=0.0, dims=None):
    """Children of the tournament winners, in pairs (0,1), (2,3), ...: with
    probability cxpb a pair is recombined by messy one-point crossover
    (concatenate, shuffle, cut; each child keeps at most max_edits), then each
    child gets one new edit (id id_base + i) with probability mutpb when it
    holds fewer than max_edits.  Generations of breeding count from 1."""
    assert gen >= 1
    children = [list(p) for p in parents]
    for i in range(0, len(children) - 1, 2):
        w = _draw(seed, 0, gen, i, STREAM_CROSS)
        if _u24(w[0]) < cxpb:
            cat = children[i] + children[i + 1]
            for t in range(len(cat) - 1, 0, -1):
                r = _draw(seed, 1 + t // 4, gen, i, STREAM_CROSS)[t % 4]
                s = _below(r, t + 1)
                cat[t], cat[s] = cat[s], cat[t]
            cut = _below(w[1], len(cat) + 1)
            children[i], children[i + 1] = cat[:cut][:max_edits], cat[cut:][:max_edits]
    for i in range(len(children)):
        w = _draw(seed, 0, gen, i, STREAM_MUT)
        if _u24(w[0]) < mutpb and len(children[i]) < max_edits:
            children[i].append(random_edit(seed, gen, i, 1, id_base + i, rho_lo, struct_p, dims))
    return children


def apply(edits, lr_base):
    """(learning rate, prune edit ids, prune thresholds, expected kept fraction)
    of an individual: the learning-rate factors multiply in order in binary32,
    the pruning edits combine as a logical and of their masks."""
    lr = _f32(lr_base)
    ids, th, dens = [], [], 1.0
    for kind, eid, value in edits:
        if kind == LR_EDIT:
            lr = _f32(lr * _bits_f32(value))
        elif kind == PRUNE_EDIT:
            ids.append(eid)
            th.append(value)
            dens = dens * (value / 16777216.0)
    return lr, ids, th, dens


def structure(edits, dims):
    """(widths [L+1], bias_keep [L]) of an individual: a hidden layer keeps the
    smallest width any of its edits asks for, inputs and classes are kept."""
    L = len(dims) - 1
    widths = [int(d) for d in dims]
    keep = [1] * L
    for kind, eid, value in edits:
        if kind == WIDTH_EDIT:
            assert 1 <= eid <= L - 1 and value >= 1
            widths[eid] = min(widths[eid], int(value))
        elif kind == BIAS_EDIT:
            assert 1 <= eid <= L
            keep[eid - 1] = 0
    for kind, eid, value in edits:                # a removed layer keeps its identity-form biases
        if kind == LAYER_EDIT:
            keep[eid - 1] = 1
    return widths, keep


def removed_layers(edits, dims):
    """[L] flags: hidden layer l (1 .. L-1) removed by a LAYER_EDIT (the
    identity map in place of the layer, frozen in training)."""
    L = len(dims) - 1
    gone = [0] * L
    for kind, eid, value in edits:
        if kind == LAYER_EDIT:
            assert 1 <= eid <= L - 1
            gone[eid - 1] = 1
    return gone


def density(edits, dims):
    """Expected kept fraction of the weights: the pruning edits' keep
    fractions in order, times the fraction the structural edits keep (a
    removed layer keeps none of its weights)."""
    dens = apply(edits, 1.0)[3]
    widths, _ = structure(edits, dims)
    gone = removed_layers(edits, dims)
    kept = sum(widths[l - 1] * widths[l] for l in range(1, len(dims)) if not gone[l - 1])
    total = sum(int(dims[l - 1]) * int(dims[l]) for l in range(1, len(dims)))
    return dens * (kept / total)
