"""GEVO-ML search loop (paper section 4) on top of the population-batched
fitness evaluation: every generation is evaluated as one population on the
GPU, then ranked, selected and bred by the library's host code.

An individual is a list of edits (patch representation, section 4.2) whose
effects are a changed learning rate (section 6.2) and pruned weights
(abstract), optionally also removed biases and removed hidden layers
(section 6.1) and narrowed hidden layers (the tensor-shrinking repair,
section 4.1) with probability struct_p per drawn edit.  Fitness (section 4.3) is minimised over two objectives:
  * model error: the training-split error of the last epoch (the paper
    computes accuracy on the training split during the search and keeps the
    test split for checking the result afterwards, section 5);
  * cost (the paper's second objective is run time), one of:
    - "kept" (default): the expected kept fraction of the weights (pruning
      densities times the fraction the structural edits keep).  Pruned
      weights still run in the dense kernels, so this stands for the time a
      pruned model would save; it is deterministic.
    - "measured": each variant's device time in the generation's training
      and prediction calls (gevo_pop_scores' time_s, summed over the calls).
      Workgroups of hidden-layer unit tiles that a narrowed variant has
      removed are skipped, so narrowed variants measure faster.  Timings vary
      from run to run, so a search on this objective is not bit-reproducible.
Each generation keeps the n_elite best unchanged and fills the rest with the
children of tournament winners (section 4.4).  The elites keep the fitness
they were selected with: the whole generation is retrained as one population,
but an unchanged individual is not scored again (a variant's rounding can
depend on its slot in the population).  All computation happens in
libgevo; this module only marshals arguments and keeps the history.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import Population, genomes_breed, genomes_initial, nsga2_rank, nsga2_select


@dataclass
class Generation:
    genomes: list                     # edit lists [(kind, id, value), ...]
    objectives: np.ndarray            # [P][2]: training error, cost (expected kept fraction or time in s)
    test_error: np.ndarray            # [P], for checking the front afterwards
    lr: np.ndarray                    # [P] learning rates of the genomes
    rank: np.ndarray = field(default=None)
    crowding: np.ndarray = field(default=None)


class Search:
    def __init__(self, pop: Population, lr_base: float, seed: int, epochs: int = 1, rho_lo: float = 0.3,
                 n_elite: int = 16, cxpb: float = 0.8, mutpb: float = 0.5, max_edits: int = 16, n_mut: int = 3,
                 struct_p: float = 0.0, time_objective: str = "kept"):
        if not 0 <= n_elite <= pop.P:
            raise ValueError("n_elite must be in [0, P]")
        if time_objective not in ("kept", "measured"):
            raise ValueError("time_objective must be 'kept' or 'measured'")
        self.time_objective = time_objective
        self.pop, self.lr_base, self.seed, self.epochs = pop, float(lr_base), int(seed), int(epochs)
        self.rho_lo, self.n_elite, self.cxpb, self.mutpb = float(rho_lo), int(n_elite), float(cxpb), float(mutpb)
        self.max_edits, self.n_mut, self.struct_p = int(max_edits), int(n_mut), float(struct_p)
        self.history: list[Generation] = []

    def evaluate(self, genomes, carried=None) -> Generation:
        """One fitness evaluation of a whole generation: rebuild, retrain, score.
        carried = (objectives, test errors) of the first individuals, kept as they are."""
        pop = self.pop
        lr, dens = pop.set_genomes(genomes, self.lr_base)
        t = np.zeros(pop.P, np.float64)
        for e in range(self.epochs):
            pop.train_epoch(e)
            if self.time_objective == "measured":
                t += pop.scores()["time_s"]
        pop.predict()
        s = pop.scores()
        train_err = 1.0 - np.asarray(s["train_acc"], np.float64)
        cost = dens if self.time_objective == "kept" else t + np.asarray(s["time_s"], np.float64)
        objs = np.stack([train_err, cost], axis=1)
        test_err = 1.0 - np.asarray(s["test_acc"], np.float64)
        if carried is not None:
            k = len(carried[0])
            objs[:k] = carried[0]
            test_err[:k] = carried[1]
        gen = Generation(genomes=[list(g) for g in genomes], objectives=objs, test_error=test_err, lr=lr)
        gen.rank, gen.crowding = nsga2_rank(objs)
        return gen

    def start(self) -> Generation:
        """Generation 0: n_mut drawn edits per individual (section 4)."""
        genomes = genomes_initial(self.pop.P, self.seed, self.rho_lo, self.n_mut, id_base=0, struct_p=self.struct_p,
                                  dims=self.pop.dims)
        self.history = [self.evaluate(genomes)]
        return self.history[-1]

    def step(self) -> Generation:
        """Next generation: elites unchanged, then bred tournament winners."""
        if not self.history:
            return self.start()
        cur = self.history[-1]
        g = len(self.history)
        P = self.pop.P
        chosen = nsga2_select(cur.rank, cur.crowding, self.n_elite, P, self.seed, g)
        elites = [cur.genomes[i] for i in chosen[:self.n_elite]]
        parents = [cur.genomes[i] for i in chosen[self.n_elite:]]
        id_base = self.n_mut * P + (g - 1) * P            # fresh edit ids every generation
        kids = genomes_breed(parents, self.seed, g, self.cxpb, self.mutpb, self.rho_lo, id_base, self.max_edits,
                             self.struct_p, self.pop.dims)
        keep = list(chosen[:self.n_elite])
        self.history.append(self.evaluate(elites + kids, (cur.objectives[keep], cur.test_error[keep])))
        return self.history[-1]

    def run(self, generations: int) -> list:
        while len(self.history) < generations:
            self.step()
        return self.history

    @staticmethod
    def front(gen: Generation):
        """Indices of the non-dominated individuals of a generation, by objective."""
        idx = [i for i in range(len(gen.rank)) if gen.rank[i] == 0]
        return sorted(idx, key=lambda i: (gen.objectives[i][0], gen.objectives[i][1], i))
