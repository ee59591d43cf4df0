"""GPU checks of the search step: populations rebuilt from genomes against the
oracle (masks, weights, learning rates bit for bit; training within the
tolerances of the fitness evaluation), and a short search run."""
import numpy as np
import pytest

import oracle
import synthetic
from oracle import nsga2 as ns

pytestmark = pytest.mark.gpu


def _pop(cfg, data):
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2310_10211_amd as g
    print(f"[gpu] Population P={cfg['P']} dims={cfg['dims']} dtype={cfg['dtype']} "
          f"n_train={len(data['y_train'])} n_test={len(data['y_test'])}", flush=True)
    return g.Population(cfg, data["x_train"], data["y_train"], data["x_test"], data["y_test"])


def _small(i, P, n_train, n_test):
    c = synthetic.config(i)
    c["P"] = P
    return c, synthetic.dataset(c, n_train, n_test)


def _genomes(P, seed):
    gs = ns.initial(P, seed, 0.3)
    gs[1] = []                                                 # the original model
    gs[2] = gs[2] + ns.initial(3, seed + 1, 0.5, id_base=900)[0] + ns.initial(3, seed + 2, 0.5, id_base=950)[1]
    gs[3] = [(ns.LR_EDIT, 5, int(np.float32(1.5).view(np.uint32)))]   # learning rate only
    return gs


@pytest.mark.parametrize("i", [1, 3])
def test_set_genomes_rebuilds_masks_weights_and_rates_exactly(i):
    cfg, data = _small(i, P=8, n_train=256, n_test=256)
    pop = _pop(cfg, data)
    genomes = _genomes(8, 31)
    lr, dens = pop.set_genomes(genomes, 0.05)
    dims = cfg["dims"]
    full, _ = oracle.variant_init(cfg["seed"], 0, dims, 1 << 24)          # initial weights, nothing pruned
    nw = oracle.weight_count(dims)
    for v in range(8):
        lr_o, ids, th, dens_o = ns.apply(genomes[v], 0.05)
        e = pop.export(v)
        mask = oracle.genome_mask(cfg["seed"], dims, ids, th)
        assert np.array_equal(e["mask"], mask), v
        want = full.copy()
        off = 0
        for l in range(1, len(dims)):
            n = dims[l - 1] * dims[l]
            want[off:off + n] *= mask[sum(dims[j - 1] * dims[j] for j in range(1, l)):][:n]
            off += n + dims[l]
        assert np.array_equal(e["params"].astype(np.float64), want), v
        assert lr[v] == np.float32(lr_o) and e["lr"] == np.float32(lr_o)
        assert dens[v] == dens_o
    assert nw == e["mask"].size
    pop.close()


def test_single_edit_genome_reproduces_the_initial_population():
    cfg, data = _small(3, P=4, n_train=256, n_test=256)
    pop = _pop(cfg, data)
    init = [pop.export(v) for v in range(4)]
    genomes = []
    for v in range(4):
        _, _, th = oracle.variant_hparams(cfg["seed"], v, cfg["lr"], cfg.get("dens", (1.0, 1.0)),
                                          cfg.get("dens_list"))
        genomes.append([(ns.PRUNE_EDIT, v, th)])
    pop.set_genomes(genomes, 0.01)
    for v in range(4):
        e = pop.export(v)
        assert np.array_equal(e["mask"], init[v]["mask"]) and np.array_equal(e["params"], init[v]["params"])
    pop.close()


@pytest.mark.parametrize("i,mode,rtol", [(1, "f32", 1e-4), (3, "bf16", 2e-2)])
def test_training_after_set_genomes_matches_oracle(i, mode, rtol):
    """One epoch after a rebuild (the fused bf16 kernel must pick up the new
    hidden layer) against the oracle's SGD on the same masks and rates."""
    cfg, data = _small(i, P=4, n_train=640, n_test=256)
    pop = _pop(cfg, data)
    pop.train_epoch(0)                                         # the old population trains first
    genomes = _genomes(4, 47)
    lr, _ = pop.set_genomes(genomes, 0.05)
    pop.train_epoch(0)
    s = pop.scores()
    dims = cfg["dims"]
    full, _ = oracle.variant_init(cfg["seed"], 0, dims, 1 << 24)
    n = len(data["y_train"])
    perm = oracle.permutation(cfg["seed"], 0, n)
    steps = -(-n // cfg["batch"])
    for v in range(4):
        _, ids, th, _ = ns.apply(genomes[v], 0.05)
        mask = oracle.genome_mask(cfg["seed"], dims, ids, th)
        params = full.copy()
        off, moff = 0, 0
        for l in range(1, len(dims)):
            k = dims[l - 1] * dims[l]
            params[off:off + k] *= mask[moff:moff + k]
            off += k + dims[l]
            moff += k
        ce, _ = oracle.train_steps(mode, dims, params, mask, float(lr[v]), data["x_train"], data["y_train"], perm,
                                   cfg["batch"], 0, steps)
        ref = ce / n
        assert abs(float(s["train_loss"][v]) - ref) <= rtol * abs(ref), (v, s["train_loss"][v], ref)
    pop.close()


def test_search_generations_are_deterministic_and_keep_elites():
    from paper_2310_10211_amd.search import Search
    cfg, data = _small(3, P=32, n_train=512, n_test=256)
    runs = []
    for _ in range(2):
        pop = _pop(cfg, data)
        s = Search(pop, lr_base=0.05, seed=5, epochs=1, n_elite=8)
        hist = s.run(3)
        runs.append([(h.genomes, h.objectives.copy(), h.test_error.copy()) for h in hist])
        import paper_2310_10211_amd as gv
        for gen, (g0, g1) in enumerate(zip(hist, hist[1:]), start=1):
            assert len(g1.genomes) == 32
            chosen = gv.nsga2_select(g0.rank, g0.crowding, 8, 32, 5, gen)
            for slot, i in enumerate(chosen[:8]):
                assert g1.genomes[slot] == g0.genomes[i]
                assert np.array_equal(g1.objectives[slot], g0.objectives[i])
        last = hist[-1]
        front = Search.front(last)
        assert front
        for a in front:
            for b in front:
                assert not ns.dominates(tuple(last.objectives[a]), tuple(last.objectives[b]))
        assert np.all((last.objectives[:, 0] >= 0) & (last.objectives[:, 0] <= 1))
        pop.close()
    for (ga, oa, ta), (gb, ob, tb) in zip(*runs):
        assert ga == gb and np.array_equal(oa, ob) and np.array_equal(ta, tb)


def _struct_genomes(P, dims, seed):
    gs = ns.initial(P, seed, 0.4, 3, 0, 0.6, dims)
    L = len(dims) - 1
    gs[0] = [(ns.BIAS_EDIT, L, 0)]                              # output biases removed
    if L > 1:
        gs[1] = [(ns.WIDTH_EDIT, 1, max(1, dims[1] // 3)), (ns.BIAS_EDIT, 1, 0)]
        gs[2] = gs[2] + [(ns.WIDTH_EDIT, 1, dims[1] - 5), (ns.WIDTH_EDIT, 1, dims[1] - 9)]
        gs[3] = [(ns.LAYER_EDIT, L - 1, 0), (ns.PRUNE_EDIT, 77, 2 ** 23)]   # the last hidden layer removed
        if L > 2:
            gs[3].append((ns.WIDTH_EDIT, 1, dims[L - 1] // 2))       # its kept input narrower than its units
    return gs


def _struct_reference(cfg, genome, lr_base):
    """(lr, mask, bias mask, params, frozen layer bits) of a genome."""
    dims = cfg["dims"]
    lr, ids, th, _ = ns.apply(genome, lr_base)
    widths, keep = ns.structure(genome, dims)
    gone = ns.removed_layers(genome, dims)
    mask, bmask = oracle.structure_masks(dims, widths, keep, oracle.genome_mask(cfg["seed"], dims, ids, th))
    full, _ = oracle.variant_init(cfg["seed"], 0, dims, 1 << 24)
    params = full.copy()
    off, moff, boff = 0, 0, 0
    for l in range(1, len(dims)):
        k = dims[l - 1] * dims[l]
        if gone[l - 1]:                                       # the identity form, frozen in training
            W, b, m = oracle.removed_layer_form(dims, widths, l)
            params[off:off + k] = W.ravel()
            params[off + k:off + k + dims[l]] = b
            mask[moff:moff + k] = m.ravel()
        else:
            params[off:off + k] *= mask[moff:moff + k]
            params[off + k:off + k + dims[l]] *= bmask[boff:boff + dims[l]]
        off += k + dims[l]
        moff += k
        boff += dims[l]
    frozen = sum(1 << l for l in range(len(gone)) if gone[l])
    return lr, mask, bmask, params, frozen


@pytest.mark.parametrize("i,dims", [(1, None), (3, None), (3, [200, 96, 64, 10]),
                                    (5, [1024, 256, 128, 10])])   # a removed 128-unit tile of the streaming kernel
def test_structural_genomes_rebuild_and_train_like_the_oracle(i, dims):
    cfg, data = _small(i, P=4, n_train=640, n_test=256)
    if dims:
        cfg["dims"] = dims
        for k in ("x_train", "x_test"):
            data[k] = np.ascontiguousarray(data[k][:, :dims[0]])
    mode = "bf16" if cfg["dtype"] == "bf16" else "f32"
    rtol = 2e-2 if mode == "bf16" else 1e-4
    pop = _pop(cfg, data)
    genomes = _struct_genomes(4, cfg["dims"], 61)
    lr, dens = pop.set_genomes(genomes, 0.05)
    refs = [_struct_reference(cfg, genomes[v], 0.05) for v in range(4)]
    for v in range(4):
        e = pop.export(v)
        r_lr, r_mask, r_bmask, r_params, _ = refs[v]
        assert np.array_equal(e["mask"], r_mask), v
        assert np.array_equal(e["params"].astype(np.float64), r_params), v
        assert lr[v] == np.float32(r_lr) and dens[v] == ns.density(genomes[v], cfg["dims"])
    pop.train_epoch(0)
    s = pop.scores()
    n = len(data["y_train"])
    perm = oracle.permutation(cfg["seed"], 0, n)
    for v in range(4):
        r_lr, r_mask, r_bmask, r_params, frozen = refs[v]
        params = r_params.copy()
        ce, _ = oracle.train_steps(mode, cfg["dims"], params, r_mask, float(r_lr), data["x_train"], data["y_train"],
                                   perm, cfg["batch"], 0, -(-n // cfg["batch"]), bmask=r_bmask, frozen=frozen)
        assert abs(float(s["train_loss"][v]) - ce / n) <= rtol * abs(ce / n), (v, s["train_loss"][v], ce / n)
        e = pop.export(v)
        if frozen:                                            # a removed layer is still its identity form
            off = 0
            for l in range(1, len(cfg["dims"])):
                k = cfg["dims"][l - 1] * cfg["dims"][l] + cfg["dims"][l]
                if (frozen >> (l - 1)) & 1:
                    assert np.array_equal(e["params"][off:off + k].astype(np.float64), r_params[off:off + k]), (v, l)
                off += k
        off, boff = 0, 0
        for l in range(1, len(cfg["dims"])):                   # removed biases are still +0
            k = cfg["dims"][l - 1] * cfg["dims"][l]
            b = e["params"][off + k:off + k + cfg["dims"][l]]
            assert np.all(b[r_bmask[boff:boff + cfg["dims"][l]] == 0] == 0.0), (v, l)
            off += k + cfg["dims"][l]
            boff += cfg["dims"][l]
    pop.close()


def test_time_s_splits_the_call_time_over_the_variants():
    cfg, data = _small(5, P=4, n_train=600, n_test=256)
    cfg["dims"] = [1024, 256, 128, 10]
    for k in ("x_train", "x_test"):
        data[k] = np.ascontiguousarray(data[k][:, :1024])
    pop = _pop(cfg, data)
    for call in (lambda: pop.train_epoch(0), pop.predict):
        call()
        s = pop.scores()
        assert np.all(s["time_s"] > 0)
        assert abs(float(np.sum(s["time_s"], dtype=np.float64)) - pop.last_time()) <= 1e-5 * pop.last_time()
    pop.close()


def test_narrowed_variants_measure_less_device_time():
    """3072-1024-512-10 in bf16: variants 4..7 keep 128 units of each hidden
    layer, so 7 of 8 and 3 of 4 unit tiles of their streaming-kernel
    workgroups are skipped; their share of the epoch's time is well below
    that of the full variants 0..3, and they still train like the oracle's
    narrowed nets (checked by the structural-genome test above)."""
    cfg, data = _small(5, P=8, n_train=1024, n_test=256)
    pop = _pop(cfg, data)
    full = [(ns.LR_EDIT, 0, ns._f32_bits(1.0))]
    narrow = full + [(ns.WIDTH_EDIT, 1, 128), (ns.WIDTH_EDIT, 2, 128)]
    pop.set_genomes([full] * 4 + [narrow] * 4, 0.01)
    pop.train_epoch(0)
    t = pop.scores()["time_s"]
    assert np.max(t[4:]) < 0.6 * np.min(t[:4]), t
    pop.close()


def test_search_on_measured_time_runs_and_scores_time():
    cfg, data = _small(5, P=8, n_train=512, n_test=256)
    cfg["dims"] = [1024, 256, 128, 10]
    for k in ("x_train", "x_test"):
        data[k] = np.ascontiguousarray(data[k][:, :1024])
    pop = _pop(cfg, data)
    from paper_2310_10211_amd.search import Search
    search = Search(pop, 0.01, seed=7, n_elite=2, struct_p=0.5, time_objective="measured")
    hist = search.run(2)
    for gen in hist:
        assert np.all(gen.objectives[:, 1] > 0) and np.all(np.isfinite(gen.objectives))
    pop.close()
