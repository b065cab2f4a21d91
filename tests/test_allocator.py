"""Host-side checks of the runtime model and the allocation solver (Eq. 7):
the solver against exhaustive search on small problems, the tile counts and
configuration choice against the oracle's tile plan."""

import itertools

import numpy as np
import pytest

from oracle import mxmoe_oracle as O
from paper_2505_05799_amd import allocator as A
from paper_2505_05799_amd import tile_cost as TC
from paper_2505_05799_amd import workloads as W


def _problem(seed, nb, nc, r, spare_units):
    rng = np.random.default_rng(seed)
    L = rng.random((nb, nc)) * 10
    T = rng.random((nb, nc)) * 100 + 1
    Wt = rng.integers(1, 4, (nb, nc)).astype(float)           # whole memory units
    M = Wt.min(axis=1).sum() + spare_units                      # a power-of-two spare: the grid is exact
    return A.Problem(L, T, Wt, M, r)


@pytest.mark.parametrize("r", [0.0, 0.5, 0.75, 1.0])
@pytest.mark.parametrize("seed", range(6))
def test_solver_matches_exhaustive_search(seed, r):
    nb, nc = 6, 3
    p = _problem(seed, nb, nc, r, spare_units=4)
    choice, info = A.solve(p)
    ref, best = A.brute_force(p)
    val, l, t, w = p.objective(choice)
    assert w <= p.M
    # time is gridded: the cell optimum may sit up to nb half-cells of time away
    span = (p.T.max(axis=1) - p.T.min(axis=1)).sum()
    tol = (1.0 - r) * nb * (span / 256) / p.T.min(axis=1).sum()
    assert val <= best * (1 + tol) + 1e-12
    if r == 1.0:
        assert val == pytest.approx(best, rel=1e-12)


def test_solver_budget_edges():
    p = _problem(3, 5, 3, 0.75, spare_units=0)     # only the smallest schemes fit
    choice, info = A.solve(p)
    assert info["W_bytes"] == p.W.min(axis=1).sum()
    p.M -= 0.5
    with pytest.raises(ValueError):
        A.solve(p)
    # a budget that fits everything: r = 1 takes the least loss everywhere
    p = _problem(4, 5, 3, 1.0, spare_units=64)
    choice, _ = A.solve(p)
    assert choice == list(p.L.argmin(axis=1))
    # r = 0 takes the least time everywhere
    p = _problem(4, 5, 3, 0.0, spare_units=64)
    choice, _ = A.solve(p)
    assert choice == list(p.T.argmin(axis=1))


def test_tile_counts_and_configuration_match_the_plan():
    """pick_cfg / n_tiles of the runtime model equal the oracle's tile plan
    (without slicing) for every scheme and a sweep of row counts."""
    rng = np.random.default_rng(0)
    counts = [0, 1, 15, 16, 17, 32, 33, 64, 65, 128, 129, 300, 1000] + rng.integers(1, 3000, 20).tolist()
    for s in W.ALL_SCHEMES:
        lins = [W.QLinear(s, 1408, 2048, None) for _ in counts]
        for phase in (0, 1):
            plan, _ = O.tile_plan(counts, lins, phase, TC.CostTable.load().device_table(), partial_floats=0)
            for m, r in zip(counts, plan):
                if m == 0:
                    continue
                c = TC.pick_cfg(m, s, phase)
                assert c == r["cfg"], (s.name, m)
                assert TC.n_tiles(m, 1408, phase, c) == r["mtiles"] * r["ntiles"]


def test_block_model_closed_form():
    cfg = W.CONFIGS["dsv2lite"]
    tab = {"P": 512, "cost": {str(ph): {s.name: [[1000.0 * (c + 1) + 7 * i, 10.0 + i] for c in range(4)]
                                        for i, s in enumerate(W.ALL_SCHEMES)} for ph in (0, 1)}}
    t = TC.CostTable(tab)
    counts = [10, 20, 40, 200] + [0] * 60
    sch = W.schemes_of(cfg)
    want = [0.0, 0.0]
    for e in range(cfg.E + cfg.n_shared):
        m = counts[e] if e < cfg.E else cfg.T
        if m == 0:
            continue
        F = cfg.F if e < cfg.E else cfg.F_shared
        for ph, (n, k) in enumerate(((F, cfg.H), (cfg.H, F))):
            c = TC.pick_cfg(m, sch[e][0 if ph == 0 else 2], ph)
            a, b = tab["cost"][str(ph)][sch[e][0 if ph == 0 else 2].name][c]
            want[ph] += -(-m // TC.BM[c]) * -(-n // TC.BN[ph][c]) * (a + b * k / 128)
    got = t.block_ns(cfg, counts, sch)
    assert got == pytest.approx([v / 512 for v in want], rel=1e-12)


def test_block_problem_memory_and_mapping():
    cfg = W.CONFIGS["qwen15_mixed"]
    cands = [W.W8A8, W.W4A4, W.W4A4G128]
    tab = TC.CostTable({"P": 512, "cost": {str(ph): {s.name: [[1000.0, 10.0]] * 4 for s in cands}
                                           for ph in (0, 1)}})
    G = cfg.E + cfg.n_shared
    delta = np.random.default_rng(0).random((G, 2, 3))
    p, blocks = A.block_problem(cfg, cands, tab, delta, budget_bits=5.0, r=0.75)
    assert p.L.shape == (2 * G, 3) and blocks[:2] == [(0, 0), (0, 1)]
    params = G * 0 + cfg.E * 3 * cfg.F * cfg.H + cfg.n_shared * 3 * cfg.F_shared * cfg.H
    assert p.M == pytest.approx(5.0 * params / 8)
    choice, info = A.solve(p)
    sch = A.allocation_to_alloc(cfg, cands, choice, blocks)
    assert len(sch) == G and all(t[0] == t[1] for t in sch)
    packed = sum(2 * W.QLinear(t[0], cfg.F if g < cfg.E else cfg.F_shared, cfg.H, None).nbytes_packed
                 + W.QLinear(t[2], cfg.H, cfg.F if g < cfg.E else cfg.F_shared, None).nbytes_packed
                 for g, t in enumerate(sch))
    assert packed == pytest.approx(info["W_bytes"]) and packed <= p.M


@pytest.mark.parametrize("s", W.ALL_SCHEMES)
def test_profiler_operands_fit_the_packer(s):
    """The profiler's random operands have the extent the packer reads for
    every scheme (regression: mxfp4 once got another format's scales)."""
    torch = pytest.importorskip("torch")
    from paper_2505_05799_amd import mxmoe as M
    g = torch.Generator(device="cpu")
    g.manual_seed(0)
    q = TC._device_linear(s, 256, 512, g, dev="cpu")
    M.check_operands(q)
    assert (q.n, q.k) == (256, 512)
