"""GPU parity on the full-size workloads (the launch configuration the
benchmark times), against the CPU oracle on every token: routing arrays and
the tile plan bit-exact over the whole block, then the stage-wise check of
tests/stagewise.py over all rows of every group (h, down-projection codes,
slot rows, combine, end-to-end output)."""

import time

import numpy as np
import pytest

from oracle import mxmoe_oracle as O
from paper_2505_05799_amd import mxmoe as M
from paper_2505_05799_amd import workloads as W
from tests.gpuhelp import say, torch_mod, upload_inputs
from tests.stagewise import check_forward

pytestmark = pytest.mark.gpu

NAMES = ["tiny", "mixtral", "dsv2lite", "qwen15_uniform", "qwen15_mixed", "qwen15_w5a5", "qwen15_float", "qwen2",
         "qwen2_f6"]


# micro-kernel ids of the schemes in the plan's tile entries
KIND = {"w16": 0, "w8a8": 1, "w4a4": 2, "w2g128": 3, "w3g128": 4, "w4g128": 5, "w8g128": 6, "w4a4g128": 7,
        "mxfp4": 8, "fp8": 9, "w4a4f6": 10}


PF_N = 12  # int32 fields per group record of the tile plan


def plan_flat(mb, T, G, cap, phase):
    torch = torch_mod()
    fcap = mb.workspace_layout(T)["plan_flat_cap"]
    o_flat = ((2 * G * PF_N + 2 * G + 3) & ~3) + 2 * 8 * cap * 3 + 64 + 16
    p = mb.ws_view("plan", torch.int32, o_flat + 2 * 8 * fcap * 4, T).cpu().numpy()
    return p[o_flat + phase * 8 * fcap * 4: o_flat + (phase + 1) * 8 * fcap * 4].reshape(8, fcap, 4)


def plan_misc(mb, T, G, cap):
    torch = torch_mod()
    o_ctr = ((2 * G * PF_N + 2 * G + 3) & ~3) + 2 * 8 * cap * 3
    p = mb.ws_view("plan", torch.int32, o_ctr + 64 + 16, T).cpu().numpy()
    return p[o_ctr + 64: o_ctr + 80]


def check_plan(mb, blk, r, costs):
    """The tile plan of the last forward, bit-exact against the oracle's plan
    under the cost table `costs`: configuration, tile counts, cost, rank, queue
    order, the per-XCD queues of super-tiles and their expansion to tiles."""
    torch = torch_mod()
    cfg = blk.cfg
    T, E, G = cfg.T, cfg.E, cfg.E + cfg.n_shared
    lay = mb.workspace_layout(T)
    cap = lay["plan_queue_cap"]
    o_ord = 2 * G * PF_N
    o_ent = (o_ord + 2 * G + 3) & ~3
    o_ctr = o_ent + 2 * 8 * cap * 3
    plan = mb.ws_view("plan", torch.int32, o_ctr + 2 * 8 * 4, T).cpu().numpy()
    rec = plan[: 2 * G * PF_N].reshape(2, G, PF_N)
    ms = list(r["counts"]) + [T] * cfg.n_shared
    nwg = int(plan_misc(mb, T, G, cap)[8])           # workgroups the slicing assumed
    assert nwg == 2 * torch.cuda.get_device_properties(0).multi_processor_count
    for phase in (0, 1):
        lins = [blk.linears[g][0 if phase == 0 else 2] for g in range(G)]
        want, order = O.tile_plan(ms, lins, phase, costs, partial_floats=lay["partial_floats"], nwg=nwg)
        for g in range(G):
            got = rec[phase, g]
            assert got[1] == ms[g] and got[2] == want[g]["cfg"], (phase, g)
            assert got[3] == want[g]["mtiles"] and got[4] == want[g]["ntiles"], (phase, g)
            assert got[6] == want[g]["cost"] and got[7] == want[g]["rank"], (phase, g)
            assert got[8] == want[g]["split"], (phase, g)
        q = plan[o_ord + phase * G: o_ord + (phase + 1) * G]
        assert q[: len(order)].tolist() == order
        queues, totals = O.xcd_queues(want, order)
        ent = plan[o_ent + phase * 8 * cap * 3: o_ent + (phase + 1) * 8 * cap * 3].reshape(8, cap, 3)
        ctr = plan[o_ctr + phase * 32: o_ctr + (phase + 1) * 32].reshape(8, 4)
        for x in range(8):
            assert ctr[x, 1] == totals[x] and ctr[x, 2] == len(queues[x]), (phase, x)
            assert [tuple(e) for e in ent[x, : len(queues[x])].tolist()] == queues[x], (phase, x)
        assert sum(totals) == sum(w["tiles"] for w in want)
        # the queues expanded to one entry per tile
        tiles = O.xcd_tiles(want, order)
        offs = r["offsets"]
        fl = plan_flat(mb, T, G, cap, phase)
        for x in range(8):
            exp = np.array([[g | (want[g]["cfg"] << 16) | (KIND[lins[g].scheme.name] << 20)
                             | ((want[g]["split"] - 1) << 24), mi | (ni << 16),
                             offs[g] if g < E else 0, ms[g]] for g, mi, ni in tiles[x]], dtype=np.int64)
            assert np.array_equal(fl[x, : len(tiles[x])].astype(np.int64), exp.reshape(-1, 4)), (phase, x)
    assert plan_misc(mb, T, G, cap)[4] == 0      # no queue overflow


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", NAMES)
def test_full_workload(name):
    torch = torch_mod()
    t0 = time.perf_counter()
    blk = W.make_block(name)
    cfg = blk.cfg
    say(f"[{name}] inputs {time.perf_counter() - t0:.1f}s")
    mb = M.MoEBlock(blk)
    x, ids, w = upload_inputs(blk)
    y = mb.forward(x, ids, w)
    torch.cuda.synchronize()
    say(f"[{name}] forward done {time.perf_counter() - t0:.1f}s")
    T, k, E, G = cfg.T, cfg.k, cfg.E, cfg.E + cfg.n_shared

    # routing, bit-exact
    r = O.route(blk.topk_ids, E)
    assert np.array_equal(mb.ws_view("counts", torch.int32, E, T).cpu().numpy(), r["counts"])
    assert np.array_equal(mb.ws_view("offsets", torch.int32, E + 1, T).cpu().numpy(), r["offsets"])
    assert np.array_equal(mb.ws_view("sorted_pair", torch.int32, T * k, T).cpu().numpy(), r["sorted_pair"])
    assert np.array_equal(mb.ws_view("inv", torch.int32, T * k, T).cpu().numpy(), r["inv"])
    assert int(mb.ws_view("status", torch.int32, 1, T).cpu().numpy()[0]) == 0

    check_plan(mb, blk, r, M.get_tile_costs())

    # every token, stage by stage
    rep = check_forward(mb, blk, y, log=say if G <= 16 else None)
    say(f"[{name}] all {T} tokens: {rep.line()}; {time.perf_counter() - t0:.1f}s")
    del mb
    torch.cuda.empty_cache()


@pytest.mark.timeout(300)
@pytest.mark.parametrize("table", ["default", "random11", "random12"])
@pytest.mark.parametrize("name", ["dsv2lite", "qwen15_mixed"])
def test_plan_follows_the_cost_table(name, table):
    """The run-time plan prices tiles with whatever cost table is installed
    (mxmoe_set_tile_costs): the library's roofline default or a seeded random
    table give the oracle's plan under that table, and the forward's output
    stays correct; the profiled table is reinstalled afterwards."""
    from paper_2505_05799_amd import tile_cost as TC
    torch = torch_mod()
    blk = W.make_block(name)
    say(f"[{name}] cost table {table}")
    try:
        if table == "default":
            M.set_tile_costs(None)
        else:
            M.set_tile_costs(W.random_tile_costs(int(table[6:])))
        costs = M.get_tile_costs()
        if table != "default":
            assert np.array_equal(costs, W.random_tile_costs(int(table[6:])))
        mb = M.MoEBlock(blk)
        x, ids, w = upload_inputs(blk)
        y = mb.forward(x, ids, w)
        torch.cuda.synchronize()
        check_plan(mb, blk, O.route(blk.topk_ids, blk.cfg.E), costs)
        rep = check_forward(mb, blk, y)
        say(f"[{name}] {table}: {rep.line()}")
        del mb
    finally:
        M.set_tile_costs(TC.CostTable.load().device_table())
    assert np.array_equal(M.get_tile_costs(), TC.CostTable.load().device_table())
