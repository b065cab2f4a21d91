"""GPU parity of the router front-end (softmax top-k of the router logits and
the sigmoid gate of shared experts) and of the forward that starts from
logits, against the CPU oracle.  Expert ids are compared bit for bit; weights
within the fp32 error bound of an exp-sum-divide: each exp within 2 ulp, the
sum of n positive terms within (n - 1) units of 2^-24, one division, so
|w - ref| <= (n + 8) 2^-24 ref with n = E (k when renormalised)."""

import dataclasses

import numpy as np
import pytest

from oracle import mxmoe_oracle as O
from paper_2505_05799_amd import mxmoe as M
from paper_2505_05799_amd import workloads as W
from tests.gpuhelp import say, torch_mod, upload_inputs
from tests.stagewise import check_forward

pytestmark = pytest.mark.gpu

CASES = [(1, 8, 2), (37, 60, 4), (300, 64, 6), (513, 65, 8), (64, 160, 6), (33, 1024, 8), (5, 1024, 64),
         (16, 64, 64), (8192, 60, 4)]


def _weights_ok(w, ref, n):
    bound = (n + 8) * 2.0 ** -24 * np.abs(ref) + 1e-45
    assert np.all(np.abs(w.astype(np.float64) - ref) <= bound), float((np.abs(w - ref) / bound).max())


@pytest.mark.parametrize("renorm", [False, True])
@pytest.mark.parametrize("T,E,k", CASES)
def test_router_topk(T, E, k, renorm):
    torch = torch_mod()
    l, sh = W.router_logits(T, E, seed=T + E, zipf_s=1.2, n_shared=2)
    l[:, 1] = l[:, 3]                                # a tie in every row
    ids, w, shw = M.router_topk(torch.from_numpy(l).cuda(), k, renorm, torch.from_numpy(sh).cuda())
    torch.cuda.synchronize()
    rids, rw = O.router_topk(l, k, renorm)
    assert np.array_equal(ids.cpu().numpy(), rids)
    _weights_ok(w.cpu().numpy(), rw, k if renorm else E)
    # sigmoid: exp within 2 ulp, one add, one division
    g = shw.cpu().numpy().astype(np.float64)
    rg = O.shared_gate(sh)
    assert np.all(np.abs(g - rg) <= 8 * 2.0 ** -24 * rg)
    say(f"router T={T} E={E} k={k} renorm={renorm}: ok")


def test_router_ties_and_nan():
    torch = torch_mod()
    rng = np.random.default_rng(5)
    l = rng.integers(-2, 3, size=(200, 64)).astype(np.float32)   # many exact ties
    l[7, 0] = np.nan                                             # a NaN is never chosen
    ids, w, _ = M.router_topk(torch.from_numpy(l).cuda(), 8)
    torch.cuda.synchronize()
    rids, rw = O.router_topk(l, 8)
    assert np.array_equal(ids.cpu().numpy(), rids)
    ok = np.ones(200, bool)
    ok[7] = False                                                 # its weights are NaN on both sides
    _weights_ok(w.cpu().numpy()[ok], rw[ok], 64)


def test_router_rejects():
    torch = torch_mod()
    l = torch.zeros((4, 8), dtype=torch.float32, device="cuda")
    for k in (0, 9):
        with pytest.raises(M.MxmoeError):
            M.router_topk(l, k)
    with pytest.raises(M.MxmoeError):
        M.router_topk(torch.zeros((4, 100), dtype=torch.float32, device="cuda"), 65)


@pytest.mark.parametrize("renorm", [False, True])
@pytest.mark.parametrize("T", [300, 2500])
def test_forward_from_logits(renorm, T):
    """Router mode of the forward: same ids and weights as the standalone
    router, the same output bit for bit as the forward given those ids, and
    the oracle's output with the sigmoid shared gates; 300 x 2 pairs route in
    the one-workgroup routing kernel, 2500 x 2 in the chunked launches."""
    torch = torch_mod()
    sch = [(W.W4G128,) * 3, (W.W8A8, W.W8A8, W.W2G128), (W.W4A4,) * 3, (W.W16,) * 3, (W.W4A4G128,) * 3,
           (W.W3G128, W.W3G128, W.W8A8), (W.W8A8,) * 3]
    blk = W.random_small_block(77, T=T, H=256, F=384, E=6, k=2, n_shared=1, F_shared=256, act="bf16",
                               schemes=sch)
    E, k = 6, 2
    l, sh = W.router_logits(T, E, seed=9, zipf_s=1.0, n_shared=1)
    lt, sht = torch.from_numpy(l).cuda(), torch.from_numpy(sh).cuda()
    mb = M.MoEBlock(blk)
    x, _, _ = upload_inputs(blk)
    y = mb.forward(x, None, None, router_logits=lt, renormalize=renorm, shared_logits=sht)
    torch.cuda.synchronize()
    y_np = M.act_numpy(y, "bf16")
    fids = mb.ws_view("router_ids", torch.int32, T * k, T).cpu().numpy().reshape(T, k)
    fw = mb.ws_view("router_w", torch.float32, T * k, T).cpu().numpy().reshape(T, k)
    fg = mb.ws_view("shared_w", torch.float32, T, T).cpu().numpy().reshape(T, 1)
    ids, w, g = M.router_topk(lt, k, renorm, sht)
    torch.cuda.synchronize()
    assert np.array_equal(fids, ids.cpu().numpy())
    assert np.array_equal(fw.view(np.uint32), w.cpu().numpy().view(np.uint32))
    assert np.array_equal(fg.view(np.uint32), g.cpu().numpy().view(np.uint32))
    # the same forward from those ids and weights, shared gates as weights
    y2 = mb.forward(x, ids, w, shared_w=g)
    torch.cuda.synchronize()
    assert np.array_equal(M.act_numpy(y2, "bf16"), y_np)
    rids, rw = O.router_topk(l, k, renorm)
    assert np.array_equal(fids, rids)
    blk2 = dataclasses.replace(blk, topk_ids=fids, topk_w=fw)
    rep = check_forward(mb, blk2, y, shared_w=fg)
    say(f"forward from logits renorm={renorm}: {rep.line()}")


def test_forward_shared_weights():
    torch = torch_mod()
    sch = [(W.W8A8,) * 3, (W.W4G128,) * 3, (W.W4A4,) * 3, (W.W2G128,) * 3, (W.W8A8, W.W8A8, W.W4A4G128),
           (W.W16,) * 3]
    blk = W.random_small_block(31, T=65, H=256, F=256, E=4, k=2, n_shared=2, F_shared=256, act="fp16",
                               schemes=sch)
    g = np.random.default_rng(2).random((65, 2)).astype(np.float32)
    mb = M.MoEBlock(blk)
    x, ids, w = upload_inputs(blk)
    y = mb.forward(x, ids, w, shared_w=torch.from_numpy(g).cuda())
    torch.cuda.synchronize()
    rep = check_forward(mb, blk, y, shared_w=g)
    say(f"shared weights: {rep.line()}")
