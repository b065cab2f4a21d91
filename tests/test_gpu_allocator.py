"""GPU checks of the allocator's sensitivity measurement (Eq. 5-6): the
per-(expert, linear block) output distortion read from the forward's slot
rows against the oracle's block output with only that expert's linear block
quantized."""

import numpy as np
import pytest

from oracle import mxmoe_oracle as O
from paper_2505_05799_amd import allocator as A
from paper_2505_05799_amd import workloads as W
from tests.gpuhelp import say, torch_mod

pytestmark = pytest.mark.gpu


def test_sensitivity_matches_the_oracle():
    torch_mod()
    cfg = W.BlockConfig("sens", T=200, H=256, F=384, E=5, k=2, n_shared=1, F_shared=256, act="bf16",
                        zipf_s=0.8, alloc=lambda e, r: (W.W16,) * 3, shared_alloc=(W.W16,) * 3)
    cands = [W.W16, W.W8A8, W.W4A4, W.W4G128, W.W4A4G128]
    delta = A.sensitivity(cfg, cands, calib_tokens=200, log=say)
    G = cfg.E + cfg.n_shared
    # 16-bit in place of 16-bit changes nothing, bit for bit
    assert np.all(delta[:, :, 0] == 0)
    base = W.make_block(cfg)
    ref_lin = base.linears
    for j in range(2):
        for ci, s in enumerate(cands[1:], start=1):
            def alloc(e, r, s=s, j=j):
                return (s, s, W.W16) if j == 0 else (W.W16, W.W16, s)
            q = W.make_block(W.BlockConfig(**{**cfg.__dict__, "alloc": alloc, "shared_alloc": alloc(0, 0)}))
            for g in range(G):
                # the oracle's block output with only expert g perturbed, on the tokens' slots of g
                lins = [q.linears[e] if e == g else ref_lin[e] for e in range(G)]
                if g < cfg.E:
                    ids = np.where(base.topk_ids == g, base.topk_ids, -1).astype(np.int32)
                    sh = [ref_lin[cfg.E]]
                    y1 = O.moe_forward(base.x, ids, base.topk_w, lins[:cfg.E] + [lins[cfg.E]], cfg.E, "bf16",
                                       shared_w=np.zeros((cfg.T, 1), np.float32))["y"]
                    y0 = O.moe_forward(base.x, ids, base.topk_w, ref_lin[:cfg.E] + sh, cfg.E, "bf16",
                                       shared_w=np.zeros((cfg.T, 1), np.float32))["y"]
                else:
                    none = np.full_like(base.topk_ids, -1)
                    y1 = O.moe_forward(base.x, none, base.topk_w, lins, cfg.E, "bf16")["y"]
                    y0 = O.moe_forward(base.x, none, base.topk_w, ref_lin, cfg.E, "bf16")["y"]
                want = float(np.sqrt(((y1 - y0) ** 2).sum()))
                got = delta[g, j, ci]
                # GPU rows carry fp32 accumulation error (and an a8/a4 code of h may
                # flip): small next to the quantization error being measured
                assert abs(got - want) <= 0.05 * want + 1e-6, (g, j, s.name, got, want)
        say(f"linear block {j}: sensitivities match the oracle")
    # fewer bits, more distortion, for every expert
    assert np.all(delta[:, :, 2] > delta[:, :, 1])
