"""GPU parity of the layer step under every recipe of paper_2606_20381_amd.recipe (Table 1, the Table 2
ablations, the E2M1 variants of Sec. 5 Q4 and the Appendix search space): the six quantized operands are
bit-exact against the oracle's layer_gemms, and the three outputs are within the GEMM tolerances
(relative Frobenius error <= 4e-3 for bf16 Y and dX, <= 1e-5 for fp32 dW)."""

import numpy as np
import pytest
import torch

from oracle import ufp4_oracle as O
from paper_2606_20381_amd import recipe as R
from paper_2606_20381_amd import workloads as WL
from paper_2606_20381_amd import ufp4 as U
from tests import parity as P

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    U.lib()


def test_recipe_tables_agree():
    assert set(R.RECIPES) == set(O.RECIPES) - {"mxufp4"}
    for name, r in R.RECIPES.items():
        cfg = O.RECIPES[name]
        assert r.fmt == cfg["fmt"] and tuple(r.rht) == tuple(cfg["rht"]), name
        assert set(r.sr) == set(cfg.get("sr", ("dy", "dyt"))), name
        assert r.max_fpx == (cfg.get("max_fpx") or 0.0) and r.rht_block == cfg.get("rht_block", 16), name
        assert all(R.LAYOUT[op][3] == O.SR_STREAMS[op] for op in R.OPERANDS)


@pytest.mark.parametrize("name", sorted(R.RECIPES))
@pytest.mark.parametrize("dual", [True, False])
def test_layer_step_matches_oracle(name, dual):
    rng = np.random.default_rng(101)
    M, N, K = 256, 384, 128  # multiples of 128 so that every RHT block fits every reduction axis
    g = torch.Generator().manual_seed(5)
    x = (torch.randn(M, K, generator=g) * 2).bfloat16()
    w = (torch.randn(N, K, generator=g) * 0.05).bfloat16()
    dy = (torch.randn(M, N, generator=g) * torch.exp(torch.randn(M, N, generator=g))).bfloat16()
    mask, seed = int(rng.integers(1, 1 << 16)), 77
    print(f"recipe {name} dual={dual}", flush=True)
    step = R.LayerStep(M, N, K, name, dual=dual)
    y, dx, dw = step.run(x.cuda(), w.cuda(), dy.cuda(), sign_mask=mask, seed=seed)
    torch.cuda.synchronize()
    q, out = O.layer_gemms(WL.bf16_bits(x), WL.bf16_bits(w), WL.bf16_bits(dy), name, sign_mask=mask, seed=seed)
    fmt = R.RECIPES[name].fmt
    for op in R.OPERANDS:
        gc, gs = P.gpu_rows(step.q[op])
        P.assert_codes_equal(gc, gs, q[op][0], q[op][1], fmt, f"{name} {op}")
    assert P.rel_fro(P.to_numpy(y), out["y"]) <= 4e-3
    assert P.rel_fro(P.to_numpy(dx), out["dx"]) <= 4e-3
    assert P.rel_fro(P.to_numpy(dw), out["dw"]) <= 1e-5
