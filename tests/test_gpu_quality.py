"""GPU parity of the quality statistics (ufp4_quant_stats) and of the range-restricted E2M1 quantizer
(ufp4_e2m1_quantize_range) against the oracle, through the C ABI (ctypes binding).

Statistics: the magnitude-code histogram is compared exactly; the three fp64 sums to a relative 1e-9 (both
sides add the same exactly computed terms in fp64; only the order of the additions differs, which moves a
sum of n terms by at most about n * 2^-53 of the sum of magnitudes)."""

import numpy as np
import pytest
import torch

from oracle import ufp4_oracle as O
from paper_2606_20381_amd import ufp4 as U
from paper_2606_20381_amd import workloads as WL
from tests import parity as P

pytestmark = pytest.mark.gpu

SUM_RTOL = 1e-9
GRIDS = [(O.UNIFORM, 0.0), (O.E2M1, 0.0), (O.E2M1, 4.0), (O.E2M1, 2.0)]


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    U.lib()


def _operand(bits: np.ndarray, transpose: bool) -> np.ndarray:
    a = O.bf16_bits_to_f32(bits)
    return np.ascontiguousarray(a.T) if transpose else a


def _assert_stats(g: U.QuantStats, o: dict, what: str):
    assert g.hist == o["hist"].tolist(), f"{what}: histogram gpu {g.hist} oracle {o['hist'].tolist()}"
    for k in ("err2", "ref2", "cross"):
        want, got = o[k], getattr(g, k)
        assert got == pytest.approx(want, rel=SUM_RTOL, abs=1e-300), f"{what}: {k} gpu {got!r} oracle {want!r}"


def _check_stats(t: torch.Tensor, transpose, fmt, mf, rounding, rht, mask, seed, stream, what=""):
    bits = WL.bf16_bits(t)
    g = U.quant_stats(t.cuda(), fmt, max_fpx=mf, transpose=transpose, rht=rht, sign_mask=mask, rounding=rounding,
                      seed=seed, stream_id=stream)
    o = O.quant_stats(_operand(bits, transpose), fmt, rounding, rht, mask, seed, stream, max_fpx=mf or None)
    _assert_stats(g, o, f"{what} t={transpose} fmt={fmt} max={mf} rnd={rounding} rht={rht}")
    return g


@pytest.mark.parametrize("fmt,mf", GRIDS)
@pytest.mark.parametrize("rounding", [O.RTNE, O.SR])
@pytest.mark.parametrize("rht", [True, False])
def test_stats_tiny_layer_tensors(fmt, mf, rounding, rht):
    wl = WL.tiny()
    for name in ("x", "w", "dy"):
        t = getattr(wl, name)
        for transpose in (False, True):
            print(f"tiny {name} {tuple(t.shape)} t={transpose} fmt={fmt} max={mf} rnd={rounding} rht={rht}", flush=True)
            _check_stats(t, transpose, fmt, mf, rounding, rht, wl.sign_mask, wl.seed, 1, what=name)


@pytest.mark.parametrize("shape", [(16, 16), (48, 80), (272, 208), (144, 400), (400, 144), (16, 2048), (2064, 16)])
def test_stats_ragged_shapes(shape):
    """Grid-stride loops over several workgroups, ragged last waves; heavy-tailed values."""
    g = torch.Generator().manual_seed(shape[0] * 7 + shape[1])
    t = (torch.randn(*shape, generator=g) * torch.exp(2.0 * torch.randn(*shape, generator=g))).bfloat16()
    print(f"ragged {shape}", flush=True)
    for transpose in (False, True):
        _check_stats(t, transpose, O.UNIFORM, 0.0, O.SR, True, 0x1357, 5, 0, what=str(shape))
        _check_stats(t, transpose, O.E2M1, 0.0, O.RTNE, True, 0x1357, 5, 0, what=str(shape))
        _check_stats(t, transpose, O.E2M1, 2.0, O.SR, False, 0x1357, 5, 1, what=str(shape))


def test_stats_edge_cases():
    rec = torch.full((U.STATS_BYTES // 8,), 7.0, dtype=torch.float64, device="cuda")
    empty = torch.zeros((0, 32), dtype=torch.bfloat16, device="cuda")
    g = U.quant_stats(empty, out=rec)
    assert (g.err2, g.ref2, g.cross, g.hist) == (0.0, 0.0, 0.0, [0] * 8)
    zeros = torch.zeros((64, 48), dtype=torch.bfloat16, device="cuda")
    for fmt, mf in GRIDS:
        g = U.quant_stats(zeros, fmt, max_fpx=mf, out=rec)
        assert (g.err2, g.ref2, g.cross) == (0.0, 0.0, 0.0) and g.hist == [64 * 48] + [0] * 7
    # values on the uniform grid (a top level in every block) are lossless; the record is overwritten
    k = torch.randint(-7, 8, (32, 64), generator=torch.Generator().manual_seed(3)).float()
    k[:, ::16] = 7.0
    g = U.quant_stats((k * 0.25).bfloat16().cuda(), O.UNIFORM, rht=False, out=rec)
    assert g.err2 == 0.0 and g.alpha == 1.0
    assert g.hist == np.bincount(k.abs().long().flatten().numpy(), minlength=8).tolist()


@pytest.mark.parametrize("cfg", ["dense", "moe124b"])
def test_stats_full_size_operands(cfg):
    """Layer tensors at full size: RTNE sums over all rows equal those over two row halves (additivity),
    and a 64-row / 64-column slice matches the oracle exactly as above."""
    wl = WL.dense_ffn() if cfg == "dense" else WL.moe_124b_share()
    for name in ("x", "dy"):
        t = getattr(wl, name).cuda()
        for fmt in (O.UNIFORM, O.E2M1):
            print(f"{cfg} {name} {tuple(t.shape)} fmt={fmt}", flush=True)
            full = U.quant_stats(t, fmt, rht=True, sign_mask=wl.sign_mask)
            h = t.shape[0] // 2
            a = U.quant_stats(t[:h], fmt, rht=True, sign_mask=wl.sign_mask)
            b = U.quant_stats(t[h:], fmt, rht=True, sign_mask=wl.sign_mask)
            assert full.hist == [x + y for x, y in zip(a.hist, b.hist)]
            assert sum(full.hist) == t.numel()
            for k in ("err2", "ref2", "cross"):
                assert getattr(full, k) == pytest.approx(getattr(a, k) + getattr(b, k), rel=SUM_RTOL)
            _check_stats(t[:64].cpu(), False, fmt, 0.0, O.SR, True, wl.sign_mask, wl.seed, 0, what=f"{cfg} {name}")
            _check_stats(t[:, 64:128].cpu(), True, fmt, 0.0, O.RTNE, True, wl.sign_mask, wl.seed, 0,
                         what=f"{cfg} {name}")
            g = U.quant_stats(t[:, 64:128], fmt, transpose=True, rht=True, sign_mask=wl.sign_mask)
            o = O.quant_stats(_operand(WL.bf16_bits(t[:, 64:128].cpu()), True), fmt, O.RTNE, True, wl.sign_mask)
            _assert_stats(g, o, f"{cfg} {name} strided slice")


@pytest.mark.parametrize("mf", [2.0, 4.0, 6.0])
@pytest.mark.parametrize("rounding", [O.RTNE, O.SR])
@pytest.mark.parametrize("layout", ["rows", "cols"])
def test_range_restricted_e2m1_quantizer(mf, rounding, layout):
    """ufp4_e2m1_quantize_range: codes and scales bit-exact against the oracle's cut grid."""
    wl = WL.tiny()
    for name, rht in (("x", False), ("w", True), ("dy", True)):
        bits = WL.bf16_bits(getattr(wl, name))
        print(f"range {name} max={mf} rnd={rounding} {layout}", flush=True)
        q = U.e2m1_quantize_range(getattr(wl, name).cuda(), mf, transpose=(layout == "cols"), rht=rht,
                                  sign_mask=wl.sign_mask, rounding=rounding, seed=wl.seed, stream_id=1)
        torch.cuda.synchronize()
        gc, gs = P.gpu_rows(q)
        a = _operand(bits, layout == "cols")
        idx, sc = O.quantize_rows(a, O.E2M1, rounding, rht, wl.sign_mask, wl.seed, 1, max_fpx=mf)
        P.assert_codes_equal(gc, gs, idx, sc, O.E2M1, f"range {name} max={mf} {layout}")
        if mf == 6.0:  # the full grid: identical to the plain E2M1 quantizer
            q6 = U.e2m1_quantize(getattr(wl, name).cuda(), transpose=(layout == "cols"), rht=rht,
                                 sign_mask=wl.sign_mask, rounding=rounding, seed=wl.seed, stream_id=1)
            assert torch.equal(q6.codes_rows(), q.codes_rows()) and torch.equal(q6.scales_rows(), q.scales_rows())
