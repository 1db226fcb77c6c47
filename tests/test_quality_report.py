"""Quality of the quantized operands and GEMMs on the synthetic layer tensors (oracle only, CPU): SQNR of each
operand in the rotated domain and the relative error of fwd_y against the unquantized product, for the UFP4
recipe (1x16 fp32 scales), the same grid with power-of-two 1x32 (E8M0) scales, and E2M1 with 1x16 fp32 scales.
Run with `pytest -s tests/test_quality_report.py` to see the table; the assertions are sanity bounds, not
the paper's numbers (those need its tensors)."""

import numpy as np
import pytest

from oracle import ufp4_oracle as O
from paper_2606_20381_amd import workloads as WL

ROWS = 256  # rows sampled from each tensor


def _rotated_reference(a_f32, mask):
    rows, red = a_f32.shape
    return O.rht_exact_f64(a_f32.reshape(rows, red // 16, 16), mask).reshape(rows, red)


def _operands(wl):
    return {
        "X": O.bf16_bits_to_f32(WL.bf16_bits(wl.x[:ROWS])),
        "W": O.bf16_bits_to_f32(WL.bf16_bits(wl.w.reshape(-1, wl.w.shape[-1])[:ROWS])),
        "dY": O.bf16_bits_to_f32(WL.bf16_bits(wl.dy[:ROWS])),
    }


def _sqnr_table(wl):
    mask, seed = wl.sign_mask, wl.seed
    out = {}
    for name, a in _operands(wl).items():
        rnd = O.SR if name == "dY" else O.RTNE
        ref = _rotated_reference(a, mask)
        iu, su = O.quantize_rows(a, O.UNIFORM, rnd, True, mask, seed, 0)
        im, em = O.quantize_rows_mx(a, rnd, True, mask, seed, 0)
        ie, se = O.quantize_rows(a, O.E2M1, rnd, True, mask, seed, 0)
        out[name] = {
            "ufp4 fp32/16": O.sqnr_db(O.dequantize(iu, su, O.UNIFORM), ref),
            "ufp4 e8m0/32": O.sqnr_db(O.dequantize_mx(im, em), ref),
            "e2m1 fp32/16": O.sqnr_db(O.dequantize(ie, se, O.E2M1), ref),
        }
    return out


def _gemm_errors(wl):
    mask = wl.sign_mask
    ops = _operands(wl)
    x, w = ops["X"], ops["W"]
    exact = x.astype(np.float64) @ w.astype(np.float64).T
    iu, su = O.quantize_rows(x, O.UNIFORM, O.RTNE, True, mask)
    ju, tu = O.quantize_rows(w, O.UNIFORM, O.RTNE, True, mask)
    im, em = O.quantize_rows_mx(x, O.RTNE, True, mask)
    jm, tm = O.quantize_rows_mx(w, O.RTNE, True, mask)
    rel = lambda c: float(np.linalg.norm(c - exact) / np.linalg.norm(exact))
    return {"ufp4 fp32/16": rel(O.gemm_nt(iu, su, ju, tu, O.UNIFORM)),
            "ufp4 e8m0/32": rel(O.gemm_nt_mx(im, em, jm, tm))}


@pytest.mark.parametrize("cfg", ["dense", "moe124b"])
def test_quality_of_scale_formats(cfg):
    wl = WL.dense_ffn() if cfg == "dense" else WL.moe_124b_share()
    table = _sqnr_table(wl)
    errs = _gemm_errors(wl)
    print(f"\n{wl.name}: operand SQNR (dB, rotated domain, {ROWS} rows)")
    for name, row in table.items():
        print(f"  {name:32s} " + "  ".join(f"{k} {v:6.2f}" for k, v in row.items()))
    print("  fwd_y relative Frobenius error vs the unquantized product: "
          + "  ".join(f"{k} {v:.4f}" for k, v in errs.items()))
    for name, row in table.items():
        # a power-of-two scale wastes at most one binade of the grid: a few dB below the fp32 scale
        assert row["ufp4 e8m0/32"] > row["ufp4 fp32/16"] - 6.0, name
        assert row["ufp4 fp32/16"] > 10.0, name
    assert errs["ufp4 e8m0/32"] < 2.0 * errs["ufp4 fp32/16"]


@pytest.mark.parametrize("cfg", ["dense", "moe124b"])
def test_rht_effect_per_grid(cfg):
    """Sec. 3.2 diagnostics from the oracle on 256 rows of X: Delta SQNR, B_eff and alpha for the uniform grid and
    E2M1, without and with the RHT. Sanity bounds only; on these outlier-heavy activations the rotation helps the
    uniform grid more than E2M1 (the paper's qualitative finding)."""
    wl = WL.dense_ffn() if cfg == "dense" else WL.moe_124b_share()
    a = _operands(wl)["X"]
    rows = {}
    for name, fmt in (("uniform", O.UNIFORM), ("e2m1", O.E2M1)):
        raw = O.quant_stats(a, fmt, O.RTNE, False, wl.sign_mask)
        rot = O.quant_stats(a, fmt, O.RTNE, True, wl.sign_mask)
        mr, mh = O.stats_metrics(raw, fmt), O.stats_metrics(rot, fmt)
        rows[name] = (O.delta_sqnr_db(mr["nmse"], mh["nmse"]), mr, mh)
        print(f"\n{wl.name} X {name}: dSQNR {rows[name][0]:+.2f} dB  B_eff {mr['beff']:.3f} -> {mh['beff']:.3f}  "
              f"alpha {mr['alpha']:.4f} -> {mh['alpha']:.4f}")
    assert rows["uniform"][0] > 0.0
    assert rows["uniform"][0] > rows["e2m1"][0]
