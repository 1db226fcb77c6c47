"""Blocks whose nonzero magnitudes span more than the kernels' fp64 butterfly sums exactly (2^41): ties at fp32
precision decided by a tiny term, large terms that cancel after a small one has been absorbed, and random spans up
to the whole bf16 range. The oracle computes the exact transform of every block (Sec. 2.2); the kernels may lose
such a block's smallest terms, an error below 2^-46 of the block's largest magnitude before the rounding to fp32.
What that leaves, and what is asserted here for the rowwise, transposed and two-operand kernels: every scale within
two fp32 ulps of the oracle's and every code within one level of it (a rounding decision near its boundary may
flip, nothing more)."""

import numpy as np
import pytest
import torch

from oracle import ufp4_oracle as O
from paper_2606_20381_amd import ufp4 as U
from paper_2606_20381_amd import workloads as WL
from tests import parity as P

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    U.lib()


BF16_MAX = (2.0 - 2.0 ** -7) * 2.0 ** 127
MASK = 0x3A5C


def _wide_rows(n_random=240, seed=3):
    """[rows, 64] bf16 bit patterns: four 16-blocks per row, every block wider than 2^41."""
    rows = []
    crafted = [
        [1.0, 2.0 ** -24, 2.0 ** -100],
        [2.0 ** 100, 2.0 ** 76, -(2.0 ** -120)],
        [2.0 ** -60, 2.0 ** -84, 2.0 ** -133, 2.0 ** -130],
        [1.0, 2.0 ** -100, 1.0],                        # cancels in the rows of H that subtract the two ones
        [1.0, 0.0, 3.0 * 2.0 ** -24, 0.0, 2.0 ** -100, 2.0 ** -100],
        [2.0 ** 126, -(2.0 ** 126), 2.0 ** 80, 2.0 ** 30],
        # the mask's own signs: the eight maxima align in the first sum, which passes FLT_MAX (24 bits, no overflow)
        [-BF16_MAX if (MASK >> j) & 1 else BF16_MAX for j in range(8)] + [2.0 ** 70],
        [2.0 ** 20, 2.0 ** -22],
    ]
    blocks = []
    for c in crafted:
        b = np.zeros(16)
        b[:len(c)] = c
        blocks.append(b)
        blocks.append(b[::-1].copy())
    rng = np.random.default_rng(seed)
    for _ in range(n_random):
        mant = rng.integers(-255, 256, size=16).astype(np.float64)
        spread = int(rng.integers(42, 250))
        base = int(rng.integers(-100, 120))
        expo = np.clip(base - (rng.random(16) * (spread + 1)).astype(np.int64), -133, 120)
        b = mant * np.exp2(expo - 7)
        b[rng.random(16) < 0.15] = 0.0
        if rng.random() < 0.3:  # equal magnitudes that cancel in some rows of H
            i, j = rng.choice(16, 2, replace=False)
            b[j] = b[i] if rng.random() < 0.5 else -b[i]
        blocks.append(b)
    while len(blocks) % 4:
        blocks.append(blocks[0])
    a = np.array(blocks).reshape(-1, 64)
    return O.f32_to_bf16_bits(a.astype(np.float32))


def _assert_within_one_level(gpu_codes, gpu_scales, idx, sc, fmt, what):
    gi = O.unpack_codes(gpu_codes, fmt)
    step = np.abs(gi - idx)
    assert step.max() <= 1, f"{what}: a code {step.max()} levels from the oracle's"
    gs = np.asarray(gpu_scales, dtype=np.float64)
    want = np.asarray(sc, dtype=np.float32).astype(np.float64)
    assert np.all(want > 0), "every test block is nonzero"
    ulp = np.spacing(np.asarray(sc, dtype=np.float32)).astype(np.float64)
    assert np.all(np.abs(gs - want) <= 2 * ulp), f"{what}: a scale more than two fp32 ulps from the oracle's"
    print(f"{what}: {int((step > 0).sum())} of {step.size} codes and {int((gs != want).sum())} of {gs.size} "
          f"scales differ from the exact transform's", flush=True)


def _wide_tensor():
    bits = _wide_rows()
    a = O.bf16_bits_to_f32(bits)
    wide = ~O._fp64_sums_exact(a.reshape(-1, 16).astype(np.float64))
    assert wide.sum() >= 200, "most blocks span more than 2^41"
    return bits


def _device(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


@pytest.mark.parametrize("layout", ["rows", "cols"])
@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
@pytest.mark.parametrize("rounding", [O.RTNE, O.SR])
def test_wide_span_blocks_within_one_level(layout, fmt, rounding):
    bits = _wide_tensor()
    if layout == "cols":  # the blocks run down the columns of T; operand row r is column r
        bits = np.ascontiguousarray(bits.T)
    q = P.gpu_operand(_device(bits), layout, fmt, rounding, True, MASK, 11, 0)
    gc, gs = P.gpu_rows(q)
    idx, sc = P.oracle_operand(bits, layout, fmt, rounding, True, MASK, 11, 0)
    _assert_within_one_level(gc, gs, idx, sc, fmt, f"{layout} fmt {fmt} rounding {rounding}")


def test_wide_span_blocks_two_operand_kernel():
    bits = _wide_tensor()
    # rows of `bits` carry the wide blocks; its transpose puts them down the columns for the transposed output
    for name, t in (("rows", bits), ("cols", np.ascontiguousarray(bits.T))):
        qr, qc = U.quantize_dual(_device(t), sign_mask_rows=MASK, sign_mask_cols=MASK)
        q = qr if name == "rows" else qc
        gc, gs = P.gpu_rows(q)
        idx, sc = P.oracle_operand(t, name, O.UNIFORM, O.RTNE, True, MASK, 0, 0)
        _assert_within_one_level(gc, gs, idx, sc, O.UNIFORM, f"two-operand {name}")


@pytest.mark.parametrize("layout", ["rows", "cols"])
@pytest.mark.parametrize("rounding", [O.RTNE, O.SR])
def test_wide_span_blocks_power_of_two_scales(layout, rounding):
    """The same blocks through the power-of-two-scale quantizer (two RHT16 halves per 1x32 block): a scale
    exponent may move by one where a rounded output crosses a power of two; where it does not, every code stays
    within one level of the exact transform's, and every dequantized value within two steps of the coarser grid."""
    bits = _wide_tensor()
    if layout == "cols":
        bits = np.ascontiguousarray(bits.T)
    q = U.mx_quantize(_device(bits), transpose=(layout == "cols"), rht=True, sign_mask=MASK, rounding=rounding,
                      seed=11, stream_id=0)
    gi = O.unpack_fp6(q.codes_rows().cpu().numpy())
    ge = q.scales_rows().cpu().numpy().astype(np.int64)
    a = O.bf16_bits_to_f32(bits) if layout == "rows" else np.ascontiguousarray(O.bf16_bits_to_f32(bits).T)
    idx, e8 = O.quantize_rows_mx(a, rounding, True, MASK, 11, 0)
    e8 = e8.astype(np.int64)
    assert np.abs(ge - e8).max() <= 1, "a scale exponent more than one from the oracle's"
    same = np.repeat(ge == e8, O.MX_BLOCK, axis=1)
    assert np.abs(gi - idx)[same].max(initial=0) <= 1, "a code more than one level from the oracle's"
    step = np.exp2(np.repeat(np.maximum(ge, e8), O.MX_BLOCK, axis=1).astype(np.float64) - 127)
    deq_g = gi * np.exp2(np.repeat(ge, O.MX_BLOCK, axis=1).astype(np.float64) - 127)
    deq_o = idx * np.exp2(np.repeat(e8, O.MX_BLOCK, axis=1).astype(np.float64) - 127)
    assert np.all(np.abs(deq_g - deq_o) <= 2 * step)
    print(f"power-of-two {layout} rounding {rounding}: {int((gi != idx).sum())} of {gi.size} codes and "
          f"{int((ge != e8).sum())} of {ge.size} exponents differ from the exact transform's", flush=True)
