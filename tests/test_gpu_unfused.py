"""GPU parity of the unfused form of RHT + quantization (ufp4_rht, then ufp4_quantize_f32): the standalone
transform is bit-exact against the oracle's correctly rounded RHT, the fp32-input quantizer bit-exact against
the oracle's quantizer on fp32 values, and the two halves together reproduce the fused kernel's codes and
scales bit for bit."""

import numpy as np
import pytest
import torch

from oracle import ufp4_oracle as O
from paper_2606_20381_amd import ufp4 as U
from paper_2606_20381_amd import workloads as WL
from tests import parity as P

pytestmark = pytest.mark.gpu

SHAPES = [(1, 16), (48, 80), (272, 208), (33, 4096), (130, 16), (700, 48)]


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    U.lib()


def _tensor(shape, seed):
    g = torch.Generator().manual_seed(seed)
    return (torch.randn(*shape, generator=g) * torch.exp(1.5 * torch.randn(*shape, generator=g))).bfloat16()


@pytest.mark.parametrize("shape", SHAPES)
def test_standalone_rht_is_correctly_rounded(shape):
    t = _tensor(shape, shape[0] * 31 + shape[1])
    print(f"rht {shape}", flush=True)
    for mask in (0x0000, 0xB3C5):
        y = U.rht(t.cuda(), sign_mask=mask).cpu().numpy()
        a = O.bf16_bits_to_f32(WL.bf16_bits(t))
        want = O.rht_blocks(a.reshape(shape[0], -1, 16), mask).reshape(shape)
        assert np.array_equal(y.view(np.uint32), want.astype(np.float32).view(np.uint32)), f"{shape} mask={mask:#x}"


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
@pytest.mark.parametrize("rounding", [O.RTNE, O.SR])
def test_unfused_equals_fused(shape, fmt, rounding):
    t = _tensor(shape, shape[0] * 17 + shape[1]).cuda()
    print(f"unfused {shape} fmt={fmt} rnd={rounding}", flush=True)
    fused = (U.rht_quantize if fmt == O.UNIFORM else U.e2m1_quantize)(t, rht=True, sign_mask=0x6A09,
                                                                     rounding=rounding, seed=11, stream_id=1)
    y = U.rht(t, sign_mask=0x6A09)
    q = U.empty_qtensor(shape[0], shape[1], fmt)
    q.codes.fill_(0xFF)
    q.scales.view(torch.int32).fill_(-1)
    U.quantize_f32(y, fmt, rounding=rounding, seed=11, stream_id=1, out=q)
    torch.cuda.synchronize()
    assert torch.equal(q.codes_rows(), fused.codes_rows()) and torch.equal(q.scales_rows(), fused.scales_rows())
    nkb, tail = shape[1] // 16, q.panels * U.PANEL_ROWS - shape[0]
    if tail:  # padding rows of the last panel are written as zeros
        assert int(q.codes[-1, : nkb * 1024].reshape(nkb, U.PANEL_ROWS, 8)[:, U.PANEL_ROWS - tail:].count_nonzero()) == 0
        assert int(q.scales[-1, : nkb * 128].reshape(nkb, U.PANEL_ROWS)[:, U.PANEL_ROWS - tail:].count_nonzero()) == 0


@pytest.mark.parametrize("shape", SHAPES)
def test_fp32_input_quantizer_against_the_oracle(shape):
    """fp32 values that are not bf16 numbers (24-bit significands), both grids and roundings."""
    g = torch.Generator().manual_seed(shape[0] + 5 * shape[1])
    x = torch.randn(*shape, generator=g, dtype=torch.float32) * 3.0
    a = x.numpy()
    print(f"f32 {shape}", flush=True)
    for fmt in (O.UNIFORM, O.E2M1):
        for rounding in (O.RTNE, O.SR):
            q = U.quantize_f32(x.cuda(), fmt, rounding=rounding, seed=21, stream_id=0)
            torch.cuda.synchronize()
            gc, gs = P.gpu_rows(q)
            idx, sc = O.quantize_rows(a, fmt, rounding, False, 0, 21, 0)
            P.assert_codes_equal(gc, gs, idx, sc, fmt, f"f32 {shape} fmt={fmt} rnd={rounding}")


def test_strided_buffers():
    """Leading dimensions larger than the row: x (bf16) and y (fp32) views into wider buffers."""
    big = _tensor((64, 96), 3).cuda()
    x = big[:, 16:80]
    ybuf = torch.full((64, 100), float("nan"), dtype=torch.float32, device="cuda")
    y = ybuf[:, 4:68]
    U.rht(x, sign_mask=0x1234, out=y)
    want = O.rht_blocks(O.bf16_bits_to_f32(WL.bf16_bits(x.cpu())).reshape(64, 4, 16), 0x1234).reshape(64, 64)
    assert np.array_equal(y.cpu().numpy().view(np.uint32), want.astype(np.float32).view(np.uint32))
    assert torch.isnan(ybuf[:, :4]).all() and torch.isnan(ybuf[:, 68:]).all()
    q = U.quantize_f32(y, O.UNIFORM)
    ref = U.rht_quantize(x, rht=True, sign_mask=0x1234)
    assert torch.equal(q.codes_rows(), ref.codes_rows()) and torch.equal(q.scales_rows(), ref.scales_rows())
