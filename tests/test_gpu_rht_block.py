"""GPU parity of the RHT over 32-, 64- and 128-element blocks followed by the 1x16 quantizer
(ufp4_quantize_rht_block): codes and scales bit-exact against the oracle, rowwise and transposed, both grids,
RTNE and SR, ragged operand rows; block 16 through this entry point equals the fused block-16 quantizer."""

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


def _tensor(shape, seed):
    g = torch.Generator().manual_seed(seed)
    return (torch.randn(*shape, generator=g) * torch.exp(torch.randn(*shape, generator=g))).bfloat16()


def _check(t, n, fmt, rounding, transpose, mask, what):
    bits = WL.bf16_bits(t)
    q = U.quantize_rht_block(t.cuda(), fmt, rht_block=n, sign_mask=mask, transpose=transpose, rounding=rounding,
                             seed=13, stream_id=1)
    torch.cuda.synchronize()
    gc, gs = P.gpu_rows(q)
    a = O.bf16_bits_to_f32(bits)
    a = np.ascontiguousarray(a.T) if transpose else a
    idx, sc = O.quantize_rows(a, fmt, rounding, True, mask, 13, 1, rht_block=n)
    P.assert_codes_equal(gc, gs, idx, sc, fmt, what)


@pytest.mark.parametrize("n", [32, 64, 128])
@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
@pytest.mark.parametrize("rounding", [O.RTNE, O.SR])
def test_rht_block_rowwise_and_transposed(n, fmt, rounding):
    rng = np.random.default_rng(n * 10 + fmt * 2 + rounding)
    mask = int.from_bytes(rng.bytes(n // 8), "little")
    for shape in ((40, 256), (3, 512), (130, 128)):
        t = _tensor(shape, shape[0] + shape[1] + n)
        print(f"rows n={n} fmt={fmt} rnd={rounding} {shape}", flush=True)
        _check(t, n, fmt, rounding, False, mask, f"rows n={n} {shape}")
    for shape in ((256, 40), (512, 24), (128, 136)):
        t = _tensor(shape, shape[0] * 3 + shape[1] + n)
        print(f"cols n={n} fmt={fmt} rnd={rounding} {shape}", flush=True)
        _check(t, n, fmt, rounding, True, mask, f"cols n={n} {shape}")


def test_rht_block_layer_tensors():
    wl = WL.tiny()
    for name in ("x", "w", "dy"):
        t = getattr(wl, name)
        for n in (32, 64, 128):
            if t.shape[1] % n == 0:
                _check(t, n, O.UNIFORM, O.SR, False, 0xDEADBEEF12345678, f"tiny {name} rows n={n}")
            if t.shape[0] % n == 0:
                _check(t, n, O.UNIFORM, O.RTNE, True, 0xDEADBEEF12345678, f"tiny {name} cols n={n}")


def test_rht_block_16_is_the_fused_quantizer():
    t = _tensor((96, 160), 7).cuda()
    for transpose in (False, True):
        a = U.quantize_rht_block(t, O.UNIFORM, rht_block=16, sign_mask=0xA5C3, transpose=transpose, rounding=O.SR,
                                 seed=3)
        b = U.rht_quantize(t, transpose=transpose, rht=True, sign_mask=0xA5C3, rounding=O.SR, seed=3)
        assert torch.equal(a.codes_rows(), b.codes_rows()) and torch.equal(a.scales_rows(), b.scales_rows())


def test_rht_block_shape_errors():
    t = _tensor((32, 48), 1).cuda()
    with pytest.raises(U.UFP4Error):
        U.quantize_rht_block(t, O.UNIFORM, rht_block=32)  # 48 is not a multiple of 32
    with pytest.raises(U.UFP4Error):
        U.quantize_rht_block(t, O.UNIFORM, rht_block=48)
