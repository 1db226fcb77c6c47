"""Maximum sizes through the C ABI: the largest rowwise operand the quantizers accept (and the first size they
refuse), reductions of 2^20 elements in both quantizer layouts, and GEMMs whose reduction is 65536 long (4096
per-16 blocks, 1024 stages of the MX kernel), each against the oracle (sampled rows where the tensor is large)."""

import numpy as np
import pytest
import torch

from oracle import ufp4_oracle as O
from paper_2606_20381_amd import ufp4 as U
from paper_2606_20381_amd import workloads as WL
from tests import parity as P

pytestmark = pytest.mark.gpu

MAX_ROWS = 2097024  # 16383 panels: the rowwise grid has at most 65535 tiles of 32 rows
MAX_ROWS_MX = 4194176  # 32767 panels: the MX rowwise grid has at most 65535 tiles of 64 rows


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    U.lib()


def _tensor(shape, seed, std=1.0):
    g = torch.Generator().manual_seed(seed)
    return (torch.randn(*shape, generator=g) * std).bfloat16()


def test_rowwise_row_limit():
    t = _tensor((MAX_ROWS, 16), 1)
    bits = WL.bf16_bits(t)
    x = t.cuda()
    print(f"rowwise {MAX_ROWS} x 16", flush=True)
    q = U.rht_quantize(x, rht=True, sign_mask=0x1357, rounding=U.SR, seed=9, stream_id=0)
    torch.cuda.synchronize()
    rows = P.sample(MAX_ROWS, 64, np.random.default_rng(0))
    gc, gs = P.gpu_rows(q, rows)
    idx, sc = P.oracle_operand(bits, "rows", O.UNIFORM, O.SR, True, 0x1357, 9, 0, rows)
    P.assert_codes_equal(gc, gs, idx, sc, O.UNIFORM, "row limit")
    with pytest.raises(U.UFP4Error) as e:
        U.rht_quantize(torch.zeros((MAX_ROWS + 1, 16), dtype=torch.bfloat16, device="cuda"))
    assert e.value.status == 5
    del q, x


def test_mx_rowwise_row_limit():
    t = _tensor((MAX_ROWS_MX, 32), 2)
    x = t.cuda()
    print(f"mx rowwise {MAX_ROWS_MX} x 32", flush=True)
    q = U.mx_quantize(x, rht=True, sign_mask=0x2468)
    torch.cuda.synchronize()
    rows = P.sample(MAX_ROWS_MX, 48, np.random.default_rng(1))
    a = O.bf16_bits_to_f32(WL.bf16_bits(t[torch.as_tensor(rows)]))
    idx, e8 = O.quantize_rows_mx(a, O.RTNE, True, 0x2468)
    codes, scales = q.codes_rows(), q.scales_rows()
    r = torch.as_tensor(rows, device="cuda")
    assert np.array_equal(codes[r].cpu().numpy(), O.pack_fp6(idx))
    assert np.array_equal(scales[r].cpu().numpy(), e8.astype(np.uint8))
    with pytest.raises(U.UFP4Error) as e:
        U.mx_quantize(torch.zeros((MAX_ROWS_MX + 1, 32), dtype=torch.bfloat16, device="cuda"))
    assert e.value.status == 5
    del q, x


@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
def test_long_reduction_both_layouts(fmt):
    red = 1 << 20
    t = _tensor((4, red), 3)
    print(f"long reduction rowwise 4 x {red} fmt={fmt}", flush=True)
    q = (U.rht_quantize if fmt == O.UNIFORM else U.e2m1_quantize)(t.cuda(), rht=True, sign_mask=0x0FF0,
                                                                  rounding=U.SR, seed=5, stream_id=1)
    gc, gs = P.gpu_rows(q)
    idx, sc = P.oracle_operand(WL.bf16_bits(t), "rows", fmt, O.SR, True, 0x0FF0, 5, 1)
    P.assert_codes_equal(gc, gs, idx, sc, fmt, "long rowwise")
    tt = _tensor((red, 16), 4)
    print(f"long reduction transposed {red} x 16 fmt={fmt}", flush=True)
    q = (U.rht_quantize if fmt == O.UNIFORM else U.e2m1_quantize)(tt.cuda(), transpose=True, rht=True,
                                                                  sign_mask=0x0FF0, rounding=U.SR, seed=5, stream_id=1)
    gc, gs = P.gpu_rows(q)
    idx, sc = P.oracle_operand(WL.bf16_bits(tt), "cols", fmt, O.SR, True, 0x0FF0, 5, 1)
    P.assert_codes_equal(gc, gs, idx, sc, fmt, "long transposed")


@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
def test_gemm_long_reduction(fmt):
    m, n, k = 130, 96, 65536
    a, b = _tensor((m, k), 6), _tensor((n, k), 7, 0.02)
    print(f"gemm long K {m}x{n}x{k} fmt={fmt}", flush=True)
    Q = U.rht_quantize if fmt == O.UNIFORM else U.e2m1_quantize
    qa, qb = Q(a.cuda(), rht=True, sign_mask=0x7777), Q(b.cuda(), rht=True, sign_mask=0x7777)
    ia, sa = O.quantize_rows(O.bf16_bits_to_f32(WL.bf16_bits(a)), fmt, O.RTNE, True, 0x7777)
    ib, sb = O.quantize_rows(O.bf16_bits_to_f32(WL.bf16_bits(b)), fmt, O.RTNE, True, 0x7777)
    want = O.gemm_nt(ia, sa, ib, sb, fmt)
    got = P.to_numpy(U.gemm_fwd_y(qa, qb, out_dtype=torch.float32))
    assert P.rel_fro(got, want) <= 1e-5


def test_mx_gemm_long_reduction():
    m, n, k = 130, 260, 65536
    a, b = _tensor((m, k), 8), _tensor((n, k), 9, 0.02)
    print(f"mx gemm long K {m}x{n}x{k}", flush=True)
    qa, qb = U.mx_quantize(a.cuda(), rht=True, sign_mask=0x5A5A), U.mx_quantize(b.cuda(), rht=True, sign_mask=0x5A5A)
    ia, ea = O.quantize_rows_mx(O.bf16_bits_to_f32(WL.bf16_bits(a)), O.RTNE, True, 0x5A5A)
    ib, eb = O.quantize_rows_mx(O.bf16_bits_to_f32(WL.bf16_bits(b)), O.RTNE, True, 0x5A5A)
    want = O.gemm_nt_mx(ia, ea, ib, eb)
    got = P.to_numpy(U.mx_gemm_fwd_y(qa, qb, out_dtype=torch.float32))
    assert P.rel_fro(got, want) <= 1e-5
