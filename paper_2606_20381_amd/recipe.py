"""Training recipes and the dense layer step built from the library's quantizers and GEMMs.

A recipe fixes, for one linear layer's training step (Sec. 2.2: fwd_y, bwd_dx, bwd_dw, each an NT GEMM on
operands quantized along its reduction axis):
  * the 4-bit grid (uniform -7..7 or E2M1, optionally cut at max_fpx, Sec. 5 Q4),
  * which GEMMs rotate their operands with the RHT (Table 1; the RHT-scope ablation of Table 2),
  * which operands are rounded stochastically (Table 1: dY only; the SR ablation of Table 2 and the SR-scope
    dimension of the E2M1 search space in the Appendix),
  * the RHT block (16 in both recipes; 32 / 64 / 128 in the Appendix search space).

The six operands and their SR streams (Philox counter word 3): X and W along K for fwd_y; dY along N (stream 0)
and W^T along N for bwd_dx; dY^T along M (stream 1) and X^T along M for bwd_dw. Operands that are not in the
recipe's usual SR set take streams 2 (X), 3 (W), 4 (W^T) and 5 (X^T) when a recipe rounds them stochastically.
Every step runs in the library's kernels; this module only chooses the calls and owns the buffers.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import torch

from . import ufp4 as U

OPERANDS = ("x", "w", "dy", "wt", "dyt", "xt")
# operand -> (source tensor, transposed, GEMM whose RHT flag applies, SR stream)
LAYOUT = {
    "x": ("x", False, 0, 2), "w": ("w", False, 0, 3),
    "dy": ("dy", False, 1, 0), "wt": ("w", True, 1, 4),
    "dyt": ("dy", True, 2, 1), "xt": ("x", True, 2, 5),
}


@dataclass(frozen=True)
class Recipe:
    name: str
    fmt: int
    rht: tuple  # (fwd_y, bwd_dx, bwd_dw)
    sr: frozenset = field(default_factory=lambda: frozenset({"dy", "dyt"}))
    max_fpx: float = 0.0  # E2M1 only: 2, 4 or 6 (0 = the full grid)
    rht_block: int = 16
    note: str = ""

    def rounding(self, op: str) -> int:
        return U.SR if op in self.sr else U.RTNE

    def rotated(self, op: str) -> bool:
        return bool(self.rht[LAYOUT[op][2]])


_T, _F = True, False
RECIPES = {
    "ufp4": Recipe("ufp4", U.UNIFORM, (_T, _T, _T), note="the method: uniform -7..7, RHT16 on all GEMMs, SR on dY"),
    "e2m1": Recipe("e2m1", U.E2M1, (_F, _F, _T), note="baseline of Table 1: E2M1, RHT16 on bwd_dw, SR on dY"),
    # Table 2: RHT scope and SR under the uniform grid
    "ufp4-rht-none": Recipe("ufp4-rht-none", U.UNIFORM, (_F, _F, _F), note="Table 2: no RHT"),
    "ufp4-rht-dw": Recipe("ufp4-rht-dw", U.UNIFORM, (_F, _F, _T), note="Table 2: RHT on bwd_dw"),
    "ufp4-rht-dx-dw": Recipe("ufp4-rht-dx-dw", U.UNIFORM, (_F, _T, _T), note="Table 2: RHT on bwd_dx, bwd_dw"),
    "ufp4-rht-y-dw": Recipe("ufp4-rht-y-dw", U.UNIFORM, (_T, _F, _T), note="Table 2: RHT on fwd_y, bwd_dw"),
    "ufp4-no-sr": Recipe("ufp4-no-sr", U.UNIFORM, (_T, _T, _T), frozenset(), note="Table 2: full RHT without SR"),
    # E2M1 variants: full RHT and the range-restricted grids of Sec. 5 Q4; SR beyond dY (Appendix)
    "e2m1-full-rht": Recipe("e2m1-full-rht", U.E2M1, (_T, _T, _T), note="E2M1 with RHT on all GEMMs"),
    "e2m1-max4": Recipe("e2m1-max4", U.E2M1, (_T, _T, _T), max_fpx=4.0, note="Sec. 5 Q4: full RHT, max_fpx = 4"),
    "e2m1-max2": Recipe("e2m1-max2", U.E2M1, (_T, _T, _T), max_fpx=2.0, note="Sec. 5 Q4: full RHT, max_fpx = 2"),
    "e2m1-sr-bwd": Recipe("e2m1-sr-bwd", U.E2M1, (_F, _F, _T), frozenset({"dy", "dyt", "xt", "wt"}),
                          note="Appendix SR scope: dY plus X_WGRAD and W_DGRAD"),
    # RHT block (Appendix search space)
    "ufp4-rht32": Recipe("ufp4-rht32", U.UNIFORM, (_T, _T, _T), rht_block=32, note="RHT over 32-blocks"),
    "ufp4-rht64": Recipe("ufp4-rht64", U.UNIFORM, (_T, _T, _T), rht_block=64, note="RHT over 64-blocks"),
    "ufp4-rht128": Recipe("ufp4-rht128", U.UNIFORM, (_T, _T, _T), rht_block=128, note="RHT over 128-blocks"),
}


def wide_mask(sign_mask: int, rht_block: int) -> int:
    """The n-bit sign mask of a wider RHT built from a 16-bit one: the same 16 signs in every sub-block."""
    return sum((sign_mask & 0xFFFF) << (16 * k) for k in range(rht_block // 16))


def quantize_operand(t: torch.Tensor, op: str, r: Recipe, sign_mask: int, seed: int, out: U.QTensor | None = None):
    """Quantize one of the six operands of a dense layer from its source tensor t under recipe r."""
    _, tr, _, stream = LAYOUT[op]
    rot, rnd = r.rotated(op), r.rounding(op)
    if rot and r.rht_block != 16:
        return U.quantize_rht_block(t, r.fmt, rht_block=r.rht_block, sign_mask=wide_mask(sign_mask, r.rht_block),
                                    transpose=tr, rounding=rnd, seed=seed, stream_id=stream, out=out)
    if r.fmt == U.E2M1 and r.max_fpx not in (0.0, 6.0):
        return U.e2m1_quantize_range(t, r.max_fpx, transpose=tr, rht=rot, sign_mask=sign_mask, rounding=rnd,
                                     seed=seed, stream_id=stream, out=out)
    fn = U.rht_quantize if r.fmt == U.UNIFORM else U.e2m1_quantize
    return fn(t, transpose=tr, rht=rot, sign_mask=sign_mask, rounding=rnd, seed=seed, stream_id=stream, out=out)


def dual_ok(r: Recipe, a: str, b: str) -> bool:
    """Whether the rowwise operand a and transposed operand b of one tensor can come from one dual pass."""
    return r.rht_block == 16 and r.max_fpx in (0.0, 6.0) and r.rounding(a) == r.rounding(b)


class LayerStep:
    """Preallocated operands and outputs of one dense layer (X [M, K], W [N, K], dY [M, N]) under a recipe.

    run() quantizes the six operands (X and W through the two-operand quantizer where the recipe allows it)
    and runs fwd_y (Y bf16), bwd_dx (dX bf16) and bwd_dw (dW fp32)."""

    def __init__(self, M: int, N: int, K: int, recipe: Recipe | str = "ufp4", dual: bool = True, device="cuda"):
        self.r = RECIPES[recipe] if isinstance(recipe, str) else recipe
        self.M, self.N, self.K, self.dual = M, N, K, dual
        shapes = {"x": (M, K), "w": (N, K), "dy": (M, N), "wt": (K, N), "dyt": (N, M), "xt": (K, M)}
        self.q = {op: U.empty_qtensor(*shapes[op], self.r.fmt, device) for op in OPERANDS}
        self.y = torch.empty(M, N, dtype=torch.bfloat16, device=device)
        self.dx = torch.empty(M, K, dtype=torch.bfloat16, device=device)
        self.dw = torch.empty(N, K, dtype=torch.float32, device=device)

    def quantize(self, x, w, dy, sign_mask: int = 0, seed: int = 0):
        r, q, src = self.r, self.q, {"x": x, "w": w, "dy": dy}
        done = set()
        if self.dual:
            for a, b in (("x", "xt"), ("w", "wt")):
                if dual_ok(r, a, b):
                    U.quantize_dual(src[a], fmt=r.fmt, rht_rows=r.rotated(a), rht_cols=r.rotated(b),
                                    sign_mask_rows=sign_mask, sign_mask_cols=sign_mask, rounding=r.rounding(a),
                                    seed=seed, stream_rows=LAYOUT[a][3], stream_cols=LAYOUT[b][3],
                                    out_rows=q[a], out_cols=q[b])
                    done |= {a, b}
        for op in OPERANDS:
            if op not in done:
                quantize_operand(src[LAYOUT[op][0]], op, r, sign_mask, seed, out=q[op])
        return q

    def gemms(self):
        q = self.q
        U.gemm_fwd_y(q["x"], q["w"], out=self.y)
        U.gemm_bwd_dx(q["dy"], q["wt"], out=self.dx)
        U.gemm_bwd_dw(q["dyt"], q["xt"], out=self.dw)
        return self.y, self.dx, self.dw

    def run(self, x, w, dy, sign_mask: int = 0, seed: int = 0):
        self.quantize(x, w, dy, sign_mask, seed)
        return self.gemms()
