"""GPU parity of the inter-model junction (eq. (1)) against the float64 oracle.

Tolerances follow from the arithmetic: row norms and the dot product g.o are
fp32 sums of at most 8192 terms (relative error far below 2^-9), so a bf16
output is within half a bf16 ulp of the float64 value plus that error
(elementwise 2^-8 relative, with an absolute floor of 1e-4 of the row's
largest value where the backward's projection cancels), and an fp32 output
is within 1e-5 relative (Frobenius, per tensor). The fresh-embedding block
of the forward is a copy and must be bit-exact.

Small cases cover every threads-per-row / chunks-per-lane shape, partial
chunks, ragged T, both channel orders, every dtype pair, accumulation and
zero-norm rows; the full-size junctions (T = 32,768, widths 1,536 / 3,072 /
4,608, and the paper's 3B-suite widths) are checked on
sampled rows (rows are independent).
"""

import numpy as np
import pytest
import torch

from oracle import junction as OJ
from paper_2608_09703_amd import api as D
from paper_2608_09703_amd import workloads as WL

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
BF16_RTOL = 2.0 ** -8
ROW_FLOOR = 1e-4
F32_RTOL = 1e-5


def _np(x):
    return x.detach().float().cpu().numpy().astype(np.float64)


def _inputs(T, dp, df, act, grad, seed, o_std=8.0, e_std=0.02):
    wl = WL.JunctionWorkload("t", T, (dp, dp + df), act_dtype=act, grad_dtype=grad, o_std=o_std,
                             e_std=e_std, g_std=1.0, seed=seed)
    return WL.make_junction_inputs(wl, 0, device=DEV)


def _close(got, ref, dtype, what):
    if dtype == torch.bfloat16:
        floor = ROW_FLOOR * np.abs(ref).max(axis=1, keepdims=True)
        bad = np.abs(got - ref) > BF16_RTOL * np.abs(ref) + floor
        assert not bad.any(), f"{what}: {bad.sum()} elements off, first at {np.argwhere(bad)[0]}"
    else:
        nrm = np.linalg.norm(ref)
        err = np.linalg.norm(got - ref) / (nrm if nrm > 0 else 1.0)
        assert err <= F32_RTOL, f"{what}: relative error {err:.2e}"
        floor = ROW_FLOOR * np.abs(ref).max(axis=1, keepdims=True)
        assert np.all(np.abs(got - ref) <= 1e-4 * np.abs(ref) + floor), what


def _check(o, e, gx, layout, what, accumulate=False):
    prev_first = layout == "prev_first"
    x = D.junction_forward(o, e, layout=layout)
    g_o0 = torch.randn(o.shape, dtype=gx.dtype, device=DEV) if accumulate else None
    g_e0 = torch.randn(e.shape, dtype=gx.dtype, device=DEV) if accumulate else None
    g_o, g_e = D.junction_backward(o, e, gx, layout=layout, accumulate=accumulate,
                                   g_o=None if g_o0 is None else g_o0.clone(),
                                   g_e=None if g_e0 is None else g_e0.clone())
    torch.cuda.synchronize()
    on, en, gn = _np(o), _np(e), _np(gx)
    xr = OJ.forward(on, en, prev_first)
    dp = o.shape[1]
    xg = _np(x)
    fresh = xg[:, dp:] if prev_first else xg[:, :e.shape[1]]
    assert np.array_equal(fresh, en), f"{what}: fresh block is not an exact copy"
    _close(xg, xr, o.dtype, f"{what} x")
    gor, ger = OJ.backward(on, en, gn, prev_first)
    if accumulate:
        gor = gor + _np(g_o0)
        ger = ger + _np(g_e0)
    _close(_np(g_o), gor, gx.dtype, f"{what} g_o")
    _close(_np(g_e), ger, gx.dtype, f"{what} g_e")


SMALL = [
    # T, d_prev, d_fresh, act, grad, layout
    # (threads per row x chunks per lane)
    (37, 8, 8, "bf16", "f32", "prev_first"),            # 64 x 1, lane 0 only
    (300, 512, 256, "bf16", "bf16", "prev_first"),      # 64 x 1
    (301, 1024, 520, "bf16", "f32", "fresh_first"),     # 64 x 2, partial chunk
    (129, 2048, 1024, "f32", "f32", "prev_first"),      # 128 x 2
    (130, 3072, 1536, "bf16", "f32", "prev_first"),     # 256 x 2 (c5 junction 2)
    (66, 4352, 2048, "f32", "bf16", "fresh_first"),     # 256 x 4
    (67, 1544, 1032, "bf16", "bf16", "prev_first"),     # 128 x 2, ragged chunk coverage
    (5, 8192, 8, "bf16", "bf16", "prev_first"),         # widest row, tiny fresh block
    (1, 64, 8192, "f32", "f32", "fresh_first"),         # T = 1, widest fresh block
]


@pytest.mark.parametrize("case", SMALL, ids=[f"t{c[0]}_p{c[1]}_f{c[2]}_{c[3]}_{c[4]}_{c[5]}"
                                              for c in SMALL])
def test_small_parity(case):
    T, dp, df, act, grad, layout = case
    print(f"[junction] T={T} d_prev={dp} d_fresh={df} {act}/{grad} {layout}", flush=True)
    o, e, gx = _inputs(T, dp, df, act, grad, seed=T + dp)
    _check(o, e, gx, layout, f"T={T} {dp}+{df}")


@pytest.mark.parametrize("grad", ["bf16", "f32"])
def test_accumulate(grad):
    print(f"[junction] accumulate {grad}", flush=True)
    o, e, gx = _inputs(77, 1024, 512, "bf16", grad, seed=5)
    _check(o, e, gx, "prev_first", "accumulate", accumulate=True)


def test_zero_norm_rows():
    print("[junction] zero-norm rows", flush=True)
    o, e, gx = _inputs(40, 256, 128, "bf16", "f32", seed=6)
    o[3] = 0
    e[7] = 0
    o[9] = 0
    e[9] = 0
    _check(o, e, gx, "prev_first", "zero rows")
    x = D.junction_forward(o, e)
    g_o, g_e = D.junction_backward(o, e, gx)
    for r in (3, 7, 9):
        assert torch.all(x[r, :256] == 0) and torch.all(g_o[r] == 0)
        assert torch.equal(g_e[r], gx[r, 256:])


def test_bitwise_deterministic():
    o, e, gx = _inputs(999, 3072, 1536, "bf16", "f32", seed=7)
    print("[junction] determinism", flush=True)
    a = [D.junction_forward(o, e), *D.junction_backward(o, e, gx)]
    b = [D.junction_forward(o, e), *D.junction_backward(o, e, gx)]
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def test_autograd_front_end():
    print("[junction] autograd", flush=True)
    o, e, gx = _inputs(64, 1024, 1024, "f32", "f32", seed=8)
    o.requires_grad_(True)
    e.requires_grad_(True)
    x = D.junction(o, e)
    (x * gx).sum().backward()
    gor, ger = OJ.backward(_np(o), _np(e), _np(gx))
    _close(_np(o.grad), gor, torch.float32, "autograd g_o")
    _close(_np(e.grad), ger, torch.float32, "autograd g_e")


@pytest.mark.parametrize("name", ["c5_junctions", "paper3b_junctions"])
def test_full_size_sampled_rows(name):
    wl = WL.JUNCTIONS[name]
    for m, (dp, df) in enumerate(wl.junctions):
        print(f"[junction] full-size {name} junction {m}: T={wl.T} {dp}+{df}", flush=True)
        o, e, gx = WL.make_junction_inputs(wl, m, device=DEV)
        x = D.junction_forward(o, e)
        g_o, g_e = D.junction_backward(o, e, gx)
        torch.cuda.synchronize()
        rows = np.unique(np.concatenate([np.random.default_rng(m).choice(wl.T, 64, replace=False),
                                         [0, wl.T - 1]]))
        ri = torch.from_numpy(rows).to(DEV)
        on, en, gn = _np(o[ri]), _np(e[ri]), _np(gx[ri])
        _close(_np(x[ri]), OJ.forward(on, en), o.dtype, f"{name}/{m} x")
        gor, ger = OJ.backward(on, en, gn)
        _close(_np(g_o[ri]), gor, gx.dtype, f"{name}/{m} g_o")
        _close(_np(g_e[ri]), ger, gx.dtype, f"{name}/{m} g_e")
        # invariants over every row: the rescaled block has ||e|| and o's direction
        xo = x[:, :dp].float()
        ne = e.float().norm(dim=1)
        rel = ((xo.norm(dim=1) - ne).abs() / ne).max().item()
        assert rel <= 2 ** -7, rel
        # (g_o . o) = 0 up to rounding of the fp32 outputs
        dot = (g_o.double() * o.double()).sum(1).abs()
        scale = (g_o.double().abs() * o.double().abs()).sum(1)
        assert (dot <= 1e-4 * scale + 1e-30).all()
