"""GPU parity: the HIP path (through the C ABI) against the float64 CPU oracle.

Small cases run the whole oracle; they span several 128 x 128 tiles, ragged
token and vocabulary tails, several backward vocabulary chunks, temperature,
ignored labels, any teacher index, M = 1..4, V = 2 and T = 1. The benchmark
workloads at full size are checked on sampled rows the oracle computes one by
one, on a reduced-T instance for the head gradients, and through invariants
that hold at any size.
"""

import numpy as np
import pytest
import torch

import oracle
from paper_2608_09703_amd import workloads as WL
from tests.gpu_helpers import (assert_grad, assert_grad_rows, assert_losses, assert_rows,
                               non_label_rows, rel_fro, run_gpu, to_np)

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _inputs(wl):
    h, W, y = WL.make_inputs(wl, device=DEV)
    return h, W, y, to_np(h), to_np(W), y.cpu().numpy()


def _coeffs(M, teacher, alpha, tau, mode="paper"):
    return oracle.coeffs(M, teacher, alpha=alpha, tau=tau, mode=mode)


SMALL = [
    # name, workload, teacher, alpha, mode, vocab_chunk
    ("m3_ragged_tau1", WL.custom(3, 300, (64, 128, 192), 1000, ignore_frac=0.1, w_std=0.05, seed=1),
     -1, 0.3, "paper", 512),
    ("m3_tau2_teacher0", WL.custom(3, 260, (128, 64, 192), 1300, tau=2.0, w_std=0.08, seed=2),
     0, 0.5, "paper", 256),
    ("m4_peaky_ignore", WL.custom(4, 200, (64, 64, 128, 256), 777, w_std=0.02, w_scale=5.0,
                                  ignore_frac=0.2, seed=3), -1, 1.0, "additive", 0),
    ("m2_tau0p7_mid_teacher", WL.custom(2, 129, (256, 96), 2049, tau=0.7, w_std=0.1, seed=4),
     0, 0.7, "paper", 1024),
    ("m1_ce_only", WL.custom(1, 130, (96,), 300, w_std=0.1, seed=5), -1, 0.0, "paper", 0),
    ("v2_binary", WL.custom(2, 64, (8, 16), 2, w_std=0.5, seed=6), -1, 0.5, "paper", 0),
    ("t1_single_token", WL.custom(2, 1, (64, 64), 300, w_std=0.1, seed=7), -1, 0.5, "paper", 0),
    ("c1_small_f32", WL.WORKLOADS["c1_small_f32"], -1, 1.0, "paper", 0),
    ("f32_ragged", WL.custom(3, 150, (32, 36, 100), 555, dtype="f32", tau=1.5, w_std=0.1,
                             ignore_frac=0.1, seed=8), -1, 0.4, "paper", 256),
    ("m8_max_models", WL.custom(8, 200, (64, 64, 128, 128, 192, 256, 256, 320), 700, tau=1.5,
                                w_std=0.05, ignore_frac=0.1, seed=9), 5, 0.6, "paper", 256),
]


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_small_full_parity(case):
    name, wl, teacher, alpha, mode, chunk = case
    print(f"[parity] {name} M={wl.M} T={wl.T} V={wl.V} dims={wl.dims} {wl.dtype}", flush=True)
    h, W, y, hn, Wn, yn = _inputs(wl)
    g_ce, g_kl = _coeffs(wl.M, teacher, alpha, wl.tau, mode)
    gpu = run_gpu(h, W, y, tau=wl.tau, teacher=teacher, g_ce=g_ce, g_kl=g_kl, vocab_chunk=chunk)
    ref = oracle.forward(hn, Wn, yn, tau=wl.tau, teacher=teacher)
    assert gpu["n_valid"] == ref["n_valid"]
    assert gpu["flags"] == 0
    assert_losses(gpu, ref, name)
    assert_rows(gpu, ref, what=name)
    gh, gW = oracle.backward(hn, Wn, yn, g_ce, g_kl, tau=wl.tau, teacher=teacher)
    check_head_grads(gpu, gh, gW, yn, wl.V, name)


def check_head_grads(gpu, gh, gW, yn, V, name):
    """Every row of grad_h and grad_W, the softmax-only rows of grad_W (no valid
    token's label) on their own, the vocabulary tail, and exact zeros on ignored rows."""
    soft = non_label_rows(V, yn)
    for i in range(len(gh)):
        e1 = assert_grad_rows(gpu["grad_h"][i], gh[i], f"{name} grad_h[{i}]")
        e2 = assert_grad_rows(gpu["grad_W"][i], gW[i], f"{name} grad_W[{i}]", softmax_rows=soft)
        # vocabulary tail (rows past the last multiple of 256)
        tail = (V // 256) * 256
        if tail < V:
            assert_grad(gpu["grad_W"][i][tail:], gW[i][tail:], f"{name} grad_W[{i}] tail")
        print(f"  sub-model {i}: grad_h err {e1['tensor']:.2e} (worst row {e1['worst_row']:.2e}), "
              f"grad_W err {e2['tensor']:.2e} (worst row {e2['worst_row']:.2e}, softmax-only rows "
              f"{e2.get('softmax_rows', 0.0):.2e})", flush=True)
        ignored = yn == oracle.IGNORE_INDEX
        assert np.all(gpu["grad_h"][i][ignored] == 0)


def test_all_labels_ignored():
    wl = WL.custom(2, 100, (64, 128), 500, w_std=0.1, seed=11, ignore_frac=1.0)
    h, W, y, hn, Wn, yn = _inputs(wl)
    assert (yn == -100).all()
    gpu = run_gpu(h, W, y, g_ce=[1.0, 1.0], g_kl=[1.0, 0.0])
    assert gpu["n_valid"] == 0
    assert np.all(gpu["ce"] == 0) and np.all(gpu["kl"] == 0) and gpu["H"] == 0
    for g in gpu["grad_h"] + gpu["grad_W"]:
        assert np.all(g == 0)


def test_identical_student_has_zero_kl():
    """A student equal to the teacher has KL = 0 and no KL gradient. The recompute
    backward holds the teacher's q as fp16 in registers (half an ulp: 2^-12 q, or
    2^-25 below the normal range), so its logit gradient there is at most that over
    tau N per entry; the gradient is bounded by it, entry by entry, through |W|. It
    is also far below a genuine student's gradient."""
    wl = WL.custom(3, 256, (128, 64, 128), 3000, tau=1.7, w_std=0.1, seed=12)
    h, W, y = WL.make_inputs(wl, device=DEV)
    h[0] = h[2].clone()
    W[0] = W[2].clone()
    gpu = run_gpu(h, W, y, tau=wl.tau, g_ce=[0.0, 0.0, 0.0], g_kl=[1.0, 1.0, 0.0])
    assert abs(gpu["kl"][0]) < 1e-5
    assert gpu["kl"][1] > 1e-2
    assert np.abs(gpu["kl_row"][0]).max() < 1e-5
    hn, Wn, yn = to_np(h), to_np(W), y.cpu().numpy()
    q = np.exp(oracle.teacher_logq(hn, Wn, tau=wl.tau))
    N = oracle.n_valid(yn)
    bound = ((2.0 ** -12 * q + 2.0 ** -25) @ np.abs(Wn[0].astype(np.float64))) / (wl.tau * N)
    g0 = np.abs(gpu["grad_h"][0].astype(np.float64))
    assert np.all(g0 <= 1.01 * bound + 1e-12), float((g0 - bound).max())
    assert g0.max() <= 1e-2 * np.abs(gpu["grad_h"][1]).max()


def test_uniform_logits_give_ln_v():
    wl = WL.custom(2, 128, (64, 128), 5000, w_std=0.1, seed=13)
    h, W, y = WL.make_inputs(wl, device=DEV)
    W = [torch.zeros_like(x) for x in W]
    gpu = run_gpu(h, W, y, grads=False)
    np.testing.assert_allclose(gpu["ce"], np.log(5000.0), rtol=1e-6)
    assert np.abs(gpu["kl"]).max() < 1e-6


def test_out_of_range_label_is_flagged_and_ignored():
    wl = WL.custom(2, 128, (64, 64), 700, w_std=0.1, seed=14)
    h, W, y = WL.make_inputs(wl, device=DEV)
    y[5] = 700
    y[9] = -7
    gpu = run_gpu(h, W, y, g_ce=[1.0, 1.0], g_kl=[0.5, 0.0])
    assert gpu["flags"] == 1
    assert gpu["n_valid"] == 126
    assert np.all(gpu["grad_h"][0][[5, 9]] == 0)


def test_deterministic_bitwise():
    wl = WL.custom(3, 384, (128, 256, 384), 4000, tau=1.3, ignore_frac=0.05, seed=15)
    h, W, y = WL.make_inputs(wl, device=DEV)
    g_ce, g_kl = _coeffs(3, -1, 0.3, wl.tau)
    a = run_gpu(h, W, y, tau=wl.tau, g_ce=g_ce, g_kl=g_kl, vocab_chunk=1024)
    b = run_gpu(h, W, y, tau=wl.tau, g_ce=g_ce, g_kl=g_kl, vocab_chunk=1024)
    for k in ("ce", "kl", "lse1", "lset", "kl_row"):
        assert np.array_equal(a[k], b[k]), k
    for i in range(3):
        assert np.array_equal(a["grad_h"][i], b["grad_h"][i])
        assert np.array_equal(a["grad_W"][i], b["grad_W"][i])


def test_default_coefficients_follow_alpha():
    """With no coefficient vectors the library uses eq. (3) with the problem's alpha and tau."""
    wl = WL.custom(3, 200, (64, 128, 128), 900, tau=2.0, w_std=0.1, seed=16)
    h, W, y, hn, Wn, yn = _inputs(wl)
    gpu = run_gpu(h, W, y, tau=2.0, alpha=0.25)
    g_ce, g_kl = oracle.coeffs(3, -1, alpha=0.25, tau=2.0)
    gh, gW = oracle.backward(hn, Wn, yn, g_ce, g_kl, tau=2.0)
    check_head_grads(gpu, gh, gW, yn, wl.V, "default coefficients")


def test_autograd_front_end():
    from paper_2608_09703_amd.api import distill
    wl = WL.custom(3, 256, (64, 128, 192), 1500, tau=1.5, w_std=0.1, ignore_frac=0.1, seed=17)
    h, W, y, hn, Wn, yn = _inputs(wl)
    hs = [x.clone().requires_grad_(True) for x in h]
    Ws = [x.clone().requires_grad_(True) for x in W]
    ce, kl, H = distill(hs, Ws, y, tau=1.5)
    w = torch.tensor([0.5, 1.0, 2.0], device=DEV)
    alpha = 0.3
    loss = (w * ((1 - alpha) * ce + alpha * 1.5 ** 2 * kl)).sum()
    loss = loss + 0.5 * ce[2]  # extra teacher weight: any linear objective works
    loss.backward()
    g_ce = np.array([0.5 * 0.7, 1.0 * 0.7, 2.0 * 0.7 + 0.5])
    g_kl = np.array([0.5 * 0.3 * 2.25, 1.0 * 0.3 * 2.25, 2.0 * 0.3 * 2.25])
    ref = oracle.forward(hn, Wn, yn, tau=1.5)
    np.testing.assert_allclose(ce.detach().cpu().numpy(), ref["ce"], rtol=1e-3)
    np.testing.assert_allclose(kl.detach().cpu().numpy()[:2], ref["kl"][:2], rtol=1e-3)
    gh, gW = oracle.backward(hn, Wn, yn, g_ce, g_kl, tau=1.5)
    soft = non_label_rows(wl.V, yn)
    for i in range(3):
        assert_grad_rows(hs[i].grad.float().cpu().numpy(), gh[i], f"grad_h[{i}]")
        assert_grad_rows(Ws[i].grad.float().cpu().numpy(), gW[i], f"grad_W[{i}]", softmax_rows=soft)


# ---------------------------------------------------------------------------
# benchmark workloads at full size
# ---------------------------------------------------------------------------

FULL = ["c2_m3_v50k", "c3_m3_v128k_tau2", "c4_m4_v128k_peaky", "c5_m3_v262k_long", "paper3b_heads"]


@pytest.mark.parametrize("name", FULL)
def test_full_size_sampled_rows(name):
    wl = WL.WORKLOADS[name]
    print(f"[parity-full] {name} M={wl.M} T={wl.T} V={wl.V} dims={wl.dims}", flush=True)
    h, W, y = WL.make_inputs(wl, device=DEV)
    g_ce, g_kl = _coeffs(wl.M, -1, wl.alpha, wl.tau)
    gpu = run_gpu(h, W, y, tau=wl.tau, g_ce=g_ce, g_kl=g_kl)
    hn, Wn, yn = to_np(h), to_np(W), y.cpu().numpy()
    del h, W
    rng = np.random.default_rng(wl.seed + 7)
    rows = np.sort(rng.choice(wl.T, size=96, replace=False))
    ref = oracle.per_row(hn, Wn, yn, rows, tau=wl.tau)
    assert_rows(gpu, ref, rows=rows, what=name)
    N = int((yn != -100).sum())
    assert gpu["n_valid"] == N
    # the means are the means of the per-row values
    for i in range(wl.M):
        np.testing.assert_allclose(gpu["ce"][i], gpu["ce_row"][i].astype(np.float64).sum() / N,
                                   rtol=1e-5)
    ghr = oracle.grad_h_rows(hn, Wn, yn, rows[:32], g_ce, g_kl, tau=wl.tau)
    for i in range(wl.M):
        assert_grad_rows(gpu["grad_h"][i][rows[:32]], ghr[i], f"{name} grad_h[{i}] rows")
    if name == "c2_m3_v50k":
        # sampled vocabulary rows of grad_W (every token's softmax in fp64: the
        # forward's cost, about a minute on the host here): some are labels,
        # most are not
        valid_labels = np.unique(yn[yn != -100])
        vrows = np.unique(np.concatenate([rng.choice(wl.V, size=20, replace=False),
                                          rng.choice(valid_labels, size=4, replace=False)]))
        gwr = oracle.grad_W_rows(hn, Wn, yn, vrows, g_ce, g_kl, tau=wl.tau)
        soft = non_label_rows(wl.V, yn)[vrows]
        for i in range(wl.M):
            assert_grad_rows(gpu["grad_W"][i][vrows], gwr[i], f"{name} grad_W[{i}] rows",
                             softmax_rows=soft)
        # every row of the logit gradient sums to zero: sum_v grad_W = 0
        colsum = gpu["grad_W"][i].astype(np.float64).sum(axis=0)
        scale = np.abs(gpu["grad_W"][i]).astype(np.float64).sum(axis=0).max()
        assert np.abs(colsum).max() <= 1e-3 * scale
        ign = yn == -100
        if ign.any():
            assert np.all(gpu["grad_h"][i][ign] == 0)


REDUCED_T = [("c2_m3_v50k", 512), ("c3_m3_v128k_tau2", 512), ("c4_m4_v128k_peaky", 256),
             ("c5_m3_v262k_long", 256), ("paper3b_heads", 512)]


@pytest.mark.parametrize("name,T", REDUCED_T, ids=[n for n, _ in REDUCED_T])
def test_reduced_T_full_head_gradient(name, T):
    """The workload's own V, widths, head scale, ignore fraction, alpha and tau with
    fewer tokens: every row of grad_h and grad_W checked against the oracle."""
    wl = WL.WORKLOADS[name].replace(T=T)
    print(f"[parity-reducedT] {name} T={wl.T} V={wl.V} dims={wl.dims}", flush=True)
    h, W, y = WL.make_inputs(wl, device=DEV)
    hn = [x.double().cpu().numpy() for x in h]
    Wn = [x.double().cpu().numpy() for x in W]
    yn = y.cpu().numpy()
    g_ce, g_kl = _coeffs(wl.M, -1, wl.alpha, wl.tau)
    gpu = run_gpu(h, W, y, tau=wl.tau, g_ce=g_ce, g_kl=g_kl)
    del h, W
    ref = oracle.forward(hn, Wn, yn, tau=wl.tau)
    assert_losses(gpu, ref, name)
    assert_rows(gpu, ref, what=name)
    gh, gW = oracle.backward(hn, Wn, yn, g_ce, g_kl, tau=wl.tau)
    check_head_grads(gpu, gh, gW, yn, wl.V, name)


@pytest.mark.parametrize("name", ["c3_m3_v128k_tau2"])
def test_full_size_backward_is_bitwise_repeatable(name):
    """Three backward passes at full size (two vocabulary chunks of up to 87k rows)
    give bitwise identical gradients, and every row of the logit gradient sums to
    zero in each (grad_W column sums vanish)."""
    wl = WL.WORKLOADS[name]
    print(f"[repeat] {name}", flush=True)
    h, W, y = WL.make_inputs(wl, device=DEV)
    g_ce, g_kl = _coeffs(wl.M, -1, wl.alpha, wl.tau)
    first = None
    for rep in range(3):
        gpu = run_gpu(h, W, y, tau=wl.tau, g_ce=g_ce, g_kl=g_kl)
        for i in range(wl.M):
            colsum = gpu["grad_W"][i].astype(np.float64).sum(axis=0)
            scale = np.abs(gpu["grad_W"][i]).astype(np.float64).sum(axis=0).max()
            assert np.abs(colsum).max() <= 1e-3 * scale, (rep, i)
        if first is None:
            first = gpu
            continue
        for i in range(wl.M):
            assert np.array_equal(gpu["grad_W"][i], first["grad_W"][i]), (rep, i)
            assert np.array_equal(gpu["grad_h"][i], first["grad_h"][i]), (rep, i)


@pytest.mark.parametrize("dtype,chunk", [("bf16", 512), ("f32", 256)])
def test_accumulate_flags_and_skipped_gradients(dtype, chunk):
    """MLS_ACCUMULATE_GRAD_W / _H add to the caller's gradients instead of
    overwriting them (over several vocabulary chunks), on the wide bf16 and
    the general fp32 paths; NULL gradient pointers skip those outputs and the
    others are still right."""
    from paper_2608_09703_amd import api as D
    from paper_2608_09703_amd import binding as B
    wl = WL.custom(3, 200, (64, 128, 192) if dtype == "bf16" else (32, 36, 100), 1100, dtype=dtype,
                   tau=1.3, w_std=0.08, ignore_frac=0.1, seed=31)
    print(f"[parity] accumulate flags {dtype} chunk {chunk}", flush=True)
    h, W, y = WL.make_inputs(wl, device=DEV)
    ref = run_gpu(h, W, y, tau=wl.tau, vocab_chunk=chunk, alpha=0.4)  # overwrite mode
    flags = B.MLS_ACCUMULATE_GRAD_W | B.MLS_ACCUMULATE_GRAD_H
    p = D.make_problem(h, W, y, tau=wl.tau, vocab_chunk=chunk, alpha=0.4, flags=flags)
    buf = D.Buffers(p, DEV)
    D.forward(p, buf, DEV)
    g = torch.Generator(device=DEV).manual_seed(5)
    # starting values of the gradients' own scale, so that the added part is checked tightly
    gh0 = [torch.randn(x.shape, generator=g, device=DEV) * float(np.std(r))
           for x, r in zip(h, ref["grad_h"])]
    gW0 = [torch.randn(x.shape, generator=g, device=DEV) * float(np.std(r))
           for x, r in zip(W, ref["grad_W"])]
    gh = [x.clone() for x in gh0]
    gW = [x.clone() for x in gW0]
    gh[1] = None   # no grad_h for sub-model 1
    gW[2] = None   # no grad_W for sub-model 2
    D.backward(p, buf, DEV, None, None, gh, gW)
    torch.cuda.synchronize()
    for i in range(3):
        if gh[i] is not None:
            added = gh[i].cpu().numpy().astype(np.float64) - gh0[i].cpu().numpy()
            assert rel_fro(added, ref["grad_h"][i]) < 1e-5, f"grad_h {i}"
        if gW[i] is not None:
            added = gW[i].cpu().numpy().astype(np.float64) - gW0[i].cpu().numpy()
            assert rel_fro(added, ref["grad_W"][i]) < 1e-5, f"grad_W {i}"


@pytest.mark.parametrize("dims,dtype,chunk", [((64, 128, 192), "bf16", 512),
                                              ((64, 128, 192), "bf16", 0),
                                              ((72, 136, 200), "bf16", 256),
                                              ((32, 36, 100), "f32", 256)],
                         ids=["wide_chunks", "wide_default", "general_bf16", "general_f32"])
def test_bf16_grad_h_is_the_rounded_fp32_gradient(dims, dtype, chunk):
    """grad_h_dtype = bf16: the fp32 sums (kept in fp32 across vocabulary chunks) rounded
    once, so the result equals the fp32 output rounded to bf16, bit for bit; with
    MLS_ACCUMULATE_GRAD_H the old bf16 value is added in fp32 before the one rounding."""
    from paper_2608_09703_amd import api as D
    from paper_2608_09703_amd import binding as B
    wl = WL.custom(3, 300, dims, 1500, dtype=dtype, tau=1.4, w_std=0.08, ignore_frac=0.1, seed=41)
    print(f"[parity] bf16 grad_h dims={dims} {dtype} chunk={chunk}", flush=True)
    h, W, y, hn, Wn, yn = _inputs(wl)
    g_ce, g_kl = _coeffs(3, -1, 0.4, wl.tau)
    gce = torch.tensor(g_ce, dtype=torch.float32, device=DEV)
    gkl = torch.tensor(g_kl, dtype=torch.float32, device=DEV)
    outs = {}
    for gdt in (torch.float32, torch.bfloat16):
        p = D.make_problem(h, W, y, tau=wl.tau, vocab_chunk=chunk, grad_h_dtype=gdt)
        buf = D.Buffers(p, DEV)
        D.forward(p, buf, DEV)
        gh = [torch.full(x.shape, float("nan"), dtype=gdt, device=DEV) for x in h]
        gW = [torch.empty(x.shape, dtype=torch.float32, device=DEV) for x in W]
        D.backward(p, buf, DEV, gce, gkl, gh, gW)
        outs[gdt] = (gh, gW)
    torch.cuda.synchronize()
    for i in range(3):
        assert torch.equal(outs[torch.float32][0][i].to(torch.bfloat16), outs[torch.bfloat16][0][i])
        assert torch.equal(outs[torch.float32][1][i], outs[torch.bfloat16][1][i])
    gh_ref, _ = oracle.backward(hn, Wn, yn, g_ce, g_kl, tau=wl.tau)
    for i in range(3):
        assert_grad_rows(outs[torch.bfloat16][0][i].float().cpu().numpy(), gh_ref[i],
                         f"bf16 grad_h[{i}]")
    # accumulate into a bf16 gradient
    p = D.make_problem(h, W, y, tau=wl.tau, vocab_chunk=chunk, grad_h_dtype=torch.bfloat16,
                       flags=B.MLS_ACCUMULATE_GRAD_H)
    buf = D.Buffers(p, DEV)
    D.forward(p, buf, DEV)
    g = torch.Generator(device=DEV).manual_seed(3)
    gh0 = [(torch.randn(x.shape, generator=g, device=DEV) * float(r.float().std())).to(torch.bfloat16)
           for x, r in zip(h, outs[torch.float32][0])]
    gh = [x.clone() for x in gh0]
    D.backward(p, buf, DEV, gce, gkl, gh, [None, None, None])
    torch.cuda.synchronize()
    for i in range(3):
        g32 = outs[torch.float32][0][i].double()
        want = gh0[i].double() + g32
        got = gh[i].double()
        # one rounding of a sum formed in fp32: a bf16 half-ulp of the result plus the
        # fp32 rounding of the terms (which shows where the old value and the gradient cancel)
        tol = 2.0 ** -8 * want.abs() + 2.0 ** -16 * (gh0[i].double().abs() + g32.abs())
        assert torch.all((got - want).abs() <= tol), i


def test_nonfinite_input_flag():
    """A NaN in a valid token's hidden state raises MLS_DEVFLAG_NONFINITE (and not the
    label flag); one in an ignored token's hidden state raises it too (that row still
    enters grad_W = G^T h) while the losses stay finite and equal the oracle's with the
    row zeroed; finite inputs raise nothing."""
    from paper_2608_09703_amd import api as D
    from paper_2608_09703_amd import binding as B
    wl = WL.custom(2, 200, (64, 128), 900, w_std=0.1, ignore_frac=0.2, seed=43)
    h, W, y = WL.make_inputs(wl, device=DEV)
    yn = y.cpu().numpy()
    valid_t = int(np.flatnonzero(yn != -100)[3])
    ign_t = int(np.flatnonzero(yn == -100)[0])

    def flags_of(hh):
        p = D.make_problem(hh, W, y)
        buf = D.Buffers(p, DEV)
        D.forward(p, buf, DEV)
        f = B.device_error(p, buf.stats.data_ptr(), torch.cuda.current_stream(DEV).cuda_stream)
        return f, buf

    f, _ = flags_of(h)
    assert f == 0
    hv = [x.clone() for x in h]
    hv[0][valid_t, 5] = float("nan")
    f, buf = flags_of(hv)
    assert f == B.MLS_DEVFLAG_NONFINITE
    assert not np.isfinite(buf.ce.cpu().numpy()[0])
    hi = [x.clone() for x in h]
    hi[1][ign_t, :] = float("inf")
    f, buf = flags_of(hi)
    assert f == B.MLS_DEVFLAG_NONFINITE
    hz = [x.clone() for x in h]
    hz[1][ign_t, :] = 0
    ref = oracle.forward(to_np(hz), to_np(W), yn)
    np.testing.assert_allclose(buf.ce.cpu().numpy(), ref["ce"], rtol=1e-3, atol=1e-5)
    np.testing.assert_allclose(buf.kl.cpu().numpy(), ref["kl"], rtol=1e-3, atol=1e-5)
    # the ignored row's gradient is an exact zero even though its logits are not finite
    gpu = run_gpu(hi, W, y, g_ce=[1.0, 1.0], g_kl=[0.5, 0.0])
    assert np.all(gpu["grad_h"][1][ign_t] == 0)
    assert np.all(np.isfinite(gpu["grad_h"][0])) and np.all(np.isfinite(gpu["grad_W"][0]))
