"""GPU parity of mls_distill_fwd_bwd, the forward + backward in one call that
stores each token chunk's logits (fp16, relative to a local maximum) instead of
recomputing them, against the float64 CPU oracle.

Small cases span several token chunks and 128 x 128 tiles with ragged token and
vocabulary tails, temperature, ignored labels, any teacher, M = 1..8 and V = 2;
the benchmark workloads are checked in full at reduced T (every row of both
gradients) and on sampled rows at full size."""

import numpy as np
import pytest
import torch

import oracle
from paper_2608_09703_amd import binding as B
from paper_2608_09703_amd import workloads as WL
from tests.gpu_helpers import (assert_grad_rows, assert_losses, assert_rows, non_label_rows,
                               rel_fro, run_fused, run_gpu, to_np)
from tests.test_parity_gpu import check_head_grads

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _inputs(wl):
    h, W, y = WL.make_inputs(wl, device=DEV)
    return h, W, y, to_np(h), to_np(W), y.cpu().numpy()


SMALL = [
    # name, workload, teacher, alpha, mode
    ("m3_ragged_tau1", WL.custom(3, 300, (64, 128, 192), 1000, ignore_frac=0.1, w_std=0.05, seed=1),
     -1, 0.3, "paper"),
    ("m3_tau2_teacher0", WL.custom(3, 520, (128, 64, 192), 1300, tau=2.0, w_std=0.08, seed=2),
     0, 0.5, "paper"),
    ("m4_peaky_ignore", WL.custom(4, 200, (64, 64, 128, 256), 777, w_std=0.02, w_scale=5.0,
                                  ignore_frac=0.2, seed=3), -1, 1.0, "additive"),
    ("m2_tau0p7_mid_teacher", WL.custom(2, 129, (256, 64), 2049, tau=0.7, w_std=0.1, seed=4),
     0, 0.7, "paper"),
    ("m1_ce_only", WL.custom(1, 1000, (128,), 300, w_std=0.1, seed=5), -1, 0.0, "paper"),
    ("v2_binary", WL.custom(2, 640, (64, 64), 2, w_std=0.5, seed=6), -1, 0.5, "paper"),
    ("m8_max_models", WL.custom(8, 260, (64, 64, 128, 128, 192, 256, 256, 320), 700, tau=1.5,
                                w_std=0.05, ignore_frac=0.1, seed=9), 5, 0.6, "paper"),
]


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_fused_small_full_parity(case):
    name, wl, teacher, alpha, mode = case
    print(f"[fused] {name} M={wl.M} T={wl.T} V={wl.V} dims={wl.dims}", flush=True)
    h, W, y, hn, Wn, yn = _inputs(wl)
    g_ce, g_kl = oracle.coeffs(wl.M, teacher, alpha=alpha, tau=wl.tau, mode=mode)
    gpu = run_fused(h, W, y, tau=wl.tau, teacher=teacher, g_ce=g_ce, g_kl=g_kl)
    ref = oracle.forward(hn, Wn, yn, tau=wl.tau, teacher=teacher)
    assert gpu["n_valid"] == ref["n_valid"] and gpu["flags"] == 0
    assert_losses(gpu, ref, name)
    assert_rows(gpu, ref, what=name)
    gh, gW = oracle.backward(hn, Wn, yn, g_ce, g_kl, tau=wl.tau, teacher=teacher)
    check_head_grads(gpu, gh, gW, yn, wl.V, name)


def test_fused_matches_separate_calls_and_bf16_grad_h():
    """Same losses and statistics as mls_distill_fwd (bit for bit: the same forward
    kernels on the same tokens), gradients within the tolerance of each other; a bf16
    grad_h is the fp32 one rounded once."""
    wl = WL.custom(3, 700, (128, 192, 256), 3000, tau=1.3, w_std=0.06, ignore_frac=0.1, seed=21)
    h, W, y, hn, Wn, yn = _inputs(wl)
    g_ce, g_kl = oracle.coeffs(3, -1, alpha=0.4, tau=wl.tau)
    a = run_fused(h, W, y, tau=wl.tau, g_ce=g_ce, g_kl=g_kl)
    b = run_gpu(h, W, y, tau=wl.tau, g_ce=g_ce, g_kl=g_kl)
    for k in ("ce", "kl", "lse1", "lset", "ce_row", "kl_row", "h_row"):
        assert np.array_equal(a[k], b[k]), k
    for i in range(3):
        assert rel_fro(a["grad_h"][i], b["grad_h"][i]) < 1e-2
        assert rel_fro(a["grad_W"][i], b["grad_W"][i]) < 1e-2
    c = run_fused(h, W, y, tau=wl.tau, g_ce=g_ce, g_kl=g_kl, grad_h_dtype=torch.bfloat16)
    for i in range(3):
        want = torch.tensor(a["grad_h"][i]).to(torch.bfloat16).float().numpy()
        assert np.array_equal(c["grad_h"][i], want), i
        assert np.array_equal(c["grad_W"][i], a["grad_W"][i]), i


def test_fused_identical_student_has_exactly_zero_kl_gradient():
    """With stored logits the student's and the teacher's probabilities are formed
    from bitwise equal values, so an identical student's KL gradient is exactly 0."""
    wl = WL.custom(3, 256, (128, 64, 128), 3000, tau=1.7, w_std=0.1, seed=12)
    h, W, y = WL.make_inputs(wl, device=DEV)
    h[0] = h[2].clone()
    W[0] = W[2].clone()
    gpu = run_fused(h, W, y, tau=wl.tau, g_ce=[0.0, 0.0, 0.0], g_kl=[1.0, 1.0, 0.0])
    assert abs(gpu["kl"][0]) < 1e-5 and gpu["kl"][1] > 1e-2
    assert np.all(gpu["grad_h"][0] == 0) and np.all(gpu["grad_W"][0] == 0)
    assert np.abs(gpu["grad_h"][1]).max() > 0


def test_fused_accumulate_flags_and_skipped_gradients():
    wl = WL.custom(3, 400, (64, 128, 192), 1100, tau=1.3, w_std=0.08, ignore_frac=0.1, seed=31)
    h, W, y = WL.make_inputs(wl, device=DEV)
    ref = run_fused(h, W, y, tau=wl.tau, alpha=0.4)
    from paper_2608_09703_amd import api as D
    p = D.make_problem(h, W, y, tau=wl.tau, alpha=0.4,
                       flags=B.MLS_ACCUMULATE_GRAD_W | B.MLS_ACCUMULATE_GRAD_H)
    buf = D.Buffers(p, DEV)
    ws_b = B.query_fwd_bwd_workspace(p)
    ws = torch.empty(ws_b, dtype=torch.uint8, device=DEV)
    g = torch.Generator(device=DEV).manual_seed(5)
    gh0 = [torch.randn(x.shape, generator=g, device=DEV) * float(np.std(r))
           for x, r in zip(h, ref["grad_h"])]
    gW0 = [torch.randn(x.shape, generator=g, device=DEV) * float(np.std(r))
           for x, r in zip(W, ref["grad_W"])]
    gh = [x.clone() for x in gh0]
    gW = [x.clone() for x in gW0]
    gh[1] = None
    gW[2] = None
    B.distill_fwd_bwd(p, buf.stats.data_ptr(), buf.ce.data_ptr(), buf.kl.data_ptr(), None, None,
                      None, [x.data_ptr() if x is not None else None for x in gh],
                      [x.data_ptr() if x is not None else None for x in gW], ws.data_ptr(), ws_b,
                      torch.cuda.current_stream(DEV).cuda_stream)
    torch.cuda.synchronize()
    for i in range(3):
        if gh[i] is not None:
            added = gh[i].cpu().numpy().astype(np.float64) - gh0[i].cpu().numpy()
            assert rel_fro(added, ref["grad_h"][i]) < 1e-5, f"grad_h {i}"
        if gW[i] is not None:
            added = gW[i].cpu().numpy().astype(np.float64) - gW0[i].cpu().numpy()
            assert rel_fro(added, ref["grad_W"][i]) < 1e-5, f"grad_W {i}"


@pytest.mark.parametrize("T,dims,dtype,flags", [(100, (64, 128), "bf16", 0),
                                                 (300, (72, 136), "bf16", 0),
                                                 (300, (32, 36), "f32", 0),
                                                 (300, (64, 128), "bf16", B.MLS_FWD_BWD_RECOMPUTE)],
                         ids=["one_tile", "general_widths", "f32", "recompute_flag"])
def test_fused_entry_point_falls_back_to_recompute(T, dims, dtype, flags):
    """One token tile, widths off the wide path, fp32 inputs or the recompute flag:
    the call runs the forward and the recomputing backward, with the same results
    as the two separate calls."""
    wl = WL.custom(2, T, dims, 900, dtype=dtype, tau=1.2, w_std=0.1, ignore_frac=0.1, seed=33)
    h, W, y, hn, Wn, yn = _inputs(wl)
    g_ce, g_kl = oracle.coeffs(2, -1, alpha=0.5, tau=wl.tau)
    a = run_fused(h, W, y, tau=wl.tau, g_ce=g_ce, g_kl=g_kl, flags=flags)
    b = run_gpu(h, W, y, tau=wl.tau, g_ce=g_ce, g_kl=g_kl)
    for k in ("ce", "kl", "lse1"):
        assert np.array_equal(a[k], b[k]), k
    for i in range(2):
        assert np.array_equal(a["grad_h"][i], b["grad_h"][i])
        assert np.array_equal(a["grad_W"][i], b["grad_W"][i])


REDUCED_T = [("c2_m3_v50k", 512), ("c3_m3_v128k_tau2", 512), ("c4_m4_v128k_peaky", 256),
             ("c5_m3_v262k_long", 256), ("paper3b_heads", 512)]


@pytest.mark.parametrize("name,T", REDUCED_T, ids=[n for n, _ in REDUCED_T])
def test_fused_reduced_T_full_head_gradient(name, T):
    wl = WL.WORKLOADS[name].replace(T=T)
    print(f"[fused-reducedT] {name} T={wl.T} V={wl.V} dims={wl.dims}", flush=True)
    h, W, y = WL.make_inputs(wl, device=DEV)
    hn = [x.double().cpu().numpy() for x in h]
    Wn = [x.double().cpu().numpy() for x in W]
    yn = y.cpu().numpy()
    g_ce, g_kl = oracle.coeffs(wl.M, -1, alpha=wl.alpha, tau=wl.tau)
    gpu = run_fused(h, W, y, tau=wl.tau, g_ce=g_ce, g_kl=g_kl)
    del h, W
    ref = oracle.forward(hn, Wn, yn, tau=wl.tau)
    assert_losses(gpu, ref, name)
    assert_rows(gpu, ref, what=name)
    gh, gW = oracle.backward(hn, Wn, yn, g_ce, g_kl, tau=wl.tau)
    check_head_grads(gpu, gh, gW, yn, wl.V, name)


@pytest.mark.parametrize("name", ["c2_m3_v50k", "c3_m3_v128k_tau2", "c4_m4_v128k_peaky"])
def test_fused_full_size_sampled_rows(name):
    wl = WL.WORKLOADS[name]
    print(f"[fused-full] {name} M={wl.M} T={wl.T} V={wl.V} dims={wl.dims}", flush=True)
    h, W, y = WL.make_inputs(wl, device=DEV)
    g_ce, g_kl = oracle.coeffs(wl.M, -1, alpha=wl.alpha, tau=wl.tau)
    gpu = run_fused(h, W, y, tau=wl.tau, g_ce=g_ce, g_kl=g_kl)
    hn, Wn, yn = to_np(h), to_np(W), y.cpu().numpy()
    del h, W
    rng = np.random.default_rng(wl.seed + 7)
    rows = np.sort(rng.choice(wl.T, size=96, replace=False))
    ref = oracle.per_row(hn, Wn, yn, rows, tau=wl.tau)
    assert_rows(gpu, ref, rows=rows, what=name)
    ghr = oracle.grad_h_rows(hn, Wn, yn, rows[:32], g_ce, g_kl, tau=wl.tau)
    for i in range(wl.M):
        assert_grad_rows(gpu["grad_h"][i][rows[:32]], ghr[i], f"{name} grad_h[{i}] rows")
        colsum = gpu["grad_W"][i].astype(np.float64).sum(axis=0)
        scale = np.abs(gpu["grad_W"][i]).astype(np.float64).sum(axis=0).max()
        assert np.abs(colsum).max() <= 1e-3 * scale
        ign = yn == -100
        if ign.any():
            assert np.all(gpu["grad_h"][i][ign] == 0)


def test_fused_five_chunks_match_the_recompute_plan_at_c5():
    """At T = 32,768, V = 262,144 the stored-logit plan runs in five token chunks (its slab
    budget), so grad_W is accumulated over five GEMM launches, a path no smaller
    case reaches. Its gradients must equal the recompute plan's within the
    gradient tolerance: two GPU paths that share no backward kernel, each
    checked against the oracle at reduced T. Compared on the device, per
    tensor and per row."""
    from paper_2608_09703_amd import api as D
    wl = WL.WORKLOADS["c5_m3_v262k_long"]
    print(f"[fused-c5] M={wl.M} T={wl.T} V={wl.V} dims={wl.dims}", flush=True)
    h, W, y = WL.make_inputs(wl, device=DEV)
    g_ce, g_kl = oracle.coeffs(wl.M, -1, alpha=wl.alpha, tau=wl.tau)
    gce = torch.tensor(g_ce, dtype=torch.float32, device=DEV)
    gkl = torch.tensor(g_kl, dtype=torch.float32, device=DEV)
    st = torch.cuda.current_stream(DEV).cuda_stream

    p = D.make_problem(h, W, y, tau=wl.tau)
    buf = D.Buffers(p, DEV)
    ws_b = B.query_fwd_bwd_workspace(p)
    ws = torch.empty(ws_b, dtype=torch.uint8, device=DEV)
    gh_f = [torch.empty(x.shape, dtype=torch.float32, device=DEV) for x in h]
    gW_f = [torch.empty(x.shape, dtype=torch.float32, device=DEV) for x in W]
    B.distill_fwd_bwd(p, buf.stats.data_ptr(), buf.ce.data_ptr(), buf.kl.data_ptr(),
                      buf.entropy.data_ptr(), gce.data_ptr(), gkl.data_ptr(),
                      [x.data_ptr() for x in gh_f], [x.data_ptr() for x in gW_f], ws.data_ptr(),
                      ws_b, st)
    torch.cuda.synchronize()
    del ws, buf

    p2 = D.make_problem(h, W, y, tau=wl.tau)
    buf2 = D.Buffers(p2, DEV)
    D.forward(p2, buf2, DEV)
    gh_r = [torch.empty(x.shape, dtype=torch.float32, device=DEV) for x in h]
    gW_r = [torch.empty(x.shape, dtype=torch.float32, device=DEV) for x in W]
    D.backward(p2, buf2, DEV, gce, gkl, gh_r, gW_r)
    torch.cuda.synchronize()
    del buf2

    for i in range(wl.M):
        for what, a, b in (("grad_h", gh_f[i], gh_r[i]), ("grad_W", gW_f[i], gW_r[i])):
            a64, b64 = a.double(), b.double()
            tensor = float(torch.linalg.norm(a64 - b64) / torch.linalg.norm(b64))
            rows = torch.linalg.norm(a64 - b64, dim=1) / torch.linalg.norm(b64, dim=1).clamp_min(1e-30)
            worst = float(rows.max())
            print(f"  sub-model {i} {what}: rel {tensor:.2e}, worst row {worst:.2e}", flush=True)
            assert tensor < 1e-2, (i, what, tensor)
            assert worst < 5e-2, (i, what, worst)
            del a64, b64, rows
