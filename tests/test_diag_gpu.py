"""GPU parity of the cross-model diagnostics (pairwise KL at temperature 1 and
top-1 agreement, paper section 3) against the float64 oracle.

Small cases run the whole oracle on every path (wide bf16, general bf16,
float32; the 128x128 tile for M <= 2 and the 128x64 tile for M = 3, 4) with
ragged token and vocabulary tails. Argmax is an integer decided by floating
point: a GPU index is accepted when its float64 logit is within the fp32
rounding bound of the float64 maximum, ties of bit-identical logits must go to
the lowest index, and agreement is compared exactly on the GPU's own argmax
and within the count of ambiguous tokens against the oracle's. Full-size
workloads are checked on sampled tokens (all other labels ignored, so the mean
covers exactly the sample) and through the identity KL(p_s || p_i) = the
forward's distillation KL at temperature 1 with teacher s.
"""

import numpy as np
import pytest
import torch

import oracle
from paper_2608_09703_amd import api as D
from paper_2608_09703_amd import workloads as WL
from tests.gpu_helpers import LOSS_ATOL, LOSS_RTOL, to_np

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
IGN = oracle.IGNORE_INDEX


def _nested(wl):
    """Sub-model i takes the first d_i features of one draw at the largest width."""
    full = WL.custom(1, wl.T, (max(wl.dims),), wl.V, dtype=wl.dtype, w_std=wl.w_std,
                     w_scale=wl.w_scale, ignore_frac=wl.ignore_frac, seed=wl.seed)
    (hf,), (Wf,), y = WL.make_inputs(full, device=DEV)
    h = [hf[:, :d].contiguous() for d in wl.dims]
    W = [Wf[:, :d].contiguous() for d in wl.dims]
    return h, W, y


def _run(h, W, y):
    kl, agree, am = D.diagnostics(h, W, y, want_argmax=True)
    torch.cuda.synchronize()
    return kl.cpu().numpy().astype(np.float64), agree.cpu().numpy().astype(np.float64), \
        am.cpu().numpy().astype(np.int64)


def _argmax_slack(hn, Wn, rows):
    """fp32 rounding bound of each logit: 2^-22 * K * sum_k |W_vk h_tk| (bounded per row)."""
    return [4.0 * 2.0 ** -24 * hn[i].shape[1] * (np.abs(hn[i][rows]) @ np.abs(Wn[i]).T).max(axis=1)
            + 1e-6 for i in range(len(hn))]


def _check_argmax(am, hn, Wn, rows):
    """Every GPU argmax is a float64 near-maximum; returns per-model ambiguity masks."""
    slack = _argmax_slack(hn, Wn, rows)
    amb = []
    for i in range(len(hn)):
        L = hn[i][rows].astype(np.float64) @ Wn[i].astype(np.float64).T
        mx = L.max(axis=1)
        got = L[np.arange(len(rows)), am[i][rows]]
        assert np.all(am[i][rows] >= 0) and np.all(am[i][rows] < L.shape[1])
        bad = got < mx - slack[i]
        assert not bad.any(), f"model {i}: argmax not a near-maximum at rows {rows[bad][:5]}"
        # a token is ambiguous when a second index comes within twice the slack
        near = (L >= (mx - 2 * slack[i])[:, None]).sum(axis=1)
        amb.append(near > 1)
    return amb


def _check_all(kl, agree, am, ref, hn, Wn, yn, what):
    M = len(hn)
    np.testing.assert_allclose(kl, ref["kl"], rtol=LOSS_RTOL, atol=LOSS_ATOL, err_msg=f"{what} kl")
    assert np.all(np.diag(kl) == 0.0)
    rows = np.arange(len(yn))
    amb = _check_argmax(am, hn, Wn, rows)
    valid = yn != IGN
    n = int(valid.sum())
    for i in range(M):
        for j in range(M):
            own = (am[i][valid] == am[j][valid]).mean() if n else 0.0
            assert abs(agree[i, j] - own) <= 1e-6, f"{what} agree[{i},{j}] vs its own argmax"
            loose = int((amb[i] | amb[j])[valid].sum())
            assert abs(agree[i, j] - ref["agree"][i, j]) * max(n, 1) <= loose + 1e-3, \
                f"{what} agree[{i},{j}] {agree[i, j]} vs oracle {ref['agree'][i, j]}"
    unamb = ~np.logical_or.reduce(amb)
    for i in range(M):
        assert np.array_equal(am[i][unamb], ref["argmax"][i][unamb]), f"{what} argmax[{i}]"


SMALL = [
    # name, workload, nested heads
    ("m2_nested_wide", WL.custom(2, 300, (64, 128), 1000, w_std=0.1, w_scale=3.0, ignore_frac=0.1,
                                 seed=21), True),
    ("m3_nested_ragged", WL.custom(3, 260, (64, 128, 192), 1300, w_std=0.1, w_scale=3.0,
                                   ignore_frac=0.1, seed=22), True),
    ("m4_random", WL.custom(4, 200, (64, 64, 128, 256), 777, w_std=0.05, ignore_frac=0.2, seed=23),
     False),
    ("m1", WL.custom(1, 130, (96,), 300, w_std=0.1, seed=24), False),
    ("m2_general_bf16", WL.custom(2, 140, (72, 136), 600, w_std=0.1, w_scale=2.0, seed=25), True),
    ("m3_general_bf16", WL.custom(3, 140, (40, 72, 136), 650, w_std=0.1, w_scale=2.0, seed=26), True),
    ("m2_f32", WL.WORKLOADS["c1_small_f32"], False),
    ("m3_f32_ragged", WL.custom(3, 150, (32, 36, 100), 555, dtype="f32", w_std=0.1, w_scale=2.0,
                                ignore_frac=0.1, seed=27), True),
    ("v2_binary", WL.custom(2, 64, (8, 16), 2, w_std=0.5, seed=28), True),
    ("t1_single_token", WL.custom(3, 1, (64, 64, 128), 300, w_std=0.1, seed=29), False),
    # logits of standard deviation ~20: every partial is normalised to its own
    # maximum, and merging rescales across lanes, waves and vocabulary tiles
    ("m3_large_logits", WL.custom(3, 200, (64, 128, 192), 1500, w_std=None, w_scale=20.0,
                                  ignore_frac=0.1, seed=30), True),
    ("m4_large_logits", WL.custom(4, 150, (64, 64, 128, 256), 1100, w_std=None, w_scale=20.0,
                                  seed=36), False),
    # more than four sub-models: passes over subsets of four that cover every pair
    ("m5_nested_subsets", WL.custom(5, 220, (64, 64, 128, 128, 192), 900, w_std=0.1, w_scale=3.0,
                                    ignore_frac=0.1, seed=37), True),
    ("m8_nested_subsets", WL.custom(8, 200, (64, 64, 128, 128, 192, 192, 256, 320), 1100,
                                    w_std=0.1, w_scale=3.0, ignore_frac=0.1, seed=38), True),
    ("m6_general_bf16", WL.custom(6, 140, (40, 72, 72, 136, 136, 200), 650, w_std=0.1, w_scale=2.0,
                                  seed=39), True),
    ("m7_f32", WL.custom(7, 130, (32, 36, 36, 64, 64, 100, 100), 555, dtype="f32", w_std=0.1,
                         w_scale=2.0, ignore_frac=0.1, seed=40), False),
]


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_small_diagnostics_parity(case):
    name, wl, nested = case
    print(f"[diag] {name} M={wl.M} T={wl.T} V={wl.V} dims={wl.dims} {wl.dtype}", flush=True)
    h, W, y = _nested(wl) if nested else WL.make_inputs(wl, device=DEV)
    hn, Wn, yn = to_np(h), to_np(W), y.cpu().numpy()
    kl, agree, am = _run(h, W, y)
    ref = oracle.diagnostics(hn, Wn, yn)
    _check_all(kl, agree, am, ref, hn, Wn, yn, name)


def test_argmax_ties_take_the_lowest_index():
    """Bit-identical dominant rows in different tiles and segments: the lowest index wins."""
    M, T, V, d = 3, 150, 420, 64
    g = torch.Generator(device=DEV).manual_seed(31)
    h = [torch.randn(T, d, generator=g, device=DEV).to(torch.bfloat16) for _ in range(M)]
    W = [(0.02 * torch.randn(V, d, generator=g, device=DEV)).to(torch.bfloat16) for _ in range(M)]
    for i in range(M):
        h[i][:, 0] = 1.0
    # model 0: rows 3 and 200 (tiles 0 and 1); model 1: 40 and 41 (one MFMA block);
    # model 2: 300 and 130 (the lower index in the later-scanned tile is 130)
    pairs = [(3, 200), (40, 41), (130, 300)]
    for i, (a, b) in enumerate(pairs):
        u = torch.zeros(d, device=DEV)
        u[0] = 8.0
        W[i][a] = u.to(torch.bfloat16)
        W[i][b] = u.to(torch.bfloat16)
    y = torch.randint(0, V, (T,), generator=g, device=DEV)
    print(f"[diag] ties M={M} T={T} V={V}", flush=True)
    kl, agree, am = _run(h, W, y)
    for i, (a, b) in enumerate(pairs):
        assert np.all(am[i] == min(a, b)), f"model {i}: {np.unique(am[i])}"
    hn, Wn, yn = to_np(h), to_np(W), y.cpu().numpy()
    ref = oracle.diagnostics(hn, Wn, yn)
    assert np.array_equal(ref["argmax"], am)
    np.testing.assert_allclose(agree, ref["agree"], atol=1e-6)
    np.testing.assert_allclose(kl, ref["kl"], rtol=LOSS_RTOL, atol=LOSS_ATOL)


def test_all_ignored_gives_zero():
    wl = WL.custom(3, 100, (64, 64, 128), 500, w_std=0.1, seed=32)
    h, W, _ = WL.make_inputs(wl, device=DEV)
    y = torch.full((wl.T,), IGN, dtype=torch.int64, device=DEV)
    print("[diag] all ignored", flush=True)
    kl, agree, am = _run(h, W, y)
    assert np.all(kl == 0.0) and np.all(agree == 0.0)
    hn, Wn = to_np(h), to_np(W)
    _check_argmax(am, hn, Wn, np.arange(wl.T))  # argmax is reported for every token


def test_identical_models_agree_fully():
    wl = WL.custom(1, 200, (128,), 900, w_std=0.1, seed=33)
    (h0,), (W0,), y = WL.make_inputs(wl, device=DEV)
    h = [h0, h0.clone(), h0.clone()]
    W = [W0, W0.clone(), W0.clone()]
    print("[diag] identical models", flush=True)
    kl, agree, am = _run(h, W, y)
    assert np.all(np.abs(kl) <= 1e-6), kl
    assert np.all(agree == 1.0)
    assert np.array_equal(am[0], am[1]) and np.array_equal(am[0], am[2])


def test_bitwise_deterministic():
    wl = WL.custom(4, 333, (64, 128, 192, 256), 2100, w_std=0.05, ignore_frac=0.1, seed=34)
    h, W, y = _nested(wl)
    print("[diag] determinism", flush=True)
    a = _run(h, W, y)
    b = _run(h, W, y)
    for x, z in zip(a, b):
        assert np.array_equal(x, z)


FULL = ["c2_m3_v50k", "c4_m4_v128k_peaky", "c5_m3_v262k_long"]  # the last: records past 4 GiB


@pytest.mark.parametrize("name", FULL)
def test_full_size_sampled_tokens(name):
    """Full shape and launch configuration; only sampled tokens carry a label."""
    wl = WL.WORKLOADS[name]
    print(f"[diag] full-size {name} M={wl.M} T={wl.T} V={wl.V}", flush=True)
    h, W, y = WL.make_inputs(wl, device=DEV)
    rng = np.random.default_rng(35)
    rows = np.sort(rng.choice(wl.T, size=48, replace=False))
    rows = np.unique(np.concatenate([rows, [0, wl.T - 1]]))
    ys = torch.full_like(y, IGN)
    yr = torch.randint(0, wl.V, (len(rows),), device=DEV)
    ys[torch.from_numpy(rows).to(DEV)] = yr
    kl, agree, am = _run(h, W, ys)
    hs = [x.float().cpu().numpy()[rows] for x in h]
    Wn = to_np(W)
    ref = oracle.diagnostics(hs, Wn, yr.cpu().numpy())
    np.testing.assert_allclose(kl, ref["kl"], rtol=LOSS_RTOL, atol=LOSS_ATOL, err_msg="kl")
    amb = _check_argmax([a[rows] for a in am], hs, Wn, np.arange(len(rows)))
    n = len(rows)
    for i in range(wl.M):
        for j in range(wl.M):
            loose = int((amb[i] | amb[j]).sum())
            assert abs(agree[i, j] - ref["agree"][i, j]) * n <= loose + 1e-3


@pytest.mark.parametrize("name", ["c2_m3_v50k", "c3_m3_v128k_tau2"])
def test_teacher_row_matches_forward_kl(name):
    """KL(p_s || p_i) from the pairwise pass equals the forward's KL term at tau = 1."""
    wl = WL.WORKLOADS[name]
    print(f"[diag] forward identity {name}", flush=True)
    h, W, y = WL.make_inputs(wl, device=DEV)
    kl, _, _ = _run(h, W, y)
    for s in range(wl.M):
        _, fkl, _ = D.distill(h, W, y, tau=1.0, teacher=s)
        fkl = fkl.detach().cpu().numpy().astype(np.float64)
        np.testing.assert_allclose(kl[s], fkl, rtol=LOSS_RTOL, atol=LOSS_ATOL,
                                   err_msg=f"teacher {s}")
