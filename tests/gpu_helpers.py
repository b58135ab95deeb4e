"""Helpers shared by the GPU tests: run the HIP path through the C ABI and
compare with the CPU oracle on the same inputs."""

from __future__ import annotations

import numpy as np
import torch

from paper_2608_09703_amd import api as D

LOSS_RTOL = 1e-3     # losses: relative 1e-3 ...
LOSS_ATOL = 1e-5     # ... with an absolute floor for values near 0 (KL of equal models)
ROW_ATOL = 5e-5      # per-row statistics: fp32 log-sum-exp of ~1e5 terms
from tests.grad_checks import (GRAD_RTOL, assert_grad, assert_grad_rows,  # noqa: F401
                                non_label_rows, rel_fro)


def to_np(xs):
    return [x.detach().float().cpu().numpy() for x in xs]


def run_gpu(h, W, labels, *, tau=1.0, teacher=-1, g_ce=None, g_kl=None, vocab_chunk=0,
            grads=True, alpha=0.0):
    dev = h[0].device
    p = D.make_problem(h, W, labels, tau=tau, teacher=teacher, vocab_chunk=vocab_chunk, alpha=alpha)
    buf = D.Buffers(p, dev)
    D.forward(p, buf, dev)
    M, T = len(h), h[0].shape[0]
    lse1, lset, ce_row, kl_row, h_row = buf.stats_view(M, T)
    out = {
        "ce": buf.ce.cpu().numpy().astype(np.float64),
        "kl": buf.kl.cpu().numpy().astype(np.float64),
        "H": float(buf.entropy.cpu().numpy()[0]),
        "lse1": lse1.cpu().numpy(),
        "lset": lset.cpu().numpy(),
        "ce_row": ce_row.cpu().numpy(),
        "kl_row": kl_row.cpu().numpy(),
        "h_row": h_row.cpu().numpy(),
    }
    if grads:
        gh = [torch.full(x.shape, float("nan"), dtype=torch.float32, device=dev) for x in h]
        gW = [torch.full(x.shape, float("nan"), dtype=torch.float32, device=dev) for x in W]
        gce = torch.tensor(g_ce, dtype=torch.float32, device=dev) if g_ce is not None else None
        gkl = torch.tensor(g_kl, dtype=torch.float32, device=dev) if g_kl is not None else None
        D.backward(p, buf, dev, gce, gkl, gh, gW)
        out["grad_h"] = [x.cpu().numpy() for x in gh]
        out["grad_W"] = [x.cpu().numpy() for x in gW]
    torch.cuda.synchronize()
    out["n_valid"], out["flags"] = __import__("paper_2608_09703_amd.binding", fromlist=["x"]) \
        .read_stats_header(p, buf.stats.data_ptr(), torch.cuda.current_stream(dev).cuda_stream)
    return out


def run_fused(h, W, labels, *, tau=1.0, teacher=-1, g_ce=None, g_kl=None, alpha=0.0, flags=0,
              grad_h_dtype=torch.float32, vocab_chunk=0):
    """mls_distill_fwd_bwd through the C ABI; the same dict as run_gpu."""
    from paper_2608_09703_amd import binding as B
    dev = h[0].device
    p = D.make_problem(h, W, labels, tau=tau, teacher=teacher, alpha=alpha, flags=flags,
                       grad_h_dtype=grad_h_dtype, vocab_chunk=vocab_chunk)
    buf = D.Buffers(p, dev)
    ws_b = B.query_fwd_bwd_workspace(p)
    ws = torch.empty(max(ws_b, 256), dtype=torch.uint8, device=dev)
    gh = [torch.full(x.shape, float("nan"), dtype=grad_h_dtype, device=dev) for x in h]
    gW = [torch.full(x.shape, float("nan"), dtype=torch.float32, device=dev) for x in W]
    gce = torch.tensor(g_ce, dtype=torch.float32, device=dev) if g_ce is not None else None
    gkl = torch.tensor(g_kl, dtype=torch.float32, device=dev) if g_kl is not None else None
    st = torch.cuda.current_stream(dev).cuda_stream
    B.distill_fwd_bwd(p, buf.stats.data_ptr(), buf.ce.data_ptr(), buf.kl.data_ptr(),
                      buf.entropy.data_ptr(), gce.data_ptr() if gce is not None else None,
                      gkl.data_ptr() if gkl is not None else None, [x.data_ptr() for x in gh],
                      [x.data_ptr() for x in gW], ws.data_ptr(), ws_b, st)
    M, T = len(h), h[0].shape[0]
    lse1, lset, ce_row, kl_row, h_row = buf.stats_view(M, T)
    out = {
        "ce": buf.ce.cpu().numpy().astype(np.float64),
        "kl": buf.kl.cpu().numpy().astype(np.float64),
        "H": float(buf.entropy.cpu().numpy()[0]),
        "lse1": lse1.cpu().numpy(), "lset": lset.cpu().numpy(), "ce_row": ce_row.cpu().numpy(),
        "kl_row": kl_row.cpu().numpy(), "h_row": h_row.cpu().numpy(),
        "grad_h": [x.float().cpu().numpy() for x in gh],
        "grad_W": [x.cpu().numpy() for x in gW],
        "ws_bytes": ws_b,
    }
    out["n_valid"], out["flags"] = B.read_stats_header(p, buf.stats.data_ptr(), st)
    return out


def assert_losses(gpu, ref, what=""):
    for k in ("ce", "kl"):
        np.testing.assert_allclose(gpu[k], ref[k], rtol=LOSS_RTOL, atol=LOSS_ATOL,
                                   err_msg=f"{what} {k}")
    np.testing.assert_allclose(gpu["H"], ref["H"], rtol=LOSS_RTOL, atol=LOSS_ATOL,
                               err_msg=f"{what} entropy")


def assert_rows(gpu, ref, rows=None, what=""):
    for k in ("lse1", "lset", "ce_row", "kl_row"):
        g = gpu[k] if rows is None else gpu[k][:, rows]
        np.testing.assert_allclose(g, ref[k], rtol=LOSS_RTOL, atol=ROW_ATOL, err_msg=f"{what} {k}")
    g = gpu["h_row"] if rows is None else gpu["h_row"][rows]
    np.testing.assert_allclose(g, ref["h_row"], rtol=LOSS_RTOL, atol=ROW_ATOL, err_msg=f"{what} H")


