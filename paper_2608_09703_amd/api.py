"""PyTorch front end of the fused multi-sub-model LM head + CE + KL.

``distill(h_list, W_list, labels, ...)`` returns the per-sub-model
cross-entropies ``ce[M]``, the distillation values ``kl[M]`` (KL from the
teacher's softmax at temperature tau) and the mean teacher entropy, with
autograd support: the backward pass feeds the upstream gradients of ``ce``
and ``kl`` to the library as the coefficients of the objective, so any
objective linear in them (eq. (3) of the paper with its sum over
sub-models, or per-sub-model weights) differentiates correctly with no host
synchronisation.

``forward`` / ``backward`` are the same two library calls without autograd,
on caller-visible buffers (used by the tests and the benchmark).
"""

from __future__ import annotations

from typing import List, Optional, Sequence

import torch

from . import binding as B


def _dtype_code(dt: torch.dtype) -> int:
    if dt == torch.bfloat16:
        return B.MLS_BF16
    if dt == torch.float32:
        return B.MLS_F32
    raise TypeError(f"unsupported dtype {dt}; use bfloat16 or float32")


def make_problem(h: Sequence[torch.Tensor], W: Sequence[torch.Tensor], labels: torch.Tensor, *,
                 alpha: float = 0.0, tau: float = 1.0, teacher: int = -1,
                 ignore_index: int = -100, flags: int = 0, vocab_chunk: int = 0,
                 grad_h_dtype: torch.dtype = torch.float32) -> B.Problem:
    M = len(h)
    if M < 1 or len(W) != M:
        raise ValueError("need one head per sub-model")
    dev = h[0].device
    if dev.type != "cuda":
        raise RuntimeError("the fused loss runs on the GPU only; got tensors on " + str(dev))
    dt = h[0].dtype
    T = h[0].shape[0]
    V = W[0].shape[0]
    for i in range(M):
        for x in (h[i], W[i]):
            if x.device != dev or x.dtype != dt or x.dim() != 2 or not x.is_contiguous():
                raise ValueError("h_i / W_i must be contiguous 2-D tensors of one dtype on one device")
        if h[i].shape[0] != T or W[i].shape[0] != V or h[i].shape[1] != W[i].shape[1]:
            raise ValueError(f"shape mismatch in sub-model {i}")
    if labels.device != dev or labels.dtype != torch.int64 or labels.shape != (T,) \
            or not labels.is_contiguous():
        raise ValueError("labels must be a contiguous int64 [T] tensor on the same device")
    return B.make_problem(M, T, V, [x.shape[1] for x in h], [x.data_ptr() for x in h],
                          [x.data_ptr() for x in W], labels.data_ptr(), dtype=_dtype_code(dt),
                          teacher=teacher, ignore_index=ignore_index, alpha=alpha, tau=tau,
                          flags=flags, vocab_chunk=vocab_chunk,
                          grad_h_dtype=_dtype_code(grad_h_dtype))


def _stream(dev) -> int:
    return torch.cuda.current_stream(dev).cuda_stream


class Buffers:
    """Caller-owned device buffers of one problem shape (workspace + statistics)."""

    def __init__(self, p: B.Problem, device):
        self.ws_bytes, self.stats_bytes = B.query_sizes(p)
        self.workspace = torch.empty(max(self.ws_bytes, 256), dtype=torch.uint8, device=device)
        self.stats = torch.empty(self.stats_bytes, dtype=torch.uint8, device=device)
        M = p.M
        self.ce = torch.empty(M, dtype=torch.float32, device=device)
        self.kl = torch.empty(M, dtype=torch.float32, device=device)
        self.entropy = torch.empty(1, dtype=torch.float32, device=device)

    def stats_view(self, M: int, T: int):
        """(lse1, lset, ce_row, kl_row, h_row) views into the statistics buffer."""
        f = self.stats[: (4 * M * T + T) * 4].view(torch.float32)
        return (f[: M * T].view(M, T), f[M * T: 2 * M * T].view(M, T),
                f[2 * M * T: 3 * M * T].view(M, T), f[3 * M * T: 4 * M * T].view(M, T),
                f[4 * M * T:])


def forward(p: B.Problem, buf: Buffers, device) -> None:
    B.distill_fwd(p, buf.stats.data_ptr(), buf.ce.data_ptr(), buf.kl.data_ptr(),
                  buf.entropy.data_ptr(), buf.workspace.data_ptr(), buf.workspace.numel(),
                  _stream(device))


def backward(p: B.Problem, buf: Buffers, device, g_ce: Optional[torch.Tensor],
             g_kl: Optional[torch.Tensor], grad_h: Sequence[Optional[torch.Tensor]],
             grad_W: Sequence[Optional[torch.Tensor]]) -> None:
    gh_dt = torch.bfloat16 if p.grad_h_dtype == B.MLS_BF16 else torch.float32
    for g in grad_h:
        if g is not None and (g.dtype != gh_dt or not g.is_contiguous()):
            raise ValueError(f"grad_h tensors are contiguous {gh_dt} tensors")
    for g in grad_W:
        if g is not None and (g.dtype != torch.float32 or not g.is_contiguous()):
            raise ValueError("grad_W tensors are contiguous float32 tensors")
    gc = g_ce.data_ptr() if g_ce is not None else None
    gk = g_kl.data_ptr() if g_kl is not None else None
    B.distill_bwd(p, buf.stats.data_ptr(), gc, gk,
                  [g.data_ptr() if g is not None else None for g in grad_h],
                  [g.data_ptr() if g is not None else None for g in grad_W],
                  buf.workspace.data_ptr(), buf.workspace.numel(), _stream(device))


class _Distill(torch.autograd.Function):
    @staticmethod
    def forward(ctx, labels, opts, *hw):
        M = len(hw) // 2
        h, W = list(hw[:M]), list(hw[M:])
        # bf16 hidden states get bf16 gradients straight from the library
        p = make_problem(h, W, labels, grad_h_dtype=h[0].dtype, **opts)
        dev = h[0].device
        buf = Buffers(p, dev)
        forward(p, buf, dev)
        ctx.p = p
        ctx.buf = buf
        ctx.M = M
        ctx.save_for_backward(labels, *hw)
        ctx.mark_non_differentiable(buf.entropy)
        return buf.ce.clone(), buf.kl.clone(), buf.entropy.clone()

    @staticmethod
    def backward(ctx, g_ce, g_kl, g_ent):
        saved = ctx.saved_tensors
        hw = saved[1:]
        M = ctx.M
        dev = hw[0].device
        if g_ce is None:
            g_ce = torch.zeros(M, dtype=torch.float32, device=dev)
        if g_kl is None:
            g_kl = torch.zeros(M, dtype=torch.float32, device=dev)
        g_ce = g_ce.to(torch.float32).contiguous()
        g_kl = g_kl.to(torch.float32).contiguous()
        need = ctx.needs_input_grad[2:]
        gh: List[Optional[torch.Tensor]] = []
        gW: List[Optional[torch.Tensor]] = []
        gh_dt = torch.bfloat16 if ctx.p.grad_h_dtype == B.MLS_BF16 else torch.float32
        for i in range(M):
            gh.append(torch.empty(hw[i].shape, dtype=gh_dt, device=dev) if need[i] else None)
            gW.append(torch.empty(hw[M + i].shape, dtype=torch.float32, device=dev)
                      if need[M + i] else None)
        backward(ctx.p, ctx.buf, dev, g_ce, g_kl, gh, gW)
        out = [None, None]
        for i in range(M):
            out.append(gh[i].to(hw[i].dtype) if gh[i] is not None else None)
        for i in range(M):
            out.append(gW[i].to(hw[M + i].dtype) if gW[i] is not None else None)
        return tuple(out)


def distill(h_list: Sequence[torch.Tensor], W_list: Sequence[torch.Tensor], labels: torch.Tensor,
            *, tau: float = 1.0, teacher: int = -1, ignore_index: int = -100,
            vocab_chunk: int = 0):
    """Per-sub-model ``(ce[M], kl[M], entropy[1])`` with autograd through the HIP kernels."""
    opts = dict(tau=tau, teacher=teacher, ignore_index=ignore_index, vocab_chunk=vocab_chunk)
    return _Distill.apply(labels, opts, *h_list, *W_list)


def run_diagnostics(p: B.Problem, buf: Buffers, device, kl_pair: torch.Tensor, agree: torch.Tensor,
                    argmax: Optional[torch.Tensor]) -> None:
    """Pairwise diagnostics into caller tensors (one pass; ``buf.workspace`` is used)."""
    B.diagnostics(p, kl_pair.data_ptr(), agree.data_ptr(),
                  argmax.data_ptr() if argmax is not None else None, buf.workspace.data_ptr(),
                  buf.workspace.numel(), _stream(device))


@torch.no_grad()
def diagnostics(h_list: Sequence[torch.Tensor], W_list: Sequence[torch.Tensor],
                labels: torch.Tensor, *, ignore_index: int = -100, want_argmax: bool = False):
    """Cross-model ``(kl[M, M], agree[M, M], argmax[M, T] or None)`` of the sub-model heads.

    ``kl[i, j]`` is the mean over valid tokens of KL(p_i || p_j) at temperature 1 and
    ``agree[i, j]`` the fraction of valid tokens whose top-1 predictions coincide.
    One self-normalising pass over the logits of all sub-models.
    """
    p = make_problem(h_list, W_list, labels, ignore_index=ignore_index)
    dev = h_list[0].device
    buf = Buffers(p, dev)
    M, T = len(h_list), h_list[0].shape[0]
    kl = torch.empty(M, M, dtype=torch.float32, device=dev)
    agree = torch.empty(M, M, dtype=torch.float32, device=dev)
    am = torch.empty(M, T, dtype=torch.int32, device=dev) if want_argmax else None
    run_diagnostics(p, buf, dev, kl, agree, am)
    return kl, agree, am


def _junction_desc(o, e, grad_dtype, layout, flags=0):
    if o.device.type != "cuda" or e.device != o.device:
        raise RuntimeError("the junction runs on the GPU only")
    if o.dim() != 2 or e.dim() != 2 or o.shape[0] != e.shape[0] or o.dtype != e.dtype:
        raise ValueError("o [T, d_prev] and e [T, d_fresh] must share T and dtype")
    if not (o.is_contiguous() and e.is_contiguous()):
        raise ValueError("o and e must be contiguous")
    lay = {"prev_first": B.MLS_JUNCTION_PREV_FIRST, "fresh_first": B.MLS_JUNCTION_FRESH_FIRST}[layout]
    return B.make_junction(o.shape[0], o.shape[1], e.shape[1], _dtype_code(o.dtype),
                           _dtype_code(grad_dtype), lay, flags)


def junction_forward(o: torch.Tensor, e: torch.Tensor, *, layout: str = "prev_first",
                     out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Eq. (1): ``x = [o * ||e|| / ||o|| | e]`` per token (no autograd)."""
    j = _junction_desc(o, e, o.dtype, layout)
    x = out if out is not None else torch.empty(o.shape[0], o.shape[1] + e.shape[1],
                                                 dtype=o.dtype, device=o.device)
    B.junction_fwd(j, o.data_ptr(), e.data_ptr(), x.data_ptr(), _stream(o.device))
    return x


def junction_backward(o: torch.Tensor, e: torch.Tensor, g_x: torch.Tensor, *,
                      layout: str = "prev_first", g_o: Optional[torch.Tensor] = None,
                      g_e: Optional[torch.Tensor] = None, accumulate: bool = False):
    """``(g_o, g_e)`` of the junction for the upstream gradient ``g_x`` (dtype of ``g_x``)."""
    if not g_x.is_contiguous() or g_x.shape != (o.shape[0], o.shape[1] + e.shape[1]):
        raise ValueError("g_x must be a contiguous [T, d_prev + d_fresh] tensor")
    j = _junction_desc(o, e, g_x.dtype, layout, B.MLS_JUNCTION_ACCUMULATE if accumulate else 0)
    if g_o is None:
        g_o = torch.empty(o.shape, dtype=g_x.dtype, device=o.device)
    if g_e is None:
        g_e = torch.empty(e.shape, dtype=g_x.dtype, device=o.device)
    for g in (g_o, g_e):
        if g.dtype != g_x.dtype or not g.is_contiguous():
            raise ValueError("g_o / g_e must be contiguous and of g_x's dtype")
    B.junction_bwd(j, o.data_ptr(), e.data_ptr(), g_x.data_ptr(), g_o.data_ptr(), g_e.data_ptr(),
                   _stream(o.device))
    return g_o, g_e


class _Junction(torch.autograd.Function):
    @staticmethod
    def forward(ctx, o, e, layout):
        ctx.save_for_backward(o, e)
        ctx.layout = layout
        return junction_forward(o, e, layout=layout)

    @staticmethod
    def backward(ctx, g_x):
        o, e = ctx.saved_tensors
        g_o, g_e = junction_backward(o, e, g_x.contiguous(), layout=ctx.layout)
        return g_o.to(o.dtype), g_e.to(e.dtype), None


def junction(o: torch.Tensor, e: torch.Tensor, *, layout: str = "prev_first") -> torch.Tensor:
    """Inter-model junction of eq. (1) with autograd through the HIP kernels."""
    return _Junction.apply(o, e, layout)


def head_logits(o: torch.Tensor, W: torch.Tensor, out: Optional[torch.Tensor] = None):
    """``logits [T, V] = o W^T`` in fp32 through the HIP head kernel (decode regime)."""
    if o.device.type != "cuda" or W.device != o.device or o.dtype != W.dtype:
        raise RuntimeError("o and W must be GPU tensors of one dtype")
    if not (o.is_contiguous() and W.is_contiguous()) or o.shape[1] != W.shape[1]:
        raise ValueError("o [T, d] and W [V, d] must be contiguous with a shared d")
    T, V = o.shape[0], W.shape[0]
    out = out if out is not None else torch.empty(T, V, dtype=torch.float32, device=o.device)
    B.head_logits(T, V, o.shape[1], _dtype_code(o.dtype), o.data_ptr(), W.data_ptr(),
                  out.data_ptr(), _stream(o.device))
    return out


def _sampling(V, temperature, top_p, greedy):
    return B.make_sampling(V, temperature, top_p, greedy)


def sample(logits: torch.Tensor, u: Optional[torch.Tensor], *, temperature: float = 1.0,
           top_p: float = 1.0, greedy: bool = False,
           params: Optional[torch.Tensor] = None) -> torch.Tensor:
    """int32 tokens, one per row of ``logits [rows, V]`` (fp32), with uniforms ``u [rows]``.

    ``params``: optional uint8 tensor of ``rows * ROW_PARAMS_BYTES`` bytes that
    receives the rows' distribution records (for ``spec_verify(draft_params=)``).
    """
    if logits.dtype != torch.float32 or not logits.is_contiguous() or logits.dim() != 2:
        raise ValueError("logits must be a contiguous float32 [rows, V] tensor")
    rows, V = logits.shape
    if u is not None and (u.dtype != torch.float32 or u.shape != (rows,) or not u.is_contiguous()):
        raise ValueError("u must be a contiguous float32 [rows] tensor")
    if params is not None and (params.dtype != torch.uint8 or not params.is_contiguous() or
                               params.numel() < rows * B.ROW_PARAMS_BYTES):
        raise ValueError("params must be a contiguous uint8 tensor of rows * ROW_PARAMS_BYTES")
    tok = torch.empty(rows, dtype=torch.int32, device=logits.device)
    B.sample(_sampling(V, temperature, top_p, greedy), rows, logits.data_ptr(),
             u.data_ptr() if u is not None else None, tok.data_ptr(), _stream(logits.device),
             params.data_ptr() if params is not None else None)
    return tok


def spec_verify(draft_logits: Optional[torch.Tensor], target_logits: torch.Tensor,
                draft_tokens: Optional[torch.Tensor], u_accept: Optional[torch.Tensor],
                u_sample: Optional[torch.Tensor], *, temperature: float = 1.0, top_p: float = 1.0,
                greedy: bool = False, draft_params: Optional[torch.Tensor] = None):
    """``(n_accepted [B], next_token [B])`` (int32) of speculative verification.

    Draft-side arrays in drafting order: ``draft_logits [gamma, B, V]`` (fp32),
    ``draft_tokens [gamma, B]`` (int32), ``u_accept [gamma, B]``; verifier side
    ``target_logits [B, gamma + 1, V]`` (fp32) and ``u_sample [B]``.
    ``draft_params``: optional uint8 records ``[gamma, B]`` from ``sample(params=)``
    on the draft rows with the same settings (then not recomputed).
    """
    Bt, G1, V = target_logits.shape
    G = G1 - 1
    dev = target_logits.device
    for x in (draft_logits, target_logits, u_accept, u_sample):
        if x is not None and (x.dtype != torch.float32 or not x.is_contiguous()):
            raise ValueError("logits and uniforms must be contiguous float32")
    if draft_tokens is not None and (draft_tokens.dtype != torch.int32 or
                                     not draft_tokens.is_contiguous()):
        raise ValueError("draft_tokens must be contiguous int32")
    if G > 0 and (draft_logits is None or draft_logits.shape != (G, Bt, V) or
                  draft_tokens is None or draft_tokens.shape != (G, Bt)):
        raise ValueError("draft_logits [gamma, B, V] and draft_tokens [gamma, B] are required")
    if G > 0 and not greedy and (u_accept is None or u_accept.shape != (G, Bt)):
        raise ValueError("u_accept [gamma, B] is required")
    n_acc = torch.empty(Bt, dtype=torch.int32, device=dev)
    nxt = torch.empty(Bt, dtype=torch.int32, device=dev)
    ws_bytes = 0 if greedy else B.spec_verify_workspace(Bt, G)
    ws = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=dev) if not greedy else None
    ptr = (lambda x: x.data_ptr() if x is not None else None)
    if draft_params is not None and (draft_params.dtype != torch.uint8 or
                                     not draft_params.is_contiguous() or
                                     draft_params.numel() < G * Bt * B.ROW_PARAMS_BYTES):
        raise ValueError("draft_params must be contiguous uint8 of gamma * B records")
    B.spec_verify(_sampling(V, temperature, top_p, greedy), Bt, G, ptr(draft_logits),
                  target_logits.data_ptr(), ptr(draft_tokens), ptr(u_accept), ptr(u_sample),
                  n_acc.data_ptr(), nxt.data_ptr(), ptr(ws), ws_bytes, _stream(dev),
                  draft_params=ptr(draft_params))
    return n_acc, nxt


def coefficients(M: int, *, alpha: float, tau: float = 1.0, teacher: int = -1,
                 mode: str = "paper", weights: Optional[Sequence[float]] = None):
    """``(g_ce, g_kl)`` lists of eq. (3) (``mode="paper"``) or the additive form."""
    m = B.MLS_MODE_PAPER if mode == "paper" else B.MLS_MODE_ADDITIVE
    return B.coeffs(M, teacher, alpha, tau, m, weights)
