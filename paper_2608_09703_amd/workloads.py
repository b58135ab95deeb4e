"""Seeded synthetic workloads for the multi-head LM loss.

This module only draws random inputs (hidden states, heads, labels) with
the shapes and value distributions of the benchmark workloads; it holds
none of the loss arithmetic, so the GPU path and the CPU oracle can both be
fed from it.

The paper trains on FineWeb-Edu with the SmolLM2 tokenizer (V = 49,152;
section 3, "Experimental Setup") and packs sequences to 2,048 tokens. That
corpus is not available here: uniform random labels and Gaussian hidden
states / heads of the same shapes stand in for it. The value distributions
change the numbers, not the cost of the computation.
"""

from __future__ import annotations

import dataclasses
import math
from typing import Optional, Sequence, Tuple

import torch

IGNORE_INDEX = -100


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape and distribution of one synthetic problem.

    ``w_std`` is the standard deviation of every head entry; ``None`` means
    ``1 / sqrt(d_i)`` per sub-model. ``w_scale`` multiplies the heads after
    drawing (used to make logits peaky). ``ignore_frac`` is the Bernoulli
    probability that a label is replaced by ``IGNORE_INDEX``.
    """

    name: str
    M: int
    T: int
    dims: Tuple[int, ...]
    V: int
    dtype: str = "bf16"          # "bf16" or "f32": the dtype of h_i and W_i
    alpha: float = 1.0
    tau: float = 1.0
    w_std: Optional[float] = 0.02
    w_scale: float = 1.0
    ignore_frac: float = 0.0
    seed: int = 0
    batch: int = 1
    seq: int = 0

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32

    def algorithmic_flops(self) -> float:
        """Dense work of one forward + backward pass: three GEMMs of 2*T*V*d_i."""
        return 6.0 * self.T * self.V * float(sum(self.dims))


# The five benchmark workloads plus the head shape of the paper's 3B suite
# (Table 1: widths 1024 / 2304 / 4352, V = 49,152; alpha_d = 0.3 from
# section 3, "Experimental Setup").
WORKLOADS = {
    "c1_small_f32": Workload("c1_small_f32", 2, 256, (128, 256), 4096, "f32",
                             alpha=1.0, tau=1.0, w_std=None, seed=1001, batch=1, seq=256),
    "c2_m3_v50k": Workload("c2_m3_v50k", 3, 4096, (1024, 2048, 3072), 50304, "bf16",
                           alpha=1.0, tau=1.0, seed=1002, batch=2, seq=2048),
    "c3_m3_v128k_tau2": Workload("c3_m3_v128k_tau2", 3, 8192, (1024, 2048, 3072), 128256,
                                 "bf16", alpha=0.5, tau=2.0, seed=1003, batch=4, seq=2048),
    "c4_m4_v128k_peaky": Workload("c4_m4_v128k_peaky", 4, 16384, (512, 1024, 2048, 4096),
                                  128256, "bf16", alpha=1.0, tau=1.0, w_scale=5.0,
                                  ignore_frac=0.1, seed=1004, batch=8, seq=2048),
    "c5_m3_v262k_long": Workload("c5_m3_v262k_long", 3, 32768, (1536, 3072, 4608), 262144,
                                 "bf16", alpha=1.0, tau=1.0, seed=1005, batch=4, seq=8192),
    "paper3b_heads": Workload("paper3b_heads", 3, 4096, (1024, 2304, 4352), 49152, "bf16",
                              alpha=0.3, tau=1.0, seed=1006, batch=2, seq=2048),
}

HEADLINE = "c2_m3_v50k"


def make_inputs(wl: Workload, device="cpu", seed: Optional[int] = None):
    """Draw ``(h_list, W_list, labels)`` for a workload on ``device``.

    Draw order from one generator: h_0..h_{M-1}, W_0..W_{M-1}, labels,
    ignore mask. Values are drawn in float32 and rounded to the workload dtype.
    """
    g = torch.Generator(device=device)
    g.manual_seed(wl.seed if seed is None else seed)
    dt = wl.torch_dtype
    hs = []
    for d in wl.dims:
        hs.append(torch.randn(wl.T, d, generator=g, device=device, dtype=torch.float32).to(dt))
    Ws = []
    for d in wl.dims:
        std = (1.0 / math.sqrt(d)) if wl.w_std is None else wl.w_std
        w = torch.randn(wl.V, d, generator=g, device=device, dtype=torch.float32)
        w.mul_(std * wl.w_scale)
        Ws.append(w.to(dt))
        del w
    labels = torch.randint(0, wl.V, (wl.T,), generator=g, device=device, dtype=torch.int64)
    if wl.ignore_frac > 0:
        drop = torch.rand(wl.T, generator=g, device=device) < wl.ignore_frac
        labels = torch.where(drop, torch.full_like(labels, IGNORE_INDEX), labels)
    return hs, Ws, labels


def custom(M: int, T: int, dims: Sequence[int], V: int, dtype="bf16", **kw) -> Workload:
    """A workload of arbitrary shape (for parity tests below full size)."""
    return Workload(kw.pop("name", f"custom_m{M}_t{T}_v{V}"), M, T, tuple(dims), V, dtype, **kw)


# ---------------------------------------------------------------------------
# inter-model junction inputs
# ---------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class JunctionWorkload:
    """Inputs of the junctions between consecutive sub-models of one suite.

    Junction m joins sub-model m (output width ``dims[m]``) and m+1 (fresh
    embedding width ``dims[m+1] - dims[m]``). Sub-model outputs are drawn
    N(0, o_std^2) and fresh embeddings N(0, e_std^2): transformer outputs have
    much larger norms than input embeddings (the mismatch the junction's
    rescaling addresses). Upstream gradients are N(0, g_std^2).
    """

    name: str
    T: int
    dims: Tuple[int, ...]
    act_dtype: str = "bf16"
    grad_dtype: str = "f32"
    o_std: float = 8.0
    e_std: float = 0.02
    g_std: float = 1e-3
    seed: int = 0

    @property
    def junctions(self):
        return [(self.dims[m], self.dims[m + 1] - self.dims[m]) for m in range(len(self.dims) - 1)]


JUNCTIONS = {
    "c2_junctions": JunctionWorkload("c2_junctions", 4096, (1024, 2048, 3072), seed=2002),
    "c5_junctions": JunctionWorkload("c5_junctions", 32768, (1536, 3072, 4608), seed=2005),
    "paper3b_junctions": JunctionWorkload("paper3b_junctions", 4096, (1024, 2304, 4352), seed=2006),
}


def _dt(name):
    return torch.bfloat16 if name == "bf16" else torch.float32


def make_junction_inputs(wl: JunctionWorkload, m: int, device="cpu", seed: Optional[int] = None,
                         T: Optional[int] = None):
    """``(o, e, g_x)`` of junction ``m``; draw order o, e, g_x from one generator."""
    d_prev, d_fresh = wl.junctions[m]
    T = wl.T if T is None else T
    g = torch.Generator(device=device)
    g.manual_seed((wl.seed if seed is None else seed) * 16 + m)
    o = (torch.randn(T, d_prev, generator=g, device=device) * wl.o_std).to(_dt(wl.act_dtype))
    e = (torch.randn(T, d_fresh, generator=g, device=device) * wl.e_std).to(_dt(wl.act_dtype))
    gx = (torch.randn(T, d_prev + d_fresh, generator=g, device=device) * wl.g_std).to(
        _dt(wl.grad_dtype))
    return o, e, gx


# ---------------------------------------------------------------------------
# speculative-decoding head step inputs
# ---------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class DecodeWorkload:
    """One decoding step of a draft / verifier pair (section 3, "Speculative
    Decoding Throughput": a 500M draft and the 3B verifier, batches of up to 102
    sequences, draft length gamma, nucleus 0.9 at temperature 0.4).

    The draft's head and hidden states are the leading ``d_draft`` columns of
    the verifier's (nested sub-models share their leading parameters). The
    verifier's hidden states are N(0, o_std^2) on those columns and
    N(0, (tail_scale * o_std)^2) on the rest, and the draft's are the verifier's
    leading columns plus N(0, (draft_noise * o_std)^2): the draft then agrees
    with its verifier about as a distilled draft does (per-token acceptance
    around 0.7 at temperature 0.4, nuclei of tens of tokens). Heads are
    N(0, w_std^2).
    """

    name: str
    batch: int
    gamma: int
    V: int
    d_draft: int
    d_target: int
    temperature: float = 0.4
    top_p: float = 0.9
    o_std: float = 3.0
    tail_scale: float = 0.15
    draft_noise: float = 0.05
    w_std: float = 0.02
    seed: int = 0


DECODE = {
    "spec_500m_3b": DecodeWorkload("spec_500m_3b", 102, 6, 49152, 1024, 4352, seed=3001),
    "spec_vanilla_b64": DecodeWorkload("spec_vanilla_b64", 64, 6, 49152, 1024, 4352, seed=3002),
}


def make_decode_inputs(wl: DecodeWorkload, device="cpu", seed: Optional[int] = None):
    """Dict of bf16 heads / hidden states and fp32 uniforms for one step.

    Draw order from one generator: W_target, o_target (rows [batch * (gamma + 1)],
    sequence-major), the draft's hidden-state noise (rows [gamma * batch],
    step-major), uniforms of the draft draws [gamma, batch], of the acceptance
    tests [batch, gamma] and of the final draws [batch]. The draft's hidden
    state at (step k, sequence b) is the leading d_draft columns of the
    verifier's at the same position plus the noise.
    """
    g = torch.Generator(device=device)
    g.manual_seed(wl.seed if seed is None else seed)
    B, G = wl.batch, wl.gamma
    Wt = (torch.randn(wl.V, wl.d_target, generator=g, device=device) * wl.w_std).to(torch.bfloat16)
    ot = torch.randn(B * (G + 1), wl.d_target, generator=g, device=device) * wl.o_std
    ot[:, wl.d_draft:] *= wl.tail_scale
    ot = ot.to(torch.bfloat16)
    noise = torch.randn(G * B, wl.d_draft, generator=g, device=device) * (wl.o_std * wl.draft_noise)
    pos = (torch.arange(B, device=device)[None, :] * (G + 1) + torch.arange(G, device=device)[:, None])
    od = (ot[pos.reshape(-1), :wl.d_draft].float() + noise).to(torch.bfloat16)
    u_draft = torch.rand(G, B, generator=g, device=device)
    u_accept = torch.rand(B, G, generator=g, device=device)
    u_sample = torch.rand(B, generator=g, device=device)
    return {"W_target": Wt, "W_draft": Wt[:, :wl.d_draft].contiguous(), "o_target": ot,
            "o_draft": od, "u_draft": u_draft, "u_accept": u_accept, "u_sample": u_sample}
