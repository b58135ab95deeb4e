"""mls_spec_verify_noalloc (static per-device scratch, no workspace) gives the
same results as mls_spec_verify with a caller workspace, bit for bit, on two
calls in a row, the second with a smaller problem, sampled and greedy, with and
without the draft's distribution records."""

import numpy as np
import pytest
import torch

from paper_2608_09703_amd import api as D
from paper_2608_09703_amd import binding as B
from paper_2608_09703_amd import workloads as WL

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _inputs(Bt, G, V, seed):
    wl = WL.DecodeWorkload("t", Bt, G, V, 128, 256, seed=seed)
    x = WL.make_decode_inputs(wl, device=DEV)
    tl = (x["o_target"].float() @ x["W_target"].float().T).reshape(Bt, G + 1, V).contiguous()
    dl = (x["o_draft"].float() @ x["W_draft"].float().T).reshape(G, Bt, V).contiguous()
    return x, dl, tl


def _both(Bt, G, V, seed, temperature, top_p, greedy, with_params):
    x, dl, tl = _inputs(Bt, G, V, seed)
    st = torch.cuda.current_stream(DEV).cuda_stream
    samp = B.make_sampling(V, temperature, top_p, greedy)
    tok = torch.empty(G, Bt, dtype=torch.int32, device=DEV)
    rec = torch.empty(max(G, 1) * Bt * B.ROW_PARAMS_BYTES, dtype=torch.uint8, device=DEV)
    for k in range(G):  # drafted tokens (and their records) from the library's sampler
        B.sample(samp, Bt, dl[k].data_ptr(), x["u_draft"][k].data_ptr(), tok[k].data_ptr(), st,
                 params=None if greedy else rec.data_ptr() + k * Bt * B.ROW_PARAMS_BYTES)
    ua = x["u_accept"].t().contiguous()  # [gamma][batch], drafting order
    us = x["u_sample"].contiguous()
    dparams = rec if (with_params and not greedy and G > 0) else None
    n_ref, x_ref = D.spec_verify(dl if G > 0 else None, tl, tok if G > 0 else None,
                                 ua if G > 0 else None, us, temperature=temperature, top_p=top_p,
                                 greedy=greedy, draft_params=dparams)
    n_acc = torch.full((Bt,), -7, dtype=torch.int32, device=DEV)
    nxt = torch.full((Bt,), -7, dtype=torch.int32, device=DEV)
    ptr = (lambda t: t.data_ptr() if t is not None else None)
    B.spec_verify_noalloc(samp, Bt, G, ptr(dl) if G > 0 else None, tl.data_ptr(),
                          ptr(tok) if G > 0 else None, ptr(ua) if G > 0 else None, us.data_ptr(),
                          n_acc.data_ptr(), nxt.data_ptr(), st, draft_params=ptr(dparams))
    torch.cuda.synchronize()
    return (n_ref.cpu().numpy(), x_ref.cpu().numpy()), (n_acc.cpu().numpy(), nxt.cpu().numpy())


@pytest.mark.parametrize("greedy,with_params", [(False, False), (False, True), (True, False)],
                         ids=["sampled", "sampled_draft_records", "greedy"])
def test_noalloc_matches_workspace_entry_point(greedy, with_params):
    # the first call fills more of the static scratch than the second one reads
    for Bt, G, V, seed in ((102, 6, 4096, 5), (13, 2, 1500, 9)):
        print(f"[noalloc] batch={Bt} gamma={G} V={V} greedy={greedy} records={with_params}",
              flush=True)
        (n_ref, x_ref), (n_got, x_got) = _both(Bt, G, V, seed, 0.4, 0.9, greedy, with_params)
        np.testing.assert_array_equal(n_got, n_ref)
        np.testing.assert_array_equal(x_got, x_ref)
        assert (n_got >= 0).all() and (n_got <= G).all() and (x_got >= 0).all() and (x_got < V).all()


def test_noalloc_rejects_problems_beyond_the_scratch():
    Bt, G = 70000, 6  # 70000 * 13 records of 20 bytes: beyond 2 MiB
    assert B.spec_verify_workspace(Bt, G) > B.SPEC_VERIFY_STATIC_BYTES
    samp = B.make_sampling(1000, 0.4, 0.9, False)
    with pytest.raises(B.MlsError) as e:
        B.spec_verify_noalloc(samp, Bt, G, 1 << 40, 1 << 40, 1 << 40, 1 << 40, 1 << 40,
                              1 << 40, 1 << 40, None)
    assert e.value.status == B.MLS_INVALID_ARG
