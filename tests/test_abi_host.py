"""Host-side checks of the C ABI (no GPU needed).

The library loads without a GPU; every argument error is detected on the
host before any device call, so these calls never touch the device.
"""

import ctypes
import math
import os
import re

import numpy as np
import pytest

import oracle
from paper_2608_09703_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "mls.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(mls_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    L = B.lib()
    names = _declared_functions()
    assert set(names) == set(B.EXPORTED)
    for n in names:
        assert hasattr(L, n), n


def test_version_and_status_strings():
    assert "gfx950" in B.version()
    L = B.lib()
    assert L.mls_status_string(B.MLS_OK) == b"ok"
    assert L.mls_status_string(B.MLS_WORKSPACE_TOO_SMALL) == b"workspace too small"


@pytest.mark.parametrize("cname,cls", [("mls_problem", B.Problem), ("mls_junction", B.Junction),
                                       ("mls_sampling", B.Sampling)])
def test_struct_layout_matches_header(tmp_path, cname, cls):
    """The ctypes mirrors of the C structs have the C compiler's layout."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    fields = [f[0] for f in cls._fields_]
    prog = tmp_path / "layout.c"
    body = "".join(f'printf("%zu\\n", offsetof({cname}, {f}));' for f in fields)
    prog.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "mls.h"\n'
                    f'int main(void){{printf("%zu\\n", sizeof({cname}));' + body + 'return 0;}')
    exe = tmp_path / "layout"
    subprocess.run([cc, "-I", os.path.join(ROOT, "include"), str(prog), "-o", str(exe)], check=True)
    out = [int(x) for x in subprocess.run([str(exe)], capture_output=True, text=True,
                                          check=True).stdout.split()]
    assert out[0] == ctypes.sizeof(cls)
    for f, off in zip(fields, out[1:]):
        assert getattr(cls, f).offset == off, f


@pytest.mark.parametrize("mode", [B.MLS_MODE_PAPER, B.MLS_MODE_ADDITIVE])
@pytest.mark.parametrize("teacher", [-1, 0, 2])
def test_coeffs_match_oracle(mode, teacher):
    w = [0.5, 1.5, 2.0]
    g_ce, g_kl = B.coeffs(3, teacher, 0.3, 2.0, mode, w)
    o_ce, o_kl = oracle.coeffs(3, teacher, 0.3, 2.0, "paper" if mode == 0 else "additive", w)
    np.testing.assert_allclose(g_ce, o_ce, rtol=1e-6)
    np.testing.assert_allclose(g_kl, o_kl, rtol=1e-6)


def _fake_problem(**kw):
    M = kw.pop("M", 3)
    dims = kw.pop("dims", [1024, 2048, 3072][:M] + [64] * max(0, M - 3))
    base = 1 << 32  # fake, 256-aligned addresses; never dereferenced by these tests
    return B.make_problem(M, kw.pop("T", 4096), kw.pop("V", 50304), dims,
                          [base + 0x100000 * i for i in range(M)],
                          [base + 0x10000000 + 0x100000 * i for i in range(M)], base + 0x20000000,
                          **kw)


def test_query_sizes_reports_workspace_and_stats():
    p = _fake_problem()
    ws, st = B.query_sizes(p)
    M, T = 3, 4096
    assert st >= (4 * M * T + T) * 4 + 8
    assert ws >= M * 2 * ((50304 + 127) // 128) * T * 16  # forward partial rows, 2 per tile
    # the default backward plan splits the vocabulary (>= 4 chunks): its bf16
    # logit-gradient slab is far below a full [T, V] slab per sub-model
    assert ws < M * T * 50304 * 2 // 2
    p1 = _fake_problem(vocab_chunk=50304)  # an explicit single chunk is the caller's choice
    assert B.query_sizes(p1)[0] >= M * T * 50304 * 2



def test_wide_backward_operands_stay_below_4_gib():
    """The wide gradient GEMM addresses each M-contiguous operand with 32-bit
    offsets: the chunk width is capped so one [T_pad][V_c] slab stays below 4 GiB,
    and a T x d_i panel that would reach 4 GiB sends the backward to the general
    kernels (which then also keep transposed copies of h_i)."""
    T, V = 1 << 22, 4096
    # explicit whole-vocabulary chunk: an uncapped slab would take T * V * 2 = 32 GiB
    ws_wide, _ = B.query_sizes(_fake_problem(M=1, dims=[64], T=T, V=V, vocab_chunk=V))
    # the forward's and the diagnostics' records (64-bit indexed) are the larger needs here
    fwd = 2 * (V // 128) * T * 16 + T * 4
    diag = 2 * (V // 128) * T * 4 * 4 + T * 2 * 4
    assert ws_wide <= max((1 << 32) - 1, fwd, diag) + 512
    # widths that are not multiples of 64 take the general kernels: no cap there
    ws_gen, _ = B.query_sizes(_fake_problem(M=1, dims=[72], T=T, V=V, vocab_chunk=V))
    assert ws_gen >= 2 * T * V * 2
    # T * d * 2 = 8 GiB: general backward, whose h^T copy alone takes 8 GiB
    ws_big, _ = B.query_sizes(_fake_problem(M=1, dims=[1024], T=T, V=V))
    assert ws_big >= T * 1024 * 2
    ws_small, _ = B.query_sizes(_fake_problem(M=1, dims=[256], T=T, V=V))
    assert ws_small < T * 256 * 2 * 4

@pytest.mark.parametrize("field,value,status", [
    ("M", 0, B.MLS_INVALID_ARG),
    ("M", 9, B.MLS_INVALID_ARG),
    ("teacher", 3, B.MLS_INVALID_ARG),
    ("T", 0, B.MLS_INVALID_ARG),
    ("V", 1, B.MLS_INVALID_ARG),
    ("tau", 0.0, B.MLS_INVALID_ARG),
    ("tau", -1.0, B.MLS_INVALID_ARG),
    ("tau", math.inf, B.MLS_INVALID_ARG),
    ("alpha", math.nan, B.MLS_INVALID_ARG),
    ("alpha", 1.5, B.MLS_INVALID_ARG),
    ("in_dtype", 7, B.MLS_UNSUPPORTED),
    ("grad_h_dtype", 2, B.MLS_UNSUPPORTED),
    ("grad_h_dtype", -1, B.MLS_UNSUPPORTED),
    ("vocab_chunk", -5, B.MLS_INVALID_ARG),
    ("labels", None, B.MLS_INVALID_ARG),
])
def test_invalid_arguments_rejected_on_host(field, value, status):
    p = _fake_problem()
    setattr(p, field, value)
    ws = ctypes.c_size_t(0)
    st = ctypes.c_size_t(0)
    got = B.lib().mls_query_sizes(ctypes.byref(p), ctypes.byref(ws), ctypes.byref(st))
    assert got == status
    assert B.lib().mls_last_error() != b""


def test_width_granularity_and_alignment():
    p = _fake_problem(dims=[1024, 2048, 3070])
    with pytest.raises(B.MlsError) as e:
        B.query_sizes(p)
    assert e.value.status == B.MLS_UNSUPPORTED
    p = _fake_problem(dtype=B.MLS_F32, dims=[1024, 2048, 3068])
    B.query_sizes(p)  # fp32 needs only multiples of 4
    p = _fake_problem()
    p.h[1] = p.h[1] + 8
    with pytest.raises(B.MlsError) as e:
        B.query_sizes(p)
    assert e.value.status == B.MLS_INVALID_ARG
    p = _fake_problem()
    p.W[0] = None
    with pytest.raises(B.MlsError):
        B.query_sizes(p)


def test_forward_rejects_small_workspace_before_device_work():
    p = _fake_problem()
    ws, st = B.query_sizes(p)
    fake = 1 << 40
    with pytest.raises(B.MlsError) as e:
        B.distill_fwd(p, fake, fake + 4096, fake + 8192, None, fake + (1 << 20), 1024, None)
    assert e.value.status == B.MLS_WORKSPACE_TOO_SMALL
    with pytest.raises(B.MlsError) as e:
        B.distill_fwd(p, None, fake, fake, None, fake, ws, None)
    assert e.value.status == B.MLS_INVALID_ARG


def test_backward_rejects_bad_arguments_before_device_work():
    p = _fake_problem()
    ws, st = B.query_sizes(p)
    fake = 1 << 40
    grads = [fake + (1 << 30) * (i + 1) for i in range(3)]
    with pytest.raises(B.MlsError) as e:  # one coefficient vector without the other
        B.distill_bwd(p, fake, fake + 256, None, grads, grads, fake + (1 << 20), ws, None)
    assert e.value.status == B.MLS_INVALID_ARG
    with pytest.raises(B.MlsError) as e:
        B.distill_bwd(p, fake, None, None, grads, grads, fake + (1 << 20), 16, None)
    assert e.value.status == B.MLS_WORKSPACE_TOO_SMALL


def test_bf16_grad_h_keeps_fp32_partial_sums_over_chunks():
    """A bf16 grad_h over several vocabulary chunks needs fp32 partial sums of every
    sub-model's grad_h in the workspace (T * sum(d) * 4 bytes); in one chunk it does not."""
    M, T, dims = 3, 4096, [1024, 2048, 3072]
    f32 = B.query_sizes(_fake_problem())[0]
    b16 = B.query_sizes(_fake_problem(grad_h_dtype=B.MLS_BF16))[0]
    assert b16 - f32 >= T * sum(dims) * 4
    one = _fake_problem(vocab_chunk=50304)
    one_b16 = _fake_problem(vocab_chunk=50304, grad_h_dtype=B.MLS_BF16)
    assert B.query_sizes(one)[0] == B.query_sizes(one_b16)[0]


def test_bf16_grad_h_alignment_checked_on_host():
    p = _fake_problem(grad_h_dtype=B.MLS_BF16)
    ws, st = B.query_sizes(p)
    fake = 1 << 40
    gW = [fake + (1 << 30) * (i + 1) for i in range(3)]
    gh = [fake + (1 << 34) + (1 << 30) * i for i in range(3)]
    gh[2] += 1  # odd address: not even 2-byte aligned
    with pytest.raises(B.MlsError) as e:
        B.distill_bwd(p, fake, None, None, gh, gW, fake + (1 << 20), ws, None)
    assert e.value.status == B.MLS_INVALID_ARG


def test_device_error_rejects_null_outputs_before_device_work():
    p = _fake_problem()
    f = ctypes.c_int32(0)
    assert B.lib().mls_device_error(ctypes.byref(p), 1 << 40, None, None) == B.MLS_INVALID_ARG
    assert B.lib().mls_device_error(ctypes.byref(p), None, None, ctypes.byref(f)) == B.MLS_INVALID_ARG
    assert B.lib().mls_last_error() != b""
    bad = _fake_problem()
    bad.M = 0
    assert B.lib().mls_device_error(ctypes.byref(bad), 1 << 40, None,
                                    ctypes.byref(f)) == B.MLS_INVALID_ARG


def test_chunk_width_is_rounded():
    p = _fake_problem(vocab_chunk=1000)
    ws1, _ = B.query_sizes(p)
    p2 = _fake_problem(vocab_chunk=1024)
    ws2, _ = B.query_sizes(p2)
    assert ws1 == ws2


def test_diagnostics_reject_bad_arguments_before_device_work():
    fake = 1 << 40
    out = fake + (1 << 30)
    p = _fake_problem(M=8)  # accepted (passes over subsets), checked like any other call
    with pytest.raises(B.MlsError) as e:
        B.diagnostics(p, out, out + 256, None, fake + (1 << 20), 1024, None)
    assert e.value.status == B.MLS_WORKSPACE_TOO_SMALL
    p = _fake_problem()
    ws, _ = B.query_sizes(p)
    with pytest.raises(B.MlsError) as e:
        B.diagnostics(p, None, out, None, fake + (1 << 20), ws, None)
    assert e.value.status == B.MLS_INVALID_ARG
    with pytest.raises(B.MlsError) as e:
        B.diagnostics(p, out, out + 256, out + 513, fake + (1 << 20), ws, None)
    assert e.value.status == B.MLS_INVALID_ARG  # misaligned argmax
    with pytest.raises(B.MlsError) as e:
        B.diagnostics(p, out, out + 256, None, fake + (1 << 20), 16, None)
    assert e.value.status == B.MLS_WORKSPACE_TOO_SMALL


@pytest.mark.parametrize("field,value,status", [
    ("T", 0, B.MLS_INVALID_ARG),
    ("d_prev", 12, B.MLS_UNSUPPORTED),
    ("d_fresh", 0, B.MLS_UNSUPPORTED),
    ("d_prev", 8200, B.MLS_UNSUPPORTED),
    ("act_dtype", 5, B.MLS_UNSUPPORTED),
    ("grad_dtype", 5, B.MLS_UNSUPPORTED),
    ("layout", 2, B.MLS_INVALID_ARG),
    ("flags", 4, B.MLS_INVALID_ARG),
])
def test_junction_rejects_bad_descriptors_before_device_work(field, value, status):
    j = B.make_junction(4096, 1024, 1024)
    setattr(j, field, value)
    fake = 1 << 40
    with pytest.raises(B.MlsError) as e:
        B.junction_fwd(j, fake, fake + (1 << 30), fake + (2 << 30), None)
    assert e.value.status == status
    with pytest.raises(B.MlsError) as e:
        B.junction_bwd(j, fake, fake + (1 << 30), fake + (2 << 30), fake + (3 << 30),
                       fake + (4 << 30), None)
    assert e.value.status == status


def test_junction_rejects_bad_pointers_before_device_work():
    j = B.make_junction(4096, 1024, 1024)
    fake = 1 << 40
    with pytest.raises(B.MlsError) as e:  # misaligned
        B.junction_fwd(j, fake + 8, fake + (1 << 30), fake + (2 << 30), None)
    assert e.value.status == B.MLS_INVALID_ARG
    with pytest.raises(B.MlsError) as e:  # x overlapping o
        B.junction_fwd(j, fake, fake + (1 << 30), fake + 4096, None)
    assert e.value.status == B.MLS_INVALID_ARG
    with pytest.raises(B.MlsError) as e:  # g_o overlapping g_x
        B.junction_bwd(j, fake, fake + (1 << 30), fake + (2 << 30), fake + (2 << 30) + 256,
                       fake + (4 << 30), None)
    assert e.value.status == B.MLS_INVALID_ARG
    with pytest.raises(B.MlsError) as e:
        B.junction_bwd(j, fake, None, fake + (2 << 30), fake + (3 << 30), fake + (4 << 30), None)
    assert e.value.status == B.MLS_INVALID_ARG


@pytest.mark.parametrize("field,value,status", [
    ("V", 1, B.MLS_UNSUPPORTED),
    ("V", 65537, B.MLS_UNSUPPORTED),
    ("temperature", 0.0, B.MLS_INVALID_ARG),
    ("temperature", math.inf, B.MLS_INVALID_ARG),
    ("top_p", 0.0, B.MLS_INVALID_ARG),
    ("top_p", 1.5, B.MLS_INVALID_ARG),
    ("reserved", 1, B.MLS_INVALID_ARG),
])
def test_sampling_rejects_bad_descriptors_before_device_work(field, value, status):
    s = B.make_sampling(49152, 0.4, 0.9)
    setattr(s, field, value)
    fake = 1 << 40
    with pytest.raises(B.MlsError) as e:
        B.sample(s, 102, fake, fake + (1 << 30), fake + (2 << 30), None)
    assert e.value.status == status
    ws = B.spec_verify_workspace(102, 6)
    with pytest.raises(B.MlsError) as e:
        B.spec_verify(s, 102, 6, fake, fake + (1 << 32), fake + (2 << 32), fake + (3 << 32),
                      fake + (4 << 32), fake + (5 << 32), fake + (6 << 32), fake + (7 << 32), ws,
                      None)
    assert e.value.status == status


def test_decode_entry_points_reject_bad_arguments_before_device_work():
    fake = 1 << 40
    s = B.make_sampling(49152, 0.4, 0.9)
    with pytest.raises(B.MlsError) as e:  # sampling without uniforms
        B.sample(s, 4, fake, None, fake + 4096, None)
    assert e.value.status == B.MLS_INVALID_ARG
    with pytest.raises(B.MlsError) as e:  # misaligned distribution records
        B.sample(s, 4, fake, fake + 8192, fake + 4096, None, params=fake + 16386)
    assert e.value.status == B.MLS_INVALID_ARG
    assert B.ROW_PARAMS_BYTES == 20
    with pytest.raises(B.MlsError) as e:  # misaligned draft records
        B.spec_verify(s, 8, 6, fake, fake + (1 << 32), fake + (2 << 32), fake + (3 << 32),
                      fake + (4 << 32), fake + (5 << 32), fake + (6 << 32), fake + (7 << 32),
                      B.spec_verify_workspace(8, 6), None, draft_params=fake + (8 << 32) + 2)
    assert e.value.status == B.MLS_INVALID_ARG
    ws = B.spec_verify_workspace(8, 6)
    assert ws >= (8 * 6 + 8 * 7) * 20
    with pytest.raises(B.MlsError) as e:
        B.spec_verify(s, 8, 6, fake, fake + (1 << 32), fake + (2 << 32), fake + (3 << 32),
                      fake + (4 << 32), fake + (5 << 32), fake + (6 << 32), fake + (7 << 32), 64,
                      None)
    assert e.value.status == B.MLS_WORKSPACE_TOO_SMALL
    with pytest.raises(B.MlsError) as e:  # drafts without their logits
        B.spec_verify(s, 8, 6, None, fake + (1 << 32), fake + (2 << 32), fake + (3 << 32),
                      fake + (4 << 32), fake + (5 << 32), fake + (6 << 32), fake + (7 << 32), ws,
                      None)
    assert e.value.status == B.MLS_INVALID_ARG
    with pytest.raises(B.MlsError) as e:
        B.head_logits(102, 49152, 1030, B.MLS_BF16, fake, fake + (1 << 32), fake + (2 << 32), None)
    assert e.value.status == B.MLS_UNSUPPORTED
    with pytest.raises(B.MlsError) as e:
        B.head_logits(102, 49152, 1024, B.MLS_BF16, fake + 8, fake + (1 << 32), fake + (2 << 32),
                      None)
    assert e.value.status == B.MLS_INVALID_ARG


def test_fused_plan_never_holds_a_full_logit_array():
    """mls_distill_fwd_bwd stores logits one token chunk at a time: at least two
    chunks, each sub-model's fp16 chunk below 4 GiB, all of them within 16 GiB."""
    for (M, T, dims, V) in [(3, 4096, [1024, 2048, 3072], 50304),
                            (3, 8192, [1024, 2048, 3072], 128256),
                            (4, 16384, [512, 1024, 2048, 4096], 128256),
                            (3, 32768, [1536, 3072, 4608], 262144)]:
        p = _fake_problem(M=M, T=T, dims=dims, V=V)
        ws = B.query_fwd_bwd_workspace(p)
        V_pad = (V + 127) // 128 * 128
        full = M * T * V_pad * 2
        assert ws < full // 2 + (1 << 30), (T, V, ws)
        tc_max = ((1 << 32) - 1) // (V_pad * 2) // 128 * 128
        assert ws >= M * min(tc_max, (T + 1) // 2) * V_pad * 2 * 0.9 or ws >= (1 << 30)
        assert ws <= (16 << 30) + (2 << 30)
    # one 128-token tile: the forward and the recomputing backward
    p = _fake_problem(M=2, T=100, dims=[64, 128], V=1000)
    assert B.query_fwd_bwd_workspace(p) <= B.query_sizes(p)[0]
