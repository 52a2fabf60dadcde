"""The C-ABI library loads, exports what include/efq_attn.h declares, and
rejects invalid arguments before touching HIP (CPU-only: no kernel runs)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "efq_attn.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(efq_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def L():
    from paper_2609_09721_amd import binding
    if not os.path.exists(binding.LIB_PATH):
        pytest.fail("libefq_attn.so is not built (run __graft_entry__.build())")
    return binding


def test_exports_every_declared_symbol(L):
    names = declared_functions()
    assert len(names) >= 12
    lib = ctypes.CDLL(L.LIB_PATH)
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing
    assert set(L.SIGNATURES) == set(names)


def test_abi_version(L):
    assert L.lib().efq_abi_version() == 1


FAKE = ctypes.c_void_p(4096)   # aligned, never dereferenced: validation fails first


def shape(**kw):
    d = dict(batch=1, seq_q=256, seq_k=256, heads_q=2, heads_kv=1, head_dim=64)
    d.update(kw)
    return L_shape(**d)


def L_shape(**d):
    from paper_2609_09721_amd.binding import Shape
    return Shape(d["batch"], d["seq_q"], d["seq_k"], d["heads_q"], d["heads_kv"], d["head_dim"])


def call_vhat(L, s, q=FAKE, k=FAKE, vh=FAKE, n=None, scale=0.125, causal=0, kind=0,
              params=(-3.06, 2.3), out=FAKE):
    lib = L.lib()
    n = lib.efq_vhat_bytes(ctypes.byref(s)) if n is None else n
    return lib.efq_attn_fwd_vhat(q, k, vh, n, scale, causal, kind, L.Params(*params), out,
                                 ctypes.byref(s), None)


def test_workspace_size_formula(L):
    s = shape(seq_k=75, heads_q=6, heads_kv=3, head_dim=128, batch=2)
    nb = 2 * ((75 + 63) // 64)
    codes = 2 * 3 * nb * 128 * 16
    off = (codes + 255) // 256 * 256
    assert L.vhat_scale_offset(s) == off
    assert L.vhat_bytes(s) == off + (2 * 3 * nb * 128 + 255) // 256 * 256
    assert L.lib().efq_attn_workspace_bytes(ctypes.byref(s)) == L.vhat_bytes(s)
    bad = shape(head_dim=96)
    assert L.vhat_bytes(bad) == 0


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=96), -2),
    (dict(head_dim=0), -1),
    (dict(heads_q=3, heads_kv=2), -1),
    (dict(seq_q=0), -1),
    (dict(batch=-1), -1),
])
def test_bad_shapes(L, kw, status):
    assert call_vhat(L, shape(**kw), n=1 << 30) == status
    msg = L.lib().efq_strerror(status).decode()
    assert msg and msg != "ok"


def test_bad_arguments(L):
    s = shape()
    assert call_vhat(L, s, q=None) == L.EFQ_EINVAL
    assert call_vhat(L, s, out=ctypes.c_void_p(4100)) == L.EFQ_EINVAL      # misaligned
    assert call_vhat(L, s, n=16) == L.EFQ_EWORKSPACE
    assert call_vhat(L, s, kind=7) == L.EFQ_EINVAL
    assert call_vhat(L, s, params=(-3.0, 0.0)) == L.EFQ_EINVAL
    assert call_vhat(L, s, params=(float("nan"), 2.0)) == L.EFQ_EINVAL
    assert call_vhat(L, s, scale=0.0) == L.EFQ_EINVAL
    assert call_vhat(L, shape(seq_q=100, seq_k=200), causal=1) == L.EFQ_EUNSUPPORTED
    lib = L.lib()
    assert lib.efq_pgen(FAKE, 0, 64, 0, L.Params(-3.06, 2.3), FAKE, FAKE, None) == L.EFQ_EINVAL
    assert lib.efq_pgen(FAKE, 4, 64, 3, L.Params(-3.06, 2.3), FAKE, FAKE, None) == L.EFQ_EINVAL
    assert lib.efq_pgen_bench(0, L.Params(-3.06, 2.3), 0, 10, FAKE, None) == L.EFQ_EINVAL
    assert lib.efq_clock_probe(0, 10, FAKE, None) == L.EFQ_EINVAL
    assert lib.efq_clock_probe(65536, 10, FAKE, None) == L.EFQ_EINVAL
    assert lib.efq_clock_probe(4, 0, FAKE, None) == L.EFQ_EINVAL
    assert lib.efq_clock_probe(4, (1 << 20) + 1, FAKE, None) == L.EFQ_EINVAL
    assert lib.efq_clock_probe(4, 10, None, None) == L.EFQ_EINVAL
    assert lib.efq_quant_v_mxfp4(FAKE, ctypes.byref(s), FAKE, 8, None) == L.EFQ_EWORKSPACE
    assert lib.efq_attn_fwd_ex(FAKE, FAKE, FAKE, 0.125, 0, 0, L.Params(-3.06, 2.3), FAKE,
                               ctypes.byref(s), None, 64, None) == L.EFQ_EWORKSPACE


def test_calibrate_arguments(L):
    """Alg. 3 entry point: every argument error is reported before any HIP call."""
    import numpy as np
    s = shape()
    lib = L.lib()
    taus = np.array([-3.06, -2.9], np.float32)
    hs = np.array([2.3, 2.0], np.float32)
    T = taus.ctypes.data_as(ctypes.c_void_p)
    H = hs.ctypes.data_as(ctypes.c_void_p)
    best = L.Params(0, 0)
    need = lib.efq_calibrate_workspace_bytes(ctypes.byref(s), 4)
    assert need > L.vhat_bytes(s)
    assert lib.efq_calibrate_workspace_bytes(ctypes.byref(s), 0) == 0

    def cal(q=FAKE, oref=FAKE, t=T, nt=2, h=H, nh=2, b=ctypes.byref(best), ws=None, nbytes=0):
        return lib.efq_calibrate(q, FAKE, FAKE, 0.125, 0, oref, ctypes.byref(s), t, nt, h, nh,
                                 None, b, ws, nbytes, None)
    assert cal(q=None) == L.EFQ_EINVAL
    assert cal(oref=None) == L.EFQ_EINVAL
    assert cal(b=None) == L.EFQ_EINVAL
    assert cal(nt=0) == L.EFQ_EINVAL
    bad = np.array([2.3, 0.0], np.float32)
    assert cal(h=bad.ctypes.data_as(ctypes.c_void_p)) == L.EFQ_EINVAL
    assert cal(ws=FAKE, nbytes=need - 1) == L.EFQ_EWORKSPACE


def test_valid_call_without_gpu_reports_hip_error(L):
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present: the GPU tests cover valid calls")
    assert call_vhat(L, shape()) == L.EFQ_EHIP
    assert "hip" in L.lib().efq_strerror(L.EFQ_EHIP).decode().lower()


def test_lowbit_sizes(L):
    """Q^ / K^ layout sizes: rows padded to 64 per (batch, head), codes then
    scales, each part a multiple of 256 bytes."""
    lib = L.lib()
    s = shape(batch=2, seq_q=75, seq_k=130, heads_q=6, heads_kv=3, head_dim=128)
    r256 = lambda n: (n + 255) // 256 * 256
    rq, rk = 2 * 6 * 128, 2 * 3 * 192
    assert lib.efq_qhat_scale_offset(ctypes.byref(s)) == r256(rq * 128)
    assert lib.efq_qhat_bytes(ctypes.byref(s)) == r256(rq * 128) + r256(rq * 4)
    assert lib.efq_khat_scale_offset(ctypes.byref(s)) == r256(rk * 128)
    assert lib.efq_khat_bytes(ctypes.byref(s)) == r256(rk * 128) + r256(rk * 4)
    assert lib.efq_attn_lowbit_workspace_bytes(ctypes.byref(s)) == (
        lib.efq_qhat_bytes(ctypes.byref(s)) + lib.efq_khat_bytes(ctypes.byref(s)) + L.vhat_bytes(s))
    assert lib.efq_qhat_bytes(ctypes.byref(shape(head_dim=96))) == 0


def test_lowbit_arguments(L):
    lib = L.lib()
    s = shape()
    nq, nk, nv = (lib.efq_qhat_bytes(ctypes.byref(s)), lib.efq_khat_bytes(ctypes.byref(s)),
                  L.vhat_bytes(s))
    P = L.Params(-3.06, 2.3)

    def qk8(qh=FAKE, a=nq, kh=FAKE, b=nk, c=nv, kind=0, causal=0, sh=s, scale=0.125):
        return lib.efq_attn_fwd_qk8(qh, a, kh, b, FAKE, c, scale, causal, kind, P, FAKE,
                                    ctypes.byref(sh), None)
    assert qk8(qh=None) == L.EFQ_EINVAL
    assert qk8(kh=ctypes.c_void_p(4104)) == L.EFQ_EINVAL
    assert qk8(a=nq - 1) == L.EFQ_EWORKSPACE
    assert qk8(b=nk - 1) == L.EFQ_EWORKSPACE
    assert qk8(c=nv - 1) == L.EFQ_EWORKSPACE
    assert qk8(kind=9) == L.EFQ_EINVAL
    assert qk8(scale=-1.0) == L.EFQ_EINVAL
    assert qk8(sh=shape(seq_q=100, seq_k=200), causal=1) == L.EFQ_EUNSUPPORTED
    assert lib.efq_attn_fwd_qk8_dump(FAKE, nq, FAKE, nk, FAKE, nv, 0.125, 0, 3, P, FAKE,
                                     ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, None) == L.EFQ_EINVAL
    assert lib.efq_attn_fwd_qk8_dump(FAKE, nq, FAKE, nk, FAKE, nv, 0.125, 0, 0, P, FAKE,
                                     ctypes.byref(s), None, FAKE, FAKE, FAKE, None) == L.EFQ_EINVAL
    assert lib.efq_quant_qk_mxfp8(FAKE, FAKE, ctypes.byref(s), FAKE, nq, FAKE, nk - 1,
                                  None) == L.EFQ_EWORKSPACE
    assert lib.efq_quant_qk_mxfp8(FAKE, None, ctypes.byref(s), FAKE, nq, FAKE, nk,
                                  None) == L.EFQ_EINVAL
    ex = lambda ws, n: lib.efq_attn_fwd_lowbit_ex(FAKE, FAKE, FAKE, 0.125, 0, 0, P, FAKE,
                                                  ctypes.byref(s), ws, n, None)
    need = lib.efq_attn_lowbit_workspace_bytes(ctypes.byref(s))
    assert ex(FAKE, need - 1) == L.EFQ_EWORKSPACE
    assert ex(ctypes.c_void_p(4096 + 16), need) == L.EFQ_EINVAL   # not 256-byte aligned
