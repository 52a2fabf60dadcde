"""efq_attn_fwd_noalloc (the entry point that allocates nothing) against
efq_attn_fwd_ex with a caller workspace, through the C ABI on the GPU: the
same kernels on the same inputs, so the outputs must be identical; two calls
in a row, the second with a smaller input (the scratch array keeps the
first call's contents), then a shape whose V~ exceeds the scratch array,
which must be rejected before anything runs."""
import ctypes

import pytest
import torch

from paper_2609_09721_amd import inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    from paper_2609_09721_amd import binding
    binding.lib()
    assert torch.cuda.is_available(), "no GPU"
    return binding


def _ref(B, q, k, v, w, kind):
    sh = B.shape_of(q, k)
    ws = torch.empty(B.vhat_bytes(sh), dtype=torch.uint8, device=q.device)
    return B.attn_fwd(q, k, v, w.scale, w.causal, kind, workspace=ws)


@pytest.mark.parametrize("kind", ["efq", "expq"])
def test_noalloc_matches_workspace_entry_point(B, kind):
    dev = torch.device("cuda:0")
    big = inputs.Workload("na1", 1, 8, 2, 2000, 128, True, "qwen", 71)
    small = inputs.Workload("na2", 1, 4, 1, 300, 64, False, "normal", 72)
    for w in (big, small):
        print(f"[noalloc] {kind} {w}", flush=True)
        q, k, v = inputs.make_qkv(w, device=dev)
        out = torch.empty(q.shape, dtype=torch.float32, device=dev)
        B.attn_fwd_noalloc(q, k, v, out, w.scale, w.causal, kind)
        ref = _ref(B, q, k, v, w, kind)
        torch.cuda.synchronize()
        assert torch.equal(out, ref), (kind, w.name, float((out - ref).abs().max()))


def test_noalloc_rejects_oversized_shapes(B):
    lib = B.lib()
    limit = 64 << 20
    sh = B.Shape(1, 131072, 131072, 32, 8, 128)
    assert B.vhat_bytes(sh) > limit
    fake = ctypes.c_void_p(4096)     # aligned, never dereferenced: rejected first
    rc = lib.efq_attn_fwd_noalloc(fake, fake, fake, 0.088, 1, 0, B.Params(-3.06, 2.3), fake,
                                  ctypes.byref(sh), None)
    assert rc == B.EFQ_EWORKSPACE
    assert b"scratch" in lib.efq_strerror(rc)
