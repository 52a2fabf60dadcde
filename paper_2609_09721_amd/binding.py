"""ctypes binding of libefq_attn.so (argument marshalling only).

Every computation runs in the HIP kernels of ``csrc/efq_attn.hip``; torch
provides device memory and the current stream.  The functions mirror the C
entry points of ``include/efq_attn.h``.  If the library is missing this
module raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libefq_attn.so")

PGEN_EFQ, PGEN_EXPQ, PGEN_LUT, PGEN_NOOP, PGEN_EXPQ6 = 0, 1, 2, 3, 4
KINDS = {"efq": PGEN_EFQ, "expq": PGEN_EXPQ, "lut": PGEN_LUT, "noop": PGEN_NOOP,
         "expq6": PGEN_EXPQ6}

# (tau, h) operating points of Sec. IV-A, and the LUT constants of Sec. II-D
PARAMS_MEAN = (-3.06, 2.30)
PARAMS_MMLU = (-2.90, 2.00)
PARAMS_BALANCE = (-2.10, 2.70)
PARAMS_LUT = (-3.17805383, 4.40521173)

EFQ_OK, EFQ_EINVAL, EFQ_EUNSUPPORTED, EFQ_EWORKSPACE, EFQ_EHIP = 0, -1, -2, -3, -4


class EfqError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"efq status {status}: {msg}")
        self.status = status


class Shape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int), ("seq_q", ctypes.c_int), ("seq_k", ctypes.c_int),
                ("heads_q", ctypes.c_int), ("heads_kv", ctypes.c_int), ("head_dim", ctypes.c_int)]


class Params(ctypes.Structure):
    _fields_ = [("tau", ctypes.c_float), ("h", ctypes.c_float)]


_lib = None
P = ctypes.c_void_p
SZ = ctypes.c_size_t
I = ctypes.c_int
F = ctypes.c_float
SP = ctypes.POINTER(Shape)

SIGNATURES = {
    "efq_abi_version": ([], I),
    "efq_strerror": ([I], ctypes.c_char_p),
    "efq_vhat_bytes": ([SP], SZ),
    "efq_vhat_scale_offset": ([SP], SZ),
    "efq_attn_workspace_bytes": ([SP], SZ),
    "efq_quant_v_mxfp4": ([P, SP, P, SZ, P], I),
    "efq_attn_fwd_vhat": ([P, P, P, SZ, F, I, I, Params, P, SP, P], I),
    "efq_attn_fwd_ex": ([P, P, P, F, I, I, Params, P, SP, P, SZ, P], I),
    "efq_attn_fwd": ([P, P, P, F, I, P, SP, P], I),
    "efq_attn_fwd_noalloc": ([P, P, P, F, I, I, Params, P, SP, P], I),
    "efq_attn_fwd_expq": ([P, P, P, F, I, P, SP, P], I),
    "efq_pgen": ([P, I, I, I, Params, P, P, P], I),
    "efq_attn_fwd_dump": ([P, P, P, SZ, F, I, I, Params, P, SP, P, P, P, P, P], I),
    "efq_pgen_bench": ([I, Params, I, I, P, P], I),
    "efq_clock_probe": ([I, I, P, P], I),
    "efq_calibrate_workspace_bytes": ([SP, I], SZ),
    "efq_calibrate": ([P, P, P, F, I, P, SP, P, I, P, I, P, ctypes.POINTER(Params), P, SZ, P], I),
    "efq_qhat_bytes": ([SP], SZ),
    "efq_qhat_scale_offset": ([SP], SZ),
    "efq_khat_bytes": ([SP], SZ),
    "efq_khat_scale_offset": ([SP], SZ),
    "efq_quant_qk_mxfp8": ([P, P, SP, P, SZ, P, SZ, P], I),
    "efq_attn_fwd_qk8": ([P, SZ, P, SZ, P, SZ, F, I, I, Params, P, SP, P], I),
    "efq_attn_fwd_qk8_dump": ([P, SZ, P, SZ, P, SZ, F, I, I, Params, P, SP, P, P, P, P, P], I),
    "efq_attn_lowbit_workspace_bytes": ([SP], SZ),
    "efq_attn_fwd_lowbit_ex": ([P, P, P, F, I, I, Params, P, SP, P, SZ, P], I),
}


def lib():
    """Load the HIP library (build it first with ``__graft_entry__.build()``)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build the HIP library first")
        L = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in SIGNATURES.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
    return _lib


def _check(status: int):
    if status != EFQ_OK:
        raise EfqError(status, lib().efq_strerror(status).decode())


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t: Optional[torch.Tensor]):
    return ctypes.c_void_p(0 if t is None else t.data_ptr())


def shape_of(q: torch.Tensor, k: torch.Tensor) -> Shape:
    B, Sq, Hq, D = q.shape
    Bk, Sk, Hkv, Dk = k.shape
    if B != Bk or D != Dk:
        raise ValueError("q and k shapes disagree")
    return Shape(B, Sq, Sk, Hq, Hkv, D)


def _params(kind: int, params) -> Params:
    if params is None:
        params = PARAMS_LUT if kind == PGEN_LUT else PARAMS_MEAN
    return Params(float(params[0]), float(params[1]))


def _kind(kind) -> int:
    return KINDS[kind] if isinstance(kind, str) else int(kind)


def _bf16(t: torch.Tensor, name: str):
    if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous bf16 CUDA tensor")


def vhat_bytes(shape: Shape) -> int:
    return int(lib().efq_vhat_bytes(ctypes.byref(shape)))


def vhat_scale_offset(shape: Shape) -> int:
    return int(lib().efq_vhat_scale_offset(ctypes.byref(shape)))


def quant_v(v: torch.Tensor, seq_q: int = 1, heads_q: Optional[int] = None,
            out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """V [B, S, Hkv, D] bf16 -> V~ byte buffer (layout in efq_attn.h)."""
    _bf16(v, "v")
    B, S, H, D = v.shape
    sh = Shape(B, seq_q, S, heads_q or H, H, D)
    n = vhat_bytes(sh)
    if out is None:
        out = torch.empty(n, dtype=torch.uint8, device=v.device)
    _check(lib().efq_quant_v_mxfp4(_ptr(v), ctypes.byref(sh), _ptr(out), out.numel(),
                                   _stream(stream)))
    return out


def attn_fwd_vhat(q, k, vhat, scale: Optional[float] = None, causal: bool = False, kind="efq",
                  params=None, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    _bf16(q, "q")
    _bf16(k, "k")
    sh = shape_of(q, k)
    kind = _kind(kind)
    if scale is None:
        scale = q.shape[-1] ** -0.5
    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    _check(lib().efq_attn_fwd_vhat(_ptr(q), _ptr(k), _ptr(vhat), vhat.numel(), float(scale),
                                   int(causal), kind, _params(kind, params), _ptr(out),
                                   ctypes.byref(sh), _stream(stream)))
    return out


def attn_fwd(q, k, v, scale: Optional[float] = None, causal: bool = False, kind="efq",
             params=None, out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
             stream=None) -> torch.Tensor:
    """O = attention(q, k, v) with the chosen probability stage (fp32 out)."""
    _bf16(q, "q")
    _bf16(k, "k")
    _bf16(v, "v")
    sh = shape_of(q, k)
    kind = _kind(kind)
    if scale is None:
        scale = q.shape[-1] ** -0.5
    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    ws_n = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().efq_attn_fwd_ex(_ptr(q), _ptr(k), _ptr(v), float(scale), int(causal), kind,
                                 _params(kind, params), _ptr(out), ctypes.byref(sh),
                                 _ptr(workspace), ws_n, _stream(stream)))
    return out


def attn_fwd_noalloc(q, k, v, out: torch.Tensor, scale: Optional[float] = None,
                     causal: bool = False, kind="efq", params=None, stream=None) -> torch.Tensor:
    """attn_fwd through the entry point that allocates nothing (V~ in the
    library's scratch array); out is the caller's fp32 BSHD tensor."""
    _bf16(q, "q")
    _bf16(k, "k")
    _bf16(v, "v")
    sh = shape_of(q, k)
    kind = _kind(kind)
    if scale is None:
        scale = q.shape[-1] ** -0.5
    _check(lib().efq_attn_fwd_noalloc(_ptr(q), _ptr(k), _ptr(v), float(scale), int(causal), kind,
                                      _params(kind, params), _ptr(out), ctypes.byref(sh),
                                      _stream(stream)))
    return out


def efq_attn_fwd(q, k, v, scale=None, causal=False, out=None, stream=None):
    """The method's entry point: EFQ-Softmax, Mean operating point."""
    sh = shape_of(q, k)
    scale = q.shape[-1] ** -0.5 if scale is None else scale
    out = torch.empty(q.shape, dtype=torch.float32, device=q.device) if out is None else out
    _check(lib().efq_attn_fwd(_ptr(q), _ptr(k), _ptr(v), float(scale), int(causal), _ptr(out),
                              ctypes.byref(sh), _stream(stream)))
    return out


def efq_attn_fwd_expq(q, k, v, scale=None, causal=False, out=None, stream=None):
    """The exp-then-quantize MXFP4 baseline."""
    sh = shape_of(q, k)
    scale = q.shape[-1] ** -0.5 if scale is None else scale
    out = torch.empty(q.shape, dtype=torch.float32, device=q.device) if out is None else out
    _check(lib().efq_attn_fwd_expq(_ptr(q), _ptr(k), _ptr(v), float(scale), int(causal),
                                   _ptr(out), ctypes.byref(sh), _stream(stream)))
    return out


def attn_fwd_dump(q, k, vhat, scale=None, causal=False, kind="efq", params=None, stream=None):
    """Attention plus the probability-stage record (codes unpacked per key)."""
    sh = shape_of(q, k)
    kind = _kind(kind)
    scale = q.shape[-1] ** -0.5 if scale is None else scale
    B, Sq, Hq, D = q.shape
    Sk = k.shape[1]
    nblk = (Sk + 31) // 32
    dev = q.device
    out = torch.empty(q.shape, dtype=torch.float32, device=dev)
    codes = torch.empty((B, Hq, Sq, nblk * 16), dtype=torch.uint8, device=dev)
    e8 = torch.empty((B, Hq, Sq, nblk), dtype=torch.uint8, device=dev)
    row_m = torch.empty((B, Hq, Sq), dtype=torch.float32, device=dev)
    row_l = torch.empty((B, Hq, Sq), dtype=torch.float32, device=dev)
    _check(lib().efq_attn_fwd_dump(_ptr(q), _ptr(k), _ptr(vhat), vhat.numel(), float(scale),
                                   int(causal), kind, _params(kind, params), _ptr(out),
                                   ctypes.byref(sh), _ptr(codes), _ptr(e8), _ptr(row_m),
                                   _ptr(row_l), _stream(stream)))
    return out, codes, e8, row_m, row_l



def quant_qk(q, k, stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Q, K (bf16 BSHD) -> the MXFP8 byte buffers Q^ and K^ (layout in efq_attn.h)."""
    _bf16(q, "q")
    _bf16(k, "k")
    sh = shape_of(q, k)
    qh = torch.empty(int(lib().efq_qhat_bytes(ctypes.byref(sh))), dtype=torch.uint8, device=q.device)
    kh = torch.empty(int(lib().efq_khat_bytes(ctypes.byref(sh))), dtype=torch.uint8, device=q.device)
    _check(lib().efq_quant_qk_mxfp8(_ptr(q), _ptr(k), ctypes.byref(sh), _ptr(qh), qh.numel(),
                                    _ptr(kh), kh.numel(), _stream(stream)))
    return qh, kh


def attn_fwd_qk8(qhat, khat, vhat, shape: Shape, scale: Optional[float] = None,
                 causal: bool = False, kind="efq", params=None, out: Optional[torch.Tensor] = None,
                 stream=None) -> torch.Tensor:
    """Attention on pre-quantised Q^, K^ (quant_qk) and V~ (quant_v); fp32 BSHD out."""
    kind = _kind(kind)
    if scale is None:
        scale = shape.head_dim ** -0.5
    if out is None:
        out = torch.empty((shape.batch, shape.seq_q, shape.heads_q, shape.head_dim),
                          dtype=torch.float32, device=qhat.device)
    _check(lib().efq_attn_fwd_qk8(_ptr(qhat), qhat.numel(), _ptr(khat), khat.numel(), _ptr(vhat),
                                  vhat.numel(), float(scale), int(causal), kind,
                                  _params(kind, params), _ptr(out), ctypes.byref(shape),
                                  _stream(stream)))
    return out


def attn_fwd_qk8_dump(qhat, khat, vhat, shape: Shape, scale=None, causal=False, kind="efq",
                      params=None, stream=None):
    """attn_fwd_qk8 plus the probability-stage record, as attn_fwd_dump."""
    kind = _kind(kind)
    scale = shape.head_dim ** -0.5 if scale is None else scale
    B, Sq, Hq, D, Sk = shape.batch, shape.seq_q, shape.heads_q, shape.head_dim, shape.seq_k
    nblk = (Sk + 31) // 32
    dev = qhat.device
    out = torch.empty((B, Sq, Hq, D), dtype=torch.float32, device=dev)
    codes = torch.empty((B, Hq, Sq, nblk * 16), dtype=torch.uint8, device=dev)
    e8 = torch.empty((B, Hq, Sq, nblk), dtype=torch.uint8, device=dev)
    row_m = torch.empty((B, Hq, Sq), dtype=torch.float32, device=dev)
    row_l = torch.empty((B, Hq, Sq), dtype=torch.float32, device=dev)
    _check(lib().efq_attn_fwd_qk8_dump(_ptr(qhat), qhat.numel(), _ptr(khat), khat.numel(),
                                       _ptr(vhat), vhat.numel(), float(scale), int(causal), kind,
                                       _params(kind, params), _ptr(out), ctypes.byref(shape),
                                       _ptr(codes), _ptr(e8), _ptr(row_m), _ptr(row_l),
                                       _stream(stream)))
    return out, codes, e8, row_m, row_l


def attn_fwd_lowbit(q, k, v, scale: Optional[float] = None, causal: bool = False, kind="efq",
                    params=None, out: Optional[torch.Tensor] = None,
                    workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Low-bit attention: MXFP8 Q K^T, the chosen probability stage, MXFP4 P~V.
    workspace: None, or a 256-byte aligned uint8 tensor of at least
    lowbit_workspace_bytes(shape) bytes."""
    _bf16(q, "q")
    _bf16(k, "k")
    _bf16(v, "v")
    sh = shape_of(q, k)
    kind = _kind(kind)
    if scale is None:
        scale = q.shape[-1] ** -0.5
    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    ws_n = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().efq_attn_fwd_lowbit_ex(_ptr(q), _ptr(k), _ptr(v), float(scale), int(causal), kind,
                                        _params(kind, params), _ptr(out), ctypes.byref(sh),
                                        _ptr(workspace), ws_n, _stream(stream)))
    return out


def lowbit_workspace_bytes(shape: Shape) -> int:
    return int(lib().efq_attn_lowbit_workspace_bytes(ctypes.byref(shape)))


def qk8_natural(buf: torch.Tensor, batch: int, heads: int, seq: int, head_dim: int, scale_off: int):
    """A Q^ or K^ buffer -> (codes [B, H, seq, D], e8m0 [B, H, seq, D/32]) without padding rows."""
    sp = 64 * ((seq + 63) // 64)
    n = batch * heads * sp
    codes = buf[: n * head_dim].view(batch, heads, sp, head_dim)[:, :, :seq]
    e8 = buf[scale_off: scale_off + n * (head_dim // 32)].view(batch, heads, sp, head_dim // 32)
    return codes, e8[:, :, :seq]


def calibrate(q, k, v, o_ref, taus, hs, scale: Optional[float] = None, causal: bool = False,
              stream=None):
    """Algorithm 3 on the GPU: returns ((tau*, h*), rho [len(taus), len(hs)]).

    q, k, v: bf16 BSHD device tensors (calibration inputs); o_ref: fp32
    reference output of the shape of q.  Waits for the stream."""
    import numpy as np
    _bf16(q, "q")
    _bf16(k, "k")
    _bf16(v, "v")
    if o_ref.dtype != torch.float32 or o_ref.shape != q.shape or not o_ref.is_contiguous():
        raise ValueError("o_ref must be a contiguous fp32 tensor of the shape of q")
    sh = shape_of(q, k)
    if scale is None:
        scale = q.shape[-1] ** -0.5
    ta = np.ascontiguousarray(taus, dtype=np.float32)
    ha = np.ascontiguousarray(hs, dtype=np.float32)
    rho = np.zeros((len(ta), len(ha)), np.float64)
    best = Params(0.0, 0.0)
    nbytes = lib().efq_calibrate_workspace_bytes(ctypes.byref(sh), len(ta) * len(ha))
    ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=q.device)
    off = (-ws.data_ptr()) % 256
    _check(lib().efq_calibrate(_ptr(q), _ptr(k), _ptr(v), float(scale), int(causal), _ptr(o_ref),
                               ctypes.byref(sh), ta.ctypes.data_as(ctypes.c_void_p), len(ta),
                               ha.ctypes.data_as(ctypes.c_void_p), len(ha),
                               rho.ctypes.data_as(ctypes.c_void_p), ctypes.byref(best),
                               ctypes.c_void_p(ws.data_ptr() + off), nbytes, _stream(stream)))
    return (best.tau, best.h), rho

def pgen(x: torch.Tensor, kind="efq", params=None, stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """P-gen unit on shifted scores x [rows, cols] fp32 (CUDA)."""
    if x.dtype != torch.float32 or not x.is_cuda or not x.is_contiguous() or x.dim() != 2:
        raise ValueError("x must be a contiguous 2-D fp32 CUDA tensor")
    rows, cols = x.shape
    kind = _kind(kind)
    codes = torch.empty((rows, (cols + 1) // 2), dtype=torch.uint8, device=x.device)
    e8 = torch.empty((rows, (cols + 31) // 32), dtype=torch.uint8, device=x.device)
    _check(lib().efq_pgen(_ptr(x), rows, cols, kind, _params(kind, params), _ptr(codes), _ptr(e8),
                          _stream(stream)))
    return codes, e8


def pgen_bench(kind="efq", params=None, waves: int = 4096, iters: int = 256,
               checksum: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    kind = _kind(kind)
    if checksum is None:
        checksum = torch.empty(waves, dtype=torch.int32, device="cuda")
    _check(lib().efq_pgen_bench(kind, _params(kind, params), int(waves), int(iters),
                                _ptr(checksum), _stream(stream)))
    return checksum


def clock_probe(blocks: int = 256, iters: int = 4000, out: Optional[torch.Tensor] = None,
                stream=None) -> torch.Tensor:
    """[blocks, 2] int64 on the GPU: per workgroup the s_memtime ticks (shader
    clock) and the s_memrealtime ticks (100 MHz) of an MFMA stream (the
    clock in GHz is 0.1 * col0 / col1); asynchronous on `stream`."""
    if out is None:
        out = torch.empty((blocks, 2), dtype=torch.int64, device="cuda")
    if out.dtype != torch.int64 or not out.is_cuda or out.numel() < 2 * blocks or not out.is_contiguous():
        raise ValueError("out must be a contiguous int64 CUDA tensor of at least 2 * blocks elements")
    _check(lib().efq_clock_probe(int(blocks), int(iters), _ptr(out), _stream(stream)))
    return out


def unpack_nibbles(packed: torch.Tensor) -> torch.Tensor:
    """[..., n] bytes -> [..., 2n] codes (low nibble first)."""
    p = packed.to(torch.int16)
    return torch.stack([p & 0xF, p >> 4], dim=-1).flatten(-2).to(torch.uint8)


def vhat_natural(vhat: torch.Tensor, shape: Shape):
    """Reorder a V~ buffer to (codes [B, Hkv, nb*32, D] one per byte, e8m0
    [B, Hkv, nb, D]) in key order (layout stated in efq_attn.h)."""
    B, H, D = shape.batch, shape.heads_kv, shape.head_dim
    nb = 2 * ((shape.seq_k + 63) // 64)
    off = vhat_scale_offset(shape)
    codes = vhat[: B * H * nb * D * 16].view(B, H, nb, D, 16)
    nib = unpack_nibbles(codes)                        # [B, H, nb, D, 32] nibble order
    t = torch.arange(32)
    e = (8 * (2 * ((t >> 2) & 1) + (t >> 4)) + 2 * (t & 3) + ((t >> 3) & 1)).to(vhat.device)
    keyed = nib[..., e]                                # [..., 32] key order
    codes_nat = keyed.permute(0, 1, 2, 4, 3).reshape(B, H, nb * 32, D)
    # scale plane: byte (d % 32) * (D / 32) + d / 32 of each block
    e8 = vhat[off: off + B * H * nb * D].view(B, H, nb, 32, D // 32)
    e8 = e8.permute(0, 1, 2, 4, 3).reshape(B, H, nb, D)
    return codes_nat, e8
