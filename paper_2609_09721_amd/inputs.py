"""Seeded synthetic attention inputs (shapes and value structure only).

This module holds no part of the attention method: it draws Q, K, V with the
shapes and distributions of the paper's three workloads (Qwen3-8B,
Qwen3-VL-8B and WAN2.2-TI2V-5B attention, Sec. IV-A) so that both the GPU
path and the CPU oracle can be fed the same bf16 tensors.  No model weights,
datasets or benchmark items are involved.

Layout: BSHD, bf16, contiguous.  Every tensor comes from its own
``torch.Generator`` seeded with ``seed + {0, 1, 2}`` for (Q, K, V), on the
requested device; values are drawn in fp32 and rounded once to bf16.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, replace
from typing import Tuple

import torch


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    heads_q: int
    heads_kv: int
    seq: int
    head_dim: int
    causal: bool
    dist: str          # "normal", "qwen", "qwen_spread", "vl", "wan", "dyadic"
    seed: int

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)

    def pairs(self) -> int:
        """Visible (query, key) pairs summed over batch and query heads."""
        per_head = self.seq * (self.seq + 1) // 2 if self.causal else self.seq * self.seq
        return per_head * self.batch * self.heads_q

    def flops(self) -> int:
        """Algorithmic flops: 2 D for Q K^T plus 2 D for P V per visible pair."""
        return 4 * self.head_dim * self.pairs()

    def with_seq(self, seq: int) -> "Workload":
        return replace(self, seq=seq)


# The five workloads the benchmark and parity tests use (plus the 32K target
# shape of the Qwen3-8B heads).
WORKLOADS = {
    "tiny": Workload("tiny", 1, 1, 1, 256, 64, False, "normal", 1000),
    "qwen3_8b_16k": Workload("qwen3_8b_16k", 1, 32, 8, 16384, 128, True, "qwen", 2000),
    "qwen3_8b_32k": Workload("qwen3_8b_32k", 1, 32, 8, 32768, 128, True, "qwen", 2500),
    "qwen3_8b_128k": Workload("qwen3_8b_128k", 1, 32, 8, 131072, 128, True, "qwen_spread", 3000),
    "qwen3_vl_32k": Workload("qwen3_vl_32k", 2, 32, 8, 32768, 128, False, "vl", 4000),
    "wan22_75600": Workload("wan22_75600", 1, 24, 24, 75600, 128, False, "wan", 5000),
}

VL_IMAGE_TOKENS = 24576   # leading image-like tokens of the Qwen3-VL workload
VL_RANK = 16              # shared low-rank component
VL_SIGMA = 3.0            # its standard deviation
WAN_OUTLIER_FRAC = 0.01   # fraction of K channels (heads x head_dim) scaled
WAN_OUTLIER_GAIN = 8.0


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def _randn(shape, g, device):
    return torch.randn(shape, generator=g, device=device, dtype=torch.float32)


def _uniform(shape, lo, hi, g, device):
    return torch.rand(shape, generator=g, device=device, dtype=torch.float32) * (hi - lo) + lo


def make_qkv(w: Workload, device="cpu") -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """Draw (Q, K, V) for workload ``w`` as bf16 BSHD tensors on ``device``."""
    B, S, Hq, Hkv, D = w.batch, w.seq, w.heads_q, w.heads_kv, w.head_dim
    gq, gk, gv = (_gen(w.seed + i, device) for i in range(3))
    if w.dist == "dyadic":
        return dyadic_qkv(w, device)
    q = _randn((B, S, Hq, D), gq, device)
    k = _randn((B, S, Hkv, D), gk, device)
    v = _randn((B, S, Hkv, D), gv, device)
    if w.dist in ("qwen", "qwen_spread"):
        # per-(tensor, head) magnitude factor a ~ U(0.5, 2)
        q *= _uniform((1, 1, Hq, 1), 0.5, 2.0, gq, device)
        k *= _uniform((1, 1, Hkv, 1), 0.5, 2.0, gk, device)
        v *= _uniform((1, 1, Hkv, 1), 0.5, 2.0, gv, device)
        if w.dist == "qwen_spread":
            # spread the per-32-key-block maxima: each 32-key block of K (per
            # batch and kv head) is scaled by 2^u, u ~ U(-3, 1)
            nblk = (S + 31) // 32
            u = _uniform((B, nblk, 1, Hkv, 1), -3.0, 1.0, gk, device)
            f = torch.exp2(u).expand(B, nblk, 32, Hkv, 1).reshape(B, nblk * 32, Hkv, 1)[:, :S]
            k *= f
    elif w.dist == "vl":
        # image-like leading tokens: q = n + U w, k = n' + U w', U in R^{D x 16}
        # with orthonormal columns per (batch, kv head), shared by K and the
        # query heads of its group; w ~ N(0, sigma^2 I)
        T = min(VL_IMAGE_TOKENS, S)
        gu = _gen(w.seed + 7, device)
        basis = torch.linalg.qr(_randn((B, Hkv, D, VL_RANK), gu, device).cpu())[0].to(device)
        group = Hq // Hkv
        wq = _randn((B, T, Hq, VL_RANK), gq, device) * VL_SIGMA
        wk = _randn((B, T, Hkv, VL_RANK), gk, device) * VL_SIGMA
        basis_q = basis.repeat_interleave(group, dim=1)          # [B, Hq, D, R]
        # fp32 batched products, transposed operands made contiguous
        bq_t = basis_q.transpose(-1, -2).contiguous()            # [B, Hq, R, D]
        bk_t = basis.transpose(-1, -2).contiguous()              # [B, Hkv, R, D]
        q[:, :T] += torch.matmul(wq.permute(0, 2, 1, 3).contiguous(), bq_t).permute(0, 2, 1, 3)
        k[:, :T] += torch.matmul(wk.permute(0, 2, 1, 3).contiguous(), bk_t).permute(0, 2, 1, 3)
    elif w.dist == "wan":
        # per-token, per-head RMS normalisation (no weight), then 1 % of the
        # K channels (over heads x head_dim) scaled by 8
        def rms(t):
            return t / torch.sqrt(t.pow(2).mean(dim=-1, keepdim=True) + 1e-6)
        q, k = rms(q), rms(k)
        nch = Hkv * D
        nout = int(WAN_OUTLIER_FRAC * nch)
        go = _gen(w.seed + 9, "cpu")
        idx = torch.randperm(nch, generator=go)[:nout].to(device)
        kf = k.view(B, S, nch)
        kf[:, :, idx] *= WAN_OUTLIER_GAIN
    elif w.dist != "normal":
        raise ValueError(f"unknown distribution {w.dist}")
    return q.to(torch.bfloat16), k.to(torch.bfloat16), v.to(torch.bfloat16)


def dyadic_qkv(w: Workload, device="cpu"):
    """Exact-score inputs: Q and K on the grid {-r, ..., r} in steps of 1/2
    (r = 2 for head_dim <= 64, else 1), V ~ N(0, 1).  Every partial sum of a
    Q.K dot product is a multiple of 1/4 below 2^10 in magnitude, so it is
    exact in fp32 whatever the summation order."""
    B, S, Hq, Hkv, D = w.batch, w.seq, w.heads_q, w.heads_kv, w.head_dim
    r = 2 if D <= 64 else 1
    gq, gk, gv = (_gen(w.seed + i, device) for i in range(3))
    n = 4 * r + 1
    q = torch.randint(0, n, (B, S, Hq, D), generator=gq, device=device).float() * 0.5 - r
    k = torch.randint(0, n, (B, S, Hkv, D), generator=gk, device=device).float() * 0.5 - r
    v = _randn((B, S, Hkv, D), gv, device)
    return q.to(torch.bfloat16), k.to(torch.bfloat16), v.to(torch.bfloat16)


def sample_rows(w: Workload, n: int, seed: int = 0) -> torch.Tensor:
    """Stratified (b, hq, i) query rows for sampled checks: every (b, hq)
    gets rows spread over the sequence, always including the first and last
    rows; int32 [n', 3]."""
    g = torch.Generator().manual_seed(seed)
    heads = [(b, h) for b in range(w.batch) for h in range(w.heads_q)]
    per = max(2, n // len(heads))
    out = []
    for (b, h) in heads:
        idx = torch.randint(0, w.seq, (per - 2,), generator=g).tolist()
        for i in sorted(set([0, w.seq - 1] + idx)):
            out.append((b, h, i))
    return torch.tensor(out, dtype=torch.int32)
