"""Seeded synthetic inputs for the gated delta rule.

This module holds no arithmetic of the method itself: it only draws random
tensors with the shapes and value distributions of a language-model layer and
is shared by the tests, the benchmark and the oracle comparisons.

Distributions (the same for every workload):
  q, k      ~ N(0, 1), then L2-normalised per (token, head) vector in fp32
              (the block normalises q and k before the rule, Sec. 3.4),
              then rounded to nearest even in the workload's dtype;
  v         ~ N(0, 1), rounded to the dtype;
  beta      = sigmoid(z),  z ~ N(0, 1)            (writing strength in (0, 1));
  log_alpha = -exp(a_h) * softplus(z),  a_h ~ U(-1, 0) per head,
              z ~ N(0, 1) per (token, head)        (Mamba2-style decay, < 0);
  h0        ~ N(0, std) fp32 when the workload has an initial state;
  dO        ~ N(0, 1) rounded to the dtype; dS_final ~ N(0, 0.01) fp32.
Draw order on one CPU ``torch.Generator`` seeded with ``seed``: packed
sequence lengths (packed workloads only), q, k, v, z_beta, a, z_alpha, h0,
dO, dS_final.  Gates are always fp32.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import torch

DTYPES = {"f32": torch.float32, "bf16": torch.bfloat16}


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int          # batch (1 for packed workloads)
    T: int          # tokens per sequence (total tokens for packed workloads)
    H: int
    dk: int
    dv: int
    dtype: str      # "f32" or "bf16"
    backward: bool  # forward only, or forward + backward
    h0_std: Optional[float] = None      # None: no initial state (zero)
    packed_mean: Optional[int] = None   # geometric mean length of packed sequences
    packed_min: int = 64
    gated: bool = True                  # False: alpha == 1 (no log_alpha input)
    recurrent: bool = False             # token-by-token form (inference), not chunked

    @property
    def tokens(self) -> int:
        return self.B * self.T


# The workloads: shapes of the gated delta rule inside 1.3B-class language
# models (4K training length, head dims 64-256, expanded value dim).
WORKLOADS = {
    w.name: w
    for w in (
        Workload("fwd_f32_b1_t256_h2_d64", 1, 256, 2, 64, 64, "f32", False),
        Workload("fwd_bf16_b4_t2048_h16_d128", 4, 2048, 16, 128, 128, "bf16", False,
                 h0_std=0.02),
        Workload("fwd_bf16_b8_t4096_h6_dk256_dv512", 8, 4096, 6, 256, 512, "bf16", False),
        Workload("fwdbwd_bf16_b8_t4096_h6_dk256_dv512", 8, 4096, 6, 256, 512, "bf16", True),
        Workload("fwdbwd_bf16_b8_t4096_h6_dk256_dv512_alpha1", 8, 4096, 6, 256, 512, "bf16",
                 True, gated=False),
        # one decode step for a serving batch, from a state left by a prefill
        Workload("decode_bf16_b256_h6_dk256_dv512", 256, 1, 6, 256, 512, "bf16", False,
                 h0_std=0.02, recurrent=True),
        Workload("fwdbwd_bf16_packed65536_h16_d128", 1, 65536, 16, 128, 128, "bf16", True,
                 packed_mean=4096, packed_min=64),
    )
}


def packed_lengths(gen: torch.Generator, total: int, mean: int, minimum: int):
    """Lengths max(minimum, Geometric(1/mean)) until they cover ``total`` tokens;
    the last one is truncated, and folded into its predecessor if that leaves
    it shorter than ``minimum``."""
    lens = []
    acc = 0
    while acc < total:
        x = int(torch.empty(1, dtype=torch.float64).geometric_(1.0 / mean, generator=gen).item())
        x = max(minimum, x)
        lens.append(x)
        acc += x
    lens[-1] -= acc - total
    if lens[-1] < minimum and len(lens) > 1:
        lens[-2] += lens.pop()
    return lens


def cu_from_lengths(lens):
    cu = [0]
    for x in lens:
        cu.append(cu[-1] + int(x))
    return torch.tensor(cu, dtype=torch.int32)


def make_inputs(B, T, H, dk, dv, dtype="bf16", seed=0, h0_std=None, backward=False,
                cu_seqlens=None, packed_mean=None, packed_min=64, dht_std=0.01,
                log_alpha_scale=1.0, beta_scale=1.0, beta_value=None, log_alpha_value=None,
                gated=True):
    """Draw one set of inputs (CPU tensors).

    Dense: q [B,T,H,dk], v [B,T,H,dv], beta/log_alpha [B,T,H] fp32.
    Packed (``cu_seqlens`` given, or ``packed_mean`` set): B must be 1 and T is
    the total token count; ``cu_seqlens`` int32 [N+1] is returned too.

    Stress knobs (defaults reproduce the distributions above):
      log_alpha_scale multiplies log_alpha (0.01 = weak decay, 0 = alpha == 1);
      beta_scale multiplies beta (2.0 gives beta in (0, 2));
      beta_value / log_alpha_value replace them by a constant;
      gated=False draws the gates as usual (same stream), then sets
      log_alpha to zero and marks the inputs ``gated: False`` (callers pass
      no log_alpha: alpha == 1).
    """
    gen = torch.Generator().manual_seed(seed)
    dt = DTYPES[dtype]
    if packed_mean is not None and cu_seqlens is None:
        if B != 1:
            raise ValueError("packed workloads have B == 1")
        cu_seqlens = cu_from_lengths(packed_lengths(gen, T, packed_mean, packed_min))
    if cu_seqlens is not None:
        cu_seqlens = torch.as_tensor(cu_seqlens, dtype=torch.int32)
        if B != 1 or int(cu_seqlens[-1]) != T:
            raise ValueError("packed inputs need B == 1 and cu_seqlens[-1] == T")
    nstate = (cu_seqlens.numel() - 1) if cu_seqlens is not None else B

    def unit(shape):
        x = torch.randn(shape, generator=gen, dtype=torch.float32)
        return x / torch.linalg.vector_norm(x, dim=-1, keepdim=True).clamp_min(1e-12)

    q = unit((B, T, H, dk)).to(dt)
    k = unit((B, T, H, dk)).to(dt)
    v = torch.randn((B, T, H, dv), generator=gen, dtype=torch.float32).to(dt)
    z_beta = torch.randn((B, T, H), generator=gen, dtype=torch.float32)
    a = torch.rand((H,), generator=gen, dtype=torch.float32) - 1.0
    z_alpha = torch.randn((B, T, H), generator=gen, dtype=torch.float32)
    beta = torch.sigmoid(z_beta) * beta_scale
    log_alpha = -torch.exp(a) * torch.nn.functional.softplus(z_alpha) * log_alpha_scale
    if beta_value is not None:
        beta = torch.full_like(beta, float(beta_value))
    if log_alpha_value is not None:
        log_alpha = torch.full_like(log_alpha, float(log_alpha_value))
    h0 = None
    if h0_std is not None:
        h0 = torch.randn((nstate, H, dk, dv), generator=gen, dtype=torch.float32) * h0_std
    if not gated:
        log_alpha = torch.zeros_like(log_alpha)
    out = dict(q=q, k=k, v=v, beta=beta.contiguous(), log_alpha=log_alpha.contiguous(), h0=h0,
               cu_seqlens=cu_seqlens, gated=gated)
    if backward:
        out["dO"] = torch.randn((B, T, H, dv), generator=gen, dtype=torch.float32).to(dt)
        out["dht"] = torch.randn((nstate, H, dk, dv), generator=gen,
                                 dtype=torch.float32) * dht_std
    return out


def workload_inputs(name: str, seed: int = 0):
    w = WORKLOADS[name]
    return make_inputs(w.B, w.T, w.H, w.dk, w.dv, w.dtype, seed=seed, h0_std=w.h0_std,
                       backward=w.backward, packed_mean=w.packed_mean, packed_min=w.packed_min,
                       gated=w.gated)


def make_block_inputs(B, T, H, dk, dv, dtype="bf16", seed=0, width=4, cu_seqlens=None):
    """Inputs of the block prologue and epilogue (CPU tensors).

    Projections xq, xk [B, T, H, dk] and xv [B, T, H, dv] ~ N(0, 1); convolution
    weights [H * d, width] ~ U(-1/sqrt(width), 1/sqrt(width)) fp32 (the default
    range of a depthwise convolution with fan-in width); gradients of the
    prologue outputs dq, dk, dv ~ N(0, 1); the rule's output o and the gate
    projection g ~ N(0, 1), the normalisation weight 1 + N(0, 0.1) fp32 [dv],
    the gradient of the block output dy ~ N(0, 1).  Draw order as listed.
    """
    gen = torch.Generator().manual_seed(seed)
    dt = DTYPES[dtype]
    n = lambda shape: torch.randn(shape, generator=gen, dtype=torch.float32).to(dt)
    bound = 1.0 / width ** 0.5
    u = lambda rows: (torch.rand((rows, width), generator=gen, dtype=torch.float32) * 2 - 1) * bound
    out = dict(xq=n((B, T, H, dk)), xk=n((B, T, H, dk)), xv=n((B, T, H, dv)),
               wq=u(H * dk), wk=u(H * dk), wv=u(H * dv),
               dq=n((B, T, H, dk)), dk=n((B, T, H, dk)), dv=n((B, T, H, dv)),
               o=n((B, T, H, dv)), g=n((B, T, H, dv)),
               wo=1.0 + 0.1 * torch.randn((dv,), generator=gen, dtype=torch.float32),
               dy=n((B, T, H, dv)))
    if cu_seqlens is not None:
        out["cu_seqlens"] = torch.as_tensor(cu_seqlens, dtype=torch.int32)
    return out
