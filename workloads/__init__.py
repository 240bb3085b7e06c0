"""Seeded synthetic inputs for the decode-op path.

This module holds shapes and random draws only: no arithmetic of the ops
themselves. It is the one piece shared by the CPU oracle's tests, the GPU
parity tests and the benchmark, so that both sides see identical inputs.

Shapes are those of Llama-family decode and prefill steps (hidden 4096/8192,
32 or 64 query heads of width 128, 8-head GQA keys, SwiGLU intermediates of
11008/14336/28672) and a Qwen3-8B-shaped decode step with per-head QK norm.
Draw order per config is fixed: x, residual, w, q, k, positions, gate, up,
then (QK-norm configs) the Q and K head-norm weights.

* activations ~ N(0, 1) drawn in float32, then rounded to bfloat16 (RNE, via
  torch's cast) when the config is bf16;
* RMSNorm weight ~ U(0.5, 1.5);
* the prefill config multiplies each activation element by 50 with
  probability 1e-3 (element-wise Bernoulli), giving heavy-tailed rows.

bf16 tensors are carried on the host as uint16 bit patterns so that nothing
in between can round them again.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Tuple

import numpy as np

F32 = "f32"
BF16 = "bf16"


@dataclasses.dataclass(frozen=True)
class ChainConfig:
    name: str
    dtype: str
    T: int
    H: int
    nq: int
    nk: int
    hd: int
    I: int
    eps: float = 1e-6
    base: float = 10000.0
    pos_mode: str = "arange"       # "arange" or "uniform"
    pos_max: int = 0               # inclusive upper bound for "uniform"
    outliers: bool = False         # element-wise Bernoulli(1e-3) x 50
    qk_norm: bool = False          # per-head RMSNorm of Q and K before RoPE
    rope: Tuple = ()               # RoPE variant as (name, value) pairs; () = plain
    seed: int = 0

    @property
    def rope_ext(self) -> Optional[dict]:
        return dict(self.rope) if self.rope else None


# The five workloads. Unstated parameters: eps 1e-6 everywhere; RoPE base
# 1e4 for the 7B decode and the mixed stream, 5e5 for the GQA decode and the
# prefill case (Llama-3 shapes); all seeds 0.
TINY_F32 = ChainConfig("tiny_f32", F32, T=4, H=256, nq=4, nk=4, hd=64, I=688)
LLAMA7B_DECODE = ChainConfig("llama7b_decode_bf16", BF16, T=1, H=4096, nq=32, nk=32,
                             hd=128, I=11008, pos_mode="uniform", pos_max=4095)
GQA_DECODE = ChainConfig("gqa_decode_bf16", BF16, T=8, H=4096, nq=32, nk=8, hd=128,
                         I=14336, base=500000.0, pos_mode="uniform", pos_max=8191)
PREFILL_8K = ChainConfig("prefill8k_bf16", BF16, T=8192, H=8192, nq=64, nk=8, hd=128,
                         I=28672, base=500000.0, pos_mode="arange", outliers=True)

# Qwen3-8B-shaped decode step (hidden 4096, 32 Q / 8 K heads of 128 with
# per-head QK-RMSNorm, intermediate 12288, RoPE base 1e6).
QWEN3_8B_DECODE = ChainConfig("qwen3_8b_decode_bf16", BF16, T=1, H=4096, nq=32, nk=8, hd=128,
                              I=12288, base=1000000.0, pos_mode="uniform", pos_max=8191,
                              qk_norm=True)

# Llama-3.1-8B-shaped decode step: Llama-3 frequency scaling (factor 8,
# low / high frequency factors 1 / 4, original context 8192), base 5e5.
LLAMA3_SCALING = (("scaling", 1), ("factor", 8.0), ("low_freq_factor", 1.0),
                  ("high_freq_factor", 4.0), ("original_max_pos", 8192))
LLAMA31_8B_DECODE = ChainConfig("llama31_8b_decode_bf16", BF16, T=1, H=4096, nq=32, nk=8, hd=128,
                                I=14336, base=500000.0, pos_mode="uniform", pos_max=131071,
                                rope=LLAMA3_SCALING)

# GPT-J-6B-shaped step: 16 heads of 256 with GPT-J pairs over the first 64
# elements of each head (hidden 4096, intermediate 16384).
GPTJ_DECODE = ChainConfig("gptj_decode_bf16", BF16, T=4, H=4096, nq=16, nk=16, hd=256, I=16384,
                          pos_mode="uniform", pos_max=2047,
                          rope=(("rotary_dim", 64), ("interleaved", 1)))

# One GPU's share of the 8192-token prefill under 8-way tensor parallelism:
# the residual stream and its norm replicated (hidden 8192), the heads and
# the SwiGLU columns split eight ways (8 Q + 1 K heads, intermediate 3584).
PREFILL_8K_TP8 = ChainConfig("prefill8k_tp8_shard_bf16", BF16, T=8192, H=8192, nq=8, nk=1, hd=128,
                             I=3584, base=500000.0, pos_mode="arange", outliers=True)

CONFIGS = {c.name: c for c in (TINY_F32, LLAMA7B_DECODE, GQA_DECODE, PREFILL_8K,
                               QWEN3_8B_DECODE, LLAMA31_8B_DECODE, GPTJ_DECODE, PREFILL_8K_TP8)}

# Mixed-shape stream: token counts, dtype mix and layout anomalies.
MIXED_T_CHOICES = (1, 2, 4, 8, 16, 32, 64, 128, 512)
MIXED_CALLS = 10_000
MIXED_H, MIXED_I, MIXED_NQ, MIXED_NK, MIXED_HD = 4096, 11008, 32, 32, 128
MIXED_BASE = 10000.0
MIXED_POS_MAX = 4095
MIXED_PAD = 64          # extra elements per row in the non-contiguous layout

LAYOUT_PLAIN = "plain"
LAYOUT_UNALIGNED = "unaligned"      # every activation pointer advanced by one element
LAYOUT_STRIDED = "strided"          # row stride = width + MIXED_PAD


def mixed_stream(seed: int = 0, n: int = MIXED_CALLS) -> List[Tuple[int, str, str]]:
    """The mixed-shape call list: (T, dtype, layout) per call, seeded.

    Token count uniform over MIXED_T_CHOICES; dtype bf16 with probability 0.9
    else f32; a layout anomaly with probability 0.05, split evenly between an
    unaligned and a padded-stride layout.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    ts = rng.integers(0, len(MIXED_T_CHOICES), size=n)
    dt = rng.random(n)
    an = rng.random(n)
    kind = rng.random(n)
    out = []
    for i in range(n):
        T = MIXED_T_CHOICES[int(ts[i])]
        dtype = BF16 if dt[i] < 0.9 else F32
        if an[i] < 0.05:
            layout = LAYOUT_UNALIGNED if kind[i] < 0.5 else LAYOUT_STRIDED
        else:
            layout = LAYOUT_PLAIN
        out.append((T, dtype, layout))
    return out


def _to_bf16_bits(a: np.ndarray) -> np.ndarray:
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def _act(rng, shape, dtype, outliers):
    a = rng.standard_normal(shape, dtype=np.float32)
    if outliers:
        m = rng.random(shape) < 1e-3
        a[m] *= np.float32(50.0)
    return _to_bf16_bits(a) if dtype == BF16 else a


def _weight(rng, H, dtype):
    w = rng.uniform(0.5, 1.5, size=H).astype(np.float32)
    return _to_bf16_bits(w) if dtype == BF16 else w


def _positions(rng, cfg: ChainConfig, T: int) -> np.ndarray:
    if cfg.pos_mode == "arange":
        return np.arange(T, dtype=np.int32)
    return rng.integers(0, cfg.pos_max + 1, size=T).astype(np.int32)


def host_inputs(cfg: ChainConfig, T: Optional[int] = None,
                seed: Optional[int] = None) -> Dict[str, np.ndarray]:
    """All chain inputs for `cfg` as host arrays (f32 values or bf16 bits).

    `T` overrides the token count (used for slices of the big configs).
    Keys: x, residual, w, q, k, pos, gate, up. q is [T, nq, hd], k [T, nk, hd].
    """
    T = cfg.T if T is None else T
    rng = np.random.Generator(np.random.PCG64(cfg.seed if seed is None else seed))
    d, o = cfg.dtype, cfg.outliers
    x = _act(rng, (T, cfg.H), d, o)
    residual = _act(rng, (T, cfg.H), d, o)
    w = _weight(rng, cfg.H, d)
    q = _act(rng, (T, cfg.nq, cfg.hd), d, o)
    k = _act(rng, (T, cfg.nk, cfg.hd), d, o)
    pos = _positions(rng, cfg, T)
    gate = _act(rng, (T, cfg.I), d, o)
    up = _act(rng, (T, cfg.I), d, o)
    out = dict(x=x, residual=residual, w=w, q=q, k=k, pos=pos, gate=gate, up=up)
    if cfg.qk_norm:
        out["q_norm_w"] = _weight(rng, cfg.hd, d)
        out["k_norm_w"] = _weight(rng, cfg.hd, d)
    return out


def cos_sin_table(rng, n: int, rd: int) -> np.ndarray:
    """A float32 [n, rd] table of (cos, sin) pairs of random angles
    U(-pi, pi): cos in the first rd/2 columns, sin in the rest."""
    th = rng.uniform(-np.pi, np.pi, size=(n, rd // 2))
    return np.concatenate([np.cos(th), np.sin(th)], axis=1).astype(np.float32)


def host_array(rng, shape, dtype, outliers=False):
    """One activation-like array drawn from `rng` (f32 values or bf16 bits)."""
    return _act(rng, shape, dtype, outliers)


def host_weight(rng, H, dtype):
    return _weight(rng, H, dtype)


def torch_dtype(dtype: str):
    import torch
    return torch.bfloat16 if dtype == BF16 else torch.float32


def to_torch(a: np.ndarray, dtype: str, device="cpu"):
    """Host array (f32 values / bf16 bits / int32) -> torch tensor on `device`."""
    import torch
    if a.dtype == np.uint16:
        t = torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(device)


def from_torch(t) -> np.ndarray:
    """torch tensor -> host array in the same representation as host_inputs."""
    import torch
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16).copy()
    return t.numpy().copy()


def device_inputs(cfg: ChainConfig, device="cuda", seed: Optional[int] = None):
    """Chain inputs drawn directly on `device` with torch's seeded generator.

    Used for sizes where drawing on the host would be slow (the 8192-token
    prefill case moves 2.2 GB). Same distributions and draw order as
    host_inputs, but a different random stream: GPU parity at these sizes
    copies sampled rows back and evaluates the oracle on them.
    """
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(cfg.seed if seed is None else seed)
    td = torch_dtype(cfg.dtype)
    T = cfg.T

    def act(shape):
        a = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
        if cfg.outliers:
            m = torch.rand(shape, generator=g, device=device) < 1e-3
            a = torch.where(m, a * 50.0, a)
        return a.to(td)

    x = act((T, cfg.H))
    residual = act((T, cfg.H))
    w = (torch.rand((cfg.H,), generator=g, device=device) + 0.5).to(td)
    q = act((T, cfg.nq, cfg.hd))
    k = act((T, cfg.nk, cfg.hd))
    if cfg.pos_mode == "arange":
        pos = torch.arange(T, device=device, dtype=torch.int32)
    else:
        pos = torch.randint(0, cfg.pos_max + 1, (T,), generator=g, device=device,
                            dtype=torch.int32)
    gate = act((T, cfg.I))
    up = act((T, cfg.I))
    out = dict(x=x, residual=residual, w=w, q=q, k=k, pos=pos, gate=gate, up=up)
    if cfg.qk_norm:
        for n in ("q_norm_w", "k_norm_w"):
            out[n] = (torch.rand((cfg.hd,), generator=g, device=device) + 0.5).to(td)
    return out
