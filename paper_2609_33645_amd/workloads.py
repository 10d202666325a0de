"""Seeded synthetic inputs for the Pruned CTC head-and-loss path.

This module only draws inputs: frame counts, target transcripts, head inputs H
and head weights W.  It holds none of the method's arithmetic, so both the CPU
oracle (through the tests) and the HIP path can be fed from it.

Shapes follow the paper's workloads:
  * Zipformer-M encoder head: D = 512, V up to 180,000 (Sec. 5.1 and App. C.2),
    25 Hz frames, utterances of 6-15 s;
  * Qwen3 LLM-CTC heads: V = 151,936 with D = 1024 / 4096 / 5120
    (Sec. 4, App. C.3, Table "qwen-config").
The paper measures on GigaSpeech audio; that data is not used.  Seeded random
draws with the same shapes, length mix and a Zipf(1.1) token-frequency law
stand in for it.

Draw order (numpy.random.default_rng(seed)): frame counts T_n, then targets,
then H, then W.  bf16 workloads round H and W to bfloat16 (round to nearest
even) on the host before either side sees them, and the values are handed over
as float32 arrays that hold exactly those bfloat16 numbers.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np


@dataclasses.dataclass
class Workload:
    name: str
    dtype: str                 # "f32" or "bf16": the type H and W are stored in on the device
    H: np.ndarray              # [M, D] float32 (bf16-exact values when dtype == "bf16")
    W: np.ndarray              # [V, D] float32 (bf16-exact values when dtype == "bf16")
    targets: np.ndarray        # [sum U_n] int32, concatenated, blank-free
    input_lengths: np.ndarray  # [N] int32, T_n >= 1
    target_lengths: np.ndarray  # [N] int32, U_n >= 0
    blank: int
    beam: float                # +inf = all alignments retained

    @property
    def N(self) -> int:
        return int(self.input_lengths.shape[0])

    @property
    def M(self) -> int:
        return int(self.H.shape[0])

    @property
    def D(self) -> int:
        return int(self.H.shape[1])

    @property
    def V(self) -> int:
        return int(self.W.shape[0])


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); return float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty_like(x)
    src = x.reshape(-1).view(np.uint32)
    dst = out.reshape(-1).view(np.uint32)
    step = 1 << 22
    for i in range(0, src.size, step):
        u = src[i:i + step]
        # finite values and infinities cannot overflow 32 bits here (|u| <= 0xFF800000)
        r = u + np.uint32(0x7FFF)
        r += (u >> np.uint32(16)) & np.uint32(1)
        r &= np.uint32(0xFFFF0000)
        dst[i:i + step] = r
    nan = np.isnan(x)
    if nan.any():
        out[nan] = np.float32("nan")
    return out


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """The upper 16 bits of bf16-exact float32 values, as uint16 (device storage)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16)


def zipf_ids(rng: np.random.Generator, n: int, V: int, s: float = 1.1) -> np.ndarray:
    """n draws from Zipf(s) truncated to ranks 1..V-1 (inverse CDF); id = rank."""
    ranks = np.arange(1, V, dtype=np.float64)
    cdf = np.cumsum(ranks ** (-s))
    cdf /= cdf[-1]
    u = rng.random(n)
    idx = np.searchsorted(cdf, u, side="right")
    return (np.minimum(idx, V - 2) + 1).astype(np.int32)


def _with_repeats(rng: np.random.Generator, fresh: np.ndarray, p_repeat: float) -> np.ndarray:
    """Each label after the first copies its predecessor with probability p_repeat."""
    y = fresh.copy()
    if y.size > 1 and p_repeat > 0:
        rep = rng.random(y.size) < p_repeat
        for i in range(1, y.size):
            if rep[i]:
                y[i] = y[i - 1]
    return y


def synthesize(*, name: str, dtype: str, T: np.ndarray, U: np.ndarray, D: int, V: int,
               rng: np.random.Generator, token_law: str = "zipf", p_repeat: float = 0.0,
               h_law: str = "normal", w_std: Optional[float] = None, blank: int = 0,
               beam: float = math.inf) -> Workload:
    """Draw targets, H and W for given frame counts T and target lengths U."""
    T = np.asarray(T, dtype=np.int32)
    U = np.asarray(U, dtype=np.int32)
    ys = []
    for u in U:
        if token_law == "zipf":
            fresh = zipf_ids(rng, int(u), V)
        else:  # uniform over [0, V) without blank
            fresh = rng.integers(0, V - 1, size=int(u)).astype(np.int32)
        if token_law != "zipf":
            fresh = np.where(fresh >= blank, fresh + 1, fresh).astype(np.int32)
        elif blank != 0:
            # Zipf ids are ranks 1..V-1; move any draw that hits the blank id to id 0
            fresh = np.where(fresh == blank, 0, fresh).astype(np.int32)
        ys.append(_with_repeats(rng, fresh, p_repeat))
    targets = np.concatenate(ys).astype(np.int32) if ys else np.zeros(0, np.int32)
    M = int(T.sum())
    H = rng.standard_normal((M, D), dtype=np.float32)
    if h_law == "rmsnorm":
        rms = np.sqrt(np.mean(H.astype(np.float64) ** 2, axis=1, keepdims=True))
        H = (H / rms).astype(np.float32)
    std = (1.0 / math.sqrt(D)) if w_std is None else w_std
    W = (rng.standard_normal((V, D), dtype=np.float32) * np.float32(std)).astype(np.float32)
    if dtype == "bf16":
        H = round_to_bf16(H)
        W = round_to_bf16(W)
    return Workload(name=name, dtype=dtype, H=H, W=W, targets=targets,
                    input_lengths=T, target_lengths=U, blank=int(blank), beam=float(beam))


# --- The five named workloads -------------------------------------------------------------

def tiny_f32(seed: int = 0) -> Workload:
    """Tiny fp32 case: N=2, T=(50,42), D=64, V=1000, U=(10,7) uniform ids, no beam."""
    rng = np.random.default_rng(seed)
    T = np.array([50, 42], np.int32)
    U = np.array([10, 7], np.int32)
    return synthesize(name="tiny_f32", dtype="f32", T=T, U=U, D=64, V=1000, rng=rng,
                      token_law="uniform", w_std=1.0 / 8.0)


def zipformer_m(seed: int = 0, beam: float = math.inf, V: int = 180_000) -> Workload:
    """Zipformer-M-like head: N=16, T~U{150..375}, U=floor(T/6) Zipf(1.1), D=512, bf16."""
    rng = np.random.default_rng(seed)
    T = rng.integers(150, 376, size=16).astype(np.int32)
    U = (T // 6).astype(np.int32)
    return synthesize(name="zipformer_m", dtype="bf16", T=T, U=U, D=512, V=V, rng=rng, beam=beam)


def qwen3_0p6b(seed: int = 0, beam: float = 32.0) -> Workload:
    """Qwen3-0.6B-style head: N=8, T~U{200..500}, U=floor(T/4), D=1024, V=151,936."""
    rng = np.random.default_rng(seed)
    T = rng.integers(200, 501, size=8).astype(np.int32)
    U = (T // 4).astype(np.int32)
    return synthesize(name="qwen3_0p6b", dtype="bf16", T=T, U=U, D=1024, V=151_936, rng=rng,
                      h_law="rmsnorm", w_std=0.02, beam=beam)


def qwen3_8b(seed: int = 0, beam: float = math.inf) -> Workload:
    """Qwen3-8B-style head: N=4, T~U{500..750}, U=floor(T/4), D=4096, V=151,936."""
    rng = np.random.default_rng(seed)
    T = rng.integers(500, 751, size=4).astype(np.int32)
    U = (T // 4).astype(np.int32)
    return synthesize(name="qwen3_8b", dtype="bf16", T=T, U=U, D=4096, V=151_936, rng=rng,
                      h_law="rmsnorm", w_std=0.02, beam=beam)


def qwen3_32b(seed: int = 0, beam: float = 16.0) -> Workload:
    """Qwen3-32B-style long utterances: N=2, T=1500, U=400 with 10% repeats, D=5120."""
    rng = np.random.default_rng(seed)
    T = np.array([1500, 1500], np.int32)
    U = np.array([400, 400], np.int32)
    return synthesize(name="qwen3_32b", dtype="bf16", T=T, U=U, D=5120, V=151_936, rng=rng,
                      p_repeat=0.1, h_law="rmsnorm", w_std=0.02, beam=beam)


def qwen3_8b_kstress(seed: int = 0, beam: float = math.inf) -> Workload:
    """The Qwen3-8B-style shape with uniform token draws instead of Zipf: nearly every
    target id distinct, so the union is as large as the targets allow (K ~ 1 + sum U)."""
    rng = np.random.default_rng(seed)
    T = rng.integers(500, 751, size=4).astype(np.int32)
    U = (T // 4).astype(np.int32)
    return synthesize(name="qwen3_8b_kstress", dtype="bf16", T=T, U=U, D=4096, V=151_936, rng=rng,
                      token_law="uniform", h_law="rmsnorm", w_std=0.02, beam=beam)


def e1_zipformer_f32(seed: int = 0, beam: float = math.inf) -> Workload:
    """The encoder benchmark's memory shape: 160 utterances x 100 frames (M = 16,000), D = 512,
    V = 180,000, fp32 head; U = floor(T/6) Zipf(1.1)."""
    rng = np.random.default_rng(seed)
    T = np.full(160, 100, np.int32)
    U = (T // 6).astype(np.int32)
    return synthesize(name="e1_zipformer_f32", dtype="f32", T=T, U=U, D=512, V=180_000, rng=rng, beam=beam)


def e3_qwen3_8b(seed: int = 0, beam: float = 32.0) -> Workload:
    """The LLM benchmark's memory shape: N = 107 utterances of at most 111 frames (M = 11,458),
    D = 4096, V = 151,936, bf16 (run with the head frozen: no dW); U = floor(T/4) Zipf(1.1)."""
    rng = np.random.default_rng(seed)
    T = np.full(107, 107, np.int32)
    T[: 11458 - 107 * 107] += 1            # 11,458 frames, lengths 107..108 (<= 111)
    U = (T // 4).astype(np.int32)
    return synthesize(name="e3_qwen3_8b", dtype="bf16", T=T, U=U, D=4096, V=151_936, rng=rng,
                      h_law="rmsnorm", w_std=0.02, beam=beam)


NAMED = {
    "tiny_f32": tiny_f32,
    "zipformer_m": zipformer_m,
    "qwen3_0p6b": qwen3_0p6b,
    "qwen3_8b": qwen3_8b,
    "qwen3_32b": qwen3_32b,
    "qwen3_8b_kstress": qwen3_8b_kstress,
    "e1_zipformer_f32": e1_zipformer_f32,
    "e3_qwen3_8b": e3_qwen3_8b,
}


def random_small(seed: int, *, N: int, T_range=(1, 40), D: int = 32, V: int = 200,
                 dtype: str = "bf16", u_frac: float = 0.25, p_repeat: float = 0.0,
                 token_law: str = "zipf", blank: int = 0, beam: float = math.inf,
                 U_override=None, w_std=None) -> Workload:
    """A small random case for parity tests (several tiles, ragged tails)."""
    rng = np.random.default_rng(seed)
    T = rng.integers(T_range[0], T_range[1] + 1, size=N).astype(np.int32)
    if U_override is not None:
        U = np.asarray(U_override, np.int32)
    else:
        U = np.floor(T * u_frac).astype(np.int32)
    return synthesize(name=f"small{seed}", dtype=dtype, T=T, U=U, D=D, V=V, rng=rng,
                      token_law=token_law, p_repeat=p_repeat, blank=blank, beam=beam,
                      w_std=w_std)


def random_scores(seed: int, M: int, K: int, scale: float = 3.0, integer: bool = False) -> np.ndarray:
    """Seeded per-frame class scores [M, K] (float32) for stand-alone tests of the
    alignment recursion: non-positive values -Exp(scale), with every 7th row shifted
    by a seeded offset so that rows do not share a common level.  integer=True rounds
    every score to an integer (sums of scores are then exact in float32)."""
    rng = np.random.default_rng(seed)
    s = -rng.exponential(scale, size=(M, K))
    s[::7] -= rng.uniform(0.0, 20.0, size=(s[::7].shape[0], 1))
    if integer:
        s = np.round(s)
    return s.astype(np.float32)
