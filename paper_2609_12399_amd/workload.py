"""Seeded synthetic GR-shaped decode workloads.

This module only draws random inputs, normalises them and rounds them to the
precision the device consumes.  It contains none of the GDN arithmetic, so
both the device path and the fp64 oracle can consume the same bits from it.

The generative-recommendation (GR) workload of the OneLA paper (arXiv
2609.12399, Sec. 2.1) is a long shared prompt followed by a few decode steps
over a wide, re-ranked beam.  The paper's own traces and its Qwen3.5 model are
not available, so these synthetic inputs stand in for them, using the paper's
GDN geometry (H = 16 heads, d_k = d_v = 128, Sec. 4.1) and its beam, request
and step ranges (Sec. 4.1).

Distributions (identical for prompt and decode tokens):
  q, k ~ N(0, 1), then L2-normalised over the key dimension (fp64);
  v ~ N(0, 1);
  beta  = sigmoid(x),            x ~ N(0, 1);
  alpha = exp(-softplus(x)),     x ~ N(mu, 1), mu = -3 (or -5: alpha near 1).
Values are drawn in fp64 and rounded once: q/k/v to the io dtype (bf16 by
round-to-nearest-even through fp32, or fp32), alpha/beta to fp32.

Parents of step t >= 1 index the previous step's beams, which are kept in rank
order by a global top-W selection; they are drawn i.i.d. with replacement,
either uniformly or Zipf(s) over ranks, P(rank r) ~ (r + 1)^-s, and are left in
draw order (unsorted).

Draw order for ``numpy.random.default_rng(seed)``: prompt k, prompt v, prompt
beta-logit, prompt alpha-logit; then for every step t: q, k, v, beta-logit,
alpha-logit and (t >= 1) parents.  Every array carries a leading request axis.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class WorkloadSpec:
    name: str
    R: int                 # independent requests (users), one S_ctx each
    HK: int                # query/key heads
    HV: int                # value heads (HV % HK == 0)
    dk: int
    dv: int
    P: int                 # prompt tokens behind S_ctx
    widths: tuple          # live beams per decode step, W_t
    io_dtype: str          # "bf16" or "f32" for q/k/v
    parents: str           # "uniform" or "zipf"
    zipf_s: float = 1.1
    alpha_mu: float = -3.0
    seed: int = 0

    @property
    def T(self) -> int:
        return len(self.widths)

    @property
    def W(self) -> int:
        return max(self.widths)


def _spec(name, R, HK, HV, d, P, W, T, io, parents, s=1.1, mu=-3.0, seed=0):
    return WorkloadSpec(name, R, HK, HV, d, d, P, (W,) * T, io, parents, s, mu, seed)


# The workload shapes used throughout (tests and benchmark).
SPECS = {
    # 1 layer, 2 heads, d = 32, fp32, 64-token prompt, 8 beams, 3 steps.
    "tiny_h2_d32_w8": _spec("tiny_h2_d32_w8", 1, 2, 2, 32, 64, 8, 3, "f32",
                            "uniform", seed=1000),
    # 16 heads, d = 128, bf16 inputs, 1024-token prompt, 128 beams, 3 steps.
    "h16_d128_w128": _spec("h16_d128_w128", 1, 16, 16, 128, 1024, 128, 3, "bf16",
                           "zipf", 1.1, seed=1001),
    # 16 heads, d = 128, bf16 inputs, 4096-token prompt, 512 beams, 4 steps.
    "h16_d128_w512": _spec("h16_d128_w512", 1, 16, 16, 128, 4096, 512, 4, "bf16",
                           "zipf", 1.1, seed=1002),
    # 8 independent users x 256 beams, 2048-token prompts, 4 steps.
    "r8_h16_d128_w256": _spec("r8_h16_d128_w256", 8, 16, 16, 128, 2048, 256, 4,
                              "bf16", "uniform", seed=1003),
    # 32 value heads over 16 query/key heads, 8192-token prompt, 1024 beams,
    # 5 steps, Zipf(1.5) parents, alpha near 1.
    "gqa_h16x32_d128_w1024": _spec("gqa_h16x32_d128_w1024", 1, 16, 32, 128, 8192,
                                   1024, 5, "bf16", "zipf", 1.5, -5.0, seed=1004),
    # The shape of the paper's recurrent-state-path breakdown: 4 requests x 512
    # beams, 16 heads, d = 128, 6 decode steps (7 output tokens), 1024-token prompts.
    "r4_h16_d128_w512_t6": _spec("r4_h16_d128_w512_t6", 4, 16, 16, 128, 1024, 512, 6,
                                 "bf16", "zipf", 1.1, seed=1007),
    # The paper's largest operator geometry: 16 requests x 512 beams, 16 heads,
    # d = 128, 1024-token prompts, 4 steps.
    "r16_h16_d128_w512": _spec("r16_h16_d128_w512", 16, 16, 16, 128, 1024, 512, 4, "bf16",
                               "zipf", 1.1, seed=1009),
    # The widest value-head count of the paper's operator suite (H_V = 64):
    # 64 value heads over 16 query/key heads, d = 128, 256 beams, 4 steps.
    "gqa_h16x64_d128_w256": _spec("gqa_h16x64_d128_w256", 1, 16, 64, 128, 2048, 256, 4,
                                  "bf16", "zipf", 1.1, seed=1008),
    # Wider heads of the paper's operator suite (key dim up to 256, value dim up
    # to 512, grouped heads): 8 heads with d_k = d_v = 256, 512 beams, 4 steps.
    "h8_k256_v256_w512": WorkloadSpec("h8_k256_v256_w512", 1, 8, 8, 256, 256, 2048,
                                      (512,) * 4, "bf16", "zipf", 1.1, seed=1005),
    # 4 query/key heads of d_k = 256 shared by 8 value heads of d_v = 512,
    # 256 beams, 4 steps.
    "h4x8_k256_v512_w256": WorkloadSpec("h4x8_k256_v512_w256", 1, 4, 8, 256, 512, 2048,
                                        (256,) * 4, "bf16", "uniform", seed=1006),
}

HEADLINE = "h16_d128_w512"


def f32_to_bf16_bits(x32: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round-to-nearest-even); returns uint16 bits."""
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32).astype(np.uint64)
    bias = 0x7FFF + ((u >> 16) & 1)
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact upcast of bf16 bit patterns."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


@dataclass
class Tensor:
    """One input array in the device's format, with its exact fp64 value."""
    dev: np.ndarray        # uint16 (bf16 bits) or float32
    dtype: str             # "bf16" or "f32"

    @property
    def f64(self) -> np.ndarray:
        if self.dtype == "bf16":
            return bf16_bits_to_f64(self.dev)
        return self.dev.astype(np.float64)

    @property
    def shape(self):
        return self.dev.shape


def _round(x64: np.ndarray, dtype: str) -> Tensor:
    x32 = x64.astype(np.float32)
    if dtype == "bf16":
        return Tensor(f32_to_bf16_bits(x32), "bf16")
    if dtype == "f32":
        return Tensor(x32, "f32")
    raise ValueError(dtype)


def _unit(x: np.ndarray) -> np.ndarray:
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def _gates(rng, shape, mu):
    b = rng.standard_normal(shape)
    a = rng.standard_normal(shape) + mu
    beta = 1.0 / (1.0 + np.exp(-b))
    alpha = np.exp(-np.logaddexp(0.0, a))
    return alpha, beta


def _draw_parents(rng, spec: WorkloadSpec, w_prev: int, w_cur: int) -> np.ndarray:
    if spec.parents == "uniform":
        return rng.integers(0, w_prev, size=(spec.R, w_cur)).astype(np.int32)
    if spec.parents == "zipf":
        p = (np.arange(w_prev, dtype=np.float64) + 1.0) ** (-spec.zipf_s)
        p /= p.sum()
        return rng.choice(w_prev, size=(spec.R, w_cur), p=p).astype(np.int32)
    raise ValueError(spec.parents)


@dataclass
class Step:
    q: Tensor              # [R][W_t][HK][dk]
    k: Tensor              # [R][W_t][HK][dk]
    v: Tensor              # [R][W_t][HV][dv]
    alpha: Tensor          # [R][W_t][HV] fp32
    beta: Tensor           # [R][W_t][HV] fp32
    parents: np.ndarray | None  # [R][W_t] int32, None at t = 0


@dataclass
class Workload:
    spec: WorkloadSpec
    prompt_k: Tensor       # [R][P][HK][dk]
    prompt_v: Tensor       # [R][P][HV][dv]
    prompt_alpha: Tensor   # [R][P][HV]
    prompt_beta: Tensor    # [R][P][HV]
    steps: list = field(default_factory=list)


def make_workload(spec: WorkloadSpec | str, seed: int | None = None,
                  with_prompt: bool = True) -> Workload:
    """Draw a workload.  ``with_prompt=False`` skips the prompt arrays but
    keeps the draw order (the prompt is still drawn, then dropped)."""
    if isinstance(spec, str):
        spec = SPECS[spec]
    if spec.HV % spec.HK:
        raise ValueError("HV must be a multiple of HK")
    rng = np.random.default_rng(spec.seed if seed is None else seed)
    R, P = spec.R, spec.P
    io = spec.io_dtype
    pk = _unit(rng.standard_normal((R, P, spec.HK, spec.dk)))
    pv = rng.standard_normal((R, P, spec.HV, spec.dv))
    pa, pb = _gates(rng, (R, P, spec.HV), spec.alpha_mu)
    if with_prompt:
        wl = Workload(spec, _round(pk, io), _round(pv, io), _round(pa, "f32"),
                      _round(pb, "f32"))
    else:
        wl = Workload(spec, None, None, None, None)
    del pk, pv
    w_prev = None
    for t, W in enumerate(spec.widths):
        q = _unit(rng.standard_normal((R, W, spec.HK, spec.dk)))
        k = _unit(rng.standard_normal((R, W, spec.HK, spec.dk)))
        v = rng.standard_normal((R, W, spec.HV, spec.dv))
        a, b = _gates(rng, (R, W, spec.HV), spec.alpha_mu)
        par = _draw_parents(rng, spec, w_prev, W) if t > 0 else None
        wl.steps.append(Step(_round(q, io), _round(k, io), _round(v, io),
                             _round(a, "f32"), _round(b, "f32"), par))
        w_prev = W
    return wl


def with_widths(spec: WorkloadSpec | str, widths, **kw) -> WorkloadSpec:
    """A copy of a spec with other per-step beam widths (and other fields)."""
    if isinstance(spec, str):
        spec = SPECS[spec]
    d = dict(spec.__dict__)
    d["widths"] = tuple(int(w) for w in widths)
    d.update(kw)
    return WorkloadSpec(**d)


# ---- beam-selection inputs ---------------------------------------------------
# The scores a model hands to global beam selection (Sec. 2.1): per live beam,
# log-probabilities over the SID codebook, plus the beam's running score.  The
# paper fixes neither the codebook size nor the model, so these stand in for
# them: logits ~ N(0, sigma^2) with sigma = 2, turned into log-probabilities
# by a numerically stable log-softmax over the codebook (fp64, then rounded
# once to fp32), and beam scores ~ -|N(0, 4)| sorted descending (the previous
# selection keeps beams in rank order).  Other kinds stress the ordering:
# "ties" draws integers in [-3, 3] (most candidates tie), "special" is
# log-softmax with 2% of the entries replaced by each of -0.0, +0.0, +inf,
# -inf, +NaN and -NaN.

SELECT_CODEBOOK = 8192


def make_select_inputs(R: int, prev_width: int, vocab: int, seed: int,
                       kind: str = "logsoftmax", with_beam: bool = True):
    """(logp fp32 [R][W_prev][V], beam fp32 [R][W_prev] or None)."""
    rng = np.random.default_rng(seed)
    shape = (R, prev_width, vocab)
    if kind == "ties":
        logp = rng.integers(-3, 4, size=shape).astype(np.float32)
    elif kind == "rising":
        # small spread inside a row, beam scores rising with the row: later
        # candidates keep beating earlier ones
        logp = (-rng.random(shape) * 0.5).astype(np.float32)
    else:
        x = rng.standard_normal(shape) * 2.0
        m = x.max(axis=-1, keepdims=True)
        logp = (x - m - np.log(np.exp(x - m).sum(axis=-1, keepdims=True))).astype(np.float32)
        if kind == "special":
            u = rng.random(shape)
            specials = [-0.0, 0.0, np.inf, -np.inf, np.nan, -np.nan]
            for j, val in enumerate(specials):
                logp[(u >= 0.02 * j) & (u < 0.02 * (j + 1))] = np.float32(val)
        elif kind not in ("logsoftmax", "rising"):
            raise ValueError(kind)
    beam = None
    if with_beam:
        if kind == "ties":
            beam = rng.integers(-2, 3, size=(R, prev_width)).astype(np.float32)
        elif kind == "rising":
            beam = np.broadcast_to(np.arange(prev_width, dtype=np.float32),
                                   (R, prev_width)).copy()
        else:
            b = -np.abs(rng.standard_normal((R, prev_width)) * 2.0)
            beam = (-np.sort(-b, axis=-1)).astype(np.float32)
    return logp, beam
