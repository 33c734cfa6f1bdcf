"""Shared helpers of the GPU tests: oracle references for a workload and the
error metric.  Everything here runs on the CPU; the device path is driven
through the C ABI by the tests themselves."""
from __future__ import annotations

import functools
import sys

import numpy as np

from oracle import oracle as orc
from paper_2609_12399_amd import workload as W

# Output tolerance: max over output vectors of ||o_gpu - o_ref||_inf /
# ||o_ref||_inf (bf16 inputs, fp32 accumulation).
REL_TOL = 2e-3


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def oracle_s0(wl: W.Workload) -> np.ndarray:
    """S_ctx per request from the fp64 oracle prefill, rounded once to fp32."""
    out = []
    for r in range(wl.spec.R):
        S = orc.prefill(wl.prompt_k.f64[r], wl.prompt_v.f64[r], wl.prompt_alpha.f64[r],
                        wl.prompt_beta.f64[r])
        out.append(S.astype(np.float32))
    return np.stack(out)


def oracle_outputs(wl: W.Workload, s0_f32: np.ndarray, heads=None):
    """fp64 oracle outputs [t] -> [R][W_t][HV][dv] (or only value heads
    ``heads``, whose query/key heads are sliced alongside)."""
    spec = wl.spec
    G = spec.HV // spec.HK
    hv_sel = list(range(spec.HV)) if heads is None else list(heads)
    hk_sel = sorted({h // G for h in hv_sel})
    # remap to a sub-problem with contiguous groups
    sub_hv = []
    for hk in hk_sel:
        sub_hv += [hk * G + g for g in range(G)]
    res = [np.zeros((spec.R, s.q.shape[1], len(sub_hv), spec.dv)) for s in wl.steps]
    for r in range(spec.R):
        o = orc.decode(s0_f32[r].astype(np.float64)[sub_hv],
                       [s.q.f64[r][:, hk_sel] for s in wl.steps],
                       [s.k.f64[r][:, hk_sel] for s in wl.steps],
                       [s.v.f64[r][:, sub_hv] for s in wl.steps],
                       [s.alpha.f64[r][:, sub_hv] for s in wl.steps],
                       [s.beta.f64[r][:, sub_hv] for s in wl.steps],
                       [s.parents[r] for s in wl.steps[1:]])
        for t in range(len(wl.steps)):
            res[t][r] = o[t]
    return res, sub_hv


def oracle_ancestry(wl: W.Workload):
    """[t] -> int32 [R][W_t][t] from the oracle's Eq. 5."""
    spec = wl.spec
    out = [np.zeros((spec.R, w, t), dtype=np.int32) for t, w in enumerate(spec.widths)]
    for r in range(spec.R):
        h = orc.ancestry(list(spec.widths), [s.parents[r] for s in wl.steps[1:]])
        for t in range(spec.T):
            out[t][r] = h[t]
    return out


def rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    num = np.max(np.abs(got - ref), axis=-1)
    den = np.maximum(np.max(np.abs(ref), axis=-1), 1e-30)
    return float(np.max(num / den)) if num.size else 0.0


@functools.lru_cache(maxsize=8)
def cached_case(name: str):
    """(workload, oracle S_ctx fp32, oracle outputs) of a named workload."""
    wl = W.make_workload(name)
    s0 = oracle_s0(wl)
    ref, heads = oracle_outputs(wl, s0)
    return wl, s0, ref
