"""Chunked prefill of S_ctx (onela_prefill_state_chunked) against the fp64
oracle's Eq. 1 recurrence over the prompt, through the C ABI.

Metric: per (request, value head), max |S_gpu - S_ref| / max |S_ref|, with
the bar 1e-4 (fp32 state against fp64; the sequential GPU prefill is held to
the same bar)."""
import numpy as np
import pytest

from oracle import oracle as orc
from paper_2609_12399_amd import onela as ab
from paper_2609_12399_amd import runner
from paper_2609_12399_amd import workload as W
from tests.gpu_common import log

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
DEV = "cuda:0"
TOL = 1e-4


def oracle_state(wl):
    return np.stack([orc.prefill(wl.prompt_k.f64[r], wl.prompt_v.f64[r],
                                 wl.prompt_alpha.f64[r], wl.prompt_beta.f64[r])
                     for r in range(wl.spec.R)])


def state_err(got, ref):
    got = np.asarray(got, dtype=np.float64)
    num = np.abs(got - ref).reshape(ref.shape[0], ref.shape[1], -1).max(-1)
    den = np.maximum(np.abs(ref).reshape(ref.shape[0], ref.shape[1], -1).max(-1), 1e-30)
    return float((num / den).max())


def run_chunked(wl, P=None):
    spec = wl.spec
    P = spec.P if P is None else P
    cfg = runner.config_for(spec)
    prompt = [runner.device_tensor(x, DEV) for x in
              (wl.prompt_k, wl.prompt_v, wl.prompt_alpha, wl.prompt_beta)]
    nbytes = ab.onela_prefill_workspace_bytes(cfg, P)
    ws = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=DEV) if nbytes else None
    s0 = torch.full((spec.R, spec.HV, spec.dv, spec.dk), float("nan"), dtype=torch.float32,
                    device=DEV)
    ab.onela_prefill_state_chunked(cfg, P, *prompt, s0, ws, nbytes)
    torch.cuda.synchronize()
    return s0.cpu().numpy()


@pytest.mark.parametrize("name", list(W.SPECS))
def test_chunked_prefill_matches_oracle(name):
    wl = W.make_workload(name)
    log(f"[prefill] {name} P={wl.spec.P}")
    ref = oracle_state(wl)
    got = run_chunked(wl)
    err = state_err(got, ref)
    log(f"[prefill] {name} err {err:.2e}")
    assert err <= TOL


@pytest.mark.parametrize("P", [1, 5, 63, 64, 65, 100, 191])
def test_chunked_prefill_ragged_prompts(P):
    spec = W.with_widths("h16_d128_w128", (8,), P=P, HK=2, HV=4)
    wl = W.make_workload(spec)
    got = run_chunked(wl)
    assert state_err(got, oracle_state(wl)) <= TOL


def test_chunked_prefill_empty_prompt_is_zero():
    spec = W.with_widths("h16_d128_w128", (8,), P=0, HK=2, HV=4)
    cfg = runner.config_for(spec)
    assert ab.onela_prefill_workspace_bytes(cfg, 0) == 0
    s0 = torch.full((1, 4, 128, 128), 7.0, dtype=torch.float32, device=DEV)
    ab.onela_prefill_state_chunked(cfg, 0, None, None, None, None, s0, None, 0)
    torch.cuda.synchronize()
    assert float(s0.abs().max()) == 0.0


def test_chunked_prefill_zero_decay_tokens():
    """alpha = 0 inside the prompt forgets everything before it exactly (no
    division by a vanishing cumulative decay)."""
    spec = W.with_widths("h16_d128_w128", (8,), P=150, HK=2, HV=4)
    wl = W.make_workload(spec)
    a = wl.prompt_alpha.dev.copy()
    a[:, [3, 70, 71, 128], :] = 0.0
    wl.prompt_alpha.dev = a
    got = run_chunked(wl)
    assert state_err(got, oracle_state(wl)) <= TOL


@pytest.mark.parametrize("dk,dv,io", [(128, 256, "bf16"), (128, 512, "bf16"), (256, 256, "bf16"),
                                       (256, 512, "bf16"), (32, 32, "f32"), (64, 64, "f32"),
                                       (128, 128, "f32"), (32, 32, "bf16"), (64, 64, "bf16")])
def test_chunked_prefill_geometries(dk, dv, io):
    spec = W.WorkloadSpec(f"pf_{dk}_{dv}", 2, 2, 4, dk, dv, 200, (8,), io, "uniform", seed=3)
    wl = W.make_workload(spec)
    got = run_chunked(wl)
    err = state_err(got, oracle_state(wl))
    log(f"[prefill] dk={dk} dv={dv} {io} err {err:.2e}")
    assert err <= TOL


def test_chunked_matches_sequential_prefill():
    wl = W.make_workload("h16_d128_w512")
    prompt = tuple(runner.device_tensor(x, DEV) for x in
                   (wl.prompt_k, wl.prompt_v, wl.prompt_alpha, wl.prompt_beta))
    seq = runner.prefill_state(wl.spec, prompt, DEV).cpu().numpy()
    got = run_chunked(wl)
    assert state_err(got, seq.astype(np.float64)) <= TOL
