"""Host-side driver of the decode path on one GPU.

Moves a :mod:`workload` to device memory (PyTorch is used only for
allocation and streams) and drives the C ABI in protocol order: for each
decode step t, ``onela_resolve_ancestry`` -> ``onela_append_records`` ->
``onela_decode_step``.  No arithmetic of the method happens here.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import onela as ab
from .workload import Tensor, Workload, WorkloadSpec


def _torch():
    import torch
    return torch


def device_tensor(x, device):
    """Copy a workload Tensor / numpy array to the device, keeping its bits."""
    torch = _torch()
    if isinstance(x, Tensor):
        arr = x.dev
        t = torch.from_numpy(np.ascontiguousarray(arr))
        if x.dtype == "bf16":
            t = t.view(torch.bfloat16)
        return t.to(device)
    return torch.from_numpy(np.ascontiguousarray(x)).to(device)


@dataclass
class DeviceStep:
    q: object
    k: object
    v: object
    alpha: object
    beta: object
    parents: object  # None at step 0
    width: int


@dataclass
class DeviceWorkload:
    spec: WorkloadSpec
    steps: list
    prompt: tuple | None  # (k, v, alpha, beta) or None


def to_device(wl: Workload, device="cuda:0", with_prompt: bool = True) -> DeviceWorkload:
    steps = []
    for t, st in enumerate(wl.steps):
        steps.append(DeviceStep(
            device_tensor(st.q, device), device_tensor(st.k, device),
            device_tensor(st.v, device), device_tensor(st.alpha, device),
            device_tensor(st.beta, device),
            None if st.parents is None else device_tensor(st.parents.astype(np.int32), device),
            int(wl.spec.widths[t])))
    prompt = None
    if with_prompt and wl.prompt_k is not None:
        prompt = tuple(device_tensor(x, device) for x in
                       (wl.prompt_k, wl.prompt_v, wl.prompt_alpha, wl.prompt_beta))
    return DeviceWorkload(wl.spec, steps, prompt)


def config_for(spec: WorkloadSpec, max_beams: int | None = None,
               max_steps: int | None = None, records: str = "inputs",
               storage: str = "copy") -> ab.onela_config_t:
    return ab.make_config(spec.R, spec.HK, spec.HV, spec.dk, spec.dv,
                          max_beams or spec.W, max_steps or spec.T, spec.io_dtype, records,
                          storage)


def prefill_state(spec: WorkloadSpec, prompt, device="cuda:0", stream=None):
    """S_ctx [R][HV][dv][dk] fp32 from the prompt, on the GPU."""
    torch = _torch()
    cfg = config_for(spec)
    s0 = torch.empty((spec.R, spec.HV, spec.dv, spec.dk), dtype=torch.float32, device=device)
    k, v, a, b = prompt
    ab.onela_prefill_state(cfg, spec.P, k, v, a, b, s0, stream)
    return s0


class Decoder:
    """One decode context (workspace + onela_ctx_t) bound to a stream."""

    def __init__(self, spec: WorkloadSpec, s0, device="cuda:0", stream=None,
                 max_beams: int | None = None, max_steps: int | None = None,
                 records: str = "inputs", storage: str = "copy"):
        """storage="borrow": the steps' k/v/alpha/beta tensors are the record
        slabs and must outlive the beam search (run() keeps them referenced)."""
        torch = _torch()
        self.spec = spec
        self.cfg = config_for(spec, max_beams, max_steps, records, storage)
        self._borrowed = []
        self.ws_bytes = ab.onela_workspace_bytes(self.cfg)
        if self.ws_bytes == 0:
            raise ab.OnelaError(ab.ONELA_EINVAL, "onela_workspace_bytes")
        self.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        self.stream = stream
        self.s0 = s0  # borrowed by the context until close()
        self.ctx = ab.onela_init(self.cfg, s0, self.workspace, self.ws_bytes, stream)

    def step(self, t: int, st: DeviceStep, o, gather_out=None, fused: bool = False):
        if self.cfg.record_storage == ab.ONELA_RECORDS_BORROW:
            self._borrowed.append(st)
        if fused:
            ab.onela_decode_step_fused(self.ctx, t, st.width, st.parents, st.k, st.v, st.alpha,
                                       st.beta, st.q, o, gather_out)
            return
        ab.onela_resolve_ancestry(self.ctx, t, st.width, st.parents, gather_out)
        ab.onela_append_records(self.ctx, t, st.k, st.v, st.alpha, st.beta)
        ab.onela_decode_step(self.ctx, t, st.q, o)

    def alloc_outputs(self, dw: DeviceWorkload):
        torch = _torch()
        s = self.spec
        return [torch.empty((s.R, st.width, s.HV, s.dv), dtype=torch.float32,
                            device=self.workspace.device) for st in dw.steps]

    def run(self, dw: DeviceWorkload, outs=None, gathers=None, fused=False):
        """Run every step; ``fused`` is a bool or a per-step list of bools."""
        if outs is None:
            outs = self.alloc_outputs(dw)
        for t, st in enumerate(dw.steps):
            f = fused[t] if isinstance(fused, (list, tuple)) else fused
            self.step(t, st, outs[t], None if gathers is None else gathers[t], f)
        return outs

    def reset(self):
        ab.onela_reset(self.ctx)
        self._borrowed = []

    def status(self) -> int:
        return ab.onela_get_device_status(self.ctx)

    def close(self):
        if self.ctx:
            ab.onela_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class FullStateBaseline:
    """The per-beam materialised-state GPU baseline (one call per step)."""

    def __init__(self, spec: WorkloadSpec, s0, device="cuda:0", stream=None):
        torch = _torch()
        self.spec = spec
        self.cfg = config_for(spec)
        self.s0 = s0
        self.ws_bytes = ab.onela_fullstate_workspace_bytes(self.cfg)
        self.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        self.status_word = torch.zeros(4, dtype=torch.int32, device=device)
        self.stream = stream

    def run(self, dw: DeviceWorkload, outs=None):
        torch = _torch()
        s = self.spec
        if outs is None:
            outs = [torch.empty((s.R, st.width, s.HV, s.dv), dtype=torch.float32,
                                device=self.workspace.device) for st in dw.steps]
        prev = 0
        for t, st in enumerate(dw.steps):
            ab.onela_fullstate_step(self.cfg, t, st.width, prev, st.parents, self.s0, st.q,
                                    st.k, st.v, st.alpha, st.beta, outs[t], self.workspace,
                                    self.ws_bytes, self.status_word, self.stream)
            prev = st.width
        return outs


class BeamSelector:
    """Global top-W beam selection (onela_select_beams) for fixed
    (R, W_prev, V, W): owns the workspace and the three output tensors."""

    def __init__(self, R: int, prev_width: int, vocab: int, width: int, device="cuda:0",
                 stream=None):
        torch = _torch()
        self.R, self.prev_width, self.vocab, self.width = R, prev_width, vocab, width
        self.ws_bytes = ab.onela_select_workspace_bytes(R, prev_width, vocab, width)
        # zero-filled once: the selection keeps its cross-workgroup state
        # here (a call counter, bound words, tagged summaries) and leaves it
        # ready for the next call
        self.workspace = torch.zeros(self.ws_bytes, dtype=torch.uint8, device=device)
        self.parents = torch.empty((R, width), dtype=torch.int32, device=device)
        self.tokens = torch.empty((R, width), dtype=torch.int32, device=device)
        self.scores = torch.empty((R, width), dtype=torch.float32, device=device)
        self.stream = stream

    def __call__(self, logp, beam_scores=None):
        ab.onela_select_beams(self.R, self.prev_width, self.vocab, self.width, logp,
                              beam_scores, self.parents, self.tokens, self.scores,
                              self.workspace, self.ws_bytes, self.stream)
        return self.parents, self.tokens, self.scores
