"""Thin ctypes binding of libonela (include/onela.h), same names as the C ABI.

This module only marshals arguments: every step of the decode path runs in
the HIP kernels of ``libonela.so``.  Device-pointer arguments accept a torch
tensor that lives on a GPU (its ``data_ptr()`` is passed), a raw integer
address, or None for an optional pointer.  Streams accept a
``torch.cuda.Stream``, a raw ``hipStream_t`` integer, or None (torch's
current stream).  A non-OK status raises :class:`OnelaError`.

There is no fallback: if ``libonela.so`` has not been built, loading raises.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libonela.so")

ONELA_OK, ONELA_EINVAL, ONELA_ESTEP, ONELA_EPARENT = 0, 1, 2, 3
ONELA_ECAPACITY, ONELA_EHIP, ONELA_ENOMEM = 4, 5, 6
ONELA_F32, ONELA_BF16 = 0, 1
ONELA_RECORD_INPUTS, ONELA_RECORD_DELTA = 0, 1
ONELA_RECORDS_COPY, ONELA_RECORDS_BORROW = 0, 1

STATUS_NAMES = {0: "ONELA_OK", 1: "ONELA_EINVAL", 2: "ONELA_ESTEP", 3: "ONELA_EPARENT",
                4: "ONELA_ECAPACITY", 5: "ONELA_EHIP", 6: "ONELA_ENOMEM"}

# every symbol declared in include/onela.h
EXPORTED = ["onela_status_str", "onela_check_config", "onela_workspace_bytes", "onela_init",
            "onela_reset", "onela_resolve_ancestry", "onela_append_records",
            "onela_decode_step", "onela_decode_step_fused", "onela_get_device_status", "onela_destroy",
            "onela_prefill_state", "onela_fullstate_workspace_bytes", "onela_fullstate_step",
            "onela_capacity_bytes", "onela_fullstate_capacity_bytes",
            "onela_select_workspace_bytes", "onela_select_beams", "onela_select_beams_noalloc",
            "onela_prefill_workspace_bytes", "onela_prefill_state_chunked"]


class OnelaError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)}")


class onela_config_t(ctypes.Structure):
    _fields_ = [("num_requests", ctypes.c_int32), ("num_qk_heads", ctypes.c_int32),
                ("num_v_heads", ctypes.c_int32), ("d_k", ctypes.c_int32),
                ("d_v", ctypes.c_int32), ("max_beams", ctypes.c_int32),
                ("max_steps", ctypes.c_int32), ("io_dtype", ctypes.c_int32),
                ("record_kind", ctypes.c_int32), ("record_storage", ctypes.c_int32)]


def make_config(num_requests, num_qk_heads, num_v_heads, d_k, d_v, max_beams, max_steps,
                io_dtype, record_kind=ONELA_RECORD_INPUTS,
                record_storage=ONELA_RECORDS_COPY) -> onela_config_t:
    if isinstance(io_dtype, str):
        io_dtype = {"bf16": ONELA_BF16, "f32": ONELA_F32}[io_dtype]
    if isinstance(record_kind, str):
        record_kind = {"inputs": ONELA_RECORD_INPUTS, "delta": ONELA_RECORD_DELTA}[record_kind]
    if isinstance(record_storage, str):
        record_storage = {"copy": ONELA_RECORDS_COPY, "borrow": ONELA_RECORDS_BORROW}[record_storage]
    return onela_config_t(num_requests, num_qk_heads, num_v_heads, d_k, d_v, max_beams,
                          max_steps, io_dtype, record_kind, record_storage)


_lib = None
_P = ctypes.c_void_p
_I32 = ctypes.c_int32


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libonela.so (raises if it is missing: there is no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"libonela.so not built at {path}; run "
                          "`python -m paper_2609_12399_amd.build`")
    # torch ships its own HIP runtime; it must be loaded before the library so
    # that the library binds to that runtime (loaded first, the library would
    # bring in a second runtime in which torch's device pointers are invalid).
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    cfgp = ctypes.POINTER(onela_config_t)
    sig = {
        "onela_status_str": ([_I32], ctypes.c_char_p),
        "onela_check_config": ([cfgp], _I32),
        "onela_workspace_bytes": ([cfgp], ctypes.c_size_t),
        "onela_init": ([cfgp, _P, _P, ctypes.c_size_t, _P, ctypes.POINTER(_P)], _I32),
        "onela_reset": ([_P], _I32),
        "onela_resolve_ancestry": ([_P, _I32, _I32, _P, _P], _I32),
        "onela_append_records": ([_P, _I32, _P, _P, _P, _P], _I32),
        "onela_decode_step": ([_P, _I32, _P, _P], _I32),
        "onela_decode_step_fused": ([_P, _I32, _I32, _P, _P, _P, _P, _P, _P, _P, _P], _I32),
        "onela_get_device_status": ([_P], _I32),
        "onela_destroy": ([_P], None),
        "onela_prefill_state": ([cfgp, _I32, _P, _P, _P, _P, _P, _P], _I32),
        "onela_fullstate_workspace_bytes": ([cfgp], ctypes.c_size_t),
        "onela_fullstate_step": ([cfgp, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                  ctypes.c_size_t, _P, _P], _I32),
        "onela_capacity_bytes": ([_I32] * 8, ctypes.c_uint64),
        "onela_fullstate_capacity_bytes": ([_I32] * 6, ctypes.c_uint64),
        "onela_select_workspace_bytes": ([_I32] * 4 + [ctypes.POINTER(ctypes.c_size_t)], _I32),
        "onela_select_beams": ([_I32] * 4 + [_P] * 6 + [ctypes.c_size_t, _P], _I32),
        "onela_select_beams_noalloc": ([_I32] * 4 + [_P] * 6, _I32),
        "onela_prefill_workspace_bytes": ([cfgp, _I32], ctypes.c_size_t),
        "onela_prefill_state_chunked": ([cfgp, _I32] + [_P] * 6 + [ctypes.c_size_t, _P], _I32),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def _dev(x, name: str, optional: bool = False):
    """Device address of a GPU tensor / raw int; None -> NULL if optional."""
    if x is None:
        if optional:
            return None
        raise ValueError(f"{name} must not be None")
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        if not getattr(x, "is_cuda", False):
            raise ValueError(f"{name} must be a GPU tensor")
        if not x.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        return x.data_ptr()
    raise TypeError(f"{name}: unsupported pointer type {type(x)}")


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(rc: int, where: str):
    if rc != ONELA_OK:
        raise OnelaError(rc, where)


def onela_status_str(status: int) -> str:
    return load_library().onela_status_str(status).decode()


def onela_check_config(cfg: onela_config_t) -> int:
    return load_library().onela_check_config(ctypes.byref(cfg))


def onela_workspace_bytes(cfg: onela_config_t) -> int:
    return load_library().onela_workspace_bytes(ctypes.byref(cfg))


def onela_init(cfg: onela_config_t, s0, workspace, workspace_bytes: int, stream=None):
    """Returns the context handle (an int)."""
    out = _P()
    _check(load_library().onela_init(ctypes.byref(cfg), _dev(s0, "s0"),
                                     _dev(workspace, "workspace"), int(workspace_bytes),
                                     _stream(stream), ctypes.byref(out)), "onela_init")
    return out.value


def onela_reset(ctx):
    _check(load_library().onela_reset(ctx), "onela_reset")


def onela_resolve_ancestry(ctx, step: int, width: int, parents=None, gather_out=None):
    _check(load_library().onela_resolve_ancestry(
        ctx, step, width, _dev(parents, "parents", optional=True),
        _dev(gather_out, "gather_out", optional=True)), "onela_resolve_ancestry")


def onela_append_records(ctx, step: int, k, v, alpha, beta):
    _check(load_library().onela_append_records(ctx, step, _dev(k, "k"), _dev(v, "v"),
                                               _dev(alpha, "alpha"), _dev(beta, "beta")),
           "onela_append_records")


def onela_decode_step(ctx, step: int, q, o):
    _check(load_library().onela_decode_step(ctx, step, _dev(q, "q"), _dev(o, "o")),
           "onela_decode_step")


def onela_decode_step_fused(ctx, step: int, width: int, parents, k, v, alpha, beta, q, o,
                            gather_out=None):
    _check(load_library().onela_decode_step_fused(
        ctx, step, width, _dev(parents, "parents", optional=True), _dev(k, "k"), _dev(v, "v"),
        _dev(alpha, "alpha"), _dev(beta, "beta"), _dev(q, "q"), _dev(o, "o"),
        _dev(gather_out, "gather_out", optional=True)), "onela_decode_step_fused")


def onela_get_device_status(ctx) -> int:
    """Synchronises; returns ONELA_OK or ONELA_EPARENT (raises on HIP errors)."""
    rc = load_library().onela_get_device_status(ctx)
    if rc not in (ONELA_OK, ONELA_EPARENT):
        raise OnelaError(rc, "onela_get_device_status")
    return rc


def onela_destroy(ctx):
    if ctx:
        load_library().onela_destroy(ctx)


def onela_prefill_state(cfg: onela_config_t, prompt_len: int, k, v, alpha, beta, s0_out,
                        stream=None):
    opt = prompt_len == 0
    _check(load_library().onela_prefill_state(
        ctypes.byref(cfg), prompt_len, _dev(k, "k", opt), _dev(v, "v", opt),
        _dev(alpha, "alpha", opt), _dev(beta, "beta", opt), _dev(s0_out, "s0_out"),
        _stream(stream)), "onela_prefill_state")


def onela_fullstate_workspace_bytes(cfg: onela_config_t) -> int:
    return load_library().onela_fullstate_workspace_bytes(ctypes.byref(cfg))


def onela_fullstate_step(cfg: onela_config_t, step: int, width: int, prev_width: int,
                         parents, s0, q, k, v, alpha, beta, o, workspace,
                         workspace_bytes: int, status_word=None, stream=None):
    _check(load_library().onela_fullstate_step(
        ctypes.byref(cfg), step, width, prev_width, _dev(parents, "parents", True),
        _dev(s0, "s0"), _dev(q, "q"), _dev(k, "k"), _dev(v, "v"), _dev(alpha, "alpha"),
        _dev(beta, "beta"), _dev(o, "o"), _dev(workspace, "workspace"),
        int(workspace_bytes), _dev(status_word, "status_word", True), _stream(stream)),
        "onela_fullstate_step")


def onela_capacity_bytes(num_requests, num_v_heads, d_k, d_v, beams, steps, state_bytes,
                         record_bytes) -> int:
    return load_library().onela_capacity_bytes(num_requests, num_v_heads, d_k, d_v, beams,
                                               steps, state_bytes, record_bytes)


def onela_fullstate_capacity_bytes(num_requests, num_v_heads, d_k, d_v, beams,
                                   state_bytes) -> int:
    return load_library().onela_fullstate_capacity_bytes(num_requests, num_v_heads, d_k, d_v,
                                                         beams, state_bytes)


def onela_select_workspace_bytes(num_requests: int, prev_width: int, vocab: int,
                                 width: int) -> int:
    out = ctypes.c_size_t(0)
    _check(load_library().onela_select_workspace_bytes(num_requests, prev_width, vocab, width,
                                                        ctypes.byref(out)),
           "onela_select_workspace_bytes")
    return out.value


def onela_select_beams(num_requests: int, prev_width: int, vocab: int, width: int, logp,
                       beam_scores, parents_out, tokens_out, scores_out, workspace=None,
                       workspace_bytes: int = 0, stream=None):
    _check(load_library().onela_select_beams(
        num_requests, prev_width, vocab, width, _dev(logp, "logp"),
        _dev(beam_scores, "beam_scores", optional=True), _dev(parents_out, "parents_out"),
        _dev(tokens_out, "tokens_out"), _dev(scores_out, "scores_out"),
        _dev(workspace, "workspace", optional=True), int(workspace_bytes), _stream(stream)),
        "onela_select_beams")


def onela_select_beams_noalloc(num_requests: int, prev_width: int, vocab: int, width: int,
                               logp, beam_scores, parents_out, tokens_out, scores_out,
                               stream=None):
    _check(load_library().onela_select_beams_noalloc(
        num_requests, prev_width, vocab, width, _dev(logp, "logp"),
        _dev(beam_scores, "beam_scores", optional=True), _dev(parents_out, "parents_out"),
        _dev(tokens_out, "tokens_out"), _dev(scores_out, "scores_out"), _stream(stream)),
        "onela_select_beams_noalloc")


def onela_prefill_workspace_bytes(cfg: onela_config_t, prompt_len: int) -> int:
    return load_library().onela_prefill_workspace_bytes(ctypes.byref(cfg), prompt_len)


def onela_prefill_state_chunked(cfg: onela_config_t, prompt_len: int, k, v, alpha, beta,
                                s0_out, workspace=None, workspace_bytes: int = 0, stream=None):
    opt = prompt_len == 0
    _check(load_library().onela_prefill_state_chunked(
        ctypes.byref(cfg), prompt_len, _dev(k, "k", opt), _dev(v, "v", opt),
        _dev(alpha, "alpha", opt), _dev(beta, "beta", opt), _dev(s0_out, "s0_out"),
        _dev(workspace, "workspace", optional=True), int(workspace_bytes), _stream(stream)),
        "onela_prefill_state_chunked")
