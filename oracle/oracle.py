"""fp64 CPU oracle for the large-beam GDN decode -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this module.  The product library never imports it
and shares no code with it.

The arithmetic lives in ``gdn_oracle.c`` (plain C, fp64, no blocking or
fusion); this file only builds that C file with gcc, loads it with ctypes and
marshals numpy arrays.  The functions follow the OneLA paper (arXiv
2609.12399):

* :func:`prefill`  -- Sec. 2.2 Eq. 1 applied over a prompt from S = 0, giving
  the shared post-prefill state S_ctx (Sec. 3.1).
* :func:`ancestry` -- Sec. 3.3 Eq. 5 on integers.
* :func:`decode`   -- per-beam materialised states: each beam copies its
  parent's state (Sec. 2.1, Sec. 3.1), applies Eq. 1 and reads out
  o = S q after the update.

Each function is pinned by tests against closed forms, exact-rational brute
force and special cases (see ``tests/test_oracle_pins.py``).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gdn_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

_D = ctypes.POINTER(ctypes.c_double)
_I = ctypes.POINTER(ctypes.c_int)


def build(src: str = _SRC, out: str = _LIB_PATH, extra_flags=()) -> str:
    """Compile the C oracle with gcc (-O2, IEEE fp64, OpenMP)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
           "-ffp-contract=off", *extra_flags, src, "-o", out]
    subprocess.run(cmd, check=True)
    return out


def load(path: str = _LIB_PATH, rebuild_if_missing: bool = True):
    """Load (building first if needed) the oracle shared library."""
    global _lib
    if path == _LIB_PATH and _lib is not None:
        return _lib
    if not os.path.exists(path) or (
            path == _LIB_PATH and os.path.getmtime(path) < os.path.getmtime(_SRC)):
        if not rebuild_if_missing:
            raise FileNotFoundError(path)
        build(out=path)
    lib = ctypes.CDLL(path)
    lib.oracle_gdn_prefill.argtypes = [ctypes.c_int] * 5 + [_D] * 5 + [ctypes.c_int]
    lib.oracle_gdn_prefill.restype = ctypes.c_int
    lib.oracle_ancestry.argtypes = [ctypes.c_int, _I, _I, _I]
    lib.oracle_ancestry.restype = ctypes.c_int
    lib.oracle_gdn_decode.argtypes = ([ctypes.c_int, _I] + [ctypes.c_int] * 4
                                      + [_D] * 6 + [_I, _D, ctypes.c_int])
    lib.oracle_gdn_decode.restype = ctypes.c_int
    lib.oracle_max_threads.argtypes = []
    lib.oracle_max_threads.restype = ctypes.c_int
    if path == _LIB_PATH:
        _lib = lib
    return lib


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


def _dp(a: np.ndarray):
    return a.ctypes.data_as(_D)


def _ip(a: np.ndarray):
    return a.ctypes.data_as(_I)


def default_threads() -> int:
    return len(os.sched_getaffinity(0))


def prefill(k, v, alpha, beta, *, nthreads: int | None = None, lib=None) -> np.ndarray:
    """S_ctx of one request from a prompt (Eq. 1 from S = 0).

    k [P][HK][dk], v [P][HV][dv], alpha/beta [P][HV]  ->  S [HV][dv][dk] fp64.
    """
    lib = lib or load()
    k, v, alpha, beta = _f64(k), _f64(v), _f64(alpha), _f64(beta)
    P, HK, dk = k.shape
    _, HV, dv = v.shape
    S = np.empty((HV, dv, dk), dtype=np.float64)
    rc = lib.oracle_gdn_prefill(P, HK, HV, dk, dv, _dp(k), _dp(v), _dp(alpha),
                                _dp(beta), _dp(S), nthreads or default_threads())
    if rc != 0:
        raise ValueError(f"oracle_gdn_prefill failed ({rc})")
    return S


def ancestry(widths, parents, *, lib=None) -> list[np.ndarray]:
    """Eq. 5 for one request.

    widths: [T] ints; parents: list of T-1 int arrays (steps 1..T-1), each
    [W_t].  Returns [h_0, ..., h_{T-1}] with h_t of shape [W_t][t].
    """
    lib = lib or load()
    widths = _i32(widths)
    T = int(widths.shape[0])
    par = _i32(np.concatenate([np.asarray(p, dtype=np.int64) for p in parents])
               if len(parents) else np.zeros(0))
    total = int(sum(int(widths[t]) * t for t in range(T)))
    h = np.zeros(max(total, 1), dtype=np.int32)
    rc = lib.oracle_ancestry(T, _ip(widths), _ip(par), _ip(h))
    if rc != 0:
        raise ValueError("oracle_ancestry: parent out of range")
    out, off = [], 0
    for t in range(T):
        n = int(widths[t]) * t
        out.append(h[off:off + n].reshape(int(widths[t]), t).copy())
        off += n
    return out


def decode(S0, q, k, v, alpha, beta, parents, *, nthreads: int | None = None,
           lib=None) -> list[np.ndarray]:
    """FullState large-beam decode of one request.

    S0 [HV][dv][dk]; q/k/v/alpha/beta: lists over steps t of [W_t][HK][dk],
    [W_t][HK][dk], [W_t][HV][dv], [W_t][HV], [W_t][HV]; parents: list over
    t = 1..T-1 of [W_t].  Returns a list over t of o_t [W_t][HV][dv] (fp64).
    """
    lib = lib or load()
    T = len(q)
    widths = _i32([np.asarray(x).shape[0] for x in q])
    S0 = _f64(S0)
    HV, dv, dk = S0.shape
    HK = np.asarray(q[0]).shape[1] if T else 1
    cat = lambda xs: _f64(np.concatenate([np.asarray(x, dtype=np.float64).reshape(-1)
                                          for x in xs]) if len(xs) else np.zeros(1))
    qc, kc, vc, ac, bc = cat(q), cat(k), cat(v), cat(alpha), cat(beta)
    par = _i32(np.concatenate([np.asarray(p, dtype=np.int64) for p in parents])
               if len(parents) else np.zeros(1))
    o = np.empty(max(int(widths.sum()) * HV * dv, 1), dtype=np.float64)
    rc = lib.oracle_gdn_decode(T, _ip(widths), HK, HV, dk, dv, _dp(S0), _dp(qc),
                               _dp(kc), _dp(vc), _dp(ac), _dp(bc), _ip(par),
                               _dp(o), nthreads or default_threads())
    if rc == -2:
        raise ValueError("oracle_gdn_decode: parent out of range")
    if rc != 0:
        raise ValueError(f"oracle_gdn_decode failed ({rc})")
    out, off = [], 0
    for t in range(T):
        n = int(widths[t]) * HV * dv
        out.append(o[off:off + n].reshape(int(widths[t]), HV, dv).copy())
        off += n
    return out


def select_beams(scores, width: int, beam_scores=None):
    """Global top-W beam selection of one request (Sec. 2.1: every live beam
    is expanded over the codebook and the global top-W candidates are kept).

    scores [W_prev][V] (fp32); beam_scores optional [W_prev] (fp32).  The
    candidate score of (p, v) is scores[p][v], or beam_scores[p] +
    scores[p][v] rounded once to fp32 when beam_scores is given.  Returns
    (parents [width], tokens [width], candidate scores [width]) in rank order.
    Order: higher score first; equal scores by lower flat index p * V + v;
    -0.0 ranks below +0.0; NaN (of either sign) below every number, NaNs among
    themselves by flat index.  Implemented as a plain sort of (score, index)
    pairs.
    """
    s = np.asarray(scores, dtype=np.float32)
    P, V = s.shape
    if beam_scores is not None:
        b = np.asarray(beam_scores, dtype=np.float32).reshape(P, 1)
        s = (b + s).astype(np.float32)
    flat = s.reshape(-1)
    if not 1 <= width <= flat.size:
        raise ValueError("width must be in [1, W_prev * V]")
    isnan = np.isnan(flat)
    sign = np.signbit(flat) & ~isnan
    idx = np.arange(flat.size)
    vals = np.where(isnan, 0.0, flat.astype(np.float64))
    # lexsort: last key is primary.  Primary: not-NaN first; then value
    # descending; then +0 before -0; then index ascending.
    order = np.lexsort((idx, sign, -vals, isnan))
    top = order[:width]
    return (top // V).astype(np.int32), (top % V).astype(np.int32), flat[top]
