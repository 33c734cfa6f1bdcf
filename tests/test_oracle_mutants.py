"""Plants plausible mistakes in a copy of the C oracle (CPU only) and checks
that the pin suite catches every one of them.  The real oracle source is not
modified; each mutant is compiled from a patched copy in a temp directory."""
import ctypes
import os

import numpy as np
import pytest

from oracle import oracle as orc
from tests import oracle_pins as pins

SRC = os.path.join(os.path.dirname(orc.__file__), "gdn_oracle.c")

# (name, original text, mutated text)
MUTANTS = [
    ("dropped_alpha_in_delta", "double w = beta * (v[i] - alpha * u[i]);",
     "double w = beta * (v[i] - u[i]);"),
    ("dropped_beta", "double w = beta * (v[i] - alpha * u[i]);",
     "double w = (v[i] - alpha * u[i]);"),
    ("wrong_sign_update", "alpha * S[(size_t)i * dk + j] + w * k[j];",
     "alpha * S[(size_t)i * dk + j] - w * k[j];"),
    ("dropped_decay", "alpha * S[(size_t)i * dk + j] + w * k[j];",
     "S[(size_t)i * dk + j] + w * k[j];"),
    ("transposed_key_projection",
     "for (int j = 0; j < dk; ++j) acc += S[(size_t)i * dk + j] * k[j];",
     "for (int j = 0; j < dk; ++j) acc += S[(size_t)j * dk + i] * k[j];"),
    ("transposed_readout",
     "for (int j = 0; j < dk; ++j) acc += S[(size_t)i * dk + j] * q[j];",
     "for (int j = 0; j < dk; ++j) acc += S[(size_t)j * dk + i] * q[j];"),
    ("readout_before_update", "gdn_readout(S, dv, dk,",
     "gdn_readout(prev + (size_t)src * ssz, dv, dk,"),
    ("wrong_gqa_head_map",
     "    const int hk = hv / group;\n    double* prev",
     "    const int hk = hv % HK;\n    double* prev"),
    ("parent_ignored", "const int src = (t == 0) ? 0 : par[b];",
     "const int src = (t == 0) ? 0 : b % widths[t - 1];"),
    ("ancestry_last_slot_is_self", "h_cur[(size_t)b * t + (t - 1)] = p;",
     "h_cur[(size_t)b * t + (t - 1)] = b % widths[t - 1];"),
    ("ancestry_reversed_inherit", "h_prev[(size_t)p * (t - 1) + j];",
     "h_prev[(size_t)p * (t - 1) + (t - 2 - j)];"),
    ("prefill_drops_first_token", "for (int p = 0; p < P; ++p) {",
     "for (int p = 1; p < P; ++p) {"),
    ("key_used_as_query", "gdn_readout(S, dv, dk, q + (row * HK + hk) * dk,",
     "gdn_readout(S, dv, dk, k + (row * HK + hk) * dk,"),
]


def _pins_fail(lib):
    failures = []
    for pin in pins.ALL_PINS:
        kw = {"n_configs": 40} if pin is pins.pin_exact_rational_bruteforce else {}
        try:
            pin(lib, **kw)
        except (AssertionError, ValueError, IndexError, FloatingPointError) as e:
            failures.append(pin.__name__)
    return failures


@pytest.mark.parametrize("name,orig,mut", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, orig, mut):
    src = open(SRC).read()
    assert src.count(orig) == 1, f"mutation anchor not unique/present: {name}"
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(orig, mut))
    so = str(tmp_path / "libmutant.so")
    orc.build(src=str(path), out=so)
    lib = orc.load(path=so)
    with np.errstate(all="ignore"):
        failed = _pins_fail(lib)
    assert failed, f"mutant {name} passed every pin"


# Mistakes planted in the beam-selection oracle (a numpy function): each is a
# textual edit of its source, executed in a scratch namespace.
SELECT_MUTANTS = [
    ("ties_by_highest_index", "np.lexsort((idx, sign, -vals, isnan))",
     "np.lexsort((-idx, sign, -vals, isnan))"),
    ("signed_zero_ignored", "np.lexsort((idx, sign, -vals, isnan))",
     "np.lexsort((idx, -vals, isnan))"),
    ("nan_ranked_first", "np.lexsort((idx, sign, -vals, isnan))",
     "np.lexsort((idx, sign, -vals, ~isnan))"),
    ("ascending_scores", "np.lexsort((idx, sign, -vals, isnan))",
     "np.lexsort((idx, sign, vals, isnan))"),
    ("nan_sign_kept", "sign = np.signbit(flat) & ~isnan", "sign = np.signbit(flat)"),
    ("beam_score_ignored", "s = (b + s).astype(np.float32)", "s = s"),
    ("parent_token_swapped", "return (top // V).astype(np.int32), (top % V)",
     "return (top % V).astype(np.int32), (top // V)"),
]


@pytest.mark.parametrize("name,orig,mut", SELECT_MUTANTS, ids=[m[0] for m in SELECT_MUTANTS])
def test_select_mutant_is_caught(name, orig, mut):
    import inspect
    import textwrap
    src = textwrap.dedent(inspect.getsource(orc.select_beams))
    assert src.count(orig) == 1, f"mutation anchor not unique/present: {name}"
    ns = {"np": np}
    exec(compile(src.replace(orig, mut), f"<mutant {name}>", "exec"), ns)
    with pytest.raises(AssertionError):
        pins.pin_select_beams(select=ns["select_beams"])
