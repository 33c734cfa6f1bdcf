"""Pins of the fp64 oracle against what the OneLA paper and the mathematics fix.

Every ``pin_*`` function takes a loaded oracle library (so that the mutation
test can run the same pins against deliberately broken copies of the oracle)
and raises AssertionError when the oracle disagrees.  None of them re-types
the oracle's loops: each checks a closed form, an exact-rational brute force,
a special case that reduces to a textbook formula, an invariant, or the
paper's alternative computation of the same quantity.

Notation (Sec. 2.2 Eq. 1 of arXiv 2609.12399): S is d_v x d_k,
S_t = alpha_t S_{t-1} + beta_t (v_t - alpha_t S_{t-1} k_t) k_t^T, o_t = S_t q_t.
Writing A_j = alpha_j (I - beta_j k_j k_j^T), Eq. 1 is
S_j = S_{j-1} A_j + beta_j v_j k_j^T, which unrolls to the closed form
S_t = S_ctx A_0 ... A_t + sum_j beta_j v_j k_j^T A_{j+1} ... A_t.
"""
from __future__ import annotations

import itertools
import math
from fractions import Fraction as Fr

import numpy as np

from oracle import oracle as orc

# ----------------------------------------------------------------------------
# exact rational linear algebra (tiny sizes only)


def _fmat(a):
    a = np.asarray(a, dtype=np.float64)
    if a.ndim == 1:
        return [Fr(float(x)) for x in a]
    return [[Fr(float(x)) for x in row] for row in a]


def _mm(A, B):
    n, m, p = len(A), len(B), len(B[0])
    return [[sum((A[i][l] * B[l][j] for l in range(m)), Fr(0)) for j in range(p)]
            for i in range(n)]


def _mv(A, x):
    return [sum((A[i][l] * x[l] for l in range(len(x))), Fr(0)) for i in range(len(A))]


def _eye(n):
    return [[Fr(int(i == j)) for j in range(n)] for i in range(n)]


def _A(k, alpha, beta):
    """A_j = alpha (I - beta k k^T), exact."""
    n = len(k)
    return [[alpha * (Fr(int(i == j)) - beta * k[i] * k[j]) for j in range(n)]
            for i in range(n)]


def closed_form_state(S0, chain):
    """S after the records in ``chain`` (oldest first), by the unrolled
    product form -- matrix products only, no step-by-step recurrence."""
    dv, dk = len(S0), len(S0[0])
    As = [_A(k, a, b) for (k, v, a, b) in chain]

    def prod(lo):
        M = _eye(dk)
        for A in As[lo:]:
            M = _mm(M, A)
        return M

    S = _mm(S0, prod(0))
    for j, (k, v, a, b) in enumerate(chain):
        outer = [[b * v[i] * k[l] for l in range(dk)] for i in range(dv)]
        T = _mm(outer, prod(j + 1))
        S = [[S[i][l] + T[i][l] for l in range(dk)] for i in range(dv)]
    return S


def _rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


# ----------------------------------------------------------------------------
# dyadic random inputs: exactly representable in fp64, so the oracle and the
# rational reference start from identical values


def dyadic_tree_inputs(rng, T, W, HK, HV, d):
    def vec(*shape):
        return rng.integers(-8, 9, size=shape).astype(np.float64) / 8.0

    S0 = rng.integers(-16, 17, size=(HV, d, d)).astype(np.float64) / 16.0
    q = [vec(W, HK, d) for _ in range(T)]
    k = [vec(W, HK, d) for _ in range(T)]
    v = [vec(W, HV, d) for _ in range(T)]
    al = [rng.integers(1, 17, size=(W, HV)).astype(np.float64) / 16.0 for _ in range(T)]
    be = [rng.integers(0, 17, size=(W, HV)).astype(np.float64) / 16.0 for _ in range(T)]
    return S0, q, k, v, al, be


def chase_path(parents, t, b):
    """Slots of beam b's ancestors at steps 0..t-1 by following parent
    pointers backwards (independent of the Eq. 5 table)."""
    path = [0] * t
    cur = b
    for s in range(t, 0, -1):
        cur = int(parents[s - 1][cur])
        path[s - 1] = cur
    return path


# ----------------------------------------------------------------------------
# pins


def pin_exact_rational_bruteforce(lib, n_configs=None, seed=7):
    """d = 4, W = 3, T = 3, HK = 2, HV = 4: every parent configuration (3^3 for
    each of steps 1 and 2, 729 trees; or a seeded subset), each beam output
    against the exact rational closed form of its own ancestry path."""
    T, W, HK, HV, d = 3, 3, 2, 4, 4
    G = HV // HK
    rng = np.random.default_rng(seed)
    S0, q, k, v, al, be = dyadic_tree_inputs(rng, T, W, HK, HV, d)
    S0f = [_fmat(S0[h]) for h in range(HV)]
    memo = {}

    def exact(t, path_slots, b, hv):
        key = (t, tuple(path_slots), b, hv)
        if key not in memo:
            hk = hv // G
            chain = []
            for j, s in enumerate(list(path_slots) + [b]):
                chain.append((_fmat(k[j][s, hk]), _fmat(v[j][s, hv]),
                              Fr(float(al[j][s, hv])), Fr(float(be[j][s, hv]))))
            S = closed_form_state(S0f[hv], chain)
            memo[key] = np.array([float(x) for x in _mv(S, _fmat(q[t][b, hk]))])
        return memo[key]

    all_par = list(itertools.product(range(W), repeat=W))
    configs = list(itertools.product(all_par, all_par))
    if n_configs is not None:
        idx = rng.choice(len(configs), size=n_configs, replace=False)
        configs = [configs[i] for i in idx]
    worst = 0.0
    for p1, p2 in configs:
        parents = [np.array(p1, dtype=np.int32), np.array(p2, dtype=np.int32)]
        o = orc.decode(S0, q, k, v, al, be, parents, nthreads=1, lib=lib)
        for t in range(T):
            for b in range(W):
                path = chase_path(parents, t, b)
                for hv in range(HV):
                    ref = exact(t, path, b, hv)
                    err = float(np.max(np.abs(o[t][b, hv] - ref)))
                    scale = max(float(np.max(np.abs(ref))), 1e-3)
                    worst = max(worst, err / scale)
    assert worst <= 1e-13, f"rational brute force: worst rel err {worst:.3e}"
    return worst


def pin_identity_gates_give_context_readout(lib, seed=11):
    """alpha = 1, beta = 0 leaves S_ctx untouched, so o = S_ctx q for every
    beam and step; checked against exactly-rounded dot products (math.fsum)."""
    rng = np.random.default_rng(seed)
    T, W, HK, HV, d = 3, 5, 2, 4, 16
    S0 = rng.standard_normal((HV, d, d))
    q = [rng.standard_normal((W, HK, d)) for _ in range(T)]
    k = [rng.standard_normal((W, HK, d)) for _ in range(T)]
    v = [rng.standard_normal((W, HV, d)) for _ in range(T)]
    al = [np.ones((W, HV)) for _ in range(T)]
    be = [np.zeros((W, HV)) for _ in range(T)]
    par = [rng.integers(0, W, size=W).astype(np.int32) for _ in range(T - 1)]
    o = orc.decode(S0, q, k, v, al, be, par, nthreads=1, lib=lib)
    G = HV // HK
    worst = 0.0
    for t in range(T):
        for b in range(W):
            for hv in range(HV):
                ref = np.array([math.fsum(S0[hv, i, :] * q[t][b, hv // G, :])
                                for i in range(d)])
                worst = max(worst, _rel(o[t][b, hv], ref))
    assert worst <= 1e-14, f"alpha=1,beta=0: rel err {worst:.3e}"
    return worst


def pin_zero_decay_forgets_history(lib, seed=12):
    """alpha_t = 0 wipes the parent state: S_t = beta_t v_t k_t^T, so
    o_t = beta_t (k_t . q_t) v_t whatever the ancestry."""
    rng = np.random.default_rng(seed)
    T, W, HK, HV, d = 3, 4, 1, 2, 8
    S0 = rng.standard_normal((HV, d, d))
    q = [rng.standard_normal((W, HK, d)) for _ in range(T)]
    k = [rng.standard_normal((W, HK, d)) for _ in range(T)]
    v = [rng.standard_normal((W, HV, d)) for _ in range(T)]
    al = [rng.uniform(0.5, 1.0, (W, HV)) for _ in range(T)]
    be = [rng.uniform(0.0, 1.0, (W, HV)) for _ in range(T)]
    al[2][:] = 0.0
    par = [rng.integers(0, W, size=W).astype(np.int32) for _ in range(T - 1)]
    o = orc.decode(S0, q, k, v, al, be, par, nthreads=1, lib=lib)
    worst = 0.0
    for b in range(W):
        for hv in range(HV):
            ref = be[2][b, hv] * math.fsum(k[2][b, 0] * q[2][b, 0]) * v[2][b, hv]
            worst = max(worst, _rel(o[2][b, hv], ref))
    assert worst <= 1e-14, f"alpha=0: rel err {worst:.3e}"
    return worst


def pin_delta_rule_write(lib, seed=13):
    """alpha = beta = 1 with k = q = e_i: the delta rule overwrites column i of
    S with v, so o_t = v_t for any history (to rounding of x + (v - x))."""
    rng = np.random.default_rng(seed)
    T, W, HK, HV, d = 4, 3, 1, 2, 8
    S0 = rng.standard_normal((HV, d, d))
    q, k, v, al, be = [], [], [], [], []
    for t in range(T):
        e = np.zeros((W, HK, d))
        cols = rng.integers(0, d, size=W)
        e[np.arange(W), 0, cols] = 1.0
        q.append(e.copy())
        k.append(e.copy())
        v.append(rng.standard_normal((W, HV, d)))
        al.append(np.ones((W, HV)))
        be.append(np.ones((W, HV)))
    # older steps use ordinary gates so the history is not trivial
    al[0] = rng.uniform(0.5, 1.0, (W, HV))
    be[0] = rng.uniform(0.0, 1.0, (W, HV))
    k[0] = rng.standard_normal((W, HK, d))
    par = [rng.integers(0, W, size=W).astype(np.int32) for _ in range(T - 1)]
    o = orc.decode(S0, q, k, v, al, be, par, nthreads=1, lib=lib)
    worst = 0.0
    for t in range(1, T):
        worst = max(worst, _rel(o[t], v[t]))
    assert worst <= 4e-16 * 8, f"delta-rule write: rel err {worst:.3e}"
    return worst


def pin_duplicated_parents_identical(lib, seed=14):
    """Children of the same parent with identical own inputs have identical
    outputs, bit for bit, through the whole subtree."""
    rng = np.random.default_rng(seed)
    T, W, HK, HV, d = 3, 6, 2, 2, 8
    S0 = rng.standard_normal((HV, d, d))

    def dup(x):
        # beams 0..2 carry inputs, beams 3..5 repeat them
        x = x.copy()
        x[3:] = x[:3]
        return x

    q = [dup(rng.standard_normal((W, HK, d))) for _ in range(T)]
    k = [dup(rng.standard_normal((W, HK, d))) for _ in range(T)]
    v = [dup(rng.standard_normal((W, HV, d))) for _ in range(T)]
    al = [dup(rng.uniform(0.5, 1, (W, HV))) for _ in range(T)]
    be = [dup(rng.uniform(0, 1, (W, HV))) for _ in range(T)]
    # at t = 1 beams b and b+3 pick the same parent; at t = 2 beam b+3 picks
    # parent b+3 while beam b picks b, so the duplicated subtrees stay apart
    p1 = np.array([2, 0, 2, 2, 0, 2], dtype=np.int32)
    p2 = np.array([0, 1, 2, 3, 4, 5], dtype=np.int32)
    o = orc.decode(S0, q, k, v, al, be, [p1, p2], nthreads=1, lib=lib)
    for t in range(T):
        assert np.array_equal(o[t][:3], o[t][3:]), f"duplicates differ at t={t}"
    # and the tree is not degenerate: distinct inputs give distinct outputs
    assert not np.array_equal(o[2][0], o[2][1])
    return 0.0


def forward_projection_replay(S0, chain, q_t, k_t, v_t, a_t, b_t):
    """The paper's projection replay (Sec. 3.2, Eqs. 2-4) in fp64: the record
    of step j is r_j = (alpha_j, delta_j, k_j); accumulators u_q = S q_t and
    u_k = S k_t are carried through the ancestral records, then delta_t and
    o_t follow from Eq. 4.  ``chain`` holds (alpha_j, delta_j, k_j), oldest
    first.  Returns (o_t, delta_t)."""
    uq = S0 @ q_t
    uk = S0 @ k_t
    for (a_j, d_j, k_j) in chain:
        uq = a_j * uq + d_j * float(k_j @ q_t)
        uk = a_j * uk + d_j * float(k_j @ k_t)
    delta = b_t * (v_t - a_t * uk)
    o = a_t * uq + delta * float(k_t @ q_t)
    return o, delta


def pin_projection_replay_matches(lib, seed=15):
    """The paper's forward projection replay with delta records (Eqs. 2-4)
    reproduces the materialised-state oracle on random trees."""
    rng = np.random.default_rng(seed)
    T, W, HK, HV, d = 4, 6, 2, 4, 16
    G = HV // HK
    S0 = rng.standard_normal((HV, d, d)) / 4
    q = [rng.standard_normal((W, HK, d)) / 4 for _ in range(T)]
    k = [rng.standard_normal((W, HK, d)) / 4 for _ in range(T)]
    v = [rng.standard_normal((W, HV, d)) for _ in range(T)]
    al = [rng.uniform(0.5, 1, (W, HV)) for _ in range(T)]
    be = [rng.uniform(0, 1, (W, HV)) for _ in range(T)]
    par = [rng.integers(0, W, size=W).astype(np.int32) for _ in range(T - 1)]
    o = orc.decode(S0, q, k, v, al, be, par, nthreads=1, lib=lib)
    # delta records of every (step, slot, value head), built step by step
    delta = {}
    worst = 0.0
    for t in range(T):
        for b in range(W):
            path = chase_path(par, t, b)
            for hv in range(HV):
                hk = hv // G
                chain = [(al[j][s, hv], delta[(j, s, hv)], k[j][s, hk])
                         for j, s in enumerate(path)]
                o_ref, d_t = forward_projection_replay(
                    S0[hv], chain, q[t][b, hk], k[t][b, hk], v[t][b, hv],
                    al[t][b, hv], be[t][b, hv])
                delta[(t, b, hv)] = d_t
                worst = max(worst, _rel(o[t][b, hv], o_ref))
    assert worst <= 1e-12, f"projection replay: rel err {worst:.3e}"
    return worst


def pin_single_beam_is_sequential(lib, seed=16):
    """With one beam per step (parents all 0) the decode is the ordinary
    sequential GDN recurrence over the decode tokens from S_ctx: checked
    against the prefill routine run over prompt + decode tokens."""
    rng = np.random.default_rng(seed)
    P, T, HK, HV, d = 5, 4, 2, 4, 8
    G = HV // HK
    pk = rng.standard_normal((P, HK, d))
    pv = rng.standard_normal((P, HV, d))
    pa = rng.uniform(0.5, 1, (P, HV))
    pb = rng.uniform(0, 1, (P, HV))
    S0 = orc.prefill(pk, pv, pa, pb, nthreads=1, lib=lib)
    q = [rng.standard_normal((1, HK, d)) for _ in range(T)]
    k = [rng.standard_normal((1, HK, d)) for _ in range(T)]
    v = [rng.standard_normal((1, HV, d)) for _ in range(T)]
    al = [rng.uniform(0.5, 1, (1, HV)) for _ in range(T)]
    be = [rng.uniform(0, 1, (1, HV)) for _ in range(T)]
    par = [np.zeros(1, dtype=np.int32) for _ in range(T - 1)]
    o = orc.decode(S0, q, k, v, al, be, par, nthreads=1, lib=lib)
    for t in range(T):
        St = orc.prefill(np.concatenate([pk] + [x[0][None] for x in k[:t + 1]]),
                         np.concatenate([pv] + [x[0][None] for x in v[:t + 1]]),
                         np.concatenate([pa] + [x[0][None] for x in al[:t + 1]]),
                         np.concatenate([pb] + [x[0][None] for x in be[:t + 1]]),
                         nthreads=1, lib=lib)
        for hv in range(HV):
            ref = St[hv] @ q[t][0, hv // G]
            assert _rel(o[t][0, hv], ref) <= 1e-14, (t, hv)
    return 0.0


def pin_prefill_closed_form(lib, seed=17):
    """Prefill from S = 0 against the exact rational closed form
    S_P = sum_p beta_p v_p k_p^T A_{p+1} ... A_{P-1} (d = 4, P = 6, dyadic
    inputs), plus the one-token case S_1 = beta v k^T."""
    rng = np.random.default_rng(seed)
    P, HK, HV, d = 6, 1, 2, 4
    pk = rng.integers(-8, 9, size=(P, HK, d)).astype(np.float64) / 8
    pv = rng.integers(-8, 9, size=(P, HV, d)).astype(np.float64) / 8
    pa = rng.integers(1, 17, size=(P, HV)).astype(np.float64) / 16
    pb = rng.integers(0, 17, size=(P, HV)).astype(np.float64) / 16
    S = orc.prefill(pk, pv, pa, pb, nthreads=1, lib=lib)
    zero = [[Fr(0)] * d for _ in range(d)]
    worst = 0.0
    for hv in range(HV):
        chain = [(_fmat(pk[p, 0]), _fmat(pv[p, hv]), Fr(float(pa[p, hv])),
                  Fr(float(pb[p, hv]))) for p in range(P)]
        ref = np.array([[float(x) for x in row] for row in closed_form_state(zero, chain)])
        worst = max(worst, _rel(S[hv], ref))
        S1 = orc.prefill(pk[:1], pv[:1], pa[:1], pb[:1], nthreads=1, lib=lib)
        assert np.array_equal(S1[hv], pb[0, hv] * np.outer(pv[0, hv], pk[0, 0]))
    assert worst <= 1e-14, f"prefill closed form: rel err {worst:.3e}"
    S_empty = orc.prefill(pk[:0], pv[:0], pa[:0], pb[:0], nthreads=1, lib=lib)
    assert not np.any(S_empty)
    return worst


def pin_ancestry_pointer_chasing(lib, seed=18):
    """Eq. 5 table against pointer chasing on random trees with changing
    widths, plus identity parents (h_t(b, j) = b) and all-zero parents
    (h_t(b, j) = 0), and an out-of-range parent is rejected."""
    rng = np.random.default_rng(seed)
    for trial in range(20):
        T = int(rng.integers(1, 7))
        widths = [int(x) for x in rng.integers(1, 40, size=T)]
        parents = [rng.integers(0, widths[t - 1], size=widths[t]).astype(np.int32)
                   for t in range(1, T)]
        h = orc.ancestry(widths, parents, lib=lib)
        for t in range(T):
            assert h[t].shape == (widths[t], t)
            for b in range(widths[t]):
                assert list(h[t][b]) == chase_path(parents, t, b), (trial, t, b)
    widths = [9] * 5
    h = orc.ancestry(widths, [np.arange(9, dtype=np.int32)] * 4, lib=lib)
    for t in range(5):
        assert np.array_equal(h[t], np.repeat(np.arange(9)[:, None], t, axis=1))
    h = orc.ancestry(widths, [np.zeros(9, dtype=np.int32)] * 4, lib=lib)
    for t in range(5):
        assert not np.any(h[t])
    try:
        orc.ancestry([3, 3], [np.array([0, 3, 1], dtype=np.int32)], lib=lib)
    except ValueError:
        pass
    else:
        raise AssertionError("out-of-range parent accepted")
    return 0.0


def backward_query_fold(S0, chain, q_t):
    """The device kernel's algebra in fp64: with records (k_j, v_j, alpha_j,
    beta_j), oldest first, fold the query newest to oldest through
    A_j = alpha_j (I - beta_j k_j k_j^T) while collecting the beta_j v_j k_j^T
    terms, then apply the shared state once."""
    p = np.array(q_t, dtype=np.float64)
    o = np.zeros(S0.shape[0])
    for (k_j, v_j, a_j, b_j) in reversed(chain):
        c = float(k_j @ p)
        o = o + b_j * c * v_j
        p = a_j * (p - b_j * c * k_j)
    return o + S0 @ p


def pin_backward_fold_matches(lib, seed=19):
    """The backward query fold (the kernel's algebra) reproduces the
    materialised-state oracle on random trees in fp64."""
    rng = np.random.default_rng(seed)
    T, W, HK, HV, d = 5, 7, 2, 4, 16
    G = HV // HK
    S0 = rng.standard_normal((HV, d, d)) / 4
    q = [rng.standard_normal((W, HK, d)) / 4 for _ in range(T)]
    k = [rng.standard_normal((W, HK, d)) / 4 for _ in range(T)]
    v = [rng.standard_normal((W, HV, d)) for _ in range(T)]
    al = [rng.uniform(0.5, 1, (W, HV)) for _ in range(T)]
    be = [rng.uniform(0, 1, (W, HV)) for _ in range(T)]
    par = [rng.integers(0, W, size=W).astype(np.int32) for _ in range(T - 1)]
    o = orc.decode(S0, q, k, v, al, be, par, nthreads=1, lib=lib)
    worst = 0.0
    for t in range(T):
        for b in range(W):
            slots = chase_path(par, t, b) + [b]
            for hv in range(HV):
                hk = hv // G
                chain = [(k[j][s, hk], v[j][s, hv], al[j][s, hv], be[j][s, hv])
                         for j, s in enumerate(slots)]
                worst = max(worst, _rel(o[t][b, hv],
                                        backward_query_fold(S0[hv], chain, q[t][b, hk])))
    assert worst <= 1e-12, f"backward fold: rel err {worst:.3e}"
    return worst




def _select_bruteforce(s, width, beam=None):
    """Python's sorted() over explicit tuples: (NaN last, value desc, +0 before
    -0, index asc).  With beam scores, each candidate is one fp32 addition of
    two fp32 scalars."""
    s = np.asarray(s, dtype=np.float32)
    P, V = s.shape
    flat = []
    for p in range(P):
        for v in range(V):
            x = s[p, v] if beam is None else np.float32(beam[p]) + s[p, v]
            assert isinstance(x, np.float32)
            flat.append(float(x))

    def key(i):
        x = flat[i]
        if math.isnan(x):
            return (1, 0.0, 0, i)
        return (0, -x, 1 if math.copysign(1.0, x) < 0 else 0, i)

    top = sorted(range(len(flat)), key=key)[:width]
    return [i // V for i in top], [i % V for i in top]


def pin_select_beams(lib=None, seed=20, select=None):
    """Top-W selection against brute force on small inputs with many ties
    (integer-valued scores), signed zeros, infinities and NaN of both signs,
    with and without beam scores; W = N keeps everything in order; all-equal
    scores keep the lowest indices."""
    select = select or orc.select_beams
    rng = np.random.default_rng(seed)
    for trial in range(80):
        P, V = int(rng.integers(1, 7)), int(rng.integers(1, 9))
        s = rng.integers(-3, 4, size=(P, V)).astype(np.float32)
        if trial % 3 == 0:
            s[rng.random((P, V)) < 0.2] = -0.0
        if trial % 4 == 0:
            s[rng.random((P, V)) < 0.1] = np.inf
            s[rng.random((P, V)) < 0.1] = -np.inf
            s[rng.random((P, V)) < 0.1] = np.nan
            s[rng.random((P, V)) < 0.1] = -np.nan
        beam = None
        if trial % 2 == 1:
            beam = rng.integers(-2, 3, size=P).astype(np.float32)
            beam[rng.random(P) < 0.3] = -0.0
            if trial % 5 == 1:
                beam += np.float32(0.375)
        width = int(rng.integers(1, P * V + 1))
        par, tok, sc = select(s, width, beam_scores=beam)
        bp, bt = _select_bruteforce(s, width, beam)
        assert list(par) == bp and list(tok) == bt, trial
        ref = s[par, tok] if beam is None else beam[par] + s[par, tok]
        assert np.array_equal(sc, ref, equal_nan=True)
    s = np.zeros((4, 5), dtype=np.float32)
    par, tok, _ = select(s, 7)
    assert list(par * 5 + tok) == list(range(7))
    s = rng.standard_normal((3, 4)).astype(np.float32)
    par, tok, sc = select(s, 12)
    assert np.all(np.diff(sc) <= 0) and sorted(par * 4 + tok) == list(range(12))
    # -0.0 + +0.0 is +0.0 under round-to-nearest: a zero beam score turns a
    # -0.0 log-probability into +0.0, which then ranks with the +0.0 entries.
    s = np.array([[-0.0, 0.0]], dtype=np.float32)
    par, tok, sc = select(s, 2, beam_scores=np.zeros(1, dtype=np.float32))
    assert list(tok) == [0, 1] and not np.signbit(sc).any()
    par, tok, _ = select(s, 2)
    assert list(tok) == [1, 0]
    return 0.0


ALL_PINS = [
    pin_exact_rational_bruteforce,
    pin_identity_gates_give_context_readout,
    pin_zero_decay_forgets_history,
    pin_delta_rule_write,
    pin_duplicated_parents_identical,
    pin_projection_replay_matches,
    pin_single_beam_is_sequential,
    pin_prefill_closed_form,
    pin_ancestry_pointer_chasing,
    pin_backward_fold_matches,
    pin_select_beams,
]
