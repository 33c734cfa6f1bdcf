"""Global top-W beam selection (Sec. 2.1) on the GPU against the oracle.

Indices and scores are compared bit for bit: the order is total (score desc,
flat index asc, -0.0 below +0.0, NaN last), so the result is unique, and the
candidate score is one fp32 addition on both sides."""
import zlib

import numpy as np
import pytest

from oracle import oracle as orc
from paper_2609_12399_amd import onela as ab
from paper_2609_12399_amd.workload import SELECT_CODEBOOK, make_select_inputs

pytestmark = pytest.mark.gpu

# (name, R, W_prev, V, W, kind, with_beam)
CASES = [
    ("tiny_direct", 1, 3, 5, 7, "ties", False),
    ("one_chunk_max_width", 2, 8, 2048, 4096, "logsoftmax", True),
    ("headline_w512", 1, 512, SELECT_CODEBOOK, 512, "logsoftmax", True),
    ("ragged_ties", 3, 37, 1001, 300, "ties", True),
    ("special_values", 2, 64, 300, 4096, "special", False),
    ("special_values_beam", 1, 300, 333, 1000, "special", True),
    ("keep_all", 1, 8, 125, 1000, "ties", True),
    ("width_one", 2, 100, 999, 1, "logsoftmax", True),
    ("many_stages_w4096", 1, 1024, 4096, 4096, "ties", True),
    ("r4_w1024", 4, 1024, 4096, 1024, "logsoftmax", True),
    ("chunk_plus_one", 1, 1, 16385, 17, "ties", False),
    # two-pass path (wave-maxima bound): heavy ties overflow one gather round
    # and some chunks their slot; special values; ragged last chunk
    ("two_pass_ties_rounds", 1, 512, SELECT_CODEBOOK, 512, "ties", True),
    ("two_pass_ties_slot_overflow", 1, 512, SELECT_CODEBOOK, 64, "ties", True),
    ("two_pass_special", 2, 600, 4096, 256, "special", True),
    ("two_pass_ragged", 3, 1023, 2047, 500, "logsoftmax", True),
    ("two_pass_width_one", 2, 700, 3000, 1, "logsoftmax", False),
    # rising beam scores: many survivors, each gather round beats the last
    ("two_pass_rising_rounds", 1, 512, SELECT_CODEBOOK, 512, "rising", True),
    ("two_pass_rising_r2_w1024", 2, 1024, 4096, 1024, "rising", True),
    # one launch with a cross-workgroup bound (all chunks resident at once):
    # ragged last chunk, ties cut off after the chunk where W tied candidates
    # are guaranteed, special values over two requests, rising scores at the
    # widest result it takes
    ("one_pass_ragged", 1, 500, 8000, 300, "logsoftmax", True),
    ("one_pass_ties_w64", 1, 300, SELECT_CODEBOOK, 64, "ties", True),
    ("one_pass_r2_special", 2, 100, SELECT_CODEBOOK, 200, "special", True),
    ("one_pass_rising_w1024", 1, 1024, 4096, 1024, "rising", True),
    # many requests in one launch: a polling workgroup and a bound word per
    # request, one epoch (64 requests: every word of the control block)
    ("one_pass_r32_ties", 32, 8, SELECT_CODEBOOK, 16, "ties", True),
    ("one_pass_r64", 64, 4, SELECT_CODEBOOK, 8, "logsoftmax", True),
    # two-pass path ranked by the placing kernel of the one-pass path: more
    # chunks than fit at once, with heavy ties (more survivors than it
    # stages), and more requests than the one-pass control block has
    ("two_pass_placed_r8_ties", 8, 256, SELECT_CODEBOOK, 256, "ties", True),
    ("two_pass_placed_r80", 80, 4, SELECT_CODEBOOK, 8, "ties", True),
    # two-pass path whose first pass also forms each request's bound (four
    # rounds of workgroups or more): 2, 4 and 8 rows of summaries per thread
    ("two_pass_summary_rising_r8", 8, 256, SELECT_CODEBOOK, 256, "rising", True),
    ("two_pass_summary_r4_w1024_ties", 4, 1024, 4096, 1024, "ties", True),
    ("two_pass_summary_rows8", 2, 1024, SELECT_CODEBOOK, 256, "logsoftmax", True),
]


def _run(R, P, V, W, kind, with_beam, seed):
    import torch
    from paper_2609_12399_amd.runner import BeamSelector
    logp, beam = make_select_inputs(R, P, V, seed, kind, with_beam)
    print(f"select R={R} W_prev={P} V={V} W={W} kind={kind} beam={with_beam}", flush=True)
    sel = BeamSelector(R, P, V, W)
    dl = torch.from_numpy(logp).cuda()
    db = None if beam is None else torch.from_numpy(beam).cuda()
    par, tok, sc = sel(dl, db)
    torch.cuda.synchronize()
    return logp, beam, par.cpu().numpy(), tok.cpu().numpy(), sc.cpu().numpy()


@pytest.mark.parametrize("name,R,P,V,W,kind,with_beam", CASES, ids=[c[0] for c in CASES])
def test_select_matches_oracle(name, R, P, V, W, kind, with_beam):
    logp, beam, par, tok, sc = _run(R, P, V, W, kind, with_beam, seed=zlib.crc32(name.encode()) % 1000)
    for r in range(R):
        op, ot, osc = orc.select_beams(logp[r], W, None if beam is None else beam[r])
        assert np.array_equal(par[r], op), f"request {r}: parents differ"
        assert np.array_equal(tok[r], ot), f"request {r}: tokens differ"
        assert np.array_equal(sc[r].view(np.int32), osc.view(np.int32)), \
            f"request {r}: scores differ"


@pytest.mark.parametrize("tied_slots", [6, 32], ids=["histogram_ranked", "exact_cut"])
def test_select_one_pass_many_tied_survivors(tied_slots):
    """Ties held by the first lane of every wave (a chunk's candidate at slot
    i of lane t sits at position 512 i + t): each wave then guarantees one
    candidate at the tied key, so all chunks up to c* (the 64th) keep every
    tied candidate of theirs, 64 x 8 x tied_slots survivors -- more than the
    final stage ranks by direct comparison (6 slots: 3072, ranked through the
    key histogram) or more than it stages at all (32 slots: 16384, the exact
    top-W cut over the slots).  The result is the W tied candidates with the
    lowest flat indices."""
    import torch
    from paper_2609_12399_amd.runner import BeamSelector
    R, P, V, W = 1, 512, SELECT_CODEBOOK, 512
    rng = np.random.default_rng(7 + tied_slots)
    logp = (-1.0 - rng.random(P * V, dtype=np.float32)).astype(np.float32)
    q = np.arange(P * V)
    logp[(q % 64 == 0) & ((q % 16384) // 512 < tied_slots)] = 0.0
    logp = logp.reshape(R, P, V)
    print(f"one-pass tied survivors: {64 * 8 * tied_slots}", flush=True)
    sel = BeamSelector(R, P, V, W)
    par, tok, sc = sel(torch.from_numpy(logp).cuda(), None)
    torch.cuda.synchronize()
    op, ot, osc = orc.select_beams(logp[0], W, None)
    assert np.array_equal(par.cpu().numpy()[0], op)
    assert np.array_equal(tok.cpu().numpy()[0], ot)
    assert np.array_equal(sc.cpu().numpy()[0].view(np.int32), osc.view(np.int32))


def test_select_all_equal_keeps_lowest_indices():
    import torch
    from paper_2609_12399_amd.runner import BeamSelector
    R, P, V, W = 2, 64, 1000, 777
    logp = np.full((R, P, V), -1.5, dtype=np.float32)
    sel = BeamSelector(R, P, V, W)
    par, tok, sc = sel(torch.from_numpy(logp).cuda())
    torch.cuda.synchronize()
    flat = par.cpu().numpy().astype(np.int64) * V + tok.cpu().numpy()
    assert np.array_equal(flat, np.tile(np.arange(W), (R, 1)))


def test_select_deterministic_and_feeds_resolve():
    """Repeated calls give identical bits; the parents it produces are valid
    input of the ancestry update (all in [0, W_prev))."""
    R, P, V, W = 1, 512, SELECT_CODEBOOK, 512
    a = _run(R, P, V, W, "logsoftmax", True, seed=5)
    b = _run(R, P, V, W, "logsoftmax", True, seed=5)
    for x, y in zip(a[2:], b[2:]):
        assert np.array_equal(x.view(np.int32), y.view(np.int32))
    assert a[2].min() >= 0 and a[2].max() < P


def _check(logp, beam, W, par, tok, sc):
    for r in range(logp.shape[0]):
        op, ot, osc = orc.select_beams(logp[r], W, None if beam is None else beam[r])
        assert np.array_equal(par[r], op), f"request {r}: parents differ"
        assert np.array_equal(tok[r], ot), f"request {r}: tokens differ"
        assert np.array_equal(sc[r].view(np.int32), osc.view(np.int32)), \
            f"request {r}: scores differ"


def test_select_shared_workspace_across_shapes():
    """One zero-filled workspace serves a sequence of calls of different
    shapes and paths (one launch with a cross-workgroup bound, reduction
    tree, wave-maxima two-pass, the one-launch path again): each call leaves
    the counters the next one relies on at zero."""
    import torch
    shapes = [(1, 512, SELECT_CODEBOOK, 512, "logsoftmax"), (3, 37, 1001, 300, "ties"),
              (2, 600, 4096, 256, "logsoftmax"), (1, 64, SELECT_CODEBOOK, 64, "rising"),
              (2, 256, SELECT_CODEBOOK, 128, "logsoftmax"), (1, 512, SELECT_CODEBOOK, 512, "ties")]
    need = max(ab.onela_select_workspace_bytes(R, P, V, W) for R, P, V, W, _ in shapes)
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
    for i, (R, P, V, W, kind) in enumerate(shapes):
        print(f"shared workspace call {i}: R={R} W_prev={P} V={V} W={W} {kind}", flush=True)
        logp, beam = make_select_inputs(R, P, V, 60 + i, kind, True)
        par = torch.empty((R, W), dtype=torch.int32, device="cuda")
        tok = torch.empty((R, W), dtype=torch.int32, device="cuda")
        sc = torch.empty((R, W), dtype=torch.float32, device="cuda")
        ab.onela_select_beams(R, P, V, W, torch.from_numpy(logp).cuda(),
                              torch.from_numpy(beam).cuda(), par, tok, sc, ws, need)
        torch.cuda.synchronize()
        _check(logp, beam, W, par.cpu().numpy(), tok.cpu().numpy(), sc.cpu().numpy())


def _mix(M, m, km):
    """The summary check word's mix (stated beside the one-pass summaries'
    tags): products with odd constants, the second rotated left by 13."""
    a = (M * 0x9E3779B1) & 0xFFFFFFFF
    b = (m * 0x85EBCA77) & 0xFFFFFFFF
    b = ((b << 13) | (b >> 19)) & 0xFFFFFFFF
    return a ^ b ^ ((km * 0xC2B2AE3D) & 0xFFFFFFFF)


def test_select_one_pass_tags_and_epoch_wrap():
    """The one-pass path's cross-call state in the workspace: a call counter
    (epoch, first word) and, from byte 1024, 8192 16-byte wave summaries
    (M, m, kM, tag ^ mix).  Planted summaries of an earlier call (older tag)
    with fields that would put the bound above every score, and summaries
    whose check word names this call's tag but whose fields it does not
    match, are not taken; the call matches the oracle and advances the
    epoch.  At the largest tag the epoch starts again at 0 and the region is
    cleared, and the call after it matches too.  Each call's survivor
    counts show that a bound was used (without one every chunk keeps W)."""
    import torch
    from paper_2609_12399_amd.runner import BeamSelector
    R, P, V, W = 1, 512, SELECT_CODEBOOK, 512
    sel = BeamSelector(R, P, V, W)
    ws = sel.workspace
    nchunks = P * V // 16384
    nseg, cap, nsum = nchunks * 8, 2 * W, 8192
    up = lambda x: -(-x // 256) * 256
    cnt_off = 1024 + nsum * 16 + up(R * nseg * 16) + up(R * 8) + up(R * nchunks * cap * 8)

    def put_u32(off, vals):
        b = torch.from_numpy(np.asarray(vals, dtype=np.uint32).reshape(-1).view(np.uint8).copy())
        ws[off:off + b.numel()].copy_(b)

    def epoch():
        return int(ws[0:4].cpu().numpy().view(np.uint32)[0])

    def call(seed):
        logp, beam = make_select_inputs(R, P, V, seed, "logsoftmax", True)
        print(f"tagged call seed={seed} epoch={epoch()}", flush=True)
        sel(torch.from_numpy(logp).cuda(), torch.from_numpy(beam).cuda())
        torch.cuda.synchronize()
        _check(logp, beam, W, sel.parents.cpu().numpy(), sel.tokens.cpu().numpy(),
               sel.scores.cpu().numpy())
        cnt = ws[cnt_off:cnt_off + nchunks * 8].cpu().numpy().view(np.uint32)[0::2]
        assert 0 < int(cnt.sum()) < 4096, int(cnt.sum())

    E, top = 5, 0xFFFFFFFF
    put_u32(0, [E])
    planted = np.zeros((nsum, 4), dtype=np.uint32)
    planted[:nseg] = [top, top, 64, E ^ _mix(top, top, 64)]              # an older call's
    planted[1:nseg:2, 3] = (E + 1) ^ _mix(0x1234, top, 64)               # fields not its own
    put_u32(1024, planted)
    call(90)
    assert epoch() == E + 1
    put_u32(0, [0xFFFFFFFE])
    call(91)
    assert epoch() == 0
    assert int(torch.count_nonzero(ws[1024:1024 + nsum * 16])) == 0
    call(92)
    assert epoch() == 1


def test_select_graph_replays_with_new_scores():
    """The headline selection captured once in a HIP graph and replayed with
    new scores copied into its input buffers between replays (eager work
    and synchronisation in between): every replay matches the oracle."""
    import torch
    from paper_2609_12399_amd.runner import BeamSelector
    R, P, V, W = 1, 512, SELECT_CODEBOOK, 512
    logp0, beam0 = make_select_inputs(R, P, V, 70, "logsoftmax", True)
    dl = torch.from_numpy(logp0).cuda()
    db = torch.from_numpy(beam0).cuda()
    s = torch.cuda.Stream()
    sel = BeamSelector(R, P, V, W, stream=s)
    with torch.cuda.stream(s):
        sel(dl, db)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        sel(dl, db)
    torch.cuda.synchronize()
    for rep, kind in enumerate(["logsoftmax", "rising", "logsoftmax", "ties"]):
        logp, beam = make_select_inputs(R, P, V, 80 + rep, kind, True)
        dl.copy_(torch.from_numpy(logp))
        db.copy_(torch.from_numpy(beam))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        print(f"graph replay {rep} ({kind})", flush=True)
        _check(logp, beam, W, sel.parents.cpu().numpy(), sel.tokens.cpu().numpy(),
               sel.scores.cpu().numpy())
