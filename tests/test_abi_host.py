"""C-ABI checks that need no GPU: the library loads, exports every symbol the
header declares, validates arguments on the host before any HIP call, and
its capacity model reproduces the paper's printed accounting."""
import ctypes
import json
import os
import re
from decimal import ROUND_HALF_UP, Decimal

import pytest

from paper_2609_12399_amd import onela as ab

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "onela.h")


@pytest.fixture(scope="module")
def lib():
    return ab.load_library()


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(onela_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    declared = header_functions()
    assert len(declared) >= 15
    for name in declared:
        assert hasattr(lib, name), name
    assert sorted(ab.EXPORTED) == declared


def cfg(**kw):
    base = dict(num_requests=1, num_qk_heads=16, num_v_heads=16, d_k=128, d_v=128,
                max_beams=512, max_steps=4, io_dtype=ab.ONELA_BF16)
    base.update(kw)
    return ab.make_config(**base)


def test_config_validation(lib):
    assert ab.onela_check_config(cfg()) == ab.ONELA_OK
    assert ab.onela_check_config(cfg(d_k=32, d_v=32, io_dtype=ab.ONELA_F32)) == ab.ONELA_OK
    assert ab.onela_check_config(cfg(num_v_heads=32)) == ab.ONELA_OK
    for dk, dv in ((128, 256), (128, 512), (256, 256), (256, 512), (64, 64)):
        assert ab.onela_check_config(cfg(d_k=dk, d_v=dv)) == ab.ONELA_OK, (dk, dv)
    for dk, dv in ((128, 256), (256, 512)):  # wide shapes are bf16-only
        assert ab.onela_check_config(cfg(d_k=dk, d_v=dv, io_dtype=ab.ONELA_F32)) == ab.ONELA_EINVAL
    for dk, dv in ((256, 128), (128, 1024), (512, 512), (128, 384)):
        assert ab.onela_check_config(cfg(d_k=dk, d_v=dv)) == ab.ONELA_EINVAL, (dk, dv)
    assert ab.onela_check_config(cfg(record_kind=ab.ONELA_RECORD_DELTA)) == ab.ONELA_OK
    assert ab.onela_check_config(cfg(record_kind=2)) == ab.ONELA_EINVAL
    assert ab.onela_check_config(cfg(record_storage=ab.ONELA_RECORDS_BORROW)) == ab.ONELA_OK
    assert ab.onela_check_config(cfg(record_storage=2)) == ab.ONELA_EINVAL
    # delta records are computed by the library: they cannot be borrowed
    assert ab.onela_check_config(cfg(record_kind=ab.ONELA_RECORD_DELTA,
                                     record_storage=ab.ONELA_RECORDS_BORROW)) == ab.ONELA_EINVAL
    bad = [dict(num_v_heads=24, num_qk_heads=16), dict(d_k=96, d_v=96), dict(d_k=128, d_v=64),
           dict(max_beams=0), dict(max_beams=65537), dict(max_steps=0), dict(max_steps=9),
           dict(io_dtype=7), dict(num_requests=0), dict(num_qk_heads=0)]
    for b in bad:
        assert ab.onela_check_config(cfg(**b)) == ab.ONELA_EINVAL, b
        assert ab.onela_workspace_bytes(cfg(**b)) == 0, b
    assert lib.onela_check_config(None) == ab.ONELA_EINVAL


def test_workspace_bytes_layout(lib):
    n = ab.onela_workspace_bytes(cfg())
    R, T, W, H, d = 1, 4, 512, 16, 128
    expect = (256 + 2 * (W * T * 4) + 2 * 2 * H * d * d + 2 * T * H * W * d * 2
              + T * H * W * 8)
    assert n == expect
    assert n % 256 == 0
    # transition records add a delta arena the size of the v arena (fp16 rows)
    # and one 32-bit word of slice scale exponents per delta row
    nd = ab.onela_workspace_bytes(cfg(record_kind=ab.ONELA_RECORD_DELTA))
    assert nd == n + T * H * W * d * 2 + T * H * W * 4
    # borrowed records: no arena at all
    nb = ab.onela_workspace_bytes(cfg(record_storage=ab.ONELA_RECORDS_BORROW))
    assert nb == 256 + 2 * (W * T * 4) + 2 * 2 * H * d * d


def test_host_errors_before_any_hip_call(lib):
    c = cfg()
    out = ctypes.c_void_p()
    # NULL pointers / misaligned pointers / short workspace: rejected on the host
    assert lib.onela_init(ctypes.byref(c), None, 256, 1 << 30, None, ctypes.byref(out)) == ab.ONELA_EINVAL
    assert lib.onela_init(ctypes.byref(c), 4096, None, 1 << 30, None, ctypes.byref(out)) == ab.ONELA_EINVAL
    assert lib.onela_init(ctypes.byref(c), 4100, 4096, 1 << 30, None, ctypes.byref(out)) == ab.ONELA_EINVAL
    assert lib.onela_init(ctypes.byref(c), 4096, 4096 + 16, 1 << 30, None, ctypes.byref(out)) == ab.ONELA_EINVAL
    assert lib.onela_init(ctypes.byref(c), 4096, 4096, 100, None, ctypes.byref(out)) == ab.ONELA_ECAPACITY
    bad = cfg(d_k=100)
    assert lib.onela_init(ctypes.byref(bad), 4096, 4096, 1 << 30, None, ctypes.byref(out)) == ab.ONELA_EINVAL
    # calls on a NULL context
    assert lib.onela_resolve_ancestry(None, 0, 4, None, None) == ab.ONELA_EINVAL
    assert lib.onela_append_records(None, 0, 16, 16, 16, 16) == ab.ONELA_EINVAL
    assert lib.onela_decode_step(None, 0, 16, 16) == ab.ONELA_EINVAL
    assert lib.onela_reset(None) == ab.ONELA_EINVAL
    assert lib.onela_get_device_status(None) == ab.ONELA_EINVAL
    lib.onela_destroy(None)
    # prefill / fullstate argument checks
    assert lib.onela_prefill_state(ctypes.byref(c), -1, 16, 16, 16, 16, 16, None) == ab.ONELA_EINVAL
    assert lib.onela_prefill_state(ctypes.byref(c), 4, None, 16, 16, 16, 16, None) == ab.ONELA_EINVAL
    fs = lib.onela_fullstate_step
    assert fs(ctypes.byref(c), 0, 513, 0, None, 16, 16, 16, 16, 16, 16, 16, 256, 1 << 40, None, None) == ab.ONELA_ECAPACITY
    assert fs(ctypes.byref(c), 1, 8, 8, None, 16, 16, 16, 16, 16, 16, 16, 256, 1 << 40, None, None) == ab.ONELA_EINVAL
    assert fs(ctypes.byref(c), 0, 8, 0, 64, 16, 16, 16, 16, 16, 16, 16, 256, 1 << 40, None, None) == ab.ONELA_EINVAL
    assert fs(ctypes.byref(c), 0, 8, 0, None, 16, 16, 16, 16, 16, 16, 16, 256, 10, None, None) == ab.ONELA_ECAPACITY


def test_status_strings(lib):
    for code in range(7):
        assert ab.onela_status_str(code)
    assert ab.onela_status_str(99) == "unknown status"


def sig3(x):
    """x rounded half-up to 3 significant digits (the paper's printing)."""
    d = Decimal(repr(float(x)))
    q = Decimal(1).scaleb(d.adjusted() - 2)
    return d.quantize(q, rounding=ROUND_HALF_UP)


def test_capacity_model_matches_paper(lib):
    g = json.load(open(os.path.join(ROOT, "tests", "golden", "capacity_e3.json")))
    w = g["workload"]
    MiB = float(1 << 20)
    record = 4 + 2 * w["d_v"] + 2 * w["d_k"]  # alpha fp32 + delta 16-bit + k 16-bit
    assert record == 516
    full = ab.onela_fullstate_capacity_bytes(w["R"], w["H"], w["d_k"], w["d_v"], w["W"], 4)
    for O in (3, 7):
        T = O - 1
        cap = ab.onela_capacity_bytes(w["R"], w["H"], w["d_k"], w["d_v"], w["W"], T, 4, record)
        writes = ab.onela_capacity_bytes(w["R"], w["H"], w["d_k"], w["d_v"], w["W"], T, 0, record)
        pr = g["printed"]
        key = f"O={O}"
        assert sig3(cap / MiB) == sig3(pr["capacity_mib"][key])
        assert sig3(full / cap) == sig3(pr["capacity_reduction_vs_fullstate"][key])
        assert sig3(writes / MiB) == sig3(pr["state_writes_mib"][key])
        assert sig3(T * full / writes) == sig3(pr["write_reduction_vs_fullstate"][key])
    assert ab.onela_capacity_bytes(-1, 1, 1, 1, 1, 1, 1, 1) == 0


def test_binding_rejects_host_tensors():
    torch = pytest.importorskip("torch")
    with pytest.raises(ValueError):
        ab._dev(torch.zeros(4), "x")
    assert ab._dev(None, "x", optional=True) is None
    assert ab._dev(1234, "x") == 1234


def _select_plan_bytes(R, P, V, W, chunk=16384):
    """Workspace model of the beam selection: a 1 KiB control block and a
    128 KiB summary region (the one-pass path's state across calls: a call
    counter, per-request bound words, 8192 16-byte wave summaries), then
    either the two-pass regions or a reduction tree whose workgroups each
    take `chunk` candidates and write one slot of `cap` (key, index) pairs
    (8 bytes each) plus a 4-byte count; stage outputs alternate between two
    buffers, every region 256-byte aligned."""
    p2 = lambda x: 1 << (x - 1).bit_length()
    cap = max(64, p2(2 * W))
    if cap > chunk // 4:
        cap = max(chunk // 4, p2(W))
    group = chunk // cap
    up = lambda x: -(-x // 256) * 256
    head = 1024 + 8192 * 16
    n = P * V
    nchunks = -(-n // chunk)
    if n > chunk and n >= 2 * W * 2048 and nchunks <= 2048:
        # two-pass / one-pass path: one 16-byte summary per wave of 2048
        # candidates, one 8-byte bound word per request, one slot of `cap`
        # pairs per chunk, one (count, largest key) pair per chunk
        return (head + up(R * nchunks * 8 * 16) + up(R * 8) + up(R * nchunks * cap * 8)
                + up(R * nchunks * 8))
    pairs, counts = [0, 0], [0, 0]
    if n > chunk:
        slots = -(-n // chunk)
        pairs[0], counts[0] = R * slots * cap * 8, R * slots * 4
        s = 1
        while slots > group:
            slots = -(-slots // group)
            pairs[s % 2] = max(pairs[s % 2], R * slots * cap * 8)
            counts[s % 2] = max(counts[s % 2], R * slots * 4)
            s += 1
    return head + sum(up(x) for x in pairs + counts)


@pytest.mark.parametrize("R,P,V,W", [(1, 3, 5, 7), (2, 8, 2048, 4096), (1, 512, 8192, 512),
                                     (3, 37, 1001, 300), (1, 1024, 4096, 4096),
                                     (4, 1024, 4096, 1024), (1, 1, 16385, 17),
                                     (7, 65536, 8192, 4096), (1, 512, 8192, 64),
                                     (2, 4096, 8192, 1), (1, 1023, 2048, 512)])
def test_select_workspace_bytes(lib, R, P, V, W):
    assert ab.onela_select_workspace_bytes(R, P, V, W) == _select_plan_bytes(R, P, V, W)


def test_select_host_errors(lib):
    out = ctypes.c_size_t(123)
    ws = lib.onela_select_workspace_bytes
    assert ws(1, 4, 4, 17, ctypes.byref(out)) == ab.ONELA_EINVAL and out.value == 0  # W > N
    assert ws(1, 4096, 4096, 4097, ctypes.byref(out)) == ab.ONELA_EINVAL  # W > 4096
    assert ws(0, 4, 4, 1, ctypes.byref(out)) == ab.ONELA_EINVAL
    assert ws(65537, 4, 4, 1, ctypes.byref(out)) == ab.ONELA_EINVAL
    assert ws(1, 1 << 15, 1 << 15, 1, ctypes.byref(out)) == ab.ONELA_EINVAL  # N > 2^29
    assert ws(1, 4, 4, 0, ctypes.byref(out)) == ab.ONELA_EINVAL
    assert ws(1, 4, 4, 1, None) == ab.ONELA_EINVAL
    sb = lib.onela_select_beams
    big = 1 << 30
    assert sb(1, 512, 8192, 513 * 0, 256, None, 256, 256, 256, 256, big, None) == ab.ONELA_EINVAL
    assert sb(1, 512, 8192, 512, None, None, 256, 256, 256, 256, big, None) == ab.ONELA_EINVAL
    assert sb(1, 512, 8192, 512, 258, None, 256, 256, 256, 256, big, None) == ab.ONELA_EINVAL
    assert sb(1, 512, 8192, 512, 256, 258, 256, 256, 256, 256, big, None) == ab.ONELA_EINVAL
    assert sb(1, 512, 8192, 512, 256, None, None, 256, 256, 256, big, None) == ab.ONELA_EINVAL
    assert sb(1, 512, 8192, 512, 256, None, 256, 256, 256, None, big, None) == ab.ONELA_EINVAL
    assert sb(1, 512, 8192, 512, 256, None, 256, 256, 256, 128, big, None) == ab.ONELA_EINVAL
    assert sb(1, 512, 8192, 512, 256, None, 256, 256, 256, 256, 1024, None) == ab.ONELA_ECAPACITY


@pytest.mark.parametrize("P,dk,dv", [(4096, 128, 128), (1, 128, 128), (65, 256, 512), (200, 32, 32)])
def test_prefill_workspace_bytes(lib, P, dk, dv):
    """Per (request, value head, 64-token chunk): fp32 W [64][d_k], Kt^T
    [d_k][64], U^T [d_v][64], then the chunk's fp32 decay repeated 16 times;
    two 256-byte aligned regions."""
    c = cfg(d_k=dk, d_v=dv, num_requests=2, num_v_heads=32)
    nch = -(-P // 64)
    up = lambda x: -(-x // 256) * 256
    units = 2 * 32
    assert ab.onela_prefill_workspace_bytes(c, P) == up(units * nch * 64 * (2 * dk + dv) * 4) + \
        up(units * nch * 16 * 4)
    assert ab.onela_prefill_workspace_bytes(c, 0) == 0
    assert ab.onela_prefill_workspace_bytes(cfg(d_k=96, d_v=96), P) == 0
    assert ab.onela_prefill_workspace_bytes(c, -1) == 0


def test_prefill_chunked_host_errors(lib):
    c = cfg()
    f = lib.onela_prefill_state_chunked
    big = 1 << 40
    assert f(ctypes.byref(c), -1, 256, 256, 256, 256, 256, 256, big, None) == ab.ONELA_EINVAL
    assert f(ctypes.byref(c), 64, None, 256, 256, 256, 256, 256, big, None) == ab.ONELA_EINVAL
    assert f(ctypes.byref(c), 64, 256, 256, 256, 256, 260, 256, big, None) == ab.ONELA_EINVAL
    assert f(ctypes.byref(c), 64, 256, 256, 256, 256, 256, None, big, None) == ab.ONELA_EINVAL
    assert f(ctypes.byref(c), 64, 256, 256, 256, 256, 256, 384, big, None) == ab.ONELA_EINVAL
    assert f(ctypes.byref(c), 64, 256, 256, 256, 256, 256, 256, 16, None) == ab.ONELA_ECAPACITY
