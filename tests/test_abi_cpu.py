"""The C-ABI library without a GPU: it loads, exports every entry point the
public header declares, and its host-side argument and call-order checks
return the documented status codes.  No call here launches a kernel or
touches device memory (pointers handed to the library are never
dereferenced on these paths)."""
from __future__ import annotations

import ctypes
import os
import re
import subprocess

import pytest

from paper_2609_33184_amd import build_lib
from paper_2609_33184_amd import specstream as ss

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "specstream.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(ss.lib_path()):
        build_lib.build(verbose=False)
    return ss.load()


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    return sorted(set(re.findall(r"\b(ss_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = _declared()
    assert set(names) == set(ss.EXPORTED), names


def test_every_declared_symbol_is_exported(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", ss.lib_path()], capture_output=True, text=True,
                         check=True).stdout
    exported = {ln.split()[-1] for ln in out.splitlines() if " T " in ln}
    missing = [n for n in _declared() if n not in exported]
    assert not missing, missing
    for n in _declared():
        assert hasattr(lib, n)
    # C linkage: no mangled spec-stream symbols
    assert not [s for s in exported if "ss_round" in s and s.startswith("_Z")]


def test_status_strings(lib):
    for code, name in [(ss.SS_OK, "SS_OK"), (ss.SS_ERR_INVALID_ARGUMENT, "SS_ERR_INVALID_ARGUMENT"),
                       (ss.SS_ERR_UNSUPPORTED, "SS_ERR_UNSUPPORTED"), (ss.SS_ERR_BAD_STATE, "SS_ERR_BAD_STATE"),
                       (ss.SS_ERR_NOT_PINNED, "SS_ERR_NOT_PINNED"), (ss.SS_ERR_WORKSPACE, "SS_ERR_WORKSPACE"),
                       (ss.SS_ERR_HIP, "SS_ERR_HIP"), (ss.SS_ERR_OUT_OF_MEMORY, "SS_ERR_OUT_OF_MEMORY")]:
        assert ss.ss_status_string(code) == name


def _ws(cands, hq, hkv):
    rows = sum(cands) * hq
    a = -(-32 * rows * 128 * 4 // 256) * 256     # 32 state slots per row
    m = -(-32 * rows * 4 // 256) * 256
    return a + 2 * m + 256                        # + the counter block (the tail's claim counter)


def test_workspace_bytes_and_descriptor_validation(lib):
    d = ss.make_desc([6] * 16, 32, 8)
    assert ss.ss_round_workspace_bytes(d) == _ws([6] * 16, 32, 8)
    d = ss.make_desc([1, 8, 3], 8, 2)
    assert ss.ss_round_workspace_bytes(d) == _ws([1, 8, 3], 8, 2)
    d = ss.make_desc([2] * 100, 8, 8)
    assert ss.ss_round_workspace_bytes(d) == _ws([2] * 100, 8, 8)
    bad = [
        (ss.make_desc([5], 32, 6), "multiple"),                          # Hq % Hkv
        (ss.make_desc([5], 8, 2, head_dim=64), "head_dim"),
        (ss.make_desc([0], 8, 2), "num_cand"),
        (ss.make_desc([9], 8, 2), "num_cand"),
        (ss.make_desc([8], 72, 8), "rows per KV head"),                  # 8 * 9 = 72 > 64
        (ss.make_desc([4], 8, 2, softmax_scale=-1.0), "softmax_scale"),
        (ss.make_desc([4], 8, 2, softmax_scale=float("inf")), "softmax_scale"),
        (ss.make_desc([4], 8, 2, split_tokens=48), "split_tokens"),
        (ss.make_desc([4], 8, 2, mfma_min_rows=6), "mfma_min_rows"),
        (ss.make_desc([4], 8, 2, kv_layout=3), "kv_layout"),
        (ss.make_desc([4], 8, 2, max_chunk_tokens=0), "max_chunk_tokens"),
        (ss.make_desc([4], 8, 2, balance_permille=501), "balance_permille"),
        (ss.make_desc([4], 8, 2, counters_zeroed=2), "counters_zeroed"),
    ]
    for desc, word in bad:
        assert ss.ss_round_workspace_bytes(desc) == 0
        assert word in ss.ss_last_error(), (word, ss.ss_last_error())


FAKE_Q = 0x7F0000000000          # aligned addresses the host checks accept; never dereferenced
FAKE_WS = 0x7F0001000000


def test_round_init_checks(lib):
    d = ss.make_desc([5], 8, 2, max_chunk_tokens=1024)
    need = ss.ss_round_workspace_bytes(d)
    cases = [
        (dict(q=0, workspace=FAKE_WS, workspace_bytes=need), ss.SS_ERR_INVALID_ARGUMENT),
        (dict(q=FAKE_Q + 8, workspace=FAKE_WS, workspace_bytes=need), ss.SS_ERR_INVALID_ARGUMENT),
        (dict(q=FAKE_Q, workspace=0, workspace_bytes=need), ss.SS_ERR_WORKSPACE),
        (dict(q=FAKE_Q, workspace=FAKE_WS + 64, workspace_bytes=need), ss.SS_ERR_WORKSPACE),
        (dict(q=FAKE_Q, workspace=FAKE_WS, workspace_bytes=need - 1), ss.SS_ERR_WORKSPACE),
    ]
    for kw, status in cases:
        with pytest.raises(ss.SpecStreamError) as e:
            ss.ss_round_init(d, **kw)
        assert e.value.status == status, (kw, e.value)
    with pytest.raises(ss.SpecStreamError) as e:
        ss.ss_round_init(ss.make_desc([4], 8, 2, head_dim=96), FAKE_Q, FAKE_WS, need)
    assert e.value.status == ss.SS_ERR_UNSUPPORTED


def test_call_order_and_chunk_arguments(lib):
    d = ss.make_desc([5, 2], 8, 2, max_chunk_tokens=1024)
    need = ss.ss_round_workspace_bytes(d)
    r = ss.ss_round_init(d, FAKE_Q, FAKE_WS, need)
    try:
        K, V = 0x7F0002000000, 0x7F0003000000

        def expect(status, fn, *a):
            with pytest.raises(ss.SpecStreamError) as e:
                fn(*a)
            assert e.value.status == status, e.value

        expect(ss.SS_ERR_BAD_STATE, ss.ss_round_finalize, r, FAKE_Q, 0)            # before candidates
        expect(ss.SS_ERR_INVALID_ARGUMENT, ss.ss_attend_history_chunk, r, K, V, [600, 600])   # > max_chunk_tokens
        expect(ss.SS_ERR_INVALID_ARGUMENT, ss.ss_attend_history_chunk, r, K, V, [-1, 3])
        expect(ss.SS_ERR_INVALID_ARGUMENT, ss.ss_attend_history_chunk, r, K + 2, V, [10, 3])  # misaligned
        expect(ss.SS_ERR_INVALID_ARGUMENT, ss.ss_attend_history_chunk, r, 0, V, [10, 3])
        expect(ss.SS_ERR_INVALID_ARGUMENT, ss.ss_attend_history_chunks, r, [K] * 33, [V] * 33, [[1, 1]] * 33)
        # the K-and-V layout takes v = k + d elements
        d2 = ss.make_desc([5, 2], 8, 2, max_chunk_tokens=1024, kv_layout=ss.SS_KV_HEAD_MAJOR_KV)
        r2 = ss.ss_round_init(d2, FAKE_Q, FAKE_WS, ss.ss_round_workspace_bytes(d2))
        try:
            expect(ss.SS_ERR_INVALID_ARGUMENT, ss.ss_attend_history_chunk, r2, K, V, [10, 3])
            expect(ss.SS_ERR_INVALID_ARGUMENT, ss.ss_attend_history_chunk, r2, K, K + 128, [10, 3])
        finally:
            ss.ss_round_destroy(r2)
        expect(ss.SS_ERR_INVALID_ARGUMENT, ss.ss_attend_local_candidates, r, 0, V)
        ss.ss_attend_local_candidates(r, K, V)                                     # records pointers only
        expect(ss.SS_ERR_BAD_STATE, ss.ss_attend_local_candidates, r, K, V)
        expect(ss.SS_ERR_INVALID_ARGUMENT, ss.ss_round_finalize, r, 0, 0)          # null out
        expect(ss.SS_ERR_INVALID_ARGUMENT, ss.ss_round_finalize, r, FAKE_Q + 4, 0)  # misaligned out
    finally:
        ss.ss_round_destroy(r)
    ss.ss_round_destroy(None)
    with pytest.raises(ss.SpecStreamError) as e:
        ss.ss_attend_history_chunk(None, 0, 0, [0, 0])
    assert e.value.status == ss.SS_ERR_INVALID_ARGUMENT


def test_pipeline_argument_checks(lib):
    d = ss.make_desc([2], 8, 2, max_chunk_tokens=1024)
    r = ss.ss_round_init(d, FAKE_Q, FAKE_WS, ss.ss_round_workspace_bytes(d))
    try:
        for call in (lambda: ss.ss_pipeline_attend_chunks(None, r, FAKE_Q, [[16]]),
                     lambda: ss.ss_pipeline_attend_chunk(None, r, FAKE_Q, [16])):
            with pytest.raises(ss.SpecStreamError) as e:
                call()
            assert e.value.status == ss.SS_ERR_INVALID_ARGUMENT
    finally:
        ss.ss_round_destroy(r)


def test_upload_argument_checks(lib):
    with pytest.raises(ss.SpecStreamError) as e:
        ss.ss_upload_chunk(0, FAKE_Q, 16)
    assert e.value.status == ss.SS_ERR_INVALID_ARGUMENT
    with pytest.raises(ss.SpecStreamError) as e:
        ss.ss_upload_chunk(FAKE_WS, FAKE_Q, 0)
    assert e.value.status == ss.SS_ERR_INVALID_ARGUMENT


def test_scratch_round_rejects_rounds_beyond_the_scratch(lib):
    """The no-allocation round start checks the workspace a round needs
    against the library's 64 MiB scratch before it touches a device."""
    big = ss.make_desc([8] * 64, 32, 8)          # 16384 rows: about 273 MB of slot states
    assert ss.ss_round_workspace_bytes(big) > 64 << 20
    with pytest.raises(ss.SpecStreamError) as e:
        ss.ss_round_init_scratch(big, FAKE_Q)
    assert e.value.status == ss.SS_ERR_WORKSPACE and "scratch" in str(e.value)
    with pytest.raises(ss.SpecStreamError) as e:
        ss.ss_round_init_scratch(ss.make_desc([0], 8, 2), FAKE_Q)
    assert e.value.status == ss.SS_ERR_INVALID_ARGUMENT


def test_read_probe_argument_checks(lib):
    """ss_probe_read refuses bad sizes, alignment and grids before it looks
    at the pointers."""
    cases = [(0, 16, FAKE_WS, 1), (FAKE_WS, 0, FAKE_WS, 1), (FAKE_WS, 24, FAKE_WS, 1), (FAKE_WS + 8, 32, FAKE_WS, 1),
             (FAKE_WS, 32, FAKE_WS, 0), (FAKE_WS, 32, FAKE_WS, 65537), (FAKE_WS, 32, FAKE_WS + 2, 1),
             (FAKE_WS, (2 << 30) + 16, FAKE_WS, 2)]
    for buf, n, sink, g in cases:
        with pytest.raises(ss.SpecStreamError) as e:
            ss.ss_probe_read(buf, n, sink, g)
        assert e.value.status == ss.SS_ERR_INVALID_ARGUMENT, (buf, n, sink, g)
