"""Host-side checks of the C ABI: the library loads, exports every symbol the
header declares, and rejects bad arguments before touching a device."""
import ctypes
import os
import re

import pytest

import paper_2609_36601_amd as saki
from paper_2609_36601_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "saki.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(binding.LIB_PATH):
        from paper_2609_36601_amd import build
        build.build()
    return saki.load()


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:[\w\s\*]+?)\b(saki_\w+)\s*\(", text, re.M)))


def test_header_and_exports_agree(lib):
    names = declared_functions()
    assert set(names) == set(binding.EXPORTED)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings(lib):
    for code in range(9):
        assert lib.saki_status_str(code)
    assert lib.saki_last_error() is not None


def _rows(**kw):
    r = dict(student=16, teacher=32, dtype=binding.SAKI_BF16, reserved=0, n_rows=4, vocab=64,
             row_stride=64, row_offset=0)
    r.update(kw)
    return binding.SakiRows(**r)


def _couple(lib, rows, eps=0.1, out=True, route=None, ws=None, ws_bytes=0):
    co = binding.SakiCoupleOut()
    return lib.saki_couple(ctypes.byref(rows) if rows is not None else None, eps, 1,
                           ctypes.byref(co) if out else None,
                           ctypes.byref(route) if route is not None else None,
                           ws, ws_bytes, None)


def test_argument_errors_without_launch(lib):
    assert _couple(lib, None) == 1                                   # NULL rows
    assert _couple(lib, _rows(), out=False) == 1                     # NULL out
    assert _couple(lib, _rows(vocab=0)) == 2                         # vocab < 1
    assert _couple(lib, _rows(vocab=(1 << 21) + 1, row_stride=(1 << 21) + 8)) == 2
    assert _couple(lib, _rows(row_stride=32)) == 2                   # stride < vocab
    assert _couple(lib, _rows(n_rows=-1)) == 2
    assert _couple(lib, _rows(), eps=-0.1) == 3
    assert _couple(lib, _rows(), eps=float("nan")) == 3
    assert _couple(lib, _rows(row_offset=-5)) == 3
    assert _couple(lib, _rows(dtype=7)) == 4
    assert _couple(lib, _rows(student=17)) == 5                      # misaligned base
    assert _couple(lib, _rows(row_stride=68)) == 5                   # pitch 136 B
    assert _couple(lib, _rows(student=0)) == 1
    rt = binding.SakiRouteArgs(None, 1.0, 0, None, 64, None, 0)     # loss_sum, no workspace
    assert _couple(lib, _rows(), route=rt) == 6
    assert _couple(lib, _rows(), route=rt, ws=256, ws_bytes=8) == 6  # too small
    # the row work counter needs a workspace on every call with rows
    assert _couple(lib, _rows()) == 6
    need = lib.saki_workspace_bytes(binding.SAKI_OP_COUPLE, 4, 64)
    assert need == 256 + 256 + 256                                   # counters + 4 doubles + 4 indices, rounded
    assert _couple(lib, _rows(), ws=256, ws_bytes=need - 1) == 6
    assert _couple(lib, _rows(), ws=260, ws_bytes=need) == 5         # not 8-byte aligned
    assert _couple(lib, _rows(n_rows=1 << 31), ws=256, ws_bytes=1 << 40) == 2
    rt = binding.SakiRouteArgs(None, float("inf"), 0, None, None, None, 0)
    assert _couple(lib, _rows(), route=rt) == 3
    rt = binding.SakiRouteArgs(None, 1.0, 0, None, None, 48, 32)    # grad stride < vocab
    assert _couple(lib, _rows(), route=rt) == 2
    assert b"vocab" in lib.saki_last_error() or lib.saki_last_error()


def test_zero_rows_returns_ok_without_device(lib):
    assert _couple(lib, _rows(n_rows=0, student=0, teacher=0)) == 0
    assert lib.saki_last_error() == b""


def test_verify_and_route_argument_errors(lib):
    rows = _rows(n_rows=6)
    acc = ctypes.c_void_p(64)
    bad_k = lib.saki_spec_verify(ctypes.byref(rows), 0, 64, 0.1, 1, -1, acc, acc, None, None, 0, None)
    assert bad_k == 2
    not_multiple = lib.saki_spec_verify(ctypes.byref(rows), 4, 64, 0.1, 1, -1, acc, acc, None, None, 0, None)
    assert not_multiple == 2
    no_draft = lib.saki_spec_verify(ctypes.byref(rows), 3, None, 0.1, 1, -1, acc, acc, None, None, 0, None)
    assert no_draft == 1
    # the block work counter lives in the caller's workspace: required, sized, aligned
    assert lib.saki_workspace_bytes(binding.SAKI_OP_VERIFY, 6, 32) == 256
    assert lib.saki_workspace_bytes(binding.SAKI_OP_VERIFY, 0, 32) == 0
    no_ws = lib.saki_spec_verify(ctypes.byref(rows), 3, 64, 0.1, 1, -1, acc, acc, None, None, 0, None)
    assert no_ws == 6 and b"workspace" in lib.saki_last_error()
    small_ws = lib.saki_spec_verify(ctypes.byref(rows), 3, 64, 0.1, 1, -1, acc, acc, None, 256, 128, None)
    assert small_ws == 6
    odd_ws = lib.saki_spec_verify(ctypes.byref(rows), 3, 64, 0.1, 1, -1, acc, acc, None, 258, 256, None)
    assert odd_ws == 5

    rt = binding.SakiRouteArgs(None, 1.0, 0, None, None, None, 0)
    assert lib.saki_route_loss(16, 9, 4, 64, 64, 64, 64, 64, 64, ctypes.byref(rt), None, 0, None) == 4
    assert lib.saki_route_loss(16, 1, 4, 64, 64, None, 64, 64, 64, ctypes.byref(rt), None, 0, None) == 1
    assert lib.saki_route_loss(16, 1, 4, 64, 64, 64, 64, 64, 64, None, None, 0, None) == 1
    # the row counter (and loss slots) live in the caller's workspace
    need = lib.saki_workspace_bytes(binding.SAKI_OP_ROUTE, 4, 64)
    assert need == 512
    assert lib.saki_route_loss(16, 1, 4, 64, 64, 64, 64, 64, 64, ctypes.byref(rt), None, 0, None) == 6
    assert lib.saki_route_loss(16, 1, 4, 64, 64, 64, 64, 64, 64, ctypes.byref(rt), 256, need - 8, None) == 6
    assert lib.saki_route_loss(16, 1, 4, 64, 64, 64, 64, 64, 64, ctypes.byref(rt), 260, need, None) == 5
    assert lib.saki_route_loss(16, 1, 1 << 31, 64, 64, 64, 64, 64, 64, ctypes.byref(rt), 256, 1 << 40, None) == 2
    assert lib.saki_route_loss(16, 1, 0, 64, 64, None, None, None, None, ctypes.byref(rt), None, 0, None) == 0


def test_workspace_sizes(lib):
    assert saki.workspace_bytes(saki.SAKI_OP_COUPLE, 0, 10) == 0
    assert saki.workspace_bytes(saki.SAKI_OP_COUPLE, 1000, 10) >= 8000
    assert saki.workspace_bytes(saki.SAKI_OP_ROUTE, 33, 10) % 256 == 0


def test_correction_target_is_checked(lib):
    rt = binding.SakiRouteArgs(None, 1.0, 0, None, None, None, 0, 7)  # unknown target
    assert _couple(lib, _rows(), route=rt) == 3
    assert b"correction_target" in lib.saki_last_error()


def test_select_positions_argument_errors(lib):
    f = lib.saki_select_positions
    p = 64
    # mode, n_traj, n_rows, offsets, tv, corrected, valid, seed, row_offset, selected, ws, ws_bytes, stream
    assert f(5, 2, 10, p, p, p, None, 1, 0, p, p, 1024, None) == 3          # unknown mode
    assert f(0, -1, 10, p, p, p, None, 1, 0, p, p, 1024, None) == 2         # n_traj < 0
    assert f(0, 2, -3, p, p, p, None, 1, 0, p, p, 1024, None) == 2          # n_rows < 0
    assert f(1, 2, 10, p, p, p, None, 1, -1, p, p, 1024, None) == 3         # row_offset < 0
    assert f(1, 2, 10, None, p, p, None, 1, 0, p, p, 1024, None) == 1       # no offsets
    assert f(1, 2, 10, p, p, p, None, 1, 0, None, p, 1024, None) == 1       # no output
    assert f(1, 2, 10, p, p, p, None, 1, 0, p, None, 0, None) == 6          # no workspace
    assert f(1, 2, 10, p, p, p, None, 1, 0, p, p, 16, None) == 6            # too small
    assert f(1, 2, 10, p, p, p, None, 1, 0, p, 68, 1024, None) == 5         # misaligned
    assert f(1, 0, 10, None, None, None, None, 1, 0, None, None, 0, None) == 0  # nothing to do
    assert saki.workspace_bytes(saki.SAKI_OP_SELECT, 100, 0) >= 800


def test_probe_metrics_argument_errors(lib):
    f = lib.saki_probe_metrics
    rows = _rows()
    assert f(None, 16, None, None, None, None, None, None, None) == 1
    assert f(ctypes.byref(rows), 0, None, None, None, None, None, None, None) == 2
    assert f(ctypes.byref(rows), 65, None, None, None, None, None, None, None) == 2
    assert f(ctypes.byref(_rows(vocab=8, row_stride=8)), 9, None, None, None, None, None, None, None) == 2
    assert f(ctypes.byref(_rows(n_rows=0, student=0, teacher=0)), 4, None, None, None, None, None, None,
             None) == 0


def test_sample_argument_errors(lib):
    f = lib.saki_sample
    tok = ctypes.c_void_p(64)
    assert f(None, 1, 0, tok, None, None) == 1
    assert f(ctypes.byref(_rows()), 0, 0, tok, None, None) == 3            # row_step < 1
    assert f(ctypes.byref(_rows(row_offset=2 ** 62)), 2 ** 62, 0, tok, None, None) == 3  # g overflows
    assert f(ctypes.byref(_rows()), 1, 0, None, None, None) == 1           # NULL token
    assert f(ctypes.byref(_rows(student=0)), 1, 0, tok, None, None) == 1   # NULL student
    assert f(ctypes.byref(_rows(student=8)), 1, 0, tok, None, None) == 5   # misaligned
    assert f(ctypes.byref(_rows(vocab=0)), 1, 0, tok, None, None) == 2
    # the teacher is not read: NULL is fine (zero rows: no device needed)
    assert f(ctypes.byref(_rows(n_rows=0, teacher=0)), 1, 0, tok, None, None) == 0


def _traj(**kw):
    t = dict(n_seq=4, max_len=8, tokens=16, length=32, done=48)
    t.update(kw)
    return binding.SakiTraj(**t)


def test_commit_argument_errors(lib):
    f = lib.saki_commit
    pp = binding.SakiCoupleOut(token=64)
    a, c = ctypes.c_void_p(80), ctypes.c_void_p(96)
    assert f(None, 4, -1, a, c, ctypes.byref(pp), None, None) == 1
    assert f(ctypes.byref(_traj()), 0, -1, a, c, ctypes.byref(pp), None, None) == 2
    assert f(ctypes.byref(_traj()), 65, -1, a, c, ctypes.byref(pp), None, None) == 2
    assert f(ctypes.byref(_traj(n_seq=-1)), 4, -1, a, c, ctypes.byref(pp), None, None) == 2
    assert f(ctypes.byref(_traj(max_len=-1)), 4, -1, a, c, ctypes.byref(pp), None, None) == 2
    assert f(ctypes.byref(_traj(max_len=2 ** 31)), 4, -1, a, c, ctypes.byref(pp), None, None) == 2
    assert f(ctypes.byref(_traj(tokens=0)), 4, -1, a, c, ctypes.byref(pp), None, None) == 1
    assert f(ctypes.byref(_traj(done=0)), 4, -1, a, c, ctypes.byref(pp), None, None) == 1
    assert f(ctypes.byref(_traj()), 4, -1, None, c, ctypes.byref(pp), None, None) == 1
    assert f(ctypes.byref(_traj()), 4, -1, a, c, None, None, None) == 1
    assert f(ctypes.byref(_traj()), 4, -1, a, c, ctypes.byref(binding.SakiCoupleOut()), None, None) == 1
    assert f(ctypes.byref(_traj(n_seq=0)), 4, -1, None, None, None, None, None) == 0


def test_static_scratch_entry_rejects_without_launch(lib):
    """saki_couple_static: the same argument checks as saki_couple, and more
    rows than its static scratch holds is SAKI_E_SHAPE before any device call."""
    co = binding.SakiCoupleOut()

    def call(rows, eps=0.1):
        return lib.saki_couple_static(ctypes.byref(rows), eps, 1, ctypes.byref(co), None, None)

    assert binding.SAKI_STATIC_MAX_ROWS == 262144
    assert call(_rows(n_rows=binding.SAKI_STATIC_MAX_ROWS + 1)) == 2
    assert b"SAKI_STATIC_MAX_ROWS" in lib.saki_last_error()
    assert call(_rows(vocab=0)) == 2
    assert call(_rows(), eps=-1.0) == 3
    assert call(_rows(student=17)) == 5
    assert call(_rows(n_rows=0)) == 0
    assert lib.saki_couple_static(None, 0.1, 1, ctypes.byref(co), None, None) == 1
