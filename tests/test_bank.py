"""The noise bank's host logic (csrc/bank.cpp) without a GPU: file format, shape index,
single-use watermark (also across reopening and across handles), exhaustion, corrupt
files, storage accounting, and argument checks of the create call.  Bank files are
written here with numpy in the documented layout; creating one from a GPU correction
is covered by test_gpu_bank.py."""
import ctypes
import os
import struct

import numpy as np
import pytest

import paper_2609_15039_amd as sp

OK, ARG, SHAPE, ALIGN, UNSUP, WS = 0, -1, -2, -4, -5, -7
IO, EXHAUSTED, FORMAT, BUSY = -8, -9, -10, -11


@pytest.fixture(scope="module")
def lib():
    return sp.load()


def write_bank(path, K, N, rows, row0=0, consumed=0, seed=7, sid=0x102, mech=1, prec=2, delta=825.27, eps=2.0,
               data=None, magic=b"SPLTBANK"):
    if data is None:
        data = np.arange(rows * N, dtype=np.float32).reshape(rows, N) * np.float32(0.5) - 3.0
    hdr = struct.pack("<8sIIqqQQiiddqqq32x", magic, 1, 128, K, N, seed, sid, mech, prec, delta, eps, row0, rows,
                      consumed)
    assert len(hdr) == 128
    with open(path, "wb") as f:
        f.write(hdr)
        f.write(np.ascontiguousarray(data, dtype=np.float32).tobytes())
    return data


def open_bank(lib, path):
    h = ctypes.c_void_p()
    rc = lib.splitee_bank_open(os.fsencode(str(path)), ctypes.byref(h))
    return rc, h.value


def load_host(lib, bank, rows, N, ldc=None):
    ldc = ldc or N
    out = np.full((max(rows, 1), ldc), np.nan, dtype=np.float32)
    r0 = ctypes.c_int64(-1)
    rc = lib.splitee_bank_load(bank, rows, out.ctypes.data, ldc, 0, ctypes.byref(r0), None)
    return rc, r0.value, out


def test_path_is_the_shape_index(lib):
    assert sp.splitee_bank_path("/banks", 3072, 5120, sp.SPLITEE_MECH_GAUSSIAN) == \
        "/banks/bank-s0000000000000001-k3072-n5120.spb"
    buf = ctypes.create_string_buffer(8)
    assert lib.splitee_bank_path(b"/banks", 1, 1, 1, buf, 8) == ARG  # does not fit


def test_open_info_and_accounting(lib, tmp_path):
    p = tmp_path / "b.spb"
    write_bank(p, K=64, N=24, rows=10, row0=1000)
    rc, b = open_bank(lib, p)
    assert rc == OK
    info = sp.splitee_bank_info(b)
    assert (info["K"], info["N"], info["rows"], info["row0"], info["consumed"]) == (64, 24, 10, 1000, 0)
    assert (info["seed"], info["stream_id"], info["mech"], info["prec"]) == (7, 0x102, 1, 2)
    assert (info["sensitivity"], info["epsilon"]) == (825.27, 2.0)
    assert info["bytes_stored"] == os.path.getsize(p) == 128 + 10 * 24 * 4
    assert info["bytes_with_masks"] == 128 + 10 * (24 + 64) * 4  # a bank that also stores eta
    sp.splitee_bank_close(b)


def test_rows_are_handed_out_once_in_order(lib, tmp_path):
    p = tmp_path / "b.spb"
    data = write_bank(p, K=8, N=12, rows=10, row0=40)
    rc, b = open_bank(lib, p)
    rc, r0, out = load_host(lib, b, 3, 12)
    assert (rc, r0) == (OK, 40) and np.array_equal(out[:3], data[0:3])
    rc, r0, out = load_host(lib, b, 4, 12, ldc=16)  # padded destination rows
    assert (rc, r0) == (OK, 43) and np.array_equal(out[:4, :12], data[3:7]) and np.all(np.isnan(out[:4, 12:]))
    rc, r0, _ = load_host(lib, b, 0, 12)  # reports the next row, takes nothing
    assert (rc, r0) == (OK, 47)
    rc, r0, out = load_host(lib, b, 4, 12)  # only 3 left: nothing taken
    assert rc == EXHAUSTED and np.all(np.isnan(out))
    assert sp.splitee_bank_info(b)["consumed"] == 7
    sp.splitee_bank_close(b)
    # the watermark is in the file: a new handle continues after it
    rc, b = open_bank(lib, p)
    assert sp.splitee_bank_info(b)["consumed"] == 7
    rc, r0, out = load_host(lib, b, 3, 12)
    assert (rc, r0) == (OK, 47) and np.array_equal(out[:3], data[7:10])
    rc, _, _ = load_host(lib, b, 1, 12)
    assert rc == EXHAUSTED
    sp.splitee_bank_close(b)
    with open(p, "rb") as f:
        assert struct.unpack_from("<q", f.read(128), 88)[0] == 10


def test_one_handle_per_file(lib, tmp_path):
    p = tmp_path / "b.spb"
    write_bank(p, K=8, N=4, rows=2)
    rc, b = open_bank(lib, p)
    assert rc == OK
    assert open_bank(lib, p)[0] == BUSY
    sp.splitee_bank_close(b)
    rc, b = open_bank(lib, p)
    assert rc == OK
    sp.splitee_bank_close(b)


@pytest.mark.parametrize("kind", ["magic", "truncated", "long", "consumed", "mech", "eps", "missing"])
def test_invalid_files_do_not_open(lib, tmp_path, kind):
    p = tmp_path / "b.spb"
    if kind == "magic":
        write_bank(p, 8, 4, 2, magic=b"\0" * 8)  # what an interrupted create leaves
    elif kind == "truncated":
        write_bank(p, 8, 4, 3)
        os.truncate(p, 128 + 2 * 4 * 4)
    elif kind == "long":
        write_bank(p, 8, 4, 3)
        with open(p, "ab") as f:
            f.write(b"\0" * 4)
    elif kind == "consumed":
        write_bank(p, 8, 4, 3, consumed=4)
    elif kind == "mech":
        write_bank(p, 8, 4, 3, mech=7)
    elif kind == "eps":
        write_bank(p, 8, 4, 3, eps=0.0)
    rc, b = open_bank(lib, p)
    assert rc == (IO if kind == "missing" else FORMAT) and not b


def test_load_argument_checks(lib, tmp_path):
    p = tmp_path / "b.spb"
    write_bank(p, 8, 12, 4)
    rc, b = open_bank(lib, p)
    r0 = ctypes.c_int64()
    buf = np.zeros((4, 12), np.float32)
    assert lib.splitee_bank_load(b, 1, buf.ctypes.data, 11, 0, ctypes.byref(r0), None) == SHAPE
    assert lib.splitee_bank_load(b, -1, buf.ctypes.data, 12, 0, ctypes.byref(r0), None) == ARG
    assert lib.splitee_bank_load(b, 1, None, 12, 0, ctypes.byref(r0), None) == ARG
    assert lib.splitee_bank_load(b, 1, buf.ctypes.data, 12, 0, None, None) == ARG
    assert sp.splitee_bank_info(b)["consumed"] == 0  # failed checks take nothing
    sp.splitee_bank_close(b)
    assert lib.splitee_bank_close(None) == ARG


def create(lib, path, W=16, K=64, N=32, rows=0, prec=2, mech=1, delta=1.0, eps=1.0, ws=None, wsb=0, ldw=None):
    return lib.splitee_bank_create(os.fsencode(str(path)), W, 1, ldw or K, K, N, mech, delta, eps, 0, 0, 0, rows,
                                   prec, ws, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(rows=-1), ARG), (dict(N=30), SHAPE), (dict(K=60), SHAPE), (dict(prec=1), UNSUP), (dict(prec=9), UNSUP),
    (dict(eps=0.0), ARG), (dict(mech=5), ARG), (dict(ldw=32), SHAPE), (dict(W=8), ALIGN),
    (dict(rows=5), WS), (dict(rows=5, W=None), ARG), (dict(rows=5, ws=16, wsb=1 << 30), ALIGN)])
def test_create_checks_arguments_before_touching_the_file(lib, tmp_path, kw, code):
    p = tmp_path / "b.spb"
    assert create(lib, p, **kw) == code
    assert not p.exists()


def test_create_empty_bank_and_never_overwrite(lib, tmp_path):
    p = tmp_path / "b.spb"
    assert create(lib, p, W=None, rows=0) == OK  # no correction to compute: no device work
    rc, b = open_bank(lib, p)
    info = sp.splitee_bank_info(b)
    assert (info["rows"], info["K"], info["N"], info["prec"]) == (0, 64, 32, 2)
    assert load_host(lib, b, 1, 32)[0] == EXHAUSTED
    sp.splitee_bank_close(b)
    before = p.read_bytes()
    assert create(lib, p, W=None, rows=0, N=64) == IO  # exists: kept as it was
    assert p.read_bytes() == before


def test_workspace_query(lib):
    q = lib.splitee_bank_workspace_bytes
    assert q(64, 32, 1) == 0 and q(60, 32, 2) == 0
    assert q(2560, 6144, 2) >= lib.splitee_fused_workspace_bytes(256, 6144, 2560, 2) + 256 * 6144 * 4
