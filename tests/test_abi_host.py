"""Host-side checks of the C ABI: the library loads, exports every entry point
the header declares, and rejects bad arguments before touching a GPU."""

import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pointid.h")


@pytest.fixture(scope="module")
def b():
    from paper_2009_04509_amd import binding
    return binding


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(pointid_[a-z_]+)\s*\(", src)))


def test_header_symbols_exported(b):
    names = _declared()
    assert "pointid_create" in names and "pointid_classify" in names
    assert set(names) == set(b.EXPORTED)
    for name in names:
        assert hasattr(b.lib, name), name


def test_version_and_empty_error(b):
    assert "gfx950" in b.pointid_version()
    assert isinstance(b.pointid_last_error(), str)


NULL = ctypes.c_void_p(0)
FAKE = ctypes.c_void_p(0x1000)      # never dereferenced: every call below fails validation first


def test_classify_validation(b):
    L = b.lib
    assert L.pointid_classify(NULL, FAKE, 10, 10, FAKE, 5, FAKE, NULL) == b.POINTID_EINVAL
    assert "handle" in b.pointid_last_error()
    assert L.pointid_classify_patches(NULL, FAKE, 5, FAKE, NULL) == b.POINTID_EINVAL
    assert L.pointid_classify_planes(NULL, None, 1, FAKE, 5, FAKE, NULL) == b.POINTID_EINVAL
    assert L.pointid_precision(NULL) == b.POINTID_EINVAL


def test_gather_validation(b):
    L = b.lib
    assert L.pointid_gather(FAKE, 10, 10, FAKE, -1, FAKE, 0, NULL) == b.POINTID_EINVAL
    assert L.pointid_gather(FAKE, 0, 10, FAKE, 3, FAKE, 0, NULL) == b.POINTID_EINVAL
    assert L.pointid_gather(FAKE, 10, -2, FAKE, 3, FAKE, 0, NULL) == b.POINTID_EINVAL
    assert L.pointid_gather(FAKE, 10, 10, FAKE, 3, FAKE, 7, NULL) == b.POINTID_EUNSUPPORTED
    assert L.pointid_gather(NULL, 10, 10, FAKE, 3, FAKE, 0, NULL) == b.POINTID_EINVAL
    assert L.pointid_gather(FAKE, 10, 10, FAKE, 3, ctypes.c_void_p(0x1004), 0, NULL) == b.POINTID_EINVAL
    assert "aligned" in b.pointid_last_error()
    # n == 0 is a no-op even with NULL pointers
    assert L.pointid_gather(NULL, 10, 10, NULL, 0, NULL, 0, NULL) == b.POINTID_OK


def test_planes_validation(b):
    L = b.lib
    P = b._Plane
    good = (P * 2)(P(0x1000, 10, 10), P(0x2000, 4, 4))
    assert L.pointid_gather_planes(good, 0, FAKE, 3, FAKE, 0, NULL) == b.POINTID_EINVAL
    assert L.pointid_gather_planes(good, 65, FAKE, 3, FAKE, 0, NULL) == b.POINTID_EINVAL
    assert "n_planes" in b.pointid_last_error()
    bad = (P * 2)(P(0x1000, 10, 10), P(0, 4, 4))
    assert L.pointid_gather_planes(bad, 2, FAKE, 3, FAKE, 0, NULL) == b.POINTID_EINVAL
    bad2 = (P * 2)(P(0x1000, 10, 10), P(0x2000, 0, 4))
    assert L.pointid_gather_planes(bad2, 2, FAKE, 3, FAKE, 0, NULL) == b.POINTID_EINVAL
    assert L.pointid_gather_planes(good, 2, NULL, 0, NULL, 0, NULL) == b.POINTID_OK


def test_requests_validation(b):
    """Batched requests: every request is checked before the handle is used
    (FAKE handles below are never dereferenced)."""
    L = b.lib
    P, R = b._Plane, b._Request
    planes = (P * 2)(P(0x1000, 10, 10), P(0x2000, 4, 4))
    ok = R(0x3000, 5, 0, 0x4000)
    assert L.pointid_classify_requests(NULL, planes, 2, (R * 1)(ok), 1, NULL) == b.POINTID_EINVAL
    assert L.pointid_classify_requests(FAKE, planes, 2, (R * 1)(ok), -1, NULL) == b.POINTID_EINVAL
    assert L.pointid_classify_requests(FAKE, planes, 2, None, 1, NULL) == b.POINTID_EINVAL
    assert L.pointid_classify_requests(FAKE, planes, 0, (R * 1)(ok), 1, NULL) == b.POINTID_EINVAL
    assert L.pointid_classify_requests(FAKE, None, 2, (R * 1)(ok), 1, NULL) == b.POINTID_EINVAL
    cases = [
        (R(0x3000, -1, 0, 0x4000), "negative"),
        (R(0x3000, 5, 2, 0x4000), "plane index"),
        (R(0, 5, 0, 0x4000), "NULL"),
        (R(0x3000, 5, -1, 0), "NULL"),
        (R(0x3000, 5, 1, 0x4004), "aligned"),
    ]
    for bad, word in cases:
        # a valid request first: nothing is classified before all are checked
        arr = (R * 2)(ok, bad)
        assert L.pointid_classify_requests(FAKE, planes, 2, arr, 2, NULL) == b.POINTID_EINVAL
        assert word in b.pointid_last_error() and "request 1" in b.pointid_last_error()
    # no requests, or only empty ones with NULL pointers, is a no-op
    assert L.pointid_classify_requests(FAKE, planes, 2, None, 0, NULL) == b.POINTID_OK
    empty = (R * 2)(R(0, 0, 0, 0), R(0, 0, -1, 0))
    assert L.pointid_classify_requests(FAKE, planes, 2, empty, 2, NULL) == b.POINTID_OK


def test_batcher_validation(b):
    """Batcher entry points reject bad arguments before using the handle."""
    L = b.lib
    P, R = b._Plane, b._Request
    planes = (P * 1)(P(0x1000, 10, 10))
    out = ctypes.c_void_p(0x1234)
    assert L.pointid_batcher_create(NULL, planes, 1, 64, 100, ctypes.byref(out)) == b.POINTID_EINVAL
    assert out.value is None                     # cleared on failure
    assert L.pointid_batcher_create(FAKE, planes, 1, 64, 100, None) == b.POINTID_EINVAL
    assert L.pointid_batcher_create(FAKE, None, 1, 64, 100, ctypes.byref(out)) == b.POINTID_EINVAL
    assert L.pointid_batcher_create(FAKE, planes, 0, 64, 100, ctypes.byref(out)) == b.POINTID_EINVAL
    assert L.pointid_batcher_create(FAKE, planes, 1, 0, 100, ctypes.byref(out)) == b.POINTID_EINVAL
    assert L.pointid_batcher_create(FAKE, planes, 1, 5000, 100, ctypes.byref(out)) == b.POINTID_EINVAL
    assert L.pointid_batcher_create(FAKE, planes, 1, 64, -1, ctypes.byref(out)) == b.POINTID_EINVAL
    bad = (P * 1)(P(0, 10, 10))
    assert L.pointid_batcher_create(FAKE, bad, 1, 64, 100, ctypes.byref(out)) == b.POINTID_EINVAL
    t = ctypes.c_uint64()
    req = R(0x3000, 5, 0, 0x4000)
    assert L.pointid_batcher_submit(NULL, ctypes.byref(req), NULL, ctypes.byref(t)) == b.POINTID_EINVAL
    assert L.pointid_trim(NULL, 0, None) == b.POINTID_EINVAL
    assert L.pointid_batcher_wait(NULL, 1) == b.POINTID_EINVAL
    assert L.pointid_batcher_destroy(NULL) == b.POINTID_OK


def test_create_validation(b):
    L = b.lib
    out = ctypes.c_void_p(123)
    assert L.pointid_create(None, 0, 0, ctypes.byref(out)) == b.POINTID_EINVAL
    assert out.value is None
    assert L.pointid_create(None, 0, 0, None) == b.POINTID_EINVAL
    arrays = {n: np.zeros(s, np.float32) for n, s in b._WEIGHT_SIZES.items()}
    fields = {n: arrays[n].ctypes.data_as(ctypes.POINTER(ctypes.c_float)) for n in arrays}
    w = b._Weights(**fields)
    assert L.pointid_create(ctypes.byref(w), 9, 0, ctypes.byref(out)) == b.POINTID_EUNSUPPORTED
    w_missing = b._Weights(**{**fields, "fc1_w": ctypes.POINTER(ctypes.c_float)()})
    assert L.pointid_create(ctypes.byref(w_missing), 0, 0, ctypes.byref(out)) == b.POINTID_EINVAL


def test_create_without_gpu_is_enodev(b):
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is visible")
    import synth
    with pytest.raises(b.PointIdError) as e:
        b.pointid_create(synth.he_normal_weights(), "fp32", 0)
    assert e.value.status == b.POINTID_ENODEV


def test_destroy_null_is_noop(b):
    assert b.lib.pointid_destroy(NULL) == b.POINTID_OK


def test_binding_shape_checks(b):
    import torch
    with pytest.raises(ValueError):
        b.pointid_create({**{n: np.zeros(s, np.float32) for n, s in b._WEIGHT_SIZES.items()},
                          "fc2_b": np.zeros(5, np.float32)})
    with pytest.raises((TypeError, ValueError)):
        b.pointid_gather(torch.zeros(4, 4), torch.zeros(3, 2, dtype=torch.int32))


def test_find_hits_validation(b):
    L = b.lib
    P = b._Plane
    good = (P * 1)(P(0x1000, 10, 10))
    n_found = ctypes.c_void_p(0x2000)
    assert L.pointid_find_hits(NULL, good, 1, 1.0, FAKE, 5, n_found, NULL) == b.POINTID_EINVAL
    assert "handle" in b.pointid_last_error()
    # handle checks come first; the remaining rules are exercised with a fake
    # non-NULL handle that validation rejects before it is ever used
    H = ctypes.c_void_p(0x3000)
    assert L.pointid_find_hits(H, good, 1, 1.0, FAKE, -1, n_found, NULL) == b.POINTID_EINVAL
    assert "capacity" in b.pointid_last_error()
    assert L.pointid_find_hits(H, good, 0, 1.0, FAKE, 5, n_found, NULL) == b.POINTID_EINVAL
    assert L.pointid_find_hits(H, None, 1, 1.0, FAKE, 5, n_found, NULL) == b.POINTID_EINVAL
    assert L.pointid_find_hits(H, good, 1, 1.0, FAKE, 5, NULL, NULL) == b.POINTID_EINVAL
    assert L.pointid_find_hits(H, good, 1, 1.0, FAKE, 5, ctypes.c_void_p(0x2004), NULL) == b.POINTID_EINVAL
    assert "aligned" in b.pointid_last_error()
    assert L.pointid_find_hits(H, good, 1, 1.0, NULL, 5, n_found, NULL) == b.POINTID_EINVAL
    assert "hits_out" in b.pointid_last_error()


def test_downsample_validation(b):
    L = b.lib
    assert L.pointid_downsample(FAKE, 0, 10, 2, FAKE, NULL) == b.POINTID_EINVAL
    assert L.pointid_downsample(FAKE, 10, 0, 2, FAKE, NULL) == b.POINTID_EINVAL
    assert L.pointid_downsample(FAKE, 10, 10, 0, FAKE, NULL) == b.POINTID_EINVAL
    assert "ticks_per_column" in b.pointid_last_error()
    assert L.pointid_downsample(NULL, 10, 10, 2, FAKE, NULL) == b.POINTID_EINVAL
    assert L.pointid_downsample(FAKE, 10, 10, 2, NULL, NULL) == b.POINTID_EINVAL
    P = b._Plane
    good = (P * 1)(P(0x1000, 10, 10))
    assert L.pointid_classify_planes_ds(NULL, good, 1, 2, FAKE, 5, FAKE, NULL) == b.POINTID_EINVAL
    H = ctypes.c_void_p(0x3000)     # rejected by validation before it is used
    assert L.pointid_classify_planes_ds(H, good, 1, 0, FAKE, 5, FAKE, NULL) == b.POINTID_EINVAL
    assert L.pointid_classify_planes_ds(H, good, 1, 2, FAKE, -1, FAKE, NULL) == b.POINTID_EINVAL
    assert L.pointid_classify_planes_ds(H, good, 1, 2, FAKE, 5, ctypes.c_void_p(0x1004), NULL) \
        == b.POINTID_EINVAL
    assert L.pointid_classify_planes_ds(H, good, 1, 2, NULL, 0, NULL, NULL) == b.POINTID_OK


def test_server_and_client_validation(b, tmp_path):
    L = b.lib
    out = ctypes.c_void_p()
    path = str(tmp_path / "s.sock").encode()
    assert L.pointid_server_start(NULL, None, 0, path, 0, 0, ctypes.byref(out)) == b.POINTID_EINVAL
    assert "handle" in b.pointid_last_error()
    H = ctypes.c_void_p(0x3000)     # rejected by validation before it is used
    assert L.pointid_server_start(H, None, 1, path, 0, 0, ctypes.byref(out)) == b.POINTID_EINVAL
    assert L.pointid_server_start(H, None, 0, None, 0, 0, ctypes.byref(out)) == b.POINTID_EINVAL
    assert L.pointid_server_start(H, None, 0, b"x" * 200, 0, 0, ctypes.byref(out)) == b.POINTID_EINVAL
    assert L.pointid_server_start(H, None, 0, path, -1, 0, ctypes.byref(out)) == b.POINTID_EINVAL
    assert L.pointid_server_stop(NULL) == b.POINTID_OK
    # no server behind the path
    assert L.pointid_client_connect(str(tmp_path / "none.sock").encode(), ctypes.byref(out)) \
        == b.POINTID_EIO
    assert "connect" in b.pointid_last_error()
    assert L.pointid_client_connect(None, ctypes.byref(out)) == b.POINTID_EINVAL
    assert L.pointid_client_classify(NULL, 0, FAKE, 1, FAKE, None) == b.POINTID_EINVAL
    assert L.pointid_client_classify_patches(NULL, FAKE, 1, FAKE, None) == b.POINTID_EINVAL
    assert L.pointid_client_close(NULL) == b.POINTID_OK


def test_client_wire_protocol_against_a_stub_server(b, tmp_path):
    # a stub speaking the documented wire format on the CPU: the client sends
    # a 32-byte header and the payload, and reads back scores, a server status
    # or, on a malformed response, fails with EIO
    import socket
    import struct
    import threading

    path = str(tmp_path / "stub.sock")
    srv = socket.socket(socket.AF_UNIX, socket.SOCK_STREAM)
    srv.bind(path)
    srv.listen(1)
    seen = []

    def stub():
        conn, _ = srv.accept()
        with conn:
            for reply in ("scores", "status", "garbage"):
                hdr = b""
                while len(hdr) < 32:
                    hdr += conn.recv(32 - len(hdr))
                magic, kind, plane, _, n, rid = struct.unpack("<IIiiqQ", hdr)
                width = 2 if plane >= 0 else 3
                body = b""
                while len(body) < 4 * width * n:
                    body += conn.recv(4 * width * n - len(body))
                seen.append((magic, kind, plane, n, np.frombuffer(body, np.int32).copy()))
                if reply == "scores":
                    sc = np.arange(4 * n, dtype=np.float32)
                    conn.sendall(struct.pack("<IiqQq", 0x52444950, 0, n, rid, 1234) + sc.tobytes())
                elif reply == "status":
                    conn.sendall(struct.pack("<IiqQq", 0x52444950, -1, n, rid, 0))
                else:
                    conn.sendall(struct.pack("<IiqQq", 0xDEADBEEF, 0, n, rid, 0))

    th = threading.Thread(target=stub)
    th.start()
    try:
        c = b.Client(path)
        hits = np.array([[3, 7], [4, 8], [5, 9]], np.int32)
        got = c.classify(hits, plane=2)
        assert np.array_equal(got, np.arange(12, dtype=np.float32).reshape(3, 4))
        assert c.server_ns == 1234
        magic, kind, plane, n, body = seen[0]
        assert (magic, kind, plane, n) == (0x51444950, 1, 2, 3)
        assert np.array_equal(body.reshape(3, 2), hits)
        with pytest.raises(b.PointIdError) as e:
            c.classify(np.array([[0, 1, 2]], np.int32), plane=-1)
        assert e.value.status == b.POINTID_EINVAL and seen[1][2] == -1
        with pytest.raises(b.PointIdError) as e:
            c.classify(hits, plane=0)
        assert e.value.status == b.POINTID_EIO
        c.close()
    finally:
        th.join(timeout=10)
        srv.close()


def test_client_request_limits(b):
    L = b.lib
    C = ctypes.c_void_p(0x3000)     # rejected by validation before it is used
    assert L.pointid_client_classify(C, 0, FAKE, (1 << 22) + 1, FAKE, None) == b.POINTID_EINVAL
    assert L.pointid_client_classify(C, 0, FAKE, -1, FAKE, None) == b.POINTID_EINVAL
    assert L.pointid_client_classify_patches(C, FAKE, (1 << 16) + 1, FAKE, None) == b.POINTID_EINVAL
    assert "65536" in b.pointid_last_error()
    assert L.pointid_client_classify(C, 0, NULL, 5, FAKE, None) == b.POINTID_EINVAL
