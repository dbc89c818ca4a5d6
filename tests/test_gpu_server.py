"""The local request server on the GPU: scores through the socket equal the
direct calls' bit for bit (hits with and without dynamic batching, multi-plane
hits, pre-cut patches), from client threads and from a client process that
never touches the GPU; a bad request is refused and a stopped server ends its
connections.  The direct calls are themselves checked against the oracle in
test_gpu_parity.py; here one sample is also checked against the oracle."""

import os
import subprocess
import sys
import tempfile
import threading

import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def say(*a):
    print(*a, flush=True, file=sys.stderr)


@pytest.fixture(scope="module")
def pid():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2009_04509_amd import binding
    return binding


@pytest.fixture(scope="module")
def setup(pid):
    planes, reqs = synth.config5_requests(n_planes=3, n_streams=4, per_stream=3, lo=200, hi=2500)
    imgs = [torch.from_numpy(p.image).to(DEV) for p in planes]
    h = pid.pointid_create(synth.he_normal_weights(), "fp16", 0)
    yield planes, reqs, imgs, h
    h.close()


def direct(pid, h, imgs, plane, hits):
    out = pid.pointid_classify(h, imgs[plane], torch.from_numpy(hits).to(DEV))
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("max_requests", [0, 8])
def test_hits_through_the_server_match_direct_calls(pid, setup, max_requests):
    planes, reqs, imgs, h = setup
    with tempfile.TemporaryDirectory() as d:
        path = os.path.join(d, "pid.sock")
        srv = pid.Server(h, imgs, path, max_requests=max_requests, max_delay_us=300)
        say(f"server max_requests={max_requests}: {len(reqs)} client threads")
        results, errors = {}, []

        def client(s):
            try:
                c = pid.Client(path)
                for k, (plane, hits) in enumerate(reqs[s]):
                    results[(s, k)] = c.classify(hits, plane=plane)
                c.close()
            except Exception as e:           # reported below
                errors.append(repr(e))

        ths = [threading.Thread(target=client, args=(s,)) for s in range(len(reqs))]
        for th in ths:
            th.start()
        for th in ths:
            th.join(timeout=120)
        srv.close()
    assert not errors, errors
    for (s, k), got in results.items():
        plane, hits = reqs[s][k]
        assert np.array_equal(got, direct(pid, h, imgs, plane, hits)), (s, k)
    assert len(results) == sum(len(r) for r in reqs)
    # one request against the oracle
    plane, hits = reqs[0][0]
    want = oracle.classify(planes[plane].image, hits[:256], synth.he_normal_weights())
    assert np.abs(results[(0, 0)][:256] - want).max() <= 2e-2


def test_multiplane_hits_and_patches(pid, setup):
    planes, reqs, imgs, h = setup
    rng = np.random.default_rng(61)
    h3 = np.concatenate([np.c_[np.full(len(x), p, np.int32), x] for p, x in
                         (reqs[0][0], reqs[1][0])]).astype(np.int32)
    h3 = h3[rng.permutation(len(h3))]
    P = oracle.gather_patches_planes([p.image for p in planes], h3[:700])
    with tempfile.TemporaryDirectory() as d:
        path = os.path.join(d, "pid.sock")
        srv = pid.Server(h, imgs, path, max_requests=4)
        c = pid.Client(path)
        got3 = c.classify(h3, plane=-1)
        gotp = c.classify_patches(P)
        assert c.server_ns > 0
        empty = c.classify(np.zeros((0, 2), np.int32), plane=0)
        c.close()
        srv.close()
    want3 = pid.pointid_classify_planes(h, imgs, torch.from_numpy(h3).to(DEV))
    wantp = pid.pointid_classify_patches(h, torch.from_numpy(P).to(DEV))
    torch.cuda.synchronize()
    assert np.array_equal(got3, want3.cpu().numpy())
    assert np.array_equal(gotp, wantp.cpu().numpy())
    assert empty.shape == (0, 4)


def test_client_process_without_gpu(pid, setup):
    planes, reqs, imgs, h = setup
    plane, hits = reqs[2][1]
    with tempfile.TemporaryDirectory() as d:
        path = os.path.join(d, "pid.sock")
        np.save(os.path.join(d, "hits.npy"), hits)
        srv = pid.Server(h, imgs, path, max_requests=8)
        code = (
            "import sys, numpy as np; sys.path.insert(0, sys.argv[1]);"
            "from paper_2009_04509_amd import binding as b;"
            "c = b.Client(sys.argv[2]);"
            "s = c.classify(np.load(sys.argv[3]), plane=int(sys.argv[4]));"
            "np.save(sys.argv[5], s); c.close()")
        env = dict(os.environ, HIP_VISIBLE_DEVICES="")      # the client needs no GPU
        r = subprocess.run([sys.executable, "-c", code, ROOT, path, os.path.join(d, "hits.npy"),
                            str(plane), os.path.join(d, "scores.npy")],
                           env=env, timeout=180, capture_output=True, text=True)
        srv.close()
        assert r.returncode == 0, r.stderr[-2000:]
        got = np.load(os.path.join(d, "scores.npy"))
    assert np.array_equal(got, direct(pid, h, imgs, plane, hits))


def test_bad_request_and_stopped_server(pid, setup):
    planes, reqs, imgs, h = setup
    with tempfile.TemporaryDirectory() as d:
        path = os.path.join(d, "pid.sock")
        srv = pid.Server(h, imgs, path)
        c = pid.Client(path)
        with pytest.raises(pid.PointIdError) as e:
            c.classify(reqs[0][0][1], plane=7)         # the server holds 3 planes
        assert e.value.status == pid.POINTID_EINVAL
        with pytest.raises(pid.PointIdError) as e:     # the server dropped the connection
            c.classify(reqs[0][0][1], plane=0)
        assert e.value.status == pid.POINTID_EIO
        c.close()
        c2 = pid.Client(path)
        assert c2.classify(reqs[0][0][1][:10], plane=0).shape == (10, 4)
        srv.close()
        assert not os.path.exists(path)
        with pytest.raises(pid.PointIdError) as e:
            c2.classify(reqs[0][0][1][:10], plane=0)
        assert e.value.status == pid.POINTID_EIO
        c2.close()


def test_finished_connections_are_reaped(pid, setup):
    # clients that come and go must not leave sockets or threads behind
    planes, reqs, imgs, h = setup
    hits = reqs[1][0][1][:50]
    with tempfile.TemporaryDirectory() as d:
        path = os.path.join(d, "pid.sock")
        srv = pid.Server(h, imgs, path, max_requests=4)
        c = pid.Client(path)
        want = c.classify(hits, plane=reqs[1][0][0])
        c.close()
        n0 = len(os.listdir("/proc/self/fd"))
        for _ in range(40):
            c = pid.Client(path)
            assert np.array_equal(c.classify(hits, plane=reqs[1][0][0]), want)
            c.close()
        n1 = len(os.listdir("/proc/self/fd"))
        srv.close()
    assert n1 - n0 <= 3, (n0, n1)
