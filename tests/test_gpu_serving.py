"""GPU: the serving pattern — many small requests classified on concurrent streams.

A reduced version of the serving workload (config 5: 1,000-8,000-hit requests
drawn from resident config-2 planes, sent on many streams).  Requests enqueued
round-robin on 8 streams, so that their kernels overlap, must give exactly the
bits each request gives when classified alone, and sampled hits must match the
fp64 oracle to the precision's tolerance (as in test_gpu_parity).
"""

import functools
import sys

import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL = {"fp32": 1e-4, "fp16": 2e-2}


def say(*a):
    print(*a, flush=True, file=sys.stderr)


@pytest.fixture(scope="module")
def pid():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2009_04509_amd import binding
    return binding


@functools.lru_cache(maxsize=None)
def weights():
    return synth.he_normal_weights()


@functools.lru_cache(maxsize=None)
def workload(n_streams, per_stream):
    return synth.config5_requests(n_planes=2, n_streams=n_streams, per_stream=per_stream)


def t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


@pytest.mark.parametrize("prec,per_stream", [("fp16", 4), ("bf16", 4), ("fp32", 1)])
def test_concurrent_streams_bitwise_and_oracle(pid, prec, per_stream):
    planes, reqs = workload(8, per_stream)
    h = pid.pointid_create(weights(), prec, 0)
    imgs = [t(p.image) for p in planes]
    hits = [[t(x) for (_, x) in rs] for rs in reqs]
    say(f"serving {prec}: {len(reqs)} streams x {per_stream} requests, "
        f"{sum(len(x) for rs in reqs for (_, x) in rs)} hits")

    # each request alone, one after another
    alone = [[pid.pointid_classify(h, imgs[p], hits[s][k]).cpu().numpy()
              for k, (p, _) in enumerate(rs)] for s, rs in enumerate(reqs)]

    # all requests in flight on 8 streams
    streams = [torch.cuda.Stream() for _ in reqs]
    outs = [[torch.full((len(x), 4), np.nan, dtype=torch.float32, device=DEV) for (_, x) in rs]
            for rs in reqs]
    torch.cuda.synchronize()
    for k in range(per_stream):
        for s, rs in enumerate(reqs):
            pid.pointid_classify(h, imgs[rs[k][0]], hits[s][k], outs[s][k], stream=streams[s])
    torch.cuda.synchronize()
    for s, rs in enumerate(reqs):
        for k in range(per_stream):
            got = outs[s][k].cpu().numpy()
            assert np.array_equal(got.view(np.uint32), alone[s][k].view(np.uint32)), \
                f"stream {s} request {k}: concurrent result differs from the request alone"

    # sampled hits of two requests against the oracle
    rng = np.random.default_rng(55)
    for s, k in ((0, 0), (len(reqs) - 1, per_stream - 1)):
        p, x = reqs[s][k]
        idx = np.sort(rng.choice(len(x), 256, replace=False))
        P = oracle.gather_patches(planes[p].image, x[idx])
        got = np.asarray(alone[s][k][idx], np.float64)
        if prec == "bf16":
            ref = oracle.classify_16bit_emulated(P, weights(), "bf16").astype(np.float64)
            tol = 2e-3
        else:
            ref = oracle.classify_patches(P, weights()).astype(np.float64)
            tol = TOL[prec]
        err = float(np.abs(got - ref).max())
        say(f"[serving {prec}] stream {s} request {k}: 256 sampled hits, max|d|={err:.3g}")
        assert err <= tol
    h.close()
