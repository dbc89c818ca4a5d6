"""GPU: batched requests (pointid_classify_requests).

Several requests classified in one batched call must each get exactly the bits
the request gets when classified alone (pointid_classify for single-plane
requests, pointid_classify_planes for multi-plane ones), whatever else is in the
batch; sampled hits must match the fp64 oracle as in test_gpu_parity.
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
def planes():
    return [synth.config2(2000 + p) for p in range(3)]


def t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def make_requests(rng, sizes):
    """(plane, hits) per size: plane >= 0 with [n][2] hits on it, or -1 with
    [n][3] hits over all planes (every 50th hit on a plane outside the table)."""
    pl = planes()
    out = []
    for k, n in enumerate(sizes):
        if k % 3 == 2:
            p = rng.integers(0, len(pl), size=n)
            h = np.stack([p] + [np.zeros(n, np.int64)] * 2, 1)
            for i in range(n):
                pool = pl[p[i]].hits
                h[i, 1:] = pool[rng.integers(0, len(pool))]
            h[::50, 0] = len(pl)
            out.append((-1, h.astype(np.int32)))
        else:
            p = int(rng.integers(0, len(pl)))
            pool = pl[p].hits
            out.append((p, np.ascontiguousarray(pool[rng.integers(0, len(pool), size=n)])))
    return out


def alone(pid, h, imgs, plane, hits):
    if plane >= 0:
        return pid.pointid_classify(h, imgs[plane], t(hits)).cpu().numpy()
    return pid.pointid_classify_planes(h, imgs, t(hits)).cpu().numpy()


@pytest.mark.parametrize("prec", ["fp32", "bf16", "fp16", "fp8"])
def test_batched_requests_bitwise(pid, prec):
    h = pid.pointid_create(weights(), prec, 0)
    imgs = [t(p.image) for p in planes()]
    rng = np.random.default_rng(11)
    sizes = [1, 17, 235, 0, 1693, 3000, 96, 97, 31, 2048]
    reqs = make_requests(rng, sizes)
    say(f"batched requests {prec}: {len(reqs)} requests, {sum(sizes)} hits")
    outs = pid.pointid_classify_requests(h, imgs, [(p, t(x), None) for p, x in reqs])
    for k, ((p, x), o) in enumerate(zip(reqs, outs)):
        got = o.cpu().numpy()
        if len(x) == 0:
            assert got.shape == (0, 4)
            continue
        ref = alone(pid, h, imgs, p, x)
        assert np.array_equal(got.view(np.uint32), ref.view(np.uint32)), f"request {k}"
    # sampled hits of the largest request (a multi-plane one) against the oracle
    p, x = reqs[5]
    assert p < 0
    idx = np.sort(rng.choice(len(x), 256, replace=False))
    P = oracle.gather_patches_planes([q.image for q in planes()], x[idx])
    got = outs[5].cpu().numpy()[idx].astype(np.float64)
    if prec == "bf16":
        ref, tol = oracle.classify_16bit_emulated(P, weights(), "bf16"), 2e-3
    elif prec == "fp8":
        ref, tol = oracle.classify_fp8_emulated(P, weights()), 5e-2
    else:
        ref, tol = oracle.classify_patches(P, weights()), {"fp32": 1e-4, "fp16": 2e-2}[prec]
    err = float(np.abs(got - np.asarray(ref, np.float64)).max())
    say(f"[requests {prec}] 256 sampled hits: max|d|={err:.3g}")
    assert err <= tol
    h.close()


def test_more_than_64_requests(pid):
    """70 non-empty requests (and some empty ones) run as two batches."""
    h = pid.pointid_create(weights(), "fp16", 0)
    imgs = [t(p.image) for p in planes()]
    rng = np.random.default_rng(12)
    sizes = [int(s) for s in rng.integers(0, 300, size=75)]
    sizes[3] = sizes[40] = 0
    reqs = make_requests(rng, sizes)
    say(f"{len(reqs)} requests, {sum(sizes)} hits")
    outs = pid.pointid_classify_requests(h, imgs, [(p, t(x), None) for p, x in reqs])
    for k, ((p, x), o) in enumerate(zip(reqs, outs)):
        if len(x):
            ref = alone(pid, h, imgs, p, x)
            assert np.array_equal(o.cpu().numpy().view(np.uint32), ref.view(np.uint32)), f"request {k}"
    h.close()


@pytest.mark.parametrize("prec", ["bf16", "fp16", "fp8"])
def test_batcher_threads_bitwise(pid, prec):
    """Requests submitted from 4 host threads through the dynamic batcher get
    the bits they get alone."""
    import threading
    h = pid.pointid_create(weights(), prec, 0)
    imgs = [t(p.image) for p in planes()]
    torch.cuda.synchronize()
    per_thread = []
    for k in range(4):
        rng = np.random.default_rng(100 + k)
        sizes = [int(s) for s in rng.integers(0, 2500, size=25)]
        sizes[0] = 0
        per_thread.append(make_requests(rng, sizes))
    b = pid.Batcher(h, imgs, max_requests=16, max_delay_us=300)
    results = [[None] * len(r) for r in per_thread]
    errors = []

    def client(k):
        try:
            # a few requests in flight per client, then wait for them in order
            tickets = []
            for i, (p, x) in enumerate(per_thread[k]):
                tickets.append((i, b.submit(p, t(x))))
                if len(tickets) == 3:
                    i0, tk = tickets.pop(0)
                    results[k][i0] = b.wait(tk).cpu().numpy()
            for i0, tk in tickets:
                results[k][i0] = b.wait(tk).cpu().numpy()
        except Exception as e:      # reported below
            errors.append(e)

    threads = [threading.Thread(target=client, args=(k,)) for k in range(4)]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    b.close()
    assert not errors, errors
    n = 0
    for k in range(4):
        for i, (p, x) in enumerate(per_thread[k]):
            got = results[k][i]
            if len(x) == 0:
                assert got.shape == (0, 4)
                continue
            ref = alone(pid, h, imgs, p, x)
            assert np.array_equal(got.view(np.uint32), ref.view(np.uint32)), f"client {k} request {i}"
            n += 1
    say(f"batcher {prec}: {n} requests from 4 threads, all equal to single calls")
    h.close()


def test_batcher_destroy_drains(pid):
    """Requests still pending when the batcher is destroyed are classified."""
    h = pid.pointid_create(weights(), "fp16", 0)
    imgs = [t(p.image) for p in planes()]
    rng = np.random.default_rng(13)
    reqs = make_requests(rng, [300, 7, 1200, 64, 5])
    b = pid.Batcher(h, imgs, max_requests=64, max_delay_us=1000000)   # never due by time
    outs = []
    for p, x in reqs:
        sc = torch.full((len(x), 4), float("nan"), device=DEV)
        b.submit(p, t(x), sc)
        outs.append(sc)
    b.close()                        # launches the partial batch and waits for it
    for (p, x), sc in zip(reqs, outs):
        ref = alone(pid, h, imgs, p, x)
        assert np.array_equal(sc.cpu().numpy().view(np.uint32), ref.view(np.uint32))
    h.close()


def test_batcher_waits_for_the_submitting_stream(pid):
    """A request's hits written on the submitting stream just before the submit
    (behind a long queue of other work there) are the hits the batch reads:
    the batch waits for the submitter's stream (pointid_batcher_submit's
    `stream`), so the scores equal those of the final hits."""
    h = pid.pointid_create(weights(), "fp16", 0)
    imgs = [t(p.image) for p in planes()]
    rng = np.random.default_rng(17)
    (p, x), = make_requests(rng, [2000])
    b = pid.Batcher(h, imgs, max_requests=1, max_delay_us=0)
    side = torch.cuda.Stream()
    hits = torch.zeros((len(x), 2), dtype=torch.int32, device=DEV)   # wrong hits until the copy
    torch.cuda.synchronize()
    with torch.cuda.stream(side):
        a = torch.randn((4096, 4096), device=DEV)
        for _ in range(8):                   # keep the side stream busy for a while
            a = a @ a
            a = a / a.norm()
        hits.copy_(t(x), non_blocking=True)
        scores = torch.empty((len(x), 4), dtype=torch.float32, device=DEV)
        ticket = b.submit(p, hits, scores, stream=side)
    got = b.wait(ticket).cpu().numpy()
    b.close()
    ref = alone(pid, h, imgs, p, x)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))
    h.close()


def test_trim_frees_idle_scratch(pid):
    """pointid_trim frees the idle cached scratch; the next call allocates
    again and gives the same bits."""
    h = pid.pointid_create(weights(), "fp16", 0)
    img = t(planes()[0].image)
    hits = t(planes()[0].hits)
    a = pid.pointid_classify(h, img, hits).cpu().numpy()
    torch.cuda.synchronize()
    assert pid.pointid_trim(h, 1 << 40) > 0          # a keep above the cache frees nothing
    assert pid.pointid_trim(h, 0) == 0               # every buffer is idle after the sync
    bb = pid.pointid_classify(h, img, hits).cpu().numpy()
    assert np.array_equal(a.view(np.uint32), bb.view(np.uint32))
    torch.cuda.synchronize()
    assert pid.pointid_trim(h, 0) == 0
    h.close()


def test_scratch_waits_for_the_call_that_used_it(pid):
    """A call's scratch buffer goes to another stream only once the call's last
    kernel has finished: its completion event is attached to that kernel's
    dispatch.  Two event-sized calls on two streams, enqueued back to back with
    no host wait between them, must each give the bits they give alone (a
    completion event that reported done too early would hand the first call's
    buffer to the second while the first still runs)."""
    h = pid.pointid_create(weights(), "fp16", 0)
    planes3, hits3 = synth.config3()
    imgs = [t(p.image) for p in planes3]
    h1 = t(hits3)
    h2 = t(np.ascontiguousarray(hits3[::-1]))
    ref1 = pid.pointid_classify_planes(h, imgs, h1).cpu().numpy().view(np.uint32)
    ref2 = pid.pointid_classify_planes(h, imgs, h2).cpu().numpy().view(np.uint32)
    torch.cuda.synchronize()
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    for rep in range(3):
        say(f"two streams, round {rep}")
        with torch.cuda.stream(sa):
            a = pid.pointid_classify_planes(h, imgs, h1)
        with torch.cuda.stream(sb):
            b = pid.pointid_classify_planes(h, imgs, h2)
        torch.cuda.synchronize()
        assert np.array_equal(a.cpu().numpy().view(np.uint32), ref1), f"round {rep}: first stream"
        assert np.array_equal(b.cpu().numpy().view(np.uint32), ref2), f"round {rep}: second stream"
    h.close()
