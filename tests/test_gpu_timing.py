"""GPU: per-kernel timing (pointid_timing_*).

The timed kernels of one call form a chain of events attached to their
dispatches: the first kernel is timed from its own start event, each later one
from the end of the kernel before it.  Every timed launch must be counted once,
the times must be positive and together no longer than the calls' own span on
the stream, and queries from another thread while calls are being enqueued
must neither fail nor lose launches (the events are reference counted, so a
query never destroys a stop event the next kernel of a call still needs).
"""

import sys
import threading

import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
KERNELS = ("gather", "conv_fc1_16", "tail")


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
    h = pid.pointid_create(synth.he_normal_weights(), "fp16", 0)
    p = synth.config2()
    img = torch.from_numpy(np.ascontiguousarray(p.image)).to(DEV)
    hits = torch.from_numpy(np.ascontiguousarray(p.hits)).to(DEV)
    pid.pointid_classify(h, img, hits)            # warm-up: scratch, code objects
    torch.cuda.synchronize()
    yield h, img, hits
    pid.pointid_timing_enable(False)
    h.close()


def test_every_launch_counted_within_the_calls_span(pid, setup):
    h, img, hits = setup
    pid.pointid_timing_reset()
    pid.pointid_timing_enable(True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        pid.pointid_classify(h, img, hits)
    e1.record()
    torch.cuda.synchronize()
    pid.pointid_timing_enable(False)
    span = e0.elapsed_time(e1)
    total = 0.0
    for k in KERNELS:
        ms, n = pid.pointid_timing_query(k)
        say(f"[timing] {k}: {n} launches, {ms:.4f} ms")
        assert n == 5, f"{k}: {n} launches"
        assert ms > 0.0, k
        total += ms
    say(f"[timing] kernels {total:.4f} ms of a {span:.4f} ms span")
    assert total <= span * 1.02 + 0.005
    pid.pointid_timing_reset()
    assert pid.pointid_timing_query("gather") == (0.0, 0)


def test_queries_from_another_thread(pid, setup):
    h, img, hits = setup
    pid.pointid_timing_reset()
    pid.pointid_timing_enable(True)
    done = threading.Event()
    errors = []

    def poll():
        try:
            while not done.is_set():
                for k in KERNELS:
                    pid.pointid_timing_query(k)
        except Exception as exc:                  # reported below
            errors.append(exc)

    th = threading.Thread(target=poll)
    th.start()
    try:
        for _ in range(40):
            pid.pointid_classify(h, img, hits)
        torch.cuda.synchronize()
    finally:
        done.set()
        th.join()
        pid.pointid_timing_enable(False)
    assert not errors, errors
    for k in KERNELS:
        ms, n = pid.pointid_timing_query(k)
        assert n == 40 and ms > 0.0, (k, n, ms)
