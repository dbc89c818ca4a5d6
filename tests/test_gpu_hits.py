"""GPU parity of hit finding (pointid_find_hits) against the CPU oracle.

Hit finding is integer output decided by exact fp32 comparisons, so the bar is
bit-exact: the same (plane, wire, tick) rows in the same order, and the same
count.  Cases: small planes with integer values (frequent plateaus and values
equal to the threshold), row lengths that are not a multiple of 4 or shorter
than one 256-tick step, an image base that is not 16-byte aligned, several
planes of different shapes, the full event workload (18 planes of 6000
ticks), capacity truncation, an empty result and special thresholds.
"""

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


@pytest.fixture(scope="module")
def handle(pid):
    h = pid.pointid_create(synth.he_normal_weights(), "fp16", 0)
    yield h
    h.close()


def run(pid, h, images_np, thr, capacity=None, views=None):
    imgs = views if views is not None else [torch.from_numpy(a).to(DEV) for a in images_np]
    cap = capacity
    if cap is None:
        cap = max(1, sum(a.size for a in images_np) // 2 + 1)
    out = torch.full((max(cap, 1), 3), -7, dtype=torch.int32, device=DEV)
    n_found = torch.full((1,), -1, dtype=torch.int64, device=DEV)
    pid.pointid_find_hits(h, imgs, thr, capacity=cap, hits_out=out, n_found=n_found)
    torch.cuda.synchronize()
    return out.cpu().numpy(), int(n_found.item())


def check_exact(pid, h, images, thr, **kw):
    ref = oracle.find_hits(images, thr)
    got, n = run(pid, h, images, thr, **kw)
    assert n == len(ref), (n, len(ref))
    assert np.array_equal(got[:n], ref)
    return ref


def test_small_integer_planes_with_ties(pid, handle):
    rng = np.random.default_rng(11)
    shapes = [(5, 40), (3, 17), (7, 256), (2, 257), (1, 1), (4, 3), (9, 1000), (1, 513)]
    imgs = [rng.integers(-3, 6, size=s).astype(np.float32) for s in shapes]
    say("find_hits small integer planes")
    for thr in (-1.0, 0.0, 2.0, 3.5, 5.0):
        check_exact(pid, handle, imgs, thr)


def test_gaussian_planes_and_odd_lengths(pid, handle):
    rng = np.random.default_rng(12)
    imgs = [rng.normal(0, 2.5, size=(33, T)).astype(np.float32) for T in (6000, 5999, 6001, 250)]
    for thr in (0.0, 7.5):
        check_exact(pid, handle, imgs, thr)


def test_worker_ranges_cross_wires_and_planes(pid, handle):
    # enough 256-tick steps that every wave owns several, so its range starts
    # and ends mid-wire and crosses wires and planes; odd lengths (4-byte loads)
    # and multiples of 4 (16-byte loads)
    rng = np.random.default_rng(17)
    odd = [rng.integers(-3, 6, size=s).astype(np.float32)
           for s in [(700, 6001), (500, 777), (900, 2000)]]
    even = [rng.integers(-3, 6, size=s).astype(np.float32) for s in [(4000, 1028), (37, 6000)]]
    say("find_hits long worker ranges")
    for imgs in (odd, even):
        steps = sum(a.shape[0] * -(-a.shape[1] // 256) for a in imgs)
        assert steps > 2 * 8192
        check_exact(pid, handle, imgs, 2.0)


def test_unaligned_image_base(pid, handle):
    rng = np.random.default_rng(13)
    W, T = 21, 700                                  # T % 4 == 0, base off by 4 bytes
    big = torch.from_numpy(rng.integers(-2, 9, size=W * T + 3).astype(np.float32)).to(DEV)
    for off in (1, 2, 3):
        view = big[off:off + W * T].view(W, T)
        ref = oracle.find_hits([view.cpu().numpy()], 1.0)
        got, n = run(pid, handle, [view.cpu().numpy()], 1.0, views=[view])
        assert n == len(ref) and np.array_equal(got[:n], ref), off


def test_event_planes(pid, handle):
    planes, _ = synth.config3()
    imgs = [p.image for p in planes]
    say("find_hits event planes (18 x 6000 ticks)")
    for thr in (10.0, 40.0):
        ref = check_exact(pid, handle, imgs, thr, capacity=4_000_000)
        assert len(ref) > 50_000


def test_capacity_truncation_and_empty(pid, handle):
    rng = np.random.default_rng(14)
    imgs = [rng.normal(0, 2.5, size=(40, 600)).astype(np.float32),
            rng.normal(0, 2.5, size=(10, 333)).astype(np.float32)]
    ref = oracle.find_hits(imgs, 1.0)
    assert len(ref) > 100
    for cap in (1, 37, len(ref) - 1, len(ref), len(ref) + 5):
        got, n = run(pid, handle, imgs, 1.0, capacity=cap)
        assert n == len(ref)
        k = min(cap, len(ref))
        assert np.array_equal(got[:k], ref[:k]), cap
        assert (got[k:] == -7).all(), cap            # rows past the hits are untouched
    # capacity 0: only the count is written
    n_found = torch.full((1,), -1, dtype=torch.int64, device=DEV)
    pid.pointid_find_hits(handle, [torch.from_numpy(a).to(DEV) for a in imgs], 1.0, capacity=0,
                          hits_out=torch.empty((0, 3), dtype=torch.int32, device=DEV),
                          n_found=n_found)
    assert int(n_found.item()) == len(ref)
    # nothing above the threshold
    got, n = run(pid, handle, imgs, 1e9, capacity=8)
    assert n == 0 and (got == -7).all()


def test_special_thresholds(pid, handle):
    rng = np.random.default_rng(15)
    imgs = [rng.integers(-3, 4, size=(6, 300)).astype(np.float32)]
    imgs[0][2, 100:110] = np.inf
    imgs[0][3, :] = -np.inf
    for thr in (-np.inf, np.float32(-3.0), np.float32(3.0)):
        check_exact(pid, handle, imgs, float(thr))
    got, n = run(pid, handle, imgs, float("nan"), capacity=8)
    assert n == 0 and len(oracle.find_hits(imgs, float("nan"))) == 0


def test_found_hits_classify_like_given_hits(pid, handle):
    # found hits feed pointid_classify_planes directly; the scores equal those
    # of the same hits handed in from the host, bit for bit
    rng = np.random.default_rng(16)
    planes, _ = synth.config3()
    imgs = [p.image for p in planes[:3]]
    thr = 40.0
    ref = oracle.find_hits(imgs, thr)
    dimgs = [torch.from_numpy(a).to(DEV) for a in imgs]
    out, n_found = pid.pointid_find_hits(handle, dimgs, thr, capacity=len(ref) + 100)
    n = int(n_found.item())
    assert n == len(ref)
    s_found = pid.pointid_classify_planes(handle, dimgs, out[:n])
    s_given = pid.pointid_classify_planes(handle, dimgs, torch.from_numpy(ref).to(DEV))
    torch.cuda.synchronize()
    assert torch.equal(s_found, s_given)
    idx = rng.choice(n, size=min(n, 256), replace=False)
    P = oracle.gather_patches_planes(imgs, ref[idx])
    want = oracle.forward(P, synth.he_normal_weights())
    assert np.abs(s_found.cpu().numpy()[idx] - want).max() <= 2e-2
