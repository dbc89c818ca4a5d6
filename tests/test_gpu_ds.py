"""GPU parity of patches with D ticks per column (pointid_downsample,
pointid_classify_planes_ds) against the CPU oracle.

A column holds the charge of its D ticks: the library sums the fp32 samples in
fp64 in tick order and rounds once, the oracle does the same in numpy, so on
ADC-like data (sums exact in fp64) the binned planes agree value for value.

Score bars.  The plain path's bars (fp32 1e-4 and fp16 2e-2 against the
oracle, bf16 2e-3 against the oracle's bf16-rounded network) are stated for
inputs on the scale of one sample.  A column sums D samples, so the inputs grow
by up to a factor D; the network is affine between ReLUs, so every
pre-activation's data part, and with it the rounding error of each fp32 sum
(and of each 16-bit operand, a relative error), grows by the same factor, and
so do the logit errors, which bound the score errors.  The bars here are
therefore the plain path's times D; the near-tie allowance of the argmax
criterion scales with them.  (Measured on the plane at D = 4 and 6: the fp16
network's own 16-bit rounding moves the scores by 0.014-0.015, inside even the
unscaled bar.)  The binning and the column arithmetic are bit-exact and have no
tolerance at all.
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
TOL = {"fp32": 1e-4, "fp16": 2e-2, "bf16": 2e-3}


def say(*a):
    print(*a, flush=True, file=sys.stderr)


def t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


@pytest.fixture(scope="module")
def pid():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2009_04509_amd import binding
    return binding


@functools.lru_cache(maxsize=None)
def weights():
    return synth.he_normal_weights()


@pytest.fixture(scope="module")
def handles(pid):
    hs = {p: pid.pointid_create(weights(), p, 0) for p in ("fp32", "fp16", "bf16")}
    yield hs
    for h in hs.values():
        h.close()


def test_downsample_matches_oracle(pid):
    rng = np.random.default_rng(41)
    p2 = synth.config2()
    planes = [p2.image, rng.normal(0, 2.5, size=(37, 5999)).astype(np.float32),
              rng.integers(-9, 9, size=(5, 7)).astype(np.float32)]
    say("downsample planes")
    for img in planes:
        for D in (1, 2, 3, 4, 6, 7, 256, img.shape[1], img.shape[1] + 5):
            got = pid.pointid_downsample(t(img), D).cpu().numpy()
            ref = oracle.downsample_plane(img, D)
            assert got.shape == ref.shape and np.array_equal(got, ref), (img.shape, D)


def test_downsample_unaligned_base(pid):
    rng = np.random.default_rng(42)
    W, T = 13, 301
    big = t(rng.normal(0, 2.5, size=W * T + 3).astype(np.float32))
    for off in (1, 2, 3):
        view = big[off:off + W * T].view(W, T)
        got = pid.pointid_downsample(view, 4).cpu().numpy()
        assert np.array_equal(got, oracle.downsample_plane(view.cpu().numpy(), 4)), off


def _compare(got, full, emu, prec, what, D):
    got = np.asarray(got, np.float64)
    ref = emu if prec == "bf16" else full
    err = np.abs(got - ref).max()
    am_g, am_f = got[:, :3].argmax(1), full[:, :3].argmax(1)
    srt = np.sort(full[:, :3], axis=1)
    gap = srt[:, 2] - srt[:, 1]
    agree = float(np.mean(am_g == am_f))
    tol = D * TOL[prec]
    say(f"[{what} {prec}] n={len(got)} max|d|={err:.3g} (bar {tol:.3g}) argmax agree={agree:.5f}")
    assert err <= tol, f"{what} {prec}: {err}"
    # bf16: a flip needs the bf16-rounded network's own gap to be a near tie
    # (the emulated network is what the path computes, up to fp32 order)
    if prec == "bf16":
        srt_e = np.sort(emu[:, :3], axis=1)
        gap, am_f = srt_e[:, 2] - srt_e[:, 1], emu[:, :3].argmax(1)
    tie = 2 * tol
    assert not ((am_g != am_f) & (gap >= tie)).any()
    if len(got) >= 1000:
        assert agree >= 0.999


@pytest.mark.parametrize("D", [4, 6])
def test_classify_planes_ds_plane(pid, handles, D):
    p2 = synth.config2()
    h3 = np.c_[np.zeros(len(p2.hits), np.int32), p2.hits].astype(np.int32)
    P = oracle.gather_patches_planes_ds([p2.image], h3, D)
    full = oracle.classify_patches(P, weights()).astype(np.float64)
    emu = oracle.classify_16bit_emulated(P, weights(), "bf16").astype(np.float64)
    for prec, h in handles.items():
        say(f"classify_planes_ds plane D={D} {prec}")
        got = pid.pointid_classify_planes_ds(h, [t(p2.image)], t(h3), D).cpu().numpy()
        _compare(got, full, emu, prec, f"plane D={D}", D)


def test_classify_planes_ds_fp8(pid):
    """The 8-bit path on D-tick columns: against the oracle's e4m3 network on
    the same binned patches at D times its bar (5e-2, tests/test_gpu_fp8.py),
    and D = 1 gives the bits of pointid_classify_planes."""
    p2 = synth.config2()
    h3 = np.c_[np.zeros(len(p2.hits), np.int32), p2.hits].astype(np.int32)
    h = pid.pointid_create(weights(), "fp8", 0)
    for D in (1, 4):
        P = oracle.gather_patches_planes_ds([p2.image], h3, D)
        emu = oracle.classify_fp8_emulated(P, weights()).astype(np.float64)
        say(f"classify_planes_ds plane D={D} fp8")
        got = pid.pointid_classify_planes_ds(h, [t(p2.image)], t(h3), D).cpu().numpy().astype(np.float64)
        err = np.abs(got - emu)
        say(f"[plane D={D} fp8] n={len(got)} max|d|={err.max():.3g} mean|d|={err.mean():.3g}")
        assert err.max() <= D * 5e-2 and err.mean() <= 1e-3
        srt = np.sort(emu[:, :3], axis=1)
        flips = (got[:, :3].argmax(1) != emu[:, :3].argmax(1)) & (srt[:, 2] - srt[:, 1] >= 2 * D * 5e-2)
        assert not flips.any()
        if D == 1:
            plain = pid.pointid_classify_planes(h, [t(p2.image)], t(h3)).cpu().numpy()
            assert np.array_equal(plain.view(np.uint32), got.astype(np.float32).view(np.uint32))
    h.close()


def test_ds_one_tick_is_classify_planes(pid, handles):
    planes, h3 = synth.config3()
    imgs = [t(p.image) for p in planes[:4]]
    sel = h3[h3[:, 0] < 4][:5000]
    for prec, h in handles.items():
        a = pid.pointid_classify_planes_ds(h, imgs, t(sel), 1)
        b = pid.pointid_classify_planes(h, imgs, t(sel))
        torch.cuda.synchronize()
        assert torch.equal(a, b), prec


def test_ds_columns_from_floor_division(pid, handles):
    # the in-kernel column floor(tick / D) against binned planes handed in with
    # host-divided ticks: same bits; ticks far outside, negative ticks and
    # out-of-range planes included
    rng = np.random.default_rng(43)
    planes, _ = synth.config3()
    imgs_np = [p.image for p in planes[:3]]
    imgs = [t(a) for a in imgs_np]
    n = 3000
    h3 = np.c_[rng.integers(-1, 4, n), rng.integers(-30, 830, n),
               rng.integers(-200, 6200, n)].astype(np.int32)
    D = 5
    binned = [pid.pointid_downsample(x, D) for x in imgs]
    cols = oracle.hits_to_columns(h3, D).astype(np.int32)
    for prec, h in handles.items():
        a = pid.pointid_classify_planes_ds(h, imgs, t(h3), D)
        b = pid.pointid_classify_planes(h, binned, t(cols))
        torch.cuda.synchronize()
        assert torch.equal(a, b), prec
    got = pid.pointid_classify_planes_ds(handles["fp32"], imgs, t(h3), D).cpu().numpy()
    idx = np.random.default_rng(44).choice(n, 512, replace=False)
    P = oracle.gather_patches_planes_ds(imgs_np, h3[idx], D)
    full = oracle.classify_patches(P, weights()).astype(np.float64)
    _compare(got[idx], full, full, "fp32", "edges D=5", D)


def test_ds_event_sampled(pid, handles):
    planes, h3 = synth.config3()
    imgs_np = [p.image for p in planes]
    imgs = [t(a) for a in imgs_np]
    D = 4
    idx = np.sort(np.random.default_rng(45).choice(len(h3), 1024, replace=False))
    P = oracle.gather_patches_planes_ds(imgs_np, h3[idx], D)
    full = oracle.classify_patches(P, weights()).astype(np.float64)
    emu = oracle.classify_16bit_emulated(P, weights(), "bf16").astype(np.float64)
    for prec in ("fp16", "bf16"):
        say(f"classify_planes_ds event D={D} {prec} (50k hits)")
        got = pid.pointid_classify_planes_ds(handles[prec], imgs, t(h3), D).cpu().numpy()
        _compare(got[idx], full, emu, prec, "event sampled D=4", D)
