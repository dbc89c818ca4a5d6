"""GPU: pointid_classify_planes_noalloc, the entry point that allocates
nothing (its scratch is the library's fixed device array), gives exactly the
bits of pointid_classify_planes on the same hits: two calls in a row, the
second with fewer hits than the first, for every precision, and sizes past
the array are refused."""

import sys

import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


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


@pytest.fixture(scope="module")
def event():
    planes, h3 = synth.config3()
    return [t(p.image) for p in planes], h3


@pytest.mark.parametrize("prec", ["fp16", "bf16", "fp32", "fp8"])
def test_noalloc_gives_the_bits_of_classify_planes(pid, event, prec):
    imgs, h3 = event
    rng = np.random.default_rng(7)
    first = h3[np.sort(rng.choice(len(h3), 8192, replace=False))].copy()     # the largest call
    first[::101, 0] = len(imgs)                                              # planes outside the table
    second = h3[np.sort(rng.choice(len(h3), 1531, replace=False))].copy()    # then a smaller one
    second[5::97, 1] = -40                                                   # wires outside the plane
    h = pid.pointid_create(synth.he_normal_weights(), prec, 0)
    for what, hh in (("first", first), ("second", second)):
        say(f"noalloc {prec} {what} call: {len(hh)} hits")
        hits = t(hh)
        got = pid.pointid_classify_planes_noalloc(h, imgs, hits)
        ref = pid.pointid_classify_planes(h, imgs, hits)
        torch.cuda.synchronize()
        assert torch.isfinite(got).all()
        assert torch.equal(got.view(torch.int32), ref.view(torch.int32)), f"{prec} {what} call"
    h.close()


def test_noalloc_refuses_more_than_its_scratch(pid, event):
    imgs, h3 = event
    h = pid.pointid_create(synth.he_normal_weights(), "fp16", 0)
    with pytest.raises(pid.PointIdError) as e:
        pid.pointid_classify_planes_noalloc(h, imgs, t(h3[:8193]))
    assert e.value.status == pid.POINTID_EINVAL and "8192" in str(e.value)
    empty = torch.zeros((0, 3), dtype=torch.int32, device=DEV)
    assert pid.pointid_classify_planes_noalloc(h, imgs, empty).shape == (0, 4)
    h.close()
