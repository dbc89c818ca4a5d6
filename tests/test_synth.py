"""The seeded input generators: reproducible, and shaped like the workloads."""

import numpy as np

import synth


def test_seeds_reproducible():
    a, b = synth.config1(), synth.config1()
    assert np.array_equal(a.image, b.image) and np.array_equal(a.hits, b.hits)
    c = synth.config1(seed=1234)
    assert not np.array_equal(a.image, c.image)
    w1, w2 = synth.he_normal_weights(), synth.he_normal_weights()
    for k in synth.WEIGHT_ORDER:
        assert np.array_equal(w1[k], w2[k])
    assert np.array_equal(synth.config4_patches(64), synth.config4_patches(64))


def test_config_shapes_and_hits_inside():
    p1 = synth.config1()
    assert p1.image.shape == (128, 512) and p1.image.dtype == np.float32
    assert p1.hits.shape == (128, 2) and p1.hits.dtype == np.int32
    p2 = synth.config2()
    assert p2.image.shape == (480, 6000) and p2.hits.shape == (3000, 2)
    for p in (p1, p2):
        assert p.hits[:, 0].min() >= 0 and p.hits[:, 0].max() < p.n_wires
        assert p.hits[:, 1].min() >= 0 and p.hits[:, 1].max() < p.n_ticks
        key = p.hits[:, 0].astype(np.int64) * p.n_ticks + p.hits[:, 1]
        assert len(np.unique(key)) == len(key)           # deduplicated


def test_noise_level_and_signal():
    p = synth.gen_plane(64, 4000, 0, 0, 0, seed=3)
    assert abs(float(p.image.std()) - 2.5) < 0.02       # paper §3.1: 2.5 ADC RMS
    p2 = synth.config2()
    vals = p2.image[p2.hits[:, 0], p2.hits[:, 1]]
    assert np.median(vals) > 10                          # hits sit on signal peaks


def test_weights_he_normal():
    w = synth.he_normal_weights()
    assert synth.n_parameters() == 11_900_420
    for name, fan in [("conv_w", 25), ("fc1_w", 92928), ("fc2_w", 128)]:
        std = float(np.std(w[name].astype(np.float64)))
        assert abs(std / np.sqrt(2.0 / fan) - 1) < 0.05
    for name in ("conv_b", "fc1_b", "fc2_b", "cls_b"):
        assert np.all(np.abs(w[name]) <= 0.1)
    z = synth.he_normal_weights(bias_scale=0.0)
    assert not z["fc1_b"].any() and np.array_equal(z["fc1_w"], w["fc1_w"])
    for k, s in synth.WEIGHT_SHAPES.items():
        assert w[k].shape == s and w[k].dtype == np.float32 and w[k].flags.c_contiguous


def test_config3_layout():
    planes, h3 = synth.config3()
    assert len(planes) == 18 and h3.shape == (50000, 3)
    assert [p.n_wires for p in planes] == list(synth.gen.CONFIG3_WIRES)
    counts = np.bincount(h3[:, 0], minlength=18)
    assert list(counts[:3]) == [3205, 3205, 1923] and counts[-1] == 1925
    for p, pl in enumerate(planes):
        sel = h3[h3[:, 0] == p]
        assert sel[:, 1].max() < pl.n_wires and sel[:, 2].max() < pl.n_ticks


def test_config5_requests():
    planes, reqs = synth.config5_requests(n_planes=2, n_streams=3, per_stream=4)
    assert len(reqs) == 3 and all(len(r) == 4 for r in reqs)
    for r in reqs:
        for p, h in r:
            assert 1000 <= len(h) <= 8000 and h.dtype == np.int32
            assert h[:, 0].max() < planes[p].n_wires
