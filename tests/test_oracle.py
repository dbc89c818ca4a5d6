"""Pins for the CPU oracle: facts fixed by the paper or by mathematics.

Each test checks the oracle against something other than itself: the paper's
architecture numbers, hand-computed patch coordinates, hand-derived closed
forms (tests/golden), brute-force loops, torch's own conv2d/linear in float64,
torch's bfloat16 rounding, and invariances of a per-hit computation.
"""

import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _zero_model():
    return {k: np.zeros(s, np.float32) for k, s in synth.WEIGHT_SHAPES.items()}


# ---------------------------------------------------------------- architecture

def test_architecture_matches_paper():
    g = _golden("paper_architecture.json")
    assert oracle.PATCH == g["patch_side"]
    assert oracle.NCH == g["filters"] and oracle.KS == g["filter_side"]
    assert oracle.FM == g["map_side"] == g["patch_side"] - g["filter_side"] + 1
    assert oracle.FC1_OUT == g["fc1_neurons"] and oracle.FC2_OUT == g["fc2_neurons"]
    assert oracle.NCLS == g["softmax_outputs"]
    # the parameter count fixes biases on all six layers and an unpadded conv
    conv = g["filters"] * (g["filter_side"] ** 2 + 1)
    fc1 = oracle.FC1_IN * g["fc1_neurons"] + g["fc1_neurons"]
    fc2 = g["fc1_neurons"] * g["fc2_neurons"] + g["fc2_neurons"]
    cls = g["fc2_neurons"] * g["softmax_outputs"] + g["softmax_outputs"]
    mic = g["fc2_neurons"] * g["sigmoid_outputs"] + g["sigmoid_outputs"]
    assert conv + fc1 + fc2 + cls + mic == g["trainable_parameters"] == 11_900_420
    assert synth.n_parameters() == g["trainable_parameters"]
    w = synth.he_normal_weights()
    assert sum(v.size for v in w.values()) == g["trainable_parameters"]


def test_patch_volume_matches_paper():
    g = _golden("paper_architecture.json")
    bytes_per_patch = g["patch_side"] ** 2 * g["bits_per_pixel"] // 8
    assert bytes_per_patch == 9216
    gbit = g["patches_per_event"] * bytes_per_patch * 8 / 1e9
    assert abs(gbit - g["gigabits_per_event"]) < 0.05
    p = oracle.gather_patches(np.zeros((8, 8), np.float32), [[0, 0]])
    assert p.dtype == np.float32 and p[0].nbytes == bytes_per_patch


# ---------------------------------------------------------------- patch gather

def test_patch_coordinates_centre():
    img = synth.coord_image(128, 512)
    P = oracle.gather_patches(img, [[64, 256]])[0]
    r = np.arange(48)[:, None]
    c = np.arange(48)[None, :]
    expect = 1 + 1000 * (40 + r) + (232 + c)
    assert np.array_equal(P, expect.astype(np.float32))
    assert P[24, 24] == 1 + 1000 * 64 + 256      # the hit sits at (24, 24)


def test_patch_corners_zero_padded():
    W, T = 128, 512
    img = synth.coord_image(W, T)
    P = oracle.gather_patches(img, [[0, 0], [W - 1, T - 1]])
    r = np.arange(48)[:, None]
    c = np.arange(48)[None, :]
    lo = np.where((r >= 24) & (c >= 24), 1 + 1000 * (r - 24) + (c - 24), 0)
    assert np.array_equal(P[0], lo.astype(np.float32))
    hi = np.where((r <= 24) & (c <= 24),
                  1 + 1000 * (W - 1 - 24 + r) + (T - 1 - 24 + c), 0)
    assert np.array_equal(P[1], hi.astype(np.float32))


def test_patch_outside_and_off_by_one():
    W, T = 64, 100
    img = synth.coord_image(W, T)
    hits = [[-100, 50], [W + 24, 50], [W + 23, 50], [30, -23], [30, -24], [30, T + 23]]
    P = oracle.gather_patches(img, hits)
    assert not P[0].any()
    assert not P[1].any()                        # centre 24 past the last wire
    assert P[2][0].all() and not P[2][1:].any()  # only row 0 = wire W-1 inside
    assert np.array_equal(P[2][0], img[W - 1, 50 - 24:50 + 24])
    assert P[3][:, 47].all() and not P[3][:, :47].any()   # only column 47 = tick 0
    assert not P[4].any()
    assert P[5][:, 0].all() and not P[5][:, 1:].any()


def test_multiplane_gather():
    a = synth.coord_image(30, 70)
    b = synth.coord_image(50, 60) + 7
    hits3 = np.array([[1, 5, 5], [0, 29, 69], [2, 3, 3], [-1, 3, 3], [1, 49, 0]])
    P = oracle.gather_patches_planes([a, b], hits3)
    assert np.array_equal(P[0], oracle.gather_patches(b, [[5, 5]])[0])
    assert np.array_equal(P[1], oracle.gather_patches(a, [[29, 69]])[0])
    assert not P[2].any() and not P[3].any()
    assert np.array_equal(P[4], oracle.gather_patches(b, [[49, 0]])[0])


def test_bf16_rne_matches_torch():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(100000) * 10 ** rng.uniform(-6, 6, 100000)).astype(np.float32)
    # exact ties with both parities of the kept bit, and values just off a tie
    base = rng.integers(0x3F800000 >> 16, 0x47000000 >> 16, 2000).astype(np.uint32) << 16
    ties = np.concatenate([base | 0x8000, base | 0x7FFF, base | 0x8001,
                           (base | 0x10000) | 0x8000]).view(np.float32)
    x = np.concatenate([x, ties, -ties, np.float32([0.0, -0.0, 1.0, 65504.0])])
    ours = oracle.to_bf16_rne(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(ours.view(np.uint32), ref.view(np.uint32))
    assert np.array_equal(oracle.bf16_bits(x),
                          (ref.view(np.uint32) >> 16).astype(np.uint16))


def test_fp16_rne_matches_torch():
    rng = np.random.default_rng(10)
    x = (rng.standard_normal(100000) * 10 ** rng.uniform(-9, 4.8, 100000)).astype(np.float32)
    x = np.concatenate([x, np.float32([0.0, -0.0, 1.0, 65504.0, 6.1e-5, 5.96e-8, 2.9e-8, 3e-8])])
    ref = torch.from_numpy(x).to(torch.float16)
    assert np.array_equal(oracle.fp16_bits(x), ref.view(torch.int16).numpy().view(np.uint16))
    assert np.array_equal(oracle.to_fp16_rne(x), ref.to(torch.float32).numpy())


# ---------------------------------------------------------------- convolution

def _conv_bruteforce(P, K, b):
    n = P.shape[0]
    nk = K.shape[0]
    out = np.zeros((n, 44, 44, nk))
    for i in range(n):
        for k in range(nk):
            for y in range(44):
                for x in range(44):
                    s = float(b[k])
                    for u in range(5):
                        for v in range(5):
                            s += float(K[k, u, v]) * float(P[i, y + u, x + v])
                    out[i, y, x, k] = s if s > 0 else 0.0
    return out


def test_conv_matches_bruteforce_loops():
    rng = np.random.default_rng(1)
    P = rng.standard_normal((2, 48, 48)).astype(np.float32) * 3
    K = rng.standard_normal((3, 5, 5)).astype(np.float32)
    b = rng.uniform(-1, 1, 3).astype(np.float32)
    got = oracle.conv_relu(P, np.concatenate([K, np.zeros((45, 5, 5), np.float32)]),
                           np.concatenate([b, np.zeros(45, np.float32)]))[..., :3]
    ref = _conv_bruteforce(P, K, b)
    np.testing.assert_allclose(got, ref, rtol=1e-13, atol=1e-12)


def test_conv_matches_torch_conv2d_fp64():
    rng = np.random.default_rng(2)
    P = rng.standard_normal((5, 48, 48)).astype(np.float32) * 4
    w = synth.he_normal_weights()
    got = oracle.conv_relu(P, w["conv_w"], w["conv_b"])
    t = torch.nn.functional.conv2d(torch.from_numpy(P).double()[:, None],
                                   torch.from_numpy(w["conv_w"]).double()[:, None],
                                   torch.from_numpy(w["conv_b"]).double())
    ref = torch.relu(t).permute(0, 2, 3, 1).numpy()       # NCHW -> NHWC
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_conv_delta_kernel_is_shifted_crop():
    rng = np.random.default_rng(3)
    P = rng.standard_normal((3, 48, 48)).astype(np.float32)
    for (k, u, v) in [(0, 0, 0), (5, 2, 3), (47, 4, 4), (11, 0, 4)]:
        K = np.zeros((48, 5, 5), np.float32)
        K[k, u, v] = 1.0
        A = oracle.conv_relu(P, K, np.zeros(48, np.float32))
        assert np.array_equal(A[..., k], np.maximum(P[:, u:u + 44, v:v + 44], 0))
        others = np.delete(A, k, axis=3)
        assert not others.any()


def test_conv_delta_image_gives_unflipped_kernel():
    K = synth.he_normal_weights()["conv_w"]
    P = np.zeros((1, 48, 48), np.float32)
    r0, c0 = 20, 30
    P[0, r0, c0] = 1.0
    A = oracle.conv_relu(P, K, np.zeros(48, np.float32))[0]
    for u in range(5):
        for v in range(5):
            np.testing.assert_array_equal(A[r0 - u, c0 - v, :], np.maximum(K[:, u, v], 0))


def test_flatten_is_channels_last():
    A = np.arange(2 * 44 * 44 * 48, dtype=np.float64).reshape(2, 44, 44, 48)
    a = oracle.flatten_hwc(A)
    for (y, x, k) in [(0, 0, 0), (3, 7, 11), (43, 43, 47), (10, 0, 5)]:
        assert a[1, (y * 44 + x) * 48 + k] == A[1, y, x, k]


# ---------------------------------------------------------------- dense + heads

def test_dense_selector_closed_form():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((6, 10))
    W = np.zeros((10, 4))
    W[3, 0] = 1.0
    W[7, 2] = -2.0
    b = np.array([0.5, -0.25, 0.0, 1.0])
    got = oracle.dense_relu(x, W, b)
    np.testing.assert_array_equal(got[:, 0], np.maximum(x[:, 3] + 0.5, 0))
    np.testing.assert_array_equal(got[:, 1], np.zeros(6))
    np.testing.assert_array_equal(got[:, 2], np.maximum(-2.0 * x[:, 7], 0))
    np.testing.assert_array_equal(got[:, 3], np.ones(6))


def test_zero_weight_model_closed_form():
    g = _golden("closed_forms.json")["zero_weights"]
    w = _zero_model()
    w["cls_b"] = np.float32([0.0, math.log(2), math.log(3)])
    w["mic_b"] = np.float32([math.log(3)])
    rng = np.random.default_rng(5)
    P = rng.standard_normal((4, 48, 48)).astype(np.float32) * 10
    s = oracle.classify_patches(P, w)
    expect = [eval(e, {}, {}) for e in g["expected"]]        # "1/6", ...
    # cls_b/mic_b are float32 roundings of ln 2, ln 3: 1e-7 relative slack
    np.testing.assert_allclose(s, np.tile(expect, (4, 1)), rtol=2e-7, atol=0)


def test_softmax_and_sigmoid_properties():
    rng = np.random.default_rng(6)
    z = rng.standard_normal((1000, 3)) * 30
    s = oracle.softmax(z)
    assert np.all(np.abs(s.sum(1) - 1) <= 1e-12)
    assert np.all(np.argmax(s, 1) == np.argmax(z, 1))
    q = np.concatenate([rng.standard_normal(1000) * 20, [-1000.0, 1000.0, 0.0]])
    m = oracle.sigmoid(q)
    assert np.all((m >= 0) & (m <= 1)) and np.all(np.isfinite(m))
    assert m[-1] == 0.5 and m[-2] == 1.0 and m[-3] == 0.0
    inner = np.abs(q) < 30
    assert np.all((m[inner] > 0) & (m[inner] < 1))
    np.testing.assert_allclose(oracle.sigmoid(q[:1000]), 1 / (1 + np.exp(-q[:1000])), rtol=1e-15)


def test_single_pixel_chains_closed_form():
    g = _golden("closed_forms.json")["single_pixel_chains"]
    W, T = g["plane"]
    e = math.e
    hit_scores = [e / (e + 1 + 1 / e), 1 / (e + 1 + 1 / e), (1 / e) / (e + 1 + 1 / e), e / (1 + e)]
    miss_scores = [1 / 3, 1 / 3, 1 / 3, 0.5]
    for case in g["cases"]:
        img = np.zeros((W, T), np.float32)
        img[case["pixel"][0], case["pixel"][1]] = 1.0
        w = _zero_model()
        k, u, v = case["tap"]
        w["conv_w"][k, u, v] = 1.0
        fy, fx, fk = case["fc1_yxk"]
        w["fc1_w"][(fy * 44 + fx) * 48 + fk, 0] = 1.0
        w["fc2_w"][0, 0] = 1.0
        w["cls_w"][0] = [1.0, 0.0, -1.0]
        w["mic_w"][0] = 1.0
        s = oracle.classify(img, np.array([case["hit"]]), w)[0]
        expect = hit_scores if case["hit_expected"] else miss_scores
        np.testing.assert_allclose(s, expect, rtol=1e-7, atol=0, err_msg=str(case))


def test_full_network_matches_torch_fp64():
    w = synth.he_normal_weights()
    P = synth.config4_patches(6, seed=77)
    got = oracle.forward(P, w)
    d = {k: torch.from_numpy(v).double() for k, v in w.items()}
    x = torch.from_numpy(P).double()[:, None]
    A = torch.relu(torch.nn.functional.conv2d(x, d["conv_w"][:, None], d["conv_b"]))
    a = A.permute(0, 2, 3, 1).reshape(6, -1)
    h1 = torch.relu(torch.nn.functional.linear(a, d["fc1_w"].T, d["fc1_b"]))
    h2 = torch.relu(torch.nn.functional.linear(h1, d["fc2_w"].T, d["fc2_b"]))
    s = torch.softmax(torch.nn.functional.linear(h2, d["cls_w"].T, d["cls_b"]), dim=1)
    m = torch.sigmoid(h2 @ d["mic_w"] + d["mic_b"])
    ref = torch.cat([s, m[:, None]], 1).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-13)


def test_scores_fp32_softmax_sum():
    p = synth.config1()
    w = synth.he_normal_weights()
    s = oracle.classify(p.image, p.hits[:64], w)
    assert s.dtype == np.float32 and s.shape == (64, 4)
    assert np.all(np.abs(s[:, :3].astype(np.float64).sum(1) - 1) <= 2 ** -22)
    assert np.all((s[:, 3] >= 0) & (s[:, 3] <= 1))


# ---------------------------------------------------------------- invariances

def test_permutation_duplicate_and_chunk_invariance():
    p = synth.config1()
    w = synth.he_normal_weights()
    hits = p.hits[:40]
    base = oracle.classify(p.image, hits, w)
    perm = np.random.default_rng(8).permutation(len(hits))
    assert np.array_equal(oracle.classify(p.image, hits[perm], w), base[perm])
    dup = np.concatenate([hits[:5], hits[:5]])
    sd = oracle.classify(p.image, dup, w)
    assert np.array_equal(sd[:5], sd[5:]) and np.array_equal(sd[:5], base[:5])
    assert np.array_equal(oracle.classify(p.image, hits, w, chunk=7), base)


def test_logits_give_the_softmax_and_their_magnitudes_are_logged():
    """The class logits the tie diagnostics use are the ones the softmax head
    turns into scores (paper section 2.2), and their magnitudes are printed:
    the fp32 path's 1e-4 score bound rests on |logit| staying moderate with
    these untrained weights (an fp32 error of about 1e-4 relative in FC1 moves
    a logit of size L by about 1e-4 L)."""
    p = synth.config2()
    w = synth.he_normal_weights()
    hits = p.hits[:48]
    P = oracle.gather_patches(p.image, hits)
    z = oracle.logits(P, w)
    s = oracle.classify_patches(P, w)
    zz = np.exp(z - z.max(axis=1, keepdims=True))
    soft = zz / zz.sum(axis=1, keepdims=True)
    assert np.abs(soft - s[:, :3]).max() < 1e-6
    a = np.abs(z)
    print(f"[oracle logits, config 2, 48 hits] max |z| = {a.max():.3g}, median {np.median(a):.3g}, "
          f"top-2 gap median {np.median(np.diff(np.sort(s[:, :3], axis=1)[:, 1:], axis=1)):.3g}")
    assert np.isfinite(z).all()


def test_planes_match_single_plane():
    a = synth.gen_plane(64, 300, 3, 1, 20, seed=11)
    b = synth.gen_plane(90, 200, 3, 1, 20, seed=12)
    w = synth.he_normal_weights()
    h3 = np.concatenate([np.c_[np.ones(len(b.hits), np.int32), b.hits],
                         np.c_[np.zeros(len(a.hits), np.int32), a.hits]])
    s = oracle.classify_planes([a.image, b.image], h3, w)
    assert np.array_equal(s[:len(b.hits)], oracle.classify(b.image, b.hits, w))
    assert np.array_equal(s[len(b.hits):], oracle.classify(a.image, a.hits, w))


def test_16bit_emulation_rounds_the_right_operands():
    """The 16-bit emulation equals the full network when every rounded operand
    is already representable, and moves away from it otherwise."""
    w = synth.he_normal_weights()
    P = synth.config4_patches(8, seed=9)
    for kind in ("bf16", "fp16"):
        q = oracle.quantize_16bit_model(w, kind)
        # representable patch and weights: only the conv output rounding remains
        Pq = oracle.round16(P, kind)
        A = oracle.conv_relu(Pq, q["conv_w"], q["conv_b"])
        Aq = oracle.round16(A.astype(np.float32), kind).astype(np.float64)
        h1 = oracle.dense_relu(oracle.flatten_hwc(Aq), q["fc1_w"], q["fc1_b"])
        h2 = oracle.dense_relu(h1, q["fc2_w"], q["fc2_b"])
        np.testing.assert_array_equal(oracle.heads(h2, q), oracle.forward_16bit_emulated(P, w, kind))
        full = oracle.forward(P, w)
        d = np.abs(full - oracle.forward_16bit_emulated(P, w, kind)).max()
        assert 0 < d < 2e-2


def _rne(x, bits):
    """A Fraction rounded to `bits` significant bits, ties to even (normal range)."""
    if x == 0:
        return Fraction(0)
    sign, x = (-1 if x < 0 else 1), abs(x)
    e = 0
    while Fraction(2) ** e > x:
        e -= 1
    while Fraction(2) ** (e + 1) <= x:
        e += 1
    ulp = Fraction(2) ** (e - bits + 1)
    q = x / ulp
    n = math.floor(q)
    r = q - n
    if r > Fraction(1, 2) or (r == Fraction(1, 2) and n % 2 == 1):
        n += 1
    return sign * n * ulp


def _chain_scores(h):
    """(softmax of (h, 0, -h), sigmoid of h) written out."""
    e, f = math.exp(h), math.exp(-h)
    return np.array([e / (e + 1 + f), 1 / (e + 1 + f), f / (e + 1 + f), 1 / (1 + f)])


def test_16bit_emulation_closed_form():
    """oracle.forward_16bit_emulated against exact closed forms of a
    single-pixel chain (tests/golden/closed_forms_16bit.json): the chain's steps
    are checked in exact rational arithmetic, the oracle must reproduce the
    resulting scores, and every listed mistake — one of the four rounding
    points dropped, or the FC1 output, the FC2 filter or the conv bias rounded
    too — moves the scores by far more than the tolerance."""
    g = _golden("closed_forms_16bit.json")
    geo = g["geometry"]
    W, T = geo["plane"]
    ch, u, v = geo["tap"]
    for case in g["cases"]:
        kind, bits = case["kind"], case["bits"]
        vals = {k: Fraction(x) for k, x in case["inputs"].items()}
        for name, op, args, value in case["chain"]:
            a = [vals[x] for x in args.split()]
            got = {"round": lambda: _rne(a[0], bits), "round32": lambda: _rne(a[0], 24),
                   "mul": lambda: a[0] * a[1], "add": lambda: a[0] + a[1]}[op]()
            assert got == Fraction(value), (kind, name)
            vals[name] = got
        h2 = Fraction(case["h2"])
        assert vals["h2"] == h2
        img = np.zeros((W, T), np.float32)
        img[tuple(geo["pixel"])] = np.float32(float(vals["a"]))
        w = _zero_model()
        w["conv_w"][ch, u, v] = float(vals["kappa"])
        w["conv_b"][ch] = float(vals["b0"])
        w["fc1_w"][geo["fc1_row"], geo["fc1_col"]] = float(vals["omega"])
        w["fc2_w"][geo["fc2"][0], geo["fc2"][1]] = float(vals["beta"])
        w["cls_w"][geo["fc2"][1]] = [1.0, 0.0, -1.0]
        w["mic_w"][geo["fc2"][1]] = 1.0
        for k in ("conv_w", "conv_b", "fc1_w", "fc2_w"):          # the inputs are float32 values
            assert np.all(w[k].astype(np.float64) == w[k])
        P = oracle.gather_patches(img, np.array([geo["hit"]]))
        got = oracle.forward_16bit_emulated(P, w, kind)[0]
        want = _chain_scores(float(h2))
        np.testing.assert_allclose(got, want, rtol=0, atol=1e-12, err_msg=kind)
        for mistake, mh in case["mutants_h2"].items():
            assert np.abs(_chain_scores(float(Fraction(mh))) - want).max() > 1e-6, (kind, mistake)


def _e4m3(x):
    """A Fraction rounded to OCP e4m3: 4 significant bits from 2^-6 up,
    multiples of 2^-9 below, ties to even, saturating at 448."""
    sign, a = (-1 if x < 0 else 1), abs(x)
    if a >= Fraction(1, 64):
        r = _rne(a, 4)
    else:
        q = a * 512
        n = math.floor(q)
        if q - n > Fraction(1, 2) or (q - n == Fraction(1, 2) and n % 2 == 1):
            n += 1
        r = Fraction(n, 512)
    return sign * min(r, Fraction(448))


def _exp448(x):
    """The largest integer k with |x| 2^k <= 448, by counting."""
    k = 0
    while abs(x) * Fraction(2) ** k > 448:
        k -= 1
    while abs(x) * Fraction(2) ** (k + 1) <= 448:
        k += 1
    return k


def test_fc1_e4m3_exponents():
    # the largest k with max |column| * 2^k <= 448, from the frexp rule,
    # against counting in exact arithmetic
    cols = [448.0, 448.00003, 224.0, 1.0, 77 / 16384, 0.875 * 2.0 ** -20, 0.8750001 * 2.0 ** -20, 3e5, 1e-30]
    w = np.zeros((5, len(cols) + 1), np.float64)
    for j, c in enumerate(cols):
        w[j % 5, j] = c if j % 2 else -c              # the sign does not matter
    k = oracle.fc1_e4m3_exponents(w)
    assert k[-1] == 0                                   # a column of zeros
    for j, c in enumerate(cols):
        assert k[j] == _exp448(Fraction(c)), (c, k[j])
    assert k[:4].tolist() == [0, -1, 1, 8]
    assert np.all(np.abs(w).max(axis=0)[:-1] * 2.0 ** k[:-1] <= 448)
    assert np.all(np.abs(w).max(axis=0)[:-1] * 2.0 ** (k[:-1] + 1) > 448)


def test_fp8_emulation_closed_form():
    """oracle.forward_fp8_emulated against exact closed forms of a single-pixel
    chain (tests/golden/closed_forms_fp8.json): the chain's steps are checked
    in exact rational arithmetic, the oracle must reproduce the resulting
    scores, and every listed mistake (the patch, conv filter, conv output or
    FC1 filter left unrounded, the FC1 column left unscaled, or fp16 rounding
    in place of e4m3) moves the scores by far more than the tolerance.  The
    conv pre-activation lies just below the e4m3 midpoint 5.25, so the fp16
    roundings of the patch and the filter decide which way it rounds."""
    g = _golden("closed_forms_fp8.json")
    geo = g["geometry"]
    W, T = geo["plane"]
    ch, u, v = geo["tap"]
    vals = {k: Fraction(x) for k, x in g["inputs"].items()}
    ops = {"round16": lambda a: _rne(a[0], 11), "round32": lambda a: _rne(a[0], 24),
           "e4m3": lambda a: _e4m3(a[0]), "exp448": lambda a: Fraction(_exp448(a[0])),
           "scale": lambda a: a[0] * Fraction(2) ** int(a[1]),
           "unscale": lambda a: a[0] * Fraction(2) ** -int(a[1]),
           "mul": lambda a: a[0] * a[1], "add": lambda a: a[0] + a[1]}
    for name, op, args, value in g["chain"]:
        got = ops[op]([vals[x] for x in args.split()])
        assert got == Fraction(value), name
        vals[name] = got
    h2 = Fraction(g["h2"])
    assert vals["h2"] == h2
    assert vals["A8"] != _rne(vals["pre32"], 11) and vals["k"] > 0
    img = np.zeros((W, T), np.float32)
    img[tuple(geo["pixel"])] = np.float32(float(vals["a"]))
    w = _zero_model()
    w["conv_w"][ch, u, v] = float(vals["kappa"])
    w["conv_b"][ch] = float(vals["b0"])
    w["fc1_w"][geo["fc1_row"], geo["fc1_col"]] = float(vals["omega"])
    w["fc2_w"][geo["fc2"][0], geo["fc2"][1]] = float(vals["beta"])
    w["cls_w"][geo["fc2"][1]] = [1.0, 0.0, -1.0]
    w["mic_w"][geo["fc2"][1]] = 1.0
    for k in ("conv_w", "conv_b", "fc1_w", "fc2_w"):          # the inputs are float32 values
        assert np.all(w[k].astype(np.float64) == w[k])
    assert oracle.fc1_e4m3_exponents(w["fc1_w"])[geo["fc1_col"]] == vals["k"]
    P = oracle.gather_patches(img, np.array([geo["hit"]]))
    got = oracle.forward_fp8_emulated(P, w)[0]
    want = _chain_scores(float(h2))
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)
    for mistake, mh in g["mutants_h2"].items():
        assert np.abs(_chain_scores(float(Fraction(mh))) - want).max() > 1e-3, mistake


def test_bf16_operands_alone_exceed_the_bf16_bar_on_adc_planes():
    """Why the 16-bit path the benchmark reports uses fp16: on raw-ADC plane
    hits (300 seeded hits of the 480 x 6000 plane) rounding the operands to
    bf16 already moves the oracle's own scores by more than the 2e-2 bf16 bar,
    while fp16 operands stay inside it; on the pre-cut N(0, 1) patches of the
    patch sweep bf16 operands stay inside it too."""
    w = synth.he_normal_weights()
    p2 = synth.config2()
    idx = np.random.default_rng(2).choice(len(p2.hits), 300, replace=False)
    P = oracle.gather_patches(p2.image, p2.hits[idx])
    full = oracle.classify_patches(P, w).astype(np.float64)
    d_bf16 = np.abs(oracle.classify_16bit_emulated(P, w, "bf16") - full).max()
    d_fp16 = np.abs(oracle.classify_16bit_emulated(P, w, "fp16") - full).max()
    assert d_bf16 > 2e-2 > d_fp16, (d_bf16, d_fp16)
    Q = synth.config4_patches(300, seed=3)
    fq = oracle.classify_patches(Q, w).astype(np.float64)
    assert np.abs(oracle.classify_16bit_emulated(Q, w, "bf16") - fq).max() < 2e-2


# ------------------------------------------------------------------ hit finding

def _hits_bruteforce(images, thr):
    """Pure-Python loops over every tick, straight from the definition."""
    out = []
    thr = float(np.float32(thr))
    for p, img in enumerate(images):
        W, T = img.shape
        for w in range(W):
            for t in range(T):
                x = float(img[w, t])
                before = float(img[w, t - 1]) if t > 0 else -np.inf
                after = float(img[w, t + 1]) if t + 1 < T else -np.inf
                if x > thr and x > before and x >= after:
                    out.append((p, w, t))
    return np.array(out, np.int32).reshape(-1, 3)


def test_hit_finding_worked_cases():
    cases = json.load(open(os.path.join(GOLDEN, "hit_finding.json")))["cases"]
    for c in cases:
        img = np.array([c["wave"]], np.float32)
        got = oracle.find_hits([img], c["threshold"])
        assert got[:, 2].tolist() == c["ticks"], c
        assert (got[:, :2] == 0).all()


def test_hit_finding_matches_bruteforce_with_ties():
    rng = np.random.default_rng(7)
    # small integers, so that equal neighbours (plateaus) and values equal to
    # the threshold are frequent
    imgs = [rng.integers(-3, 6, size=(5, 40)).astype(np.float32),
            rng.integers(0, 3, size=(3, 17)).astype(np.float32),
            rng.normal(0, 2.5, size=(4, 64)).astype(np.float32)]
    for thr in (-1.0, 0.0, 2.0, 3.5):
        got = oracle.find_hits(imgs, thr)
        ref = _hits_bruteforce(imgs, thr)
        assert np.array_equal(got, ref), thr


def test_hit_finding_single_pulse_and_order():
    # one Gaussian pulse per wire on a quiet waveform: exactly one hit, at the
    # peak; hits come out in plane, wire, tick order
    T = 200
    t = np.arange(T)
    a = np.stack([50 * np.exp(-0.5 * ((t - c) / 3.0) ** 2) for c in (20, 150, 77)]).astype(np.float32)
    b = np.zeros((2, T), np.float32)
    b[1, [5, 190]] = 9.0
    got = oracle.find_hits([a, b], 1.0)
    assert got.tolist() == [[0, 0, 20], [0, 1, 150], [0, 2, 77], [1, 1, 5], [1, 1, 190]]
    assert oracle.find_hits([b], 9.0).shape == (0, 3)       # equal to the threshold


# ------------------------------------------------------- columns of D ticks

def test_downsample_worked_cases():
    row = np.array([[1, 2, 3, 4, 5, 6, 7]], np.float32)
    # a column holds the charge of its interval; the ragged last column's
    # missing ticks count as 0
    assert oracle.downsample_plane(row, 3).tolist() == [[6, 15, 7]]
    assert oracle.downsample_plane(row, 7).tolist() == [[28]]
    assert oracle.downsample_plane(row, 10).tolist() == [[28]]
    assert oracle.downsample_plane(row, 2).tolist() == [[3, 7, 11, 7]]
    assert np.array_equal(oracle.downsample_plane(row, 1), row)         # one tick per column
    with pytest.raises(ValueError):
        oracle.downsample_plane(row, 0)


def test_downsample_one_tick_is_the_plain_gather():
    rng = np.random.default_rng(21)
    imgs = [rng.normal(0, 2.5, size=(60, 300)).astype(np.float32),
            rng.normal(0, 2.5, size=(30, 77)).astype(np.float32)]
    hits = np.c_[rng.integers(0, 2, 200), rng.integers(-30, 90, 200), rng.integers(-40, 340, 200)]
    assert np.array_equal(oracle.gather_patches_planes_ds(imgs, hits, 1),
                          oracle.gather_patches_planes(imgs, hits))


def test_downsample_coordinate_image_closed_form():
    # I[w][t] = 1 + 1000 w + t: a full column j of D ticks sums to
    # D (1 + 1000 w + D j) + D (D - 1) / 2, exactly
    W, T, D = 100, 500, 4
    img = synth.coord_image(W, T)
    ds = oracle.downsample_plane(img, D)
    assert ds.shape == (W, 125)
    w, j = np.meshgrid(np.arange(W), np.arange(125), indexing="ij")
    assert np.array_equal(ds, (D * (1 + 1000 * w + D * j) + D * (D - 1) // 2).astype(np.float32))
    # hit (plane 0, wire 50, tick 203) -> column 50; patch (r, c) is binned
    # pixel (26 + r, 26 + c), all inside the plane
    P = oracle.gather_patches_planes_ds([img], [[0, 50, 203]], D)[0]
    r, c = np.meshgrid(np.arange(48), np.arange(48), indexing="ij")
    want = D * (1 + 1000 * (26 + r) + D * (26 + c)) + 6
    assert np.array_equal(P, want.astype(np.float32))
    # ticks 200..203 all give column 50; tick 204 gives column 51
    for t in (200, 201, 202):
        assert np.array_equal(oracle.gather_patches_planes_ds([img], [[0, 50, t]], D)[0], P)
    assert not np.array_equal(oracle.gather_patches_planes_ds([img], [[0, 50, 204]], D)[0], P)


def test_downsample_negative_tick_and_edges():
    # floor division: tick -5 with D = 4 is column -2, so patch column c holds
    # binned column c - 26 and columns c < 26 are zero
    W, T, D = 10, 30, 4
    img = synth.coord_image(W, T)
    ds = oracle.downsample_plane(img, D)                     # 8 columns, the last of 2 ticks
    assert ds[3, 7] == (1 + 3000 + 28) + (1 + 3000 + 29)
    P = oracle.gather_patches_planes_ds([img], [[0, 3, -5]], D)[0]
    assert (P[:, :26] == 0).all()
    assert P[24, 26] == ds[3, 0] and P[24, 33] == ds[3, 7]
    assert (P[:, 34:] == 0).all()                            # past the 8 columns
    assert (P[:21, :] == 0).all() and (P[31:, :] == 0).all()  # wires outside 0..9


def test_downsample_bruteforce_and_charge_conservation():
    rng = np.random.default_rng(22)
    imgs = [rng.normal(0, 2.5, size=(9, 61)).astype(np.float32),
            rng.normal(5, 2.5, size=(4, 13)).astype(np.float32)]
    D = 6
    hits = np.c_[rng.integers(-1, 3, 40), rng.integers(-3, 12, 40), rng.integers(-20, 80, 40)]
    got = oracle.gather_patches_planes_ds(imgs, hits, D)
    for i, (p, w, t) in enumerate(hits):
        for r in range(48):
            for c in range(48):
                v = 0.0
                if 0 <= p < len(imgs):
                    img = imgs[p]
                    ww = w - 24 + r
                    col = t // D - 24 + c                    # Python // is floor division
                    if 0 <= ww < img.shape[0] and col >= 0:
                        ticks = [tt for tt in range(col * D, col * D + D) if tt < img.shape[1]]
                        v = float(np.float32(sum(float(img[ww, tt]) for tt in ticks)))
                assert got[i, r, c] == np.float32(v), (i, r, c)
    for img in imgs:                                         # the binning keeps the charge
        assert abs(oracle.downsample_plane(img, D).astype(np.float64).sum()
                   - img.astype(np.float64).sum()) < 1e-4


# --------------------------------------------------- fp8 precision study (MX)

def test_e4m3_rounding_matches_the_format():
    # the OCP e4m3 grid: 3 mantissa bits, bias 7, max 448, min normal 2^-6,
    # subnormal step 2^-9; nearest even on ties; saturation past 448
    f = oracle.to_e4m3_rne
    assert f([448.0, 480.0, 1e6, -1e6]).tolist() == [448.0, 448.0, 448.0, -448.0]
    assert f([1.0, 1.125, 1.0625, 1.1875]).tolist() == [1.0, 1.125, 1.0, 1.25]   # ties to even
    assert f([2.0 ** -6, 2.0 ** -9, 3 * 2.0 ** -10, 2.0 ** -11]).tolist() == \
        [2.0 ** -6, 2.0 ** -9, 2.0 ** -8, 0.0]
    assert f([240.0, 232.0, 17.0, 0.0]).tolist() == [240.0, 224.0, 16.0, 0.0]
    # every value of the format is a fixed point; there are 126 positive finite values
    vals = sorted({m * 2.0 ** (e - 3) for e in range(-6, 9) for m in range(8, 16)} |
                  {m * 2.0 ** -9 for m in range(1, 8)})
    vals = [v for v in vals if v <= 448]
    assert len(vals) == 126 and np.array_equal(f(vals), vals)
    # block scale: the largest magnitude lands in [256, 512) before rounding
    b = np.array([[3.0, -700.0, 0.001, 5.5]])
    X = 2.0 ** (np.floor(np.log2(700.0)) - 8)
    assert np.array_equal(oracle.mx_e4m3(b), oracle.to_e4m3_rne(b / X) * X)
    assert oracle.mx_e4m3(np.zeros((2, 32))).tolist() == np.zeros((2, 32)).tolist()


@pytest.mark.slow
def test_fp8_emulation_cost_on_event_hits():
    # what e4m3 FC1 operands cost on event patches with these (untrained)
    # weights: the scores move by more than the 2e-2 the 16-bit path is held
    # to on some hits, by about 5e-3 on average, and the class decision agrees
    planes, h3 = synth.config3()
    idx = np.random.default_rng(0).choice(len(h3), 120, replace=False)
    P = oracle.gather_patches_planes([p.image for p in planes], h3[idx])
    w = synth.he_normal_weights()
    full = oracle.forward(P, w)
    e8 = oracle.forward_fp8_emulated(P, w)
    d = np.abs(e8 - full)
    assert d.max() > 2e-2 and d.mean() < 1e-2, (d.max(), d.mean())
    assert (e8[:, :3].argmax(1) == full[:, :3].argmax(1)).mean() >= 0.99


@pytest.mark.slow
def test_mx_fp8_moves_scores_beyond_the_16bit_budget():
    # why the library has no fp8 path: on event patches with these (untrained)
    # weights, microscaled e4m3 FC1 operands move the scores by far more than
    # the 2e-2 the 16-bit path is held to, while fp16 operands stay inside it
    planes, h3 = synth.config3()
    idx = np.random.default_rng(0).choice(len(h3), 120, replace=False)
    P = oracle.gather_patches_planes([p.image for p in planes], h3[idx])
    w = synth.he_normal_weights()
    full = oracle.forward(P, w)
    d8 = np.abs(oracle.forward_mx_fp8_emulated(P, w) - full).max()
    d16 = np.abs(oracle.forward_16bit_emulated(P, w, "fp16") - full).max()
    assert d16 < 2e-2 < d8
