"""Seeded synthetic workloads standing in for ProtoDUNE-SP data (paper §2.1, §3.1).

The paper measures on Corsika cosmic-ray Monte Carlo of ProtoDUNE-SP: a 3 ms
readout sampled every 0.5 us (6000 ticks), white noise of 2.5 ADC RMS, and about
55,000 hits per event, each classified from a 48x48 wire-by-tick patch (paper
§2.1 and §3.1).  Neither that sample nor the trained network weights exist here,
so this module draws stand-ins with the same shapes, sizes and value
distributions:

* a plane image is float32 ``[n_wires][n_ticks]`` (tick fastest) of Gaussian
  noise (sigma 2.5 ADC) plus straight "cosmic" tracks with a Gaussian transverse
  profile and 2-D Gaussian "showers";
* hits are integer ``(wire, tick)`` pairs taken at signal peaks on the tracks
  and inside the showers;
* weights follow He-normal initialisation, N(0, 2/fan_in), for the network of
  paper §2.2 (conv 48@5x5, FC 128, FC 32, softmax 3 + sigmoid 1), with biases
  U(-0.1, 0.1) so that every bias add is exercised.

Every routine takes an explicit seed and uses numpy's PCG64 ``default_rng``;
the draw order is fixed so that a seed always gives identical bytes.
Nothing here evaluates the network.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

# Network shape, paper §2.2: 48x48 patch -> 48 maps of 44x44 (5x5, stride 1)
# -> FC 128 -> FC 32 -> {softmax 3, sigmoid 1}.
PATCH = 48
KSIZE = 5
NCH = 48
FMAP = PATCH - KSIZE + 1          # 44
FC1_IN = FMAP * FMAP * NCH        # 92928
FC1_OUT = 128
FC2_OUT = 32
NCLS = 3

WEIGHT_ORDER = ("conv_w", "conv_b", "fc1_w", "fc1_b", "fc2_w", "fc2_b",
                "cls_w", "cls_b", "mic_w", "mic_b")
WEIGHT_SHAPES = {
    "conv_w": (NCH, KSIZE, KSIZE),   # [k][u = wire offset][v = tick offset]
    "conv_b": (NCH,),
    "fc1_w": (FC1_IN, FC1_OUT),      # row (y*44 + x)*48 + k
    "fc1_b": (FC1_OUT,),
    "fc2_w": (FC1_OUT, FC2_OUT),
    "fc2_b": (FC2_OUT,),
    "cls_w": (FC2_OUT, NCLS),
    "cls_b": (NCLS,),
    "mic_w": (FC2_OUT,),
    "mic_b": (1,),
}
_FAN_IN = {"conv_w": KSIZE * KSIZE, "fc1_w": FC1_IN, "fc2_w": FC1_OUT,
           "cls_w": FC2_OUT, "mic_w": FC2_OUT}

WEIGHT_SEED = 4509


def n_parameters() -> int:
    """Number of trainable parameters implied by ``WEIGHT_SHAPES``."""
    return int(sum(int(np.prod(s)) for s in WEIGHT_SHAPES.values()))


def he_normal_weights(seed: int = WEIGHT_SEED, bias_scale: float = 0.1) -> dict:
    """He-normal weights N(0, 2/fan_in), untruncated; biases U(-b, b).

    Drawn in ``WEIGHT_ORDER`` from one PCG64 stream and stored as float32
    C-contiguous arrays in the layouts of ``WEIGHT_SHAPES``.  ``bias_scale=0``
    gives an all-zero-bias model (the bias draws are still consumed so the
    weights are unchanged).
    """
    rng = np.random.default_rng(seed)
    out = {}
    for name in WEIGHT_ORDER:
        shape = WEIGHT_SHAPES[name]
        if name.endswith("_w"):
            std = np.sqrt(2.0 / _FAN_IN[name])
            arr = rng.normal(0.0, std, size=shape)
        else:
            arr = rng.uniform(-0.1, 0.1, size=shape) * (bias_scale / 0.1)
        out[name] = np.ascontiguousarray(arr, dtype=np.float32)
    return out


@dataclass
class Plane:
    """One wire plane: float32 image [n_wires][n_ticks] and int32 hits [n][2]."""
    image: np.ndarray
    hits: np.ndarray

    @property
    def n_wires(self) -> int:
        return int(self.image.shape[0])

    @property
    def n_ticks(self) -> int:
        return int(self.image.shape[1])


def _render_track(img, rng, amp, w0, t0, w1, t1, width):
    """Add amp*exp(-d^2 / (2 width^2)) for every pixel within 3*width of the segment.

    Distances are in pixel units (one wire == one tick).  For each wire column the
    pixels that can lie within reach are bounded first, then masked exactly.
    """
    W, T = img.shape
    r = 3.0 * width
    wlo = max(0, int(np.ceil(min(w0, w1) - r)))
    whi = min(W - 1, int(np.floor(max(w0, w1) + r)))
    if whi < wlo:
        return
    wires = np.arange(wlo, whi + 1, dtype=np.float64)
    dw = w1 - w0
    if abs(dw) < 1e-9:
        s_lo = np.zeros_like(wires)
        s_hi = np.ones_like(wires)
    else:
        sa = (wires - r - w0) / dw
        sb = (wires + r - w0) / dw
        s_lo = np.clip(np.minimum(sa, sb), 0.0, 1.0)
        s_hi = np.clip(np.maximum(sa, sb), 0.0, 1.0)
    ta = t0 + s_lo * (t1 - t0)
    tb = t0 + s_hi * (t1 - t0)
    tlo = np.clip(np.ceil(np.minimum(ta, tb) - r), 0, T - 1).astype(np.int64)
    thi = np.clip(np.floor(np.maximum(ta, tb) + r), 0, T - 1).astype(np.int64)
    lens = np.maximum(thi - tlo + 1, 0)
    total = int(lens.sum())
    if total == 0:
        return
    ws = np.repeat(wires.astype(np.int64), lens)
    starts = np.repeat(np.cumsum(lens) - lens, lens)
    ts = np.repeat(tlo, lens) + (np.arange(total) - starts)
    # exact point-to-segment distance
    ab_w, ab_t = w1 - w0, t1 - t0
    ab2 = ab_w * ab_w + ab_t * ab_t
    pw = ws - w0
    pt = ts - t0
    if ab2 > 0:
        s = np.clip((pw * ab_w + pt * ab_t) / ab2, 0.0, 1.0)
    else:
        s = np.zeros(total)
    dw_ = pw - s * ab_w
    dt_ = pt - s * ab_t
    d2 = dw_ * dw_ + dt_ * dt_
    keep = d2 <= r * r
    img[ws[keep], ts[keep]] += amp * np.exp(-0.5 * d2[keep] / (width * width))


def _track_hits(img, w0, t0, w1, t1):
    """Peak hits of one track: for each wire the segment crosses, the argmax tick
    of the finished image within +-5 ticks of the track centre (lowest tick on ties)."""
    W, T = img.shape
    lo = int(np.ceil(min(w0, w1)))
    hi = int(np.floor(max(w0, w1)))
    lo, hi = max(lo, 0), min(hi, W - 1)
    if hi < lo or abs(w1 - w0) < 1e-9:
        return np.zeros((0, 2), np.int64)
    wires = np.arange(lo, hi + 1)
    centre = np.rint(t0 + (wires - w0) * (t1 - t0) / (w1 - w0)).astype(np.int64)
    offs = np.arange(-5, 6)
    ticks = centre[:, None] + offs[None, :]
    valid = (ticks >= 0) & (ticks < T)
    vals = np.where(valid, img[wires[:, None], np.clip(ticks, 0, T - 1)], -np.inf)
    best = ticks[np.arange(len(wires)), np.argmax(vals, axis=1)]
    return np.stack([wires, best], axis=1)


def gen_plane(n_wires: int, n_ticks: int, n_tracks: int, n_showers: int,
              n_hits: int, seed: int, track_amp=None,
              shower_draws: int = 400) -> Plane:
    """Synthetic deconvolved plane plus hits.

    Draw order (one PCG64 stream): noise N(0, 2.5^2) for the whole image; per
    track (w0, t0, w1, t1) uniform over the plane, amplitude U(20, 80) unless
    ``track_amp`` is given, width U(1, 2); per shower amplitude U(20, 60),
    centre uniform, sigma_w U(3, 10), sigma_t U(10, 40); then ``shower_draws``
    Gaussian hit draws per shower; then the subsample and the permutation.
    Hits are deduplicated, subsampled without replacement to ``n_hits`` (all of
    them if fewer exist) and returned in a random order.
    """
    rng = np.random.default_rng(seed)
    W, T = n_wires, n_ticks
    img = rng.normal(0.0, 2.5, size=(W, T))
    tracks = []
    for _ in range(n_tracks):
        w0, w1 = rng.uniform(0, W, size=2)
        t0, t1 = rng.uniform(0, T, size=2)
        amp = float(track_amp) if track_amp is not None else rng.uniform(20, 80)
        width = rng.uniform(1.0, 2.0)
        _render_track(img, rng, amp, w0, t0, w1, t1, width)
        tracks.append((w0, t0, w1, t1))
    showers = []
    for _ in range(n_showers):
        amp = rng.uniform(20, 60)
        wc, tc = rng.uniform(0, W), rng.uniform(0, T)
        sw, st = rng.uniform(3, 10), rng.uniform(10, 40)
        wa = max(0, int(np.floor(wc - 4 * sw)))
        wb = min(W - 1, int(np.ceil(wc + 4 * sw)))
        ta = max(0, int(np.floor(tc - 4 * st)))
        tb = min(T - 1, int(np.ceil(tc + 4 * st)))
        if wb >= wa and tb >= ta:
            ww = np.arange(wa, wb + 1)[:, None]
            tt = np.arange(ta, tb + 1)[None, :]
            img[wa:wb + 1, ta:tb + 1] += amp * np.exp(
                -0.5 * (((ww - wc) / sw) ** 2 + ((tt - tc) / st) ** 2))
        showers.append((wc, tc, sw, st))
    img32 = np.ascontiguousarray(img, dtype=np.float32)

    cand = [np.zeros((0, 2), np.int64)]
    for (w0, t0, w1, t1) in tracks:
        cand.append(_track_hits(img32, w0, t0, w1, t1))
    for (wc, tc, sw, st) in showers:
        dw = rng.normal(wc, sw, size=shower_draws)
        dt = rng.normal(tc, st, size=shower_draws)
        hw = np.clip(np.rint(dw), 0, W - 1).astype(np.int64)
        ht = np.clip(np.rint(dt), 0, T - 1).astype(np.int64)
        cand.append(np.stack([hw, ht], axis=1))
    allh = np.concatenate(cand, axis=0)
    key = np.unique(allh[:, 0] * T + allh[:, 1])
    take = min(n_hits, len(key))
    sel = rng.choice(len(key), size=take, replace=False)
    key = key[sel][rng.permutation(take)]
    hits = np.stack([key // T, key % T], axis=1).astype(np.int32)
    return Plane(img32, np.ascontiguousarray(hits))


def config1(seed: int = 1001) -> Plane:
    """Tiny: one 128-wire x 512-tick plane, 3 tracks of amplitude 40, 1 shower, 128 hits."""
    return gen_plane(128, 512, 3, 1, 128, seed, track_amp=40.0, shower_draws=60)


def config2(seed: int = 1002) -> Plane:
    """One collection plane 480 x 6000, 40 tracks (A 20-80), 5 showers, 3000 hits."""
    return gen_plane(480, 6000, 40, 5, 3000, seed)


CONFIG3_WIRES = (800, 800, 480) * 6    # 18 planes, 12,480 wires
CONFIG3_HITS = 50_000


def config3(seed: int = 1003):
    """Event: 18 planes of 800/800/480 wires x 6000 ticks, ~50k hits in one call.

    Plane p is drawn as ``config2`` with seed ``seed + p`` and its own wire
    count; it receives ``floor(50000 * W_p / 12480)`` hits, the remainder going
    to the last plane.  Returns ``(planes, hits3)`` where ``hits3`` is int32
    ``[n][3] = (plane, wire, tick)``, plane-grouped as the detector reads out.
    """
    total_w = sum(CONFIG3_WIRES)
    quota = [CONFIG3_HITS * w // total_w for w in CONFIG3_WIRES]
    quota[-1] += CONFIG3_HITS - sum(quota)
    planes, parts = [], []
    for p, (w, q) in enumerate(zip(CONFIG3_WIRES, quota)):
        pl = gen_plane(w, 6000, 40, 5, q, seed + p)
        planes.append(pl)
        h = np.empty((len(pl.hits), 3), np.int32)
        h[:, 0] = p
        h[:, 1:] = pl.hits
        parts.append(h)
    return planes, np.ascontiguousarray(np.concatenate(parts, axis=0))


def config4_patches(batch: int, seed: int = 1004, chunk: int = 4096) -> np.ndarray:
    """Pre-cut patch batch: float32 [batch][48][48] of N(0,1) plus one line each.

    Each line passes through (24 + o_r, 24 + o_c) with offsets U(-4, 4) px at an
    angle U(0, pi), with amplitude U(3, 10) and a Gaussian profile of sigma 1 px.
    """
    rng = np.random.default_rng(seed)
    out = np.empty((batch, PATCH, PATCH), np.float32)
    r = np.arange(PATCH, dtype=np.float32)[:, None]
    c = np.arange(PATCH, dtype=np.float32)[None, :]
    for s in range(0, batch, chunk):
        n = min(chunk, batch - s)
        noise = rng.standard_normal((n, PATCH, PATCH), dtype=np.float32)
        off = rng.uniform(-4, 4, size=(n, 2)).astype(np.float32)
        ang = rng.uniform(0, np.pi, size=n).astype(np.float32)
        amp = rng.uniform(3, 10, size=n).astype(np.float32)
        r0 = (24 + off[:, 0])[:, None, None]
        c0 = (24 + off[:, 1])[:, None, None]
        sn = np.sin(ang)[:, None, None]
        cs = np.cos(ang)[:, None, None]
        d = (r[None] - r0) * sn - (c[None] - c0) * cs
        out[s:s + n] = noise + amp[:, None, None] * np.exp(-0.5 * d * d)
    return out


def config5_requests(n_planes: int = 8, n_streams: int = 64, per_stream: int = 32,
                     seed: int = 1005, lo: int = 1000, hi: int = 8000):
    """Serving pattern: ``n_planes`` config-2 planes and a request list.

    Returns ``(planes, requests)``; ``requests[s]`` is the list of requests
    sent on stream ``s``, each ``(plane_index, hits int32 [n][2])`` with
    ``n ~ U{lo..hi}`` hits drawn with replacement from that plane's hit pool.
    """
    planes = [config2(seed + 100 + p) for p in range(n_planes)]
    rng = np.random.default_rng(seed)
    reqs = []
    for _ in range(n_streams):
        mine = []
        for _ in range(per_stream):
            p = int(rng.integers(0, n_planes))
            n = int(rng.integers(lo, hi + 1))
            pool = planes[p].hits
            idx = rng.integers(0, len(pool), size=n)
            mine.append((p, np.ascontiguousarray(pool[idx])))
        reqs.append(mine)
    return planes, reqs


def coord_image(n_wires: int, n_ticks: int) -> np.ndarray:
    """Coordinate-encoded image I[w][t] = 1 + 1000*w + t (exact in float32 for w < 16k)."""
    w = np.arange(n_wires, dtype=np.float64)[:, None]
    t = np.arange(n_ticks, dtype=np.float64)[None, :]
    return np.ascontiguousarray(1.0 + 1000.0 * w + t, dtype=np.float32)
