"""Plain fp64 CPU oracle for per-hit track/shower/Michel classification.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import or call this module.  The
product path (the HIP library and its Python binding) never touches it, and it
shares no code with that path: it needs only numpy.

What it computes, with the passage each step follows:

* Patch construction, paper §2.1 (EmTrackMichelId / PointIdAlg): a 48x48 image
  centred on the hit's wire and peak time, rows indexing the wire and columns
  the time.  Reading used here: row r, column c of the patch of hit (w, t) is
  the plane pixel (w - 24 + r, t - 24 + c), and 0 wherever that pixel lies
  outside the plane.
* The network of paper §2.2: 48 separate 5x5 filters, stride 1, giving 48 maps
  of 44x44 (so no padding), ReLU; a fully connected layer of 128 with ReLU; one
  of 32 with ReLU; then two branches from the 32: three outputs through a
  softmax and one through a sigmoid.  Dropout is the identity at inference.
  Readings: the filter is a cross-correlation (no kernel flip), every layer
  has a bias (the paper's parameter count of 11,900,420 requires all six), and
  the 44x44x48 maps are flattened channels-last, index (y*44 + x)*48 + k.

* Time-interval columns, paper §2.1: each pixel holds the charge that the
  deconvolved waveform of its wire deposits in the time interval of its column.
  With one tick per column this is the plane pixel itself (the reading above).
  Reading used for D ticks per column: the waveform is binned once into
  columns of D ticks aligned to tick 0, column j covering ticks jD .. jD + D - 1,
  and a column's value is the charge deposited in that interval, the sum of
  its samples; ticks past the end of the plane deposit nothing (0), as pixels
  outside the plane read 0.  The patch of hit (w, t) is then cut from the
  binned plane around column floor(t / D), with the same centring and zero
  fill as above.

* Hit finding, paper §2.1: the reconstruction finds wire hits on the
  deconvolved waveforms (giving peak time and charge) before they are
  classified; the paper names no algorithm.  Reading used here: a hit is a tick
  whose value exceeds a threshold and is a local maximum along its wire's
  waveform — greater than the tick before it and not less than the tick after
  it, with ticks outside the waveform counting as minus infinity (a plateau
  gives one hit, at its first tick).  Comparisons are exact in float32.

All arithmetic is float64 with no intermediate rounding; each output is rounded
to float32 once at the end.  Matrix products use numpy's ``@`` (a library
primitive) with no blocking or reordering of our own.  Large inputs are
processed in chunks of hits; chunking never changes a result bit because every
hit is computed independently.

Pins: ``tests/test_oracle.py`` checks each function against facts fixed by the
paper or by mathematics (hand-computed patch coordinates, brute-force
convolution, a library convolution, closed forms of the heads, the parameter
count, invariances).  The physical meaning of the scores (trained weights on
ProtoDUNE-SP data) is parity unpinned: neither exists here.
"""

from __future__ import annotations

import numpy as np

PATCH = 48                 # patch side, paper §2.1
HALF = PATCH // 2          # the hit sits at patch pixel (24, 24)
KS = 5                     # filter side, paper §2.2
NCH = 48                   # number of filters, paper §2.2
FM = PATCH - KS + 1        # 44: map side of a stride-1 unpadded 5x5 filter
FC1_IN = FM * FM * NCH     # 92,928
FC1_OUT = 128
FC2_OUT = 32
NCLS = 3

CHUNK = 256


# --------------------------------------------------------------------------
# Patch construction (paper §2.1)
# --------------------------------------------------------------------------

def gather_patches(image, hits) -> np.ndarray:
    """float32 [n][48][48]: P[r][c] = image[w-24+r][t-24+c], 0 outside the plane.

    ``image`` is [n_wires][n_ticks]; ``hits`` is int [n][2] = (wire, tick).
    The values are copied, never computed, so the result is exact.
    """
    image = np.asarray(image, dtype=np.float32)
    hits = np.asarray(hits, dtype=np.int64).reshape(-1, 2)
    W, T = image.shape
    n = hits.shape[0]
    rows = hits[:, 0:1] - HALF + np.arange(PATCH)[None, :]      # [n][48] wires
    cols = hits[:, 1:2] - HALF + np.arange(PATCH)[None, :]      # [n][48] ticks
    inside = ((rows >= 0) & (rows < W))[:, :, None] & ((cols >= 0) & (cols < T))[:, None, :]
    vals = image[np.clip(rows, 0, W - 1)[:, :, None], np.clip(cols, 0, T - 1)[:, None, :]]
    out = np.where(inside, vals, np.float32(0.0)).astype(np.float32)
    return out.reshape(n, PATCH, PATCH)


def gather_patches_planes(images, hits3) -> np.ndarray:
    """Multi-plane gather: ``hits3`` is int [n][3] = (plane, wire, tick).

    A plane index outside [0, len(images)) gives an all-zero patch.
    """
    hits3 = np.asarray(hits3, dtype=np.int64).reshape(-1, 3)
    out = np.zeros((hits3.shape[0], PATCH, PATCH), np.float32)
    for p, img in enumerate(images):
        sel = np.nonzero(hits3[:, 0] == p)[0]
        if sel.size:
            out[sel] = gather_patches(img, hits3[sel, 1:3])
    return out


# --------------------------------------------------------------------------
# Columns of D ticks (paper §2.1; the reading is in the module docstring)
# --------------------------------------------------------------------------

def downsample_plane(image, ticks_per_column) -> np.ndarray:
    """float32 [n_wires][ceil(n_ticks / D)]: column j is the sum of ticks
    jD .. jD + D - 1 (missing ticks past the end count as 0), in float64,
    rounded once."""
    D = int(ticks_per_column)
    if D < 1:
        raise ValueError("ticks_per_column must be >= 1")
    x = np.asarray(image, dtype=np.float32).astype(np.float64)
    W, T = x.shape
    J = -(-T // D)
    padded = np.zeros((W, J * D), np.float64)
    padded[:, :T] = x
    return padded.reshape(W, J, D).sum(axis=2).astype(np.float32)


def hits_to_columns(hits3, ticks_per_column) -> np.ndarray:
    """(plane, wire, column) of each hit: column = floor(tick / D)."""
    h = np.array(hits3, dtype=np.int64).reshape(-1, 3)
    h[:, 2] = np.floor_divide(h[:, 2], int(ticks_per_column))
    return h


def gather_patches_planes_ds(images, hits3, ticks_per_column) -> np.ndarray:
    """Patches with D ticks per column: cut from the binned planes around the
    hit's column."""
    binned = [downsample_plane(img, ticks_per_column) for img in images]
    return gather_patches_planes(binned, hits_to_columns(hits3, ticks_per_column))


# --------------------------------------------------------------------------
# Hit finding (paper §2.1; the reading is in the module docstring)
# --------------------------------------------------------------------------

def find_hits(images, threshold) -> np.ndarray:
    """int32 [n][3] = (plane, wire, tick) of every hit of every plane image
    ([n_wires][n_ticks] float32), in plane, then wire, then tick order.

    A tick t of wire w is a hit when x[t] > threshold, x[t] > x[t-1] and
    x[t] >= x[t+1], where x[-1] and x[n_ticks] are minus infinity.
    """
    thr = np.float32(threshold)
    out = []
    for p, img in enumerate(images):
        x = np.asarray(img, dtype=np.float32)
        before = np.full_like(x, -np.inf)
        before[:, 1:] = x[:, :-1]
        after = np.full_like(x, -np.inf)
        after[:, :-1] = x[:, 1:]
        w, t = np.nonzero((x > thr) & (x > before) & (x >= after))    # row-major order
        out.append(np.stack([np.full_like(w, p), w, t], axis=1))
    if not out:
        return np.zeros((0, 3), np.int32)
    return np.concatenate(out, axis=0).astype(np.int32)


def to_bf16_rne(x) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even).

    Returned as float32 holding exactly the bfloat16 value.  Finite inputs only.
    A bfloat16 keeps the top 16 bits of the float32 encoding; the discarded low
    16 bits decide the rounding: above half rounds up, below half down, exactly
    half rounds to the neighbour whose last kept bit is 0.
    """
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    low = b & 0xFFFF
    keep = b >> 16
    up = (low > 0x8000) | ((low == 0x8000) & ((keep & 1) == 1))
    keep = keep + up.astype(np.uint64)
    return (keep << 16).astype(np.uint32).view(np.float32).reshape(np.shape(x))


def bf16_bits(x) -> np.ndarray:
    """uint16 bit patterns of ``to_bf16_rne(x)``."""
    return (to_bf16_rne(x).view(np.uint32) >> 16).astype(np.uint16)


def to_fp16_rne(x) -> np.ndarray:
    """Round float32 values to IEEE binary16 (nearest, ties to even), returned
    as float32 holding the fp16 value (numpy's correctly rounded conversion)."""
    return np.asarray(x, dtype=np.float32).astype(np.float16).astype(np.float32)


def fp16_bits(x) -> np.ndarray:
    """uint16 bit patterns of ``to_fp16_rne(x)``."""
    return np.asarray(x, dtype=np.float32).astype(np.float16).view(np.uint16)


def round16(x, kind: str) -> np.ndarray:
    """Round to the 16-bit operand type ``kind`` ('bf16' or 'fp16')."""
    return to_bf16_rne(x) if kind == "bf16" else to_fp16_rne(x)


# --------------------------------------------------------------------------
# The network (paper §2.2)
# --------------------------------------------------------------------------

def conv_relu(patches, conv_w, conv_b) -> np.ndarray:
    """48 maps of 44x44 per patch, channels-last: A[n][y][x][k] (float64).

    A[y][x][k] = ReLU(b_k + sum_{u,v<5} K[k][u][v] * P[y+u][x+v]): a stride-1
    cross-correlation over the valid region.  The 25 taps of every output are
    laid out by a sliding-window view (no arithmetic), then contracted with the
    filters by one matrix product.
    """
    P = np.asarray(patches, dtype=np.float64).reshape(-1, PATCH, PATCH)
    K = np.asarray(conv_w, dtype=np.float64).reshape(NCH, KS * KS)
    win = np.lib.stride_tricks.sliding_window_view(P, (KS, KS), axis=(1, 2))
    taps = win.reshape(P.shape[0], FM, FM, KS * KS)         # [n][y][x][u*5+v]
    pre = taps @ K.T + np.asarray(conv_b, dtype=np.float64)  # [n][y][x][k]
    return np.maximum(pre, 0.0)


def flatten_hwc(A) -> np.ndarray:
    """[n][44][44][48] -> [n][92928] with index (y*44 + x)*48 + k."""
    return np.asarray(A).reshape(A.shape[0], FC1_IN)


def dense_relu(x, w, b) -> np.ndarray:
    """ReLU(b + x @ W) in float64."""
    return np.maximum(np.asarray(x, np.float64) @ np.asarray(w, np.float64)
                      + np.asarray(b, np.float64), 0.0)


def softmax(z) -> np.ndarray:
    """exp(z - max z) / sum exp(z - max z) along the last axis."""
    z = np.asarray(z, np.float64)
    e = np.exp(z - z.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def sigmoid(q) -> np.ndarray:
    """1 / (1 + e^-q), evaluated without overflow for either sign of q."""
    q = np.asarray(q, np.float64)
    e = np.exp(-np.abs(q))
    return np.where(q >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def heads(h2, weights) -> np.ndarray:
    """Scores [n][4] float64 = (softmax(cls), sigmoid(mic)) from the 32-wide layer."""
    z = h2 @ np.asarray(weights["cls_w"], np.float64) + np.asarray(weights["cls_b"], np.float64)
    q = h2 @ np.asarray(weights["mic_w"], np.float64) + np.asarray(weights["mic_b"], np.float64)[0]
    return np.concatenate([softmax(z), sigmoid(q)[:, None]], axis=1)


def forward(patches, weights, return_hidden: bool = False):
    """Scores for a batch of patches, float64 [n][4] (no final rounding).

    ``return_hidden`` also returns (A, h1, h2) for diagnostics.
    """
    A = conv_relu(patches, weights["conv_w"], weights["conv_b"])
    a = flatten_hwc(A)
    h1 = dense_relu(a, weights["fc1_w"], weights["fc1_b"])
    h2 = dense_relu(h1, weights["fc2_w"], weights["fc2_b"])
    s = heads(h2, weights)
    if return_hidden:
        return s, (A, h1, h2)
    return s


def logits(patches, weights) -> np.ndarray:
    """Pre-softmax class logits [n][3] (float64), for tie diagnostics."""
    A = conv_relu(patches, weights["conv_w"], weights["conv_b"])
    h1 = dense_relu(flatten_hwc(A), weights["fc1_w"], weights["fc1_b"])
    h2 = dense_relu(h1, weights["fc2_w"], weights["fc2_b"])
    return h2 @ np.asarray(weights["cls_w"], np.float64) + np.asarray(weights["cls_b"], np.float64)


def classify_patches(patches, weights, chunk: int = CHUNK) -> np.ndarray:
    """float32 [n][4] = (p_track, p_em, p_none, p_michel) for pre-cut patches."""
    patches = np.asarray(patches, dtype=np.float32).reshape(-1, PATCH, PATCH)
    n = patches.shape[0]
    out = np.empty((n, 4), np.float32)
    for s in range(0, n, chunk):
        out[s:s + chunk] = forward(patches[s:s + chunk], weights).astype(np.float32)
    return out


def classify(image, hits, weights, chunk: int = CHUNK) -> np.ndarray:
    """Scores for every hit of one plane, in hit order."""
    hits = np.asarray(hits).reshape(-1, 2)
    out = np.empty((hits.shape[0], 4), np.float32)
    for s in range(0, hits.shape[0], chunk):
        out[s:s + chunk] = forward(gather_patches(image, hits[s:s + chunk]),
                                   weights).astype(np.float32)
    return out


def classify_planes(images, hits3, weights, chunk: int = CHUNK) -> np.ndarray:
    """Scores for (plane, wire, tick) hits over several planes, in hit order."""
    hits3 = np.asarray(hits3).reshape(-1, 3)
    out = np.empty((hits3.shape[0], 4), np.float32)
    for s in range(0, hits3.shape[0], chunk):
        out[s:s + chunk] = forward(gather_patches_planes(images, hits3[s:s + chunk]),
                                   weights).astype(np.float32)
    return out


def classify_planes_ds(images, hits3, weights, ticks_per_column, chunk: int = CHUNK) -> np.ndarray:
    """Scores of hits (plane, wire, tick) with patches of D ticks per column."""
    binned = [downsample_plane(img, ticks_per_column) for img in images]
    return classify_planes(binned, hits_to_columns(hits3, ticks_per_column), weights, chunk)


def quantize_16bit_model(weights, kind: str = "bf16") -> dict:
    """Weights as a 16-bit path holds them: conv and FC1 filters rounded to
    ``kind`` (RNE), everything else unchanged."""
    q = dict(weights)
    q["conv_w"] = round16(weights["conv_w"], kind)
    q["fc1_w"] = round16(weights["fc1_w"], kind)
    return q


def forward_16bit_emulated(patches, weights, kind: str = "bf16") -> np.ndarray:
    """The network with a 16-bit path's roundings applied — patch, conv filter,
    conv output (after ReLU, through float32) and FC1 filter rounded to
    ``kind`` — and float64 accumulation; the conv bias, FC1 bias, FC2 and the
    heads stay as given.  This is what a 16-bit path computes up to its fp32
    accumulation order; the full-precision ``forward`` remains the reference.
    Pinned by exact closed forms of a single-pixel chain in which each of these
    roundings, and each rounding the reading leaves out, changes the scores
    (tests/golden/closed_forms_16bit.json)."""
    q = quantize_16bit_model(weights, kind)
    P = round16(np.asarray(patches, np.float32), kind)
    A = conv_relu(P, q["conv_w"], q["conv_b"])
    A = round16(A.astype(np.float32), kind).astype(np.float64)
    h1 = dense_relu(flatten_hwc(A), q["fc1_w"], q["fc1_b"])
    h2 = dense_relu(h1, q["fc2_w"], q["fc2_b"])
    return heads(h2, q)


def to_e4m3_rne(x) -> np.ndarray:
    """Round to the OCP 8-bit float e4m3 (4 exponent bits, bias 7, 3 mantissa
    bits, largest finite 448, subnormal step 2^-9), nearest even, values beyond
    448 saturating to +-448; returned as float64."""
    x = np.asarray(x, np.float64)
    a = np.abs(x)
    e = np.maximum(np.floor(np.log2(np.maximum(a, 2.0 ** -40))), -6.0)   # -6: subnormal range
    q = 2.0 ** (e - 3)
    r = np.minimum(np.round(a / q) * q, 448.0)                          # np.round: half to even
    return np.copysign(r, x)


def mx_e4m3(blocks) -> np.ndarray:
    """Microscaled e4m3 along the last axis (OCP MX): each block of values
    shares the power-of-two scale X = 2^(floor(log2 max|v|) - 8) (8 = the
    largest e4m3 exponent), and v / X is rounded to e4m3.  Returns the
    dequantized values X * e4m3(v / X)."""
    b = np.asarray(blocks, np.float64)
    m = np.abs(b).max(axis=-1, keepdims=True)
    X = np.where(m > 0, 2.0 ** (np.floor(np.log2(np.where(m > 0, m, 1.0))) - 8), 1.0)
    return to_e4m3_rne(b / X) * X


def forward_mx_fp8_emulated(patches, weights) -> np.ndarray:
    """The network with FC1 in microscaled e4m3 (the fp8 MFMA operands of
    gfx950): the conv as on the fp16 path (fp16 patch and filter), its ReLU
    output and the FC1 weights quantized in blocks of 32 FC1 inputs — 8
    consecutive map positions x 4 consecutive channels, one block per output
    neuron for the weights — then float64 accumulation.  A precision study
    only: no kernel computes this."""
    q = quantize_16bit_model(weights, "fp16")
    P = round16(np.asarray(patches, np.float32), "fp16")
    A = conv_relu(P, q["conv_w"], q["conv_b"])
    n = A.shape[0]
    a = flatten_hwc(A).reshape(n, FM * FM // 8, 8, NCH // 4, 4).transpose(0, 1, 3, 2, 4)
    a = mx_e4m3(a.reshape(n, FM * FM // 8, NCH // 4, 32))
    a = a.reshape(n, FM * FM // 8, NCH // 4, 8, 4).transpose(0, 1, 3, 2, 4).reshape(n, FC1_IN)
    W1 = np.asarray(weights["fc1_w"], np.float64).T.reshape(FC1_OUT, FM * FM // 8, 8, NCH // 4, 4)
    W1 = mx_e4m3(W1.transpose(0, 1, 3, 2, 4).reshape(FC1_OUT, FM * FM // 8, NCH // 4, 32))
    W1 = W1.reshape(FC1_OUT, FM * FM // 8, NCH // 4, 8, 4).transpose(0, 1, 3, 2, 4)
    W1 = W1.reshape(FC1_OUT, FC1_IN).T
    h1 = dense_relu(a, W1, weights["fc1_b"])
    h2 = dense_relu(h1, weights["fc2_w"], weights["fc2_b"])
    return heads(h2, weights)


def fc1_e4m3_exponents(fc1_w) -> np.ndarray:
    """Per FC1 output n, the power-of-two exponent k_n by which an 8-bit path
    scales column n of the FC1 weights before rounding them to e4m3: the
    largest integer with max_k |W1[k][n]| * 2^k_n <= 448, the format's largest
    value (0 for a column of zeros).  Exact: with max = f * 2^e, f in
    [1/2, 1), and 448 = (7/8) * 2^9, k_n = 9 - e when f <= 7/8, else 8 - e."""
    m = np.abs(np.asarray(fc1_w, np.float64)).max(axis=0)
    f, e = np.frexp(m)
    k = np.where(f <= 0.875, 9 - e, 8 - e).astype(np.float64)
    return np.where(m > 0, k, 0.0)


def quantize_fp8_model(weights) -> dict:
    """Weights as the 8-bit path holds them: the conv filters rounded to fp16
    (its conv runs as on the fp16 path), FC1 column n multiplied by 2^k_n
    (``fc1_e4m3_exponents``) and rounded to e4m3 (``fc1_w8``, with the exponents
    in ``fc1_exp``); everything else unchanged."""
    q = quantize_16bit_model(weights, "fp16")
    k = fc1_e4m3_exponents(weights["fc1_w"])
    q["fc1_exp"] = k
    q["fc1_w8"] = to_e4m3_rne(np.asarray(weights["fc1_w"], np.float64) * 2.0 ** k)
    return q


def forward_fp8_emulated(patches, weights) -> np.ndarray:
    """The network with FC1 on e4m3 operands (the 8-bit operation of the
    paper's outlook, section 4): the conv as on the fp16 path (fp16 patch and
    filter, exact bias); its ReLU output through float32, then rounded to e4m3
    (nearest even, saturating at 448); FC1 column n as ``quantize_fp8_model``
    holds it; float64 accumulation of the e4m3 products, the sum for output n
    multiplied by 2^-k_n, then the FC1 bias, ReLU, FC2 and the heads as given.
    This is what the 8-bit path computes up to its accumulation order."""
    q = quantize_fp8_model(weights)
    P = round16(np.asarray(patches, np.float32), "fp16")
    A = conv_relu(P, q["conv_w"], q["conv_b"])
    A = to_e4m3_rne(A.astype(np.float32))
    h1 = (flatten_hwc(A) @ q["fc1_w8"]) * 2.0 ** -q["fc1_exp"] + np.asarray(q["fc1_b"], np.float64)
    h1 = np.maximum(h1, 0.0)
    h2 = dense_relu(h1, q["fc2_w"], q["fc2_b"])
    return heads(h2, q)


def classify_fp8_emulated(patches, weights, chunk: int = CHUNK) -> np.ndarray:
    """float32 [n][4] from ``forward_fp8_emulated``, chunked."""
    patches = np.asarray(patches, dtype=np.float32).reshape(-1, PATCH, PATCH)
    out = np.empty((patches.shape[0], 4), np.float32)
    for s in range(0, patches.shape[0], chunk):
        out[s:s + chunk] = forward_fp8_emulated(patches[s:s + chunk], weights).astype(np.float32)
    return out


def forward_bf16_emulated(patches, weights) -> np.ndarray:
    """``forward_16bit_emulated`` with bfloat16 operands."""
    return forward_16bit_emulated(patches, weights, "bf16")


def classify_16bit_emulated(patches, weights, kind: str, chunk: int = CHUNK) -> np.ndarray:
    """float32 [n][4] from ``forward_16bit_emulated``, chunked."""
    patches = np.asarray(patches, dtype=np.float32).reshape(-1, PATCH, PATCH)
    out = np.empty((patches.shape[0], 4), np.float32)
    for s in range(0, patches.shape[0], chunk):
        out[s:s + chunk] = forward_16bit_emulated(patches[s:s + chunk], weights, kind).astype(np.float32)
    return out
