"""Plain CPU oracle for batched policy/value evaluation of search leaves.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this module; the GPU library never does, and this
module imports nothing from it.

What it computes.  The forward pass of the residual policy/value network that
the paper's inference worker evaluates for every search leaf (Section 3.3 "One
learning cycle", Section 3.5 "Chess representation and outputs", Section 5.2
"Batching and host-side submission"):

  stem      h = act(conv3x3(x) + b)                        ("start block", Section 5.3)
  block j   t = act(conv3x3(h) + b1)
            h = act(h + conv3x3(t) + b2)                   (post-activation block, Section 4.3
                                                            "Quantization as an architectural
                                                            constraint": conv, norm, act, conv,
                                                            norm, residual add, act; norms are
                                                            folded into the biases, Appendix D)
  policy    z[p*64 + r*8 + c] = b_p[p] + sum_f Wp[p,f] h[f,r,c]   (move-plane head, Section 4.3
                                                            "Three policy representations":
                                                            move types at board squares)
            P = softmax of z over the legal cells, exactly 0 elsewhere (Section 3.5, Appendix D:
                                                            illegal actions are masked before
                                                            the softmax)
  value     u[s] = b_v + sum_f w_v[f] h[f,s]   (optionally ReLU)
            V = tanh(w2 . relu(W1 u + b1) + b2)

act is ReLU, or ReLU capped at act_cap when act_cap > 0 (the capped activation of
Section 4.3).  conv3x3 is a stride-1 cross-correlation over one 8x8 board with a
zero pad of one square; boards never see each other.

Modes.
  forward(..., mode="f64")     exact definition in float64 (parity reference for
                               the fp32 and bf16 paths).
  forward(..., mode="bf16emu") float64 arithmetic with every inter-layer
                               activation rounded to bfloat16 (diagnostic).
  forward_quant(...)           the int8 / fp8-e4m3 network defined by its
                               quantisation: residual-conv weights quantised per
                               output channel, every activation tensor between
                               layers quantised per tensor, stem in bf16, heads
                               in floating point (Section 5.3 "Inference runtimes
                               and precision": most trunk convolutions in INT8,
                               the start block and heads at higher precision,
                               explicit quantise/dequantise operations).
                               Products and sums are exact (float64 holds every
                               integer and e4m3 product sum here); the steps that
                               decide a quantised code (rescale, bias, residual,
                               activation, requantise) are taken in float32 in a
                               fixed order, the same order the GPU kernels use.

The softmax, value head and quantisers are written from their definitions; the
convolution is the sum over the nine taps of a channel contraction (a matrix
product per tap), which is the definition of a 3x3 cross-correlation.
"""

from __future__ import annotations

import numpy as np

N_SQUARES = 64
E4M3_MAX = 448.0
INT8_MAX = 127.0


# --------------------------------------------------------------------------- #
# Weight blob (canonical order: stem W[F][C][3][3], b[F]; per block W1, b1, W2, b2;
# policy W[P][F], b[P]; value conv W[1][F], b[1]; fc1 W[H][64], b[H]; fc2 W[1][H], b[1])
# --------------------------------------------------------------------------- #
def unpack(spec, blob):
    """Split a flat canonical blob into named float64 arrays."""
    C, F, P, H = spec.in_planes, spec.filters, spec.policy_planes, spec.value_hidden
    blob = np.asarray(blob, dtype=np.float64).ravel()
    sizes = [("stem.w", (F, C, 3, 3)), ("stem.b", (F,))]
    for j in range(spec.blocks):
        sizes += [(f"w1.{j}", (F, F, 3, 3)), (f"b1.{j}", (F,)),
                  (f"w2.{j}", (F, F, 3, 3)), (f"b2.{j}", (F,))]
    sizes += [("policy.w", (P, F)), ("policy.b", (P,)), ("value.w", (1, F)),
              ("value.b", (1,)), ("fc1.w", (H, N_SQUARES)), ("fc1.b", (H,)),
              ("fc2.w", (1, H)), ("fc2.b", (1,))]
    out, off = {}, 0
    for name, shp in sizes:
        n = int(np.prod(shp))
        out[name] = blob[off:off + n].reshape(shp)
        off += n
    if off != blob.size:
        raise ValueError(f"blob has {blob.size} values, layer list needs {off}")
    return out


# --------------------------------------------------------------------------- #
# Building blocks
# --------------------------------------------------------------------------- #
def conv3x3(x, w, b=None):
    """3x3 stride-1 cross-correlation, zero pad 1, per 8x8 board.

    x: [B, C, 8, 8], w: [F, C, 3, 3], b: [F] or None -> [B, F, 8, 8], float64.
    y[f, r, c] = b[f] + sum_{i, dy, dx} w[f, i, dy, dx] * x[i, r+dy-1, c+dx-1].
    """
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    B, C = x.shape[:2]
    F = w.shape[0]
    xp = np.zeros((C, B, 10, 10))
    xp[:, :, 1:9, 1:9] = x.transpose(1, 0, 2, 3)
    y = np.zeros((F, B * N_SQUARES))
    for dy in range(3):
        for dx in range(3):
            tap = np.ascontiguousarray(xp[:, :, dy:dy + 8, dx:dx + 8]).reshape(C, B * N_SQUARES)
            y += np.ascontiguousarray(w[:, :, dy, dx]) @ tap
    y = y.reshape(F, B, 8, 8).transpose(1, 0, 2, 3)
    if b is not None:
        y = y + np.asarray(b, dtype=np.float64)[None, :, None, None]
    return y


def act(y, cap):
    y = np.maximum(y, 0.0)
    return np.minimum(y, cap) if cap and cap > 0 else y


def policy_logits(h, wp, bp):
    """1x1 conv F->P over every square, flattened plane-major: idx = p*64 + r*8 + c."""
    B, F = h.shape[:2]
    hs = h.reshape(B, F, N_SQUARES)
    z = np.einsum("pf,bfs->bps", wp, hs) + bp[None, :, None]
    return z.reshape(B, -1)


def softmax_legal(z, legal):
    """Softmax over legal cells only; illegal cells get exactly 0; a row with no
    legal cell is all zero."""
    z = np.asarray(z, dtype=np.float64)
    m = np.asarray(legal) != 0
    out = np.zeros_like(z)
    for i in range(z.shape[0]):
        if not m[i].any():
            continue
        zl = z[i, m[i]]
        e = np.exp(zl - zl.max())
        out[i, m[i]] = e / e.sum()
    return out


def value_head(h, wv, bv, w1, b1, w2, b2, conv_relu):
    """u = 1x1 conv F->1 per square (64-vector); V = tanh(w2 . relu(W1 u + b1) + b2)."""
    B, F = h.shape[:2]
    u = np.einsum("f,bfs->bs", wv[0], h.reshape(B, F, N_SQUARES)) + bv[0]
    if conv_relu:
        u = np.maximum(u, 0.0)
    g = np.maximum(u @ w1.T + b1[None, :], 0.0)
    return np.tanh(g @ w2[0] + b2[0])


def heads(spec, W, h, legal):
    z = policy_logits(h, W["policy.w"], W["policy.b"])
    P = softmax_legal(z, legal)
    V = value_head(h, W["value.w"], W["value.b"], W["fc1.w"], W["fc1.b"], W["fc2.w"],
                   W["fc2.b"], spec.value_conv_relu)
    return P, V


# --------------------------------------------------------------------------- #
# bfloat16 rounding (for the diagnostic mode and for bf16 ingest)
# --------------------------------------------------------------------------- #
def to_bf16(x):
    """Round to the nearest bfloat16 (ties to even) via float32; returns float64."""
    f = np.asarray(x, dtype=np.float32)
    bits = f.view(np.uint32).astype(np.uint64)
    lsb = (bits >> 16) & 1
    bits = ((bits + 0x7FFF + lsb) >> 16) << 16
    return bits.astype(np.uint32).view(np.float32).astype(np.float64)


# --------------------------------------------------------------------------- #
# Float network
# --------------------------------------------------------------------------- #
def tower(spec, W, x, round_fn=None, record=None):
    """Stem + residual blocks.  round_fn rounds each inter-layer activation;
    record (a list) receives every tensor that feeds a residual conv, plus the
    final tower output, in order h0, t0, h1, t1, ..., h_N."""
    rnd = round_fn if round_fn is not None else (lambda a: a)
    cap = spec.act_cap
    h = rnd(act(conv3x3(x, W["stem.w"], W["stem.b"]), cap))
    if record is not None:
        record.append(h)
    for j in range(spec.blocks):
        t = rnd(act(conv3x3(h, W[f"w1.{j}"], W[f"b1.{j}"]), cap))
        if record is not None:
            record.append(t)
        h = rnd(act(h + conv3x3(t, W[f"w2.{j}"], W[f"b2.{j}"]), cap))
        if record is not None:
            record.append(h)
    return h


def forward(spec, blob, planes, legal, mode="f64"):
    """Policy priors [B, P*64] and values [B] in float64."""
    W = unpack(spec, blob)
    x = np.asarray(planes, dtype=np.float64)
    if mode == "f64":
        h = tower(spec, W, x)
    elif mode == "bf16emu":
        h = tower(spec, W, to_bf16(x), round_fn=to_bf16)
    else:
        raise ValueError(mode)
    return heads(spec, W, h, legal)


def calibrate_absmax(spec, blob, planes, chunk=128):
    """Per-tensor absolute maxima of h0, t0, h1, ..., h_N over a calibration set,
    on the float64 network.  Absmax calibration is this implementation's reading:
    the paper calibrates on 516 real positions but names no calibrator."""
    W = unpack(spec, blob)
    amax = np.zeros(spec.blocks * 2 + 1)
    for s in range(0, planes.shape[0], chunk):
        rec = []
        tower(spec, W, np.asarray(planes[s:s + chunk], dtype=np.float64), record=rec)
        amax = np.maximum(amax, [np.abs(a).max() for a in rec])
    return amax


# --------------------------------------------------------------------------- #
# Quantisers
# --------------------------------------------------------------------------- #
def quant_int8(v):
    """Symmetric int8 code of a float32 value: round half to even, saturate to
    [-127, 127] (-128 unused)."""
    return np.clip(np.rint(np.asarray(v, dtype=np.float32)), -INT8_MAX, INT8_MAX).astype(np.float32)


def e4m3_round(v):
    """Nearest OCP fp8 e4m3fn value (1 sign, 4 exponent bits with bias 7, 3 mantissa
    bits, no infinities, max finite 448), ties to even, saturating to +-448.
    Normal numbers in [2^e, 2^(e+1)) with e >= -6 are spaced 2^(e-3); below 2^-6
    the spacing is the subnormal step 2^-9."""
    v = np.asarray(v, dtype=np.float64)
    a = np.abs(v)
    _, ex = np.frexp(np.where(a > 0, a, 1.0))       # a = m * 2^ex, m in [0.5, 1)
    e = np.maximum(ex.astype(np.float64) - 1.0, -6.0)   # floor(log2 a), clamped to the normal range
    step = np.exp2(e - 3.0)
    r = np.rint(a / step) * step
    r = np.minimum(r, E4M3_MAX)
    return np.where(a > 0, np.copysign(r, v), 0.0 * v)


def e4m3_decode(code):
    """Value of an e4m3fn byte (0..255); NaN for the two NaN codes."""
    code = np.asarray(code, dtype=np.int64)
    s = np.where(code & 0x80, -1.0, 1.0)
    e = (code >> 3) & 0xF
    m = code & 0x7
    val = np.where(e == 0, m * 2.0 ** -9, (1.0 + m / 8.0) * np.exp2(e - 7.0))
    val = np.where((e == 0xF) & (m == 0x7), np.nan, val)
    return s * val


def quant_code(v, fmt):
    """Quantised value (as float) of a float32 value already divided by its scale."""
    if fmt == "int8":
        return quant_int8(v)
    if fmt == "fp8":
        return e4m3_round(np.asarray(v, dtype=np.float32)).astype(np.float32)
    raise ValueError(fmt)


def qmax(fmt):
    return INT8_MAX if fmt == "int8" else E4M3_MAX


def weight_scales(spec, blob, fmt):
    """Per-output-channel absmax weight scales of the 2*blocks residual convs,
    s_w[f] = max|W[f]| / qmax (1 where the channel is all zero), as float32."""
    W = unpack(spec, blob)
    out = []
    for j in range(spec.blocks):
        for key in (f"w1.{j}", f"w2.{j}"):
            a = np.abs(W[key]).reshape(spec.filters, -1).max(axis=1) / qmax(fmt)
            out.append(np.where(a > 0, a, 1.0))
    return np.concatenate(out).astype(np.float32)


def act_scales_from_absmax(amax, fmt):
    a = np.asarray(amax, dtype=np.float64) / qmax(fmt)
    return np.where(a > 0, a, 1.0).astype(np.float32)


def quantize_weights(w, s, fmt):
    """Weight codes q = sat(rne(w / s[f])), with the division in float32."""
    w32 = np.asarray(w, dtype=np.float32)
    s32 = np.asarray(s, dtype=np.float32).reshape((-1,) + (1,) * (w32.ndim - 1))
    return quant_code(w32 / s32, fmt).astype(np.float64)


# --------------------------------------------------------------------------- #
# Quantised network
# --------------------------------------------------------------------------- #
def _requant(y32, cap, inv_out, fmt):
    """Activation then requantisation of a float32 tensor: q = sat(rne(act(y) * inv))."""
    y32 = np.maximum(y32, np.float32(0.0))
    if cap and cap > 0:
        y32 = np.minimum(y32, np.float32(cap))
    return quant_code((y32 * np.float32(inv_out)).astype(np.float32), fmt)


def forward_quant(spec, blob, w_scales, act_scales, fmt, planes, legal, record=None):
    """int8 (fmt="int8") or fp8-e4m3 (fmt="fp8") network.

    Tensors h0, t0, h1, ..., h_N are stored as codes q with per-tensor scales
    a[0..2N] (value = q * a[k]).  Residual conv n (n = 2j for conv1, 2j+1 for
    conv2 of block j) uses weight codes with per-channel scales s_w[n, f].
    Per output element, in float32 and in this order:
        m_f = a_in * s_w[f]                (float32 product)
        y   = float32(acc) * m_f
        y   = y + b[f]
        y   = y + float32(q_res) * a_res   (conv2 only; q_res is the block input)
        q   = sat(rne(act(y) * inv_out))   with inv_out = float32(1 / a_out)
    The stem runs on bf16 inputs and weights: y = float32(acc) + b[f], then the
    same activation and requantisation at a[0].  The heads take the float value
    q * a[2N] of the final tower tensor.
    """
    F, nb = spec.filters, spec.blocks
    W = unpack(spec, blob)
    a = np.asarray(act_scales, dtype=np.float32)
    sw = np.asarray(w_scales, dtype=np.float32).reshape(2 * nb, F)
    inv = (1.0 / a.astype(np.float64)).astype(np.float32)
    cap = spec.act_cap
    f32 = np.float32

    x = to_bf16(np.asarray(planes, dtype=np.float64))
    acc = conv3x3(x, W["stem.w"])
    y = acc.astype(f32) + W["stem.b"].astype(f32)[None, :, None, None]
    q = _requant(y, cap, inv[0], fmt)
    if record is not None:
        record.append(q)
    for j in range(nb):
        q_in = q
        for n, (wk, bk, a_in, a_out) in enumerate(
                [(f"w1.{j}", f"b1.{j}", 2 * j, 2 * j + 1),
                 (f"w2.{j}", f"b2.{j}", 2 * j + 1, 2 * j + 2)]):
            ci = 2 * j + n
            wq = quantize_weights(W[wk], sw[ci], fmt)
            acc = conv3x3(q, wq)
            m = (a[a_in] * sw[ci]).astype(f32)
            y = (acc.astype(f32) * m[None, :, None, None]).astype(f32)
            y = (y + W[bk].astype(f32)[None, :, None, None]).astype(f32)
            if n == 1:
                y = (y + (q_in.astype(f32) * a[2 * j]).astype(f32)).astype(f32)
            q = _requant(y, cap, inv[a_out], fmt)
            if record is not None:
                record.append(q)
    h = q.astype(np.float64) * np.float64(a[2 * nb])
    return heads(spec, W, h, legal)
