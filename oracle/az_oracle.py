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
  forward(..., mode="bf16emu") the bf16 storage scheme of the GPU library
                               (diagnostic): every convolution input rounded to
                               bfloat16, the residual stream kept in float32, the
                               heads fed the float32 tower output.
  forward_quant(...)           the int8 / fp8-e4m3 network defined by its
                               quantisation, in float64: residual-conv weights
                               quantised per output channel, every activation
                               tensor between layers quantised per tensor, stem in
                               bf16, heads in floating point (Section 5.3
                               "Inference runtimes and precision": most trunk
                               convolutions in INT8, the start block and heads at
                               higher precision, explicit quantise/dequantise
                               operations).  Products of codes are summed exactly
                               and every rescale, bias, residual, activation and
                               rounding is taken in float64 from its definition.
                               forward_quant(..., sums="fp8_mfma") is a
                               diagnostic only (the measured summation of the
                               gfx950 fp8 matrix instruction).

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


def tower_bf16_operands(spec, W, x):
    """Tower with bfloat16 convolution inputs and a float32 residual stream."""
    f32 = lambda a: a.astype(np.float32).astype(np.float64)  # noqa: E731
    cap = spec.act_cap
    h = f32(act(conv3x3(x, W["stem.w"], W["stem.b"]), cap))
    for j in range(spec.blocks):
        t = act(conv3x3(to_bf16(h), W[f"w1.{j}"], W[f"b1.{j}"]), cap)
        h = f32(act(h + conv3x3(to_bf16(t), W[f"w2.{j}"], W[f"b2.{j}"]), cap))
    return h


def forward(spec, blob, planes, legal, mode="f64"):
    """Policy priors [B, P*64] and values [B] in float64."""
    W = unpack(spec, blob)
    x = np.asarray(planes, dtype=np.float64)
    if mode == "f64":
        h = tower(spec, W, x)
    elif mode == "bf16emu":
        h = tower_bf16_operands(spec, W, to_bf16(x))
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
    """Symmetric int8 code of a value (already divided by its scale): round half
    to even, saturate to [-127, 127] (-128 unused).  Computed in float64."""
    return np.clip(np.rint(np.asarray(v, dtype=np.float64)), -INT8_MAX, INT8_MAX)


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
    """sat(rne(v)) on the format's grid, v already divided by its scale (float64)."""
    if fmt == "int8":
        return quant_int8(v)
    if fmt == "fp8":
        return e4m3_round(v)
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
    """Weight codes q_w[f, ...] = sat(rne(w[f, ...] / s[f])), float64 throughout
    (the quotient of two float32 values is decided exactly: float64 rounds it
    only where it is not a tie of the integer or e4m3 grid)."""
    w = np.asarray(w, dtype=np.float64)
    s = np.asarray(s, dtype=np.float64).reshape((-1,) + (1,) * (w.ndim - 1))
    return quant_code(w / s, fmt)


def requant(y, s_out, cap, fmt):
    """Code of the next tensor: q = sat(rne(act(y) / s_out)), float64."""
    return quant_code(act(y, cap) / np.float64(s_out), fmt)


# --------------------------------------------------------------------------- #
# fp8 sums as gfx950's fp8 matrix instructions take them (diagnostic only)
# --------------------------------------------------------------------------- #
def _native():
    from . import native
    return native.lib()


def conv3x3_fp8_mfma(x, w):
    """DIAGNOSTIC, never a parity reference.  3x3 convolution of fp8 values
    (given as floats) summed the way the gfx950 fp8 matrix instruction was
    measured to sum them: per group of eight input channels at one tap,
    products truncated toward zero to 2^-13 of the group's largest exponent sum
    and added exactly, group sums added to a float32 accumulator
    (oracle/fp8_groups.c).  It tells how far a GPU fp8 path built on that
    instruction can be from the definition, whose sums are exact."""
    import ctypes
    B, C = x.shape[:2]
    F = w.shape[0]
    x = np.ascontiguousarray(np.asarray(x, dtype=np.float32).reshape(B, C, 64))
    w = np.ascontiguousarray(np.asarray(w, dtype=np.float32).reshape(F, C, 9))
    out = np.empty((B, F, 64), dtype=np.float32)
    P = ctypes.POINTER(ctypes.c_float)
    _native().fp8_conv3x3_groups(x.ctypes.data_as(P), w.ctypes.data_as(P), B, C, F,
                                 out.ctypes.data_as(P))
    return out.reshape(B, F, 8, 8).astype(np.float64)


def quant_conv_sum(q, wq, fmt, sums):
    """Exact sum of code products (the definition), or with sums="fp8_mfma" the
    diagnostic fp8 matrix-instruction sum."""
    if sums == "fp8_mfma" and fmt == "fp8":
        return conv3x3_fp8_mfma(q, wq)
    if sums not in ("exact", "fp8_mfma"):
        raise ValueError(sums)
    return conv3x3(q, wq)


# --------------------------------------------------------------------------- #
# Quantised network
# --------------------------------------------------------------------------- #
def forward_quant(spec, blob, w_scales, act_scales, fmt, planes, legal, record=None, sums="exact"):
    """int8 (fmt="int8") or fp8-e4m3 (fmt="fp8") network, the plain definition in
    float64 (Section 5.3 "Inference runtimes and precision": explicit quantise /
    dequantise operations around the INT8 trunk convolutions, the start block and
    heads at higher precision; Section 4.3 "Quantization as an architectural
    constraint" for the block).

    Tensors h0, t0, h1, ..., h_N are stored as codes q (integers for int8, e4m3
    values for fp8) with per-tensor scales a[0..2N]: value = q * a[k].

      stem     y = conv3x3(bf16(x), W_s) + b_s       (bf16-valued weights, exact sum)
               q0 = sat(rne(act(y) / a[0]))
      conv n   q_w = sat(rne(W_n / s_w[n][f]))        (per output channel f)
               acc = conv3x3(q_in, q_w)               (exact: integer or e4m3 products,
                                                       every partial sum is a float64)
               y = acc * a[n] * s_w[n][f] + b_n[f]
               second conv of a block: y += q_res * a[n-1]   (dequantised block input)
               q = sat(rne(act(y) / a[n+1]))
      heads    in float64 on the dequantised h = q_N * a[2N].

    sat clamps to +-127 (int8) or +-448 (e4m3); rne rounds half to even (for e4m3
    to the nearest e4m3fn value).  sums="fp8_mfma" replaces the exact fp8 sums by
    the diagnostic model of the matrix instruction (conv3x3_fp8_mfma); it is
    never a parity reference."""
    F, nb = spec.filters, spec.blocks
    W = unpack(spec, blob)
    sw = np.asarray(w_scales, dtype=np.float32).astype(np.float64).reshape(2 * nb, F)
    a = np.asarray(act_scales, dtype=np.float32).astype(np.float64)
    cap = spec.act_cap
    bc = lambda v: v[None, :, None, None]  # noqa: E731  per-channel broadcast

    x = to_bf16(np.asarray(planes, dtype=np.float64))
    q = requant(conv3x3(x, W["stem.w"], W["stem.b"]), a[0], cap, fmt)
    if record is not None:
        record.append(q)
    for j in range(nb):
        q_in = q
        for second, (wk, bk) in enumerate([(f"w1.{j}", f"b1.{j}"), (f"w2.{j}", f"b2.{j}")]):
            n = 2 * j + second
            wq = quantize_weights(W[wk], sw[n], fmt)
            acc = quant_conv_sum(q, wq, fmt, sums)
            y = acc * a[n] * bc(sw[n]) + bc(W[bk])
            if second:
                y = y + q_in * a[n - 1]
            q = requant(y, a[n + 1], cap, fmt)
            if record is not None:
                record.append(q)
    h = q * a[2 * nb]
    return heads(spec, W, h, legal)


# --------------------------------------------------------------------------- #
# Deployment validation metrics
# --------------------------------------------------------------------------- #
P_FLOOR = 1e-30


def compare_outputs(P_ref, V_ref, P_test, V_test, legal):
    """Per-position agreement of a test evaluation with a reference one, the checks
    applied to a deployed engine against its source network (Section "Prediction
    drift under TensorRT refitting": top-one legal-move agreement, legal-policy KL
    divergence, value error).  Returns float64 arrays (top1_equal, kl, dv):
      top1_equal[b] = 1 if the first maximising legal cell of P_ref[b] equals that of
                      P_test[b] (1 for a row without legal cells), else 0;
      kl[b]         = sum over legal cells with P_ref > 0 of
                      P_ref * (ln P_ref - ln max(P_test, 1e-30));
      dv[b]         = |V_ref[b] - V_test[b]|."""
    Pr = np.asarray(P_ref, dtype=np.float64)
    Pt = np.asarray(P_test, dtype=np.float64)
    m = np.asarray(legal) != 0
    ir = np.argmax(np.where(m, Pr, -np.inf), axis=1)
    it = np.argmax(np.where(m, Pt, -np.inf), axis=1)
    has = m.any(axis=1)
    top1 = np.where(has, (ir == it).astype(np.float64), 1.0)
    use = m & (Pr > 0)
    terms = np.where(use, Pr * (np.log(np.where(use, Pr, 1.0)) - np.log(np.maximum(Pt, P_FLOOR))), 0.0)
    kl = terms.sum(axis=1)
    dv = np.abs(np.asarray(V_ref, dtype=np.float64) - np.asarray(V_test, dtype=np.float64))
    return top1, kl, dv
