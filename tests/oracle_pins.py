"""Pins of the CPU oracle: checks against what the paper and the mathematics
fix, not against the oracle itself.

Each pin takes an oracle.Oracle and raises AssertionError on a mismatch.  The
same pins run against the real oracle (all must pass) and against builds
with a planted mistake (at least one must fail for each).

Sources of truth used here:
  * hand-worked blocks under tests/golden (Sec. 3.2 Eq. 3-4, Sec. 4.3 Eq. 9-12);
  * the E2M1 magnitudes {0, 0.5, 1, 1.5, 2, 3, 4, 6} (Sec. 3.2.2 format);
  * brute force: nearest grid point by exhaustive distance comparison, block
    exponent by counting, fp64 matrix products with numpy of values decoded
    here from the literal table;
  * invariants of the method (zero residual on grid values, power-of-two
    equivariance, idempotence, negation symmetry, monotone improvement, the
    half-error bound of the second stage);
  * closed forms for the SwiGLU intermediate and bf16 rounding;
  * HiF4 (Sec. 3.3): the decode of Eq. 6 worked by hand and implemented
    here independently; the encoder is the library's reading (parity
    unpinned) and is pinned by its defining properties (smallest macro scale
    with no saturation, smallest non-saturating micro-exponents under the
    shared 8-element bit, nearest element with ties to even) checked by
    brute force, and by a hand-worked block.
"""
import math
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
E2M1 = (0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0)


# ---------------------------------------------------------------- helpers
def read_golden(name):
    d = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            k, v = line.split(":", 1)
            d[k.strip()] = v.split()
    return d


def padded_floats(vals, n=32):
    a = [float(v) for v in vals]
    return np.array(a + [0.0] * (n - len(a)), dtype=np.float64)


def padded_bytes(vals, n=16):
    a = [int(v, 16) for v in vals]
    return np.array(a + [0] * (n - len(a)), dtype=np.uint8)


def decode_codes(codes, scales):
    """Independent decode: literal table, nibble 2j low, scale 2^(s-127)."""
    codes = np.asarray(codes, np.uint8)
    rows, K = codes.shape[0], codes.shape[1] * 2
    nib = np.empty((rows, K), np.int64)
    nib[:, 0::2] = codes & 0x0F
    nib[:, 1::2] = codes >> 4
    mag = np.array(E2M1)[nib & 7]
    val = np.where(nib & 8, -mag, mag)
    sc = np.repeat(np.asarray(scales, np.float64) - 127.0, 32, axis=1)
    return val * np.exp2(sc)


def brute_code(y):
    """Nearest E2M1 magnitude by exhaustive comparison, ties to the even
    index, values beyond 6 saturate; the sign bit follows y's sign."""
    a = min(abs(y), 6.0)
    cands = sorted(range(8), key=lambda i: (abs(a - E2M1[i]), i % 2))
    return (8 if math.copysign(1.0, y) < 0 else 0) | cands[0]


def brute_exponent(amax):
    """Smallest e in [-127, 127] with amax < 8 * 2^e (the E2M1 range
    [0, 8) of x / 2^e before saturation), found by counting."""
    e = -127
    while e < 127 and amax >= 8.0 * 2.0 ** e:
        e += 1
    return e


def brute_block(x):
    """Quantize one block by brute force; returns (codes, scale byte)."""
    e = brute_exponent(max(abs(v) for v in x))
    return [brute_code(v / 2.0 ** e) for v in x], e + 127


def pack(codes):
    return bytes(codes[2 * j] | (codes[2 * j + 1] << 4) for j in range(len(codes) // 2))


def bf16_ulp(v):
    if v == 0:
        return 2.0 ** -133
    return 2.0 ** (math.floor(math.log2(abs(v))) - 7)


# Scale bytes swept by the converter-convention tests: the lower clamp and
# the subnormal range of the scale (0-2), the first byte whose grid is normal
# (3), unit scale (127), a large scale (200) and the largest byte a finite
# fp32 or bf16 block can reach (252: amax below 2^128 gives at most
# exponent field 254, minus the offset 2).
SWEEP_SCALE_BYTES = (0, 1, 2, 3, 127, 200, 252)


def _neighbours(v, bf16):
    """The two fp32 (or bf16) neighbours of a positive value v of that format
    (by incrementing its bit pattern, subnormals included)."""
    shift = 16 if bf16 else 0
    u = int(np.array([v], np.float32).view(np.uint32)[0])
    assert (u >> shift) << shift == u, v
    out = []
    for d in (-1, 1):
        w = np.array([((u >> shift) + d) << shift], np.uint32).view(np.float32)[0]
        out.append(float(w))
    return out


def _below(v, bf16):
    """The largest fp32 (or bf16) value below v (a power of two up to 2^128,
    where the bit pattern just below v's is the largest finite value)."""
    if v == 2.0 ** 128:
        return float(np.array([0x7F7FFFFF if not bf16 else 0x7F7F0000], np.uint32)
                     .view(np.float32)[0])
    return _neighbours(v, bf16)[0]


def scale_sweep_blocks(bf16=False):
    """Blocks that pin the element conversions at the scale bytes of
    SWEEP_SCALE_BYTES.  Returns x float64 [rows][128]; row i holds four
    32-element blocks of scale byte SWEEP_SCALE_BYTES[i], S = 2^(byte-127):
    every E2M1 grid point from 0.5, every midpoint and its two fp32 (bf16)
    neighbours, zero, and 6.25, 7.5 and the largest value below 8 (which
    sets the block maximum in [4S, 8S)), all times S, in that order, then
    negated, with alternating signs, and reversed.  The last row holds
    clamped blocks at byte 0 (maximum below 2^-125, so x / 2^-127 < 4): the
    sweep values below 4S, those below 2S (all subnormal), a block of mixed
    small values with zeros, and the first block with signs flipped on every
    third element.  Every value is exactly representable in fp32 (in bf16
    when bf16 is set)."""
    grid = [v for v in E2M1 if v > 0]
    mids = [(a + b) / 2 for a, b in zip(E2M1, E2M1[1:])]

    def sweep(S, limit=None):
        vals = [g * S for g in grid] + [m * S for m in mids]
        for m in mids:
            vals += _neighbours(m * S, bf16)
        vals += [0.0, 6.25 * S, 7.5 * S]
        if limit is None:
            vals.append(_below(8.0 * S, bf16))
        else:
            vals = [v for v in vals if v < limit * S] + [_below(limit * S, bf16)]
        assert len(vals) <= 32
        return np.array(vals + [0.0] * (32 - len(vals)))

    sign_alt = np.where(np.arange(32) % 2 == 0, 1.0, -1.0)
    rows = []
    for byte in SWEEP_SCALE_BYTES:
        b = sweep(2.0 ** (byte - 127))
        rows.append(np.concatenate([b, -b, b * sign_alt, b[::-1]]))
    S0 = 2.0 ** -127
    small, tiny = sweep(S0, 4.0), sweep(S0, 2.0)
    mixed = [_below(2.0 ** -125, bf16), 1.5 * 2.0 ** -126, 3 * 2.0 ** -128, -(2.0 ** -128),
             _below(2.0 ** -126, bf16), -1.25 * 2.0 ** -128]
    mixed = np.array(mixed + [0.0] * (32 - len(mixed)))
    flip = np.where(np.arange(32) % 3 == 0, -1.0, 1.0)
    rows.append(np.concatenate([small, -tiny, mixed, small * flip]))
    x = np.array(rows, np.float64)
    f = x.astype(np.float32)
    assert np.array_equal(f.astype(np.float64), x)
    if bf16:
        assert ((f.view(np.uint32) & 0xFFFF) == 0).all(), "sweep value not a bf16 value"
    return x


# ---------------------------------------------------------------- pins
def pin_e2m1_table(o):
    """The 16 code values are the E2M1 magnitudes with the sign bit."""
    for c in range(16):
        want = E2M1[c & 7] * (-1.0 if c & 8 else 1.0)
        got = o.e2m1_value(c)
        assert got == want and math.copysign(1, got) == math.copysign(1, want), (c, got)


def pin_encode_boundaries(o):
    """Every grid point, every midpoint and one ulp either side of each, both
    signs, plus values beyond saturation, against brute force."""
    ys = set(E2M1)
    for a, b in zip(E2M1, E2M1[1:]):
        mid = (a + b) / 2
        ys.update([mid, math.nextafter(mid, 0), math.nextafter(mid, 10)])
        ys.update([float(np.nextafter(np.float32(mid), np.float32(0))),
                   float(np.nextafter(np.float32(mid), np.float32(10)))])
    ys.update([6.5, 7.0, 7.99, 1e-30, 0.0])
    for y in sorted(ys):
        for s in (1.0, -1.0):
            v = s * y
            assert o.e2m1_encode(v) == brute_code(v), (v, o.e2m1_encode(v), brute_code(v))


def pin_block_exponent(o):
    """e = floor(log2 amax) - 2 by construction amax = f * 2^j, against
    counting, including both clamps and zero."""
    assert o.block_exponent(0.0) == -127
    for j in range(-149, 128):
        for f in (1.0, 1.5, 1.9999999):
            amax = f * 2.0 ** j
            want = max(-127, min(127, j - 2))
            assert o.block_exponent(amax) == want == brute_exponent(amax), (amax, j)


def pin_scale_byte_sweep(o):
    """The RFQ quantizer (primary and residual) at the scale bytes of
    SWEEP_SCALE_BYTES, the lower clamp and subnormal elements included, fp32
    and bf16 values, against brute force: exponent by counting, nearest grid
    point by exhaustive comparison, residual x - deq(q) exact in Python."""
    for bf16 in (False, True):
        x = scale_sweep_blocks(bf16)
        qc, qs, rc, rs = o.quantize(x)
        want_bytes = list(SWEEP_SCALE_BYTES) + [0]
        for i in range(x.shape[0]):
            for b in range(x.shape[1] // 32):
                blk = [float(v) for v in x[i, 32 * b:32 * b + 32]]
                codes, byte = brute_block(blk)
                assert byte == qs[i, b] and (b != 0 or byte == want_bytes[i]), (i, b, byte)
                assert pack(codes) == bytes(qc[i, 16 * b:16 * b + 16]), (bf16, i, b)
                scale = 2.0 ** (byte - 127)
                res = [v - (-1.0 if c & 8 else 1.0) * E2M1[c & 7] * scale
                       for v, c in zip(blk, codes)]
                rcodes, rbyte = brute_block(res)
                assert rbyte == rs[i, b], (bf16, i, b, rbyte, rs[i, b])
                assert pack(rcodes) == bytes(rc[i, 16 * b:16 * b + 16]), (bf16, i, b)
        # The clamped row really is clamped and still has nonzero codes.
        assert x[-1].max() < 2.0 ** -125 and qc[-1].any() and rc[-1].any()


def _check_golden_block(o, name):
    g = read_golden(name)
    x = padded_floats(g["x"])
    if "x" in g and len(g["x"]) == 1 and g["x"][0] in ("0", "-0"):
        x = np.full(32, float(g["x"][0]))
    qc, qs, rc, rs = o.quantize(x[None, :])
    assert qs[0, 0] == int(g["q_scale"][0], 16), (name, "q_scale", hex(qs[0, 0]))
    assert bytes(qc[0]) == bytes(padded_bytes(g["q_codes"])), (name, "q_codes", qc[0])
    assert rs[0, 0] == int(g["r_scale"][0], 16), (name, "r_scale", hex(rs[0, 0]))
    assert bytes(rc[0]) == bytes(padded_bytes(g["r_codes"])), (name, "r_codes", rc[0])
    recon = o.dequant(qc, qs) + o.dequant(rc, rs)
    want = padded_floats(g["recon"]) if len(g["recon"]) > 1 else np.zeros(32)
    assert np.array_equal(recon[0], want), (name, recon[0])


def pin_golden_h1(o):
    _check_golden_block(o, "h1_mixed_block.txt")


def pin_golden_h2(o):
    _check_golden_block(o, "h2_outlier_block.txt")


def pin_golden_h3(o):
    _check_golden_block(o, "h3_representable_block.txt")


def pin_golden_h4(o):
    _check_golden_block(o, "h4_zero_blocks.txt")
    _check_golden_block(o, "h4_negative_zero_block.txt")


def pin_golden_h5_identity_gemm(o):
    g = read_golden("h5_identity_weight.txt")
    x = padded_floats(g["x"])[None, :]
    qc, qs, rc, rs = o.quantize(x)
    wc, ws, _, _ = o.quantize(np.eye(32), residual=False)
    assert np.all(ws == int(g["w_scale"][0], 16))
    z, _ = o.gemm(qc, qs, rc, rs, wc, ws)
    assert np.array_equal(z[0], padded_floats(g["z_rfq"])), z[0]
    z0, _ = o.gemm(qc, qs, None, None, wc, ws)
    assert np.array_equal(z0[0], padded_floats(g["z_plain"])), z0[0]


def _random_blocks(seed, n=400):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((n, 32))
    x *= np.exp2(rng.integers(-20, 20, (n, 1)))
    x[::7, rng.integers(0, 32)] *= 60.0                    # outliers
    x[::11] = np.round(x[::11] * 4) / 4                     # coarse values
    x[::13, ::3] = 0.0                                      # zeros
    return x.astype(np.float32).astype(np.float64)


def pin_brute_force_blocks(o):
    """Random blocks (fp32 values) quantized by brute force in pure Python."""
    x = _random_blocks(1, 300)
    qc, qs, rc, rs = o.quantize(x)
    for i in range(x.shape[0]):
        codes, sb = brute_block(list(x[i]))
        assert qs[i, 0] == sb, (i, qs[i, 0], sb)
        assert bytes(qc[i]) == pack(codes), i
        deq = [E2M1[c & 7] * (-1 if c & 8 else 1) * 2.0 ** (sb - 127) for c in codes]
        res = [a - b for a, b in zip(x[i], deq)]
        rcodes, rsb = brute_block(res)
        assert rs[i, 0] == rsb, (i, rs[i, 0], rsb)
        assert bytes(rc[i]) == pack(rcodes), i


def pin_dequant_independent(o):
    """Oracle dequant equals the literal-table decode written here."""
    x = _random_blocks(2, 200).reshape(50, 128)
    qc, qs, rc, rs = o.quantize(x)
    assert np.array_equal(o.dequant(qc, qs), decode_codes(qc, qs))
    assert np.array_equal(o.dequant(rc, rs), decode_codes(rc, rs))


def pin_zero_residual_on_grid(o):
    """I1: blocks made of grid values times 2^e, with the block maximum 4 or 6,
    reproduce exactly and leave an all-zero residual."""
    rng = np.random.default_rng(3)
    for t in range(200):
        e = int(rng.integers(-100, 100))
        mags = rng.choice(E2M1, 32)
        mags[rng.integers(0, 32)] = rng.choice([4.0, 6.0])
        x = (mags * rng.choice([-1.0, 1.0], 32) * 2.0 ** e)[None, :]
        qc, qs, rc, rs = o.quantize(x)
        assert qs[0, 0] == e + 127
        assert np.array_equal(o.dequant(qc, qs), x)
        assert rs[0, 0] == 0 and not rc.any()


def pin_power_of_two_equivariance(o):
    """I2: scaling a block by 2^j shifts both scale bytes by j and keeps every
    code (no clamp in range)."""
    x = _random_blocks(4, 200)
    qc, qs, rc, rs = o.quantize(x)
    ok = (qs.astype(int) > 40) & (qs.astype(int) < 200) & (rs.astype(int) > 40) & (rs.astype(int) < 200)
    for j in (-7, -1, 1, 13):
        qc2, qs2, rc2, rs2 = o.quantize(x * 2.0 ** j)
        sel = ok[:, 0]
        assert np.array_equal(qc2[sel], qc[sel]) and np.array_equal(rc2[sel], rc[sel])
        assert np.array_equal(qs2[sel].astype(int), qs[sel].astype(int) + j)
        assert np.array_equal(rs2[sel].astype(int), rs[sel].astype(int) + j)


def pin_idempotence(o):
    """I3: quantizing the dequantized code gives the same code back, and its
    residual is zero."""
    x = _random_blocks(5, 300)
    qc, qs, _, _ = o.quantize(x)
    d = o.dequant(qc, qs)
    qc2, qs2, rc2, rs2 = o.quantize(d)
    assert np.array_equal(qc2, qc) and np.array_equal(qs2, qs)
    assert not rc2.any()


def pin_negation(o):
    """I4: deq Q(-x) = -deq Q(x) for both stages."""
    x = _random_blocks(6, 300)
    a = o.quantize(x)
    b = o.quantize(-x)
    assert np.array_equal(o.dequant(b[0], b[1]), -o.dequant(a[0], a[1]))
    assert np.array_equal(o.dequant(b[2], b[3]), -o.dequant(a[2], a[3]))


def pin_residual_improves(o):
    """I5 and I6: the two-stage error never exceeds the one-stage error, and
    per block it is at most half of the largest one-stage error (blocks whose
    residual scale is not clamped)."""
    x = _random_blocks(7, 400)
    qc, qs, rc, rs = o.quantize(x)
    q = o.dequant(qc, qs)
    r = o.dequant(rc, rs)
    e1 = np.abs(x - q)
    e2 = np.abs(x - (q + r))
    assert np.all(e2 <= e1)
    unclamped = rs[:, 0] > 0
    assert np.all(e2.max(axis=1)[unclamped] <= 0.5 * e1.max(axis=1)[unclamped])
    # and the residual is exactly x - deq(q)
    assert np.array_equal(o.residual(x), x - q)


def pin_gemm_bruteforce(o):
    """Eq. 11 on small shapes against numpy fp64 products of values decoded
    here; also the phi = 0 product and linearity in the residual term."""
    rng = np.random.default_rng(8)
    for (M, N, K) in ((3, 5, 32), (7, 9, 96), (16, 16, 256)):
        x = rng.standard_normal((M, K))
        x[:, rng.integers(0, K)] *= 40
        w = rng.normal(0, 0.02, (N, K))
        qc, qs, rc, rs = o.quantize(x)
        wc, ws, _, _ = o.quantize(w, residual=False)
        dq, dr, dw = decode_codes(qc, qs), decode_codes(rc, rs), decode_codes(wc, ws)
        z, bound = o.gemm(qc, qs, rc, rs, wc, ws)
        want = dq @ dw.T + dr @ dw.T
        assert np.all(np.abs(z - want) <= 1e-12 * bound + 1e-300), (M, N, K)
        assert np.allclose(bound, np.abs(dq) @ np.abs(dw).T + np.abs(dr) @ np.abs(dw).T,
                           rtol=1e-12, atol=0)
        z0, _ = o.gemm(qc, qs, None, None, wc, ws)
        assert np.all(np.abs(z0 - dq @ dw.T) <= 1e-12 * bound + 1e-300)
        zs, bs = o.gemm_sampled(qc, qs, rc, rs, wc, ws, [0, M - 1, M // 2], [N - 1, 0, N // 2])
        assert np.array_equal(zs, z[[0, M - 1, M // 2], [N - 1, 0, N // 2]])


def pin_rfq_beats_mxfp4(o):
    """On outlier-bearing activations the RFQ product is closer to the exact
    product than plain MXFP4 (the accuracy claim of Sec. 4.3)."""
    rng = np.random.default_rng(9)
    x = rng.standard_normal((32, 256))
    x[:, rng.choice(256, 4, replace=False)] *= 50
    w = rng.normal(0, 0.02, (64, 256))
    qc, qs, rc, rs = o.quantize(x)
    wc, ws, _, _ = o.quantize(w, residual=False)
    exact = x @ decode_codes(wc, ws).T
    z1, _ = o.gemm(qc, qs, rc, rs, wc, ws)
    z0, _ = o.gemm(qc, qs, None, None, wc, ws)
    e_rfq = np.linalg.norm(z1 - exact)
    e_mx = np.linalg.norm(z0 - exact)
    assert e_rfq < 0.25 * e_mx, (e_rfq, e_mx)


def pin_round_bf16(o):
    """bf16 rounding: ties to even, above-tie rounds up, subnormal grid 2^-133,
    overflow to infinity."""
    cases = [
        (1.0 + 2.0 ** -8, 1.0),
        (1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -6),
        (1.0 + 2.0 ** -8 + 2.0 ** -30, 1.0 + 2.0 ** -7),
        (-(1.0 + 2.0 ** -8 + 2.0 ** -30), -(1.0 + 2.0 ** -7)),
        (1.5 * 2.0 ** -133, 2.0 ** -132),
        (0.5 * 2.0 ** -133, 0.0),
        (3.0, 3.0),
        ((2.0 - 2.0 ** -7) * 2.0 ** 127, (2.0 - 2.0 ** -7) * 2.0 ** 127),
        ((2.0 - 2.0 ** -9) * 2.0 ** 127, math.inf),
        (0.1, 0.10009765625),
    ]
    for v, want in cases:
        assert o.round_bf16(v) == want, (v, o.round_bf16(v), want)


def pin_swiglu_closed_forms(o):
    """silu(0) = 0; silu(g) - silu(-g) = g; u = 0 gives 0; large g gives g*u;
    every output is a bf16 value within half a bf16 ulp of the exact one."""
    g = np.array([0.0, 1.0, -1.0, 2.5, -2.5, 30.0, -30.0, 0.125, 3.0])
    u = np.array([1.0, 1.0, 1.0, 1.0, 1.0, 2.0, 2.0, 0.0, 1.0])
    h = o.swiglu(g, u)
    assert h[0] == 0.0 and h[7] == 0.0
    assert h[5] == 60.0 and abs(h[6]) < 1e-10
    s1 = 1.0 / (1.0 + math.exp(-1.0))
    exact = [0, s1, -(1 - s1), 2.5 / (1 + math.exp(-2.5)), -2.5 / (1 + math.exp(2.5))]
    for i, e in enumerate(exact):
        assert abs(h[i] - e) <= 0.5 * bf16_ulp(e), (i, h[i], e)
    # h(1) - h(-1) = 1 up to the two roundings
    assert abs((h[1] - h[2]) - 1.0) <= bf16_ulp(1.0)
    # outputs are bf16 values
    for v in h:
        if v != 0:
            m, p = math.frexp(v)
            assert (m * 2 ** 8) == int(m * 2 ** 8), v


def pin_gemm_phi_tiles(o):
    """Eq. 11 with a phi map (Algorithm 1's phi(p, r) over tiles of 64 rows
    by 256 reduction columns): brute force from values decoded here, for
    random maps on shapes with ragged tiles; phi = 1 and phi = 0 reduce to the
    RFQ and the plain products."""
    rng = np.random.default_rng(12)
    for (M, N, K) in ((130, 6, 544), (64, 3, 256), (7, 5, 96)):
        x = rng.standard_normal((M, K))
        x[:, rng.integers(0, K, 3)] *= 30
        w = rng.normal(0, 0.02, (N, K))
        qc, qs, rc, rs = o.quantize(x)
        wc, ws, _, _ = o.quantize(w, residual=False)
        dq, dr, dw = decode_codes(qc, qs), decode_codes(rc, rs), decode_codes(wc, ws)
        pr, pc = (M + 63) // 64, (K + 255) // 256
        for trial in range(4):
            phi = rng.integers(0, 2, (pr, pc)).astype(np.uint8)
            if trial == 0:
                phi[:] = 1
            if trial == 1:
                phi[:] = 0
            mask = np.zeros((M, K))
            for m in range(M):
                for k in range(K):
                    mask[m, k] = phi[m // 64, k // 256]
            z, bound = o.gemm_phi(qc, qs, rc, rs, wc, ws, phi)
            want = dq @ dw.T + (dr * mask) @ dw.T
            assert np.all(np.abs(z - want) <= 1e-12 * bound + 1e-300), (M, N, K, trial)
            if trial == 0:
                assert np.array_equal(z, o.gemm(qc, qs, rc, rs, wc, ws)[0])
            if trial == 1:
                assert np.array_equal(z, o.gemm(qc, qs, None, None, wc, ws)[0])


def pin_fallback_map_rules(o):
    """The two phi rules by brute force over tiles: rule 0 marks tiles with a
    residual code of nonzero magnitude, rule 1 tiles with a primary scale
    byte at least the threshold; on grid-valued rows the residual is zero, so
    rule 0 leaves their tiles off, and phi from rule 0 gives exactly the
    phi = 1 product."""
    rng = np.random.default_rng(13)
    M, K = 150, 800
    x = rng.standard_normal((M, K))
    # Rows 64..127 hold E2M1 grid values only: their residual is exactly zero.
    grid = np.array([0, 0.5, 1, 1.5, 2, 3, 4, 6])
    x[64:128] = rng.choice(grid, (64, K)) * rng.choice([-1, 1], (64, K))
    x[:64, 700] *= 100
    x[128:, 700] *= 100
    qc, qs, rc, rs = o.quantize(x)
    top00 = int(qs[:64, :8].max())          # a threshold met with equality by tile (0, 0)
    for rule, thr in ((0, 0), (1, int(np.median(qs)) + 3), (1, top00), (1, 255), (1, 0)):
        phi = o.fallback_map(rc, qs, rule, thr)
        assert phi.shape == ((M + 63) // 64, (K + 255) // 256)
        for p in range(phi.shape[0]):
            for c in range(phi.shape[1]):
                rows = slice(64 * p, min(64 * p + 64, M))
                if rule == 0:
                    nib = np.stack([rc[rows] & 15, rc[rows] >> 4], -1).reshape(
                        rc[rows].shape[0], K)[:, 256 * c:256 * c + 256]
                    want = bool(np.any(nib & 7))
                else:
                    want = bool(np.any(qs[rows, 8 * c:8 * c + 8] >= thr))
                assert phi[p, c] == want, (rule, thr, p, c)
    phi = o.fallback_map(rc, qs, 0)
    assert not phi[1].any() and phi[0].all()
    w = rng.normal(0, 0.02, (4, K))
    wc, ws, _, _ = o.quantize(w, residual=False)
    assert np.array_equal(o.gemm_phi(qc, qs, rc, rs, wc, ws, phi)[0],
                          o.gemm(qc, qs, rc, rs, wc, ws)[0])


# -------------------------------------------------------------------- HiF4
def hif4_macro_py(byte):
    """E6M2 macro scale (Eq. 5): exponent field bias 48, two mantissa bits."""
    return (1.0 + (byte & 3) / 4.0) * 2.0 ** ((byte >> 2) - 48)


def hif4_decode_py(codes, meta):
    """Independent Eq. 6 decode: V_i = S 2^(E1_8[i/8] + E1_16[i/4]) (+-) k/4."""
    codes = np.asarray(codes, np.uint8)
    meta = np.asarray(meta, np.uint64)
    rows, K = codes.shape[0], codes.shape[1] * 2
    nib = np.empty((rows, K), np.int64)
    nib[:, 0::2] = codes & 0x0F
    nib[:, 1::2] = codes >> 4
    i = np.arange(K) % 64
    blk = np.arange(K) // 64
    m = meta[:, blk]                                            # [rows][K]
    s = np.vectorize(hif4_macro_py)((m & 255).astype(np.int64))
    e8 = ((m >> (8 + i // 8).astype(np.uint64)) & 1).astype(np.int64)
    e16 = ((m >> (16 + i // 4).astype(np.uint64)) & 1).astype(np.int64)
    mag = s * np.ldexp((nib & 7) / 4.0, e8 + e16)
    return np.where(nib & 8, -mag, mag)


def _hif4_golden(o, name):
    g = read_golden(name)
    meta = np.array([[int(g["meta"][0], 16)]], np.uint32)
    codes = padded_bytes(g["codes"], 32).reshape(1, 32)
    want = padded_floats(g["values"], 64)
    return g, meta, codes, want


def pin_hif4_golden_decode(o):
    """H6: the decode of Eq. 6 on a block worked by hand (signs of zero too)."""
    _, meta, codes, want = _hif4_golden(o, "h6_hif4_decode.txt")
    for got in (o.hif4_dequant(codes, meta)[0], hif4_decode_py(codes, meta)[0]):
        assert np.array_equal(got, want) and np.array_equal(np.signbit(got), np.signbit(want))
    for i in (0, 4, 20, 63):
        c = (codes[0, i // 2] >> (4 * (i & 1))) & 15
        assert o.hif4_value(int(meta[0, 0]), i, int(c)) == want[i]


def pin_hif4_golden_encode(o):
    """H7: one block encoded by hand under the library's reading."""
    g, meta, codes, want = _hif4_golden(o, "h7_hif4_encode.txt")
    x = padded_floats(g["x"], 64).reshape(1, 64)
    qc, qm, _, _ = o.hif4_quantize(x, residual=False)
    assert int(qm[0, 0]) == int(meta[0, 0]), hex(int(qm[0, 0]))
    assert np.array_equal(qc, codes), qc
    got = o.hif4_dequant(qc, qm)[0]
    assert np.array_equal(got, want) and np.array_equal(np.signbit(got), np.signbit(want))


def pin_hif4_macro_scale_brute_force(o):
    """Reading 1: the macro byte is the smallest of the 256 E6M2 values S with
    7 S >= amax (exhaustive), values ordered with the byte."""
    vals = [hif4_macro_py(b) for b in range(256)]
    assert all(vals[b] < vals[b + 1] for b in range(255))
    for b in range(256):
        assert o.hif4_macro_value(b) == vals[b]
    rng = np.random.default_rng(41)
    amaxes = list(rng.lognormal(0, 8, 2000)) + [0.0, 1e-30, 7 * vals[0], 7 * vals[0] * 1.01,
                                                7 * vals[255], 7 * vals[255] * 2, 1e30]
    amaxes += [7 * v for v in vals[::5]] + [np.nextafter(7 * v, np.inf) for v in vals[::7]]
    for a in amaxes:
        want = next((b for b in range(256) if 7 * vals[b] >= a), 255)
        assert o.hif4_macro_byte(a) == want, (a, want)


def _hif4_blocks(seed, n):
    """Blocks with varied spreads, outliers, zeros, exact ties and negative
    zeros, for the brute-force pins."""
    rng = np.random.default_rng(seed)
    xs = []
    for t in range(n):
        x = rng.standard_normal(64) * np.exp(rng.uniform(-6, 6))
        if t % 3 == 0:
            x[rng.integers(0, 64, 3)] *= rng.uniform(5, 60)
        if t % 4 == 1:
            x[rng.integers(0, 64, 20)] = 0.0
        if t % 5 == 2:
            x[rng.integers(0, 64, 5)] = -0.0
        xs.append(x)
    # Blocks whose elements sit exactly on midpoints of their encoding grid.
    for t in range(n // 4):
        s = hif4_macro_py(int(rng.integers(150, 210)))
        e = rng.integers(0, 3, 16)
        k = rng.integers(0, 7, 64)
        x = (2 * k + 1) / 8.0 * s * 2.0 ** np.repeat(e, 4) * rng.choice([-1.0, 1.0], 64)
        x[0] = 7 * s * rng.choice([-1.0, 1.0])
        xs.append(x)
    return np.array(xs)


def pin_hif4_encode_brute_force(o):
    """Readings 1-3 by their defining properties, exhaustively: the macro
    scale is the smallest with 7 S >= amax; per 8-element group, among the
    eight settings of (E1_8, E1_16a, E1_16b) that saturate no element, the
    one with the smallest total exponent, E1_8 = 0 on a tie; each element the
    nearest of the eight grid values (ties to even k), sign kept."""
    x = _hif4_blocks(43, 240)
    qc, qm, _, _ = o.hif4_quantize(x, residual=False)
    vals = [hif4_macro_py(b) for b in range(256)]
    for r in range(x.shape[0]):
        xb = x[r]
        amax = np.abs(xb).max()
        sb = next((b for b in range(256) if 7 * vals[b] >= amax), 255)
        meta = int(qm[r, 0])
        assert meta & 255 == sb, (r, meta & 255, sb)
        s = vals[sb]
        gmax = np.abs(xb).reshape(16, 4).max(1)
        for g in range(8):
            best = None
            for e8 in (0, 1):
                for ea in (0, 1):
                    for eb in (0, 1):
                        ta, tb = e8 + ea, e8 + eb
                        if 1.75 * s * 2 ** ta < gmax[2 * g] or 1.75 * s * 2 ** tb < gmax[2 * g + 1]:
                            continue
                        key = (ta + tb, e8)
                        if best is None or key < best[0]:
                            best = (key, e8, ea, eb)
            _, e8, ea, eb = best
            assert (meta >> (8 + g)) & 1 == e8, (r, g)
            assert (meta >> (16 + 2 * g)) & 1 == ea and (meta >> (17 + 2 * g)) & 1 == eb, (r, g)
        for i in range(64):
            c = (int(qc[r, i // 2]) >> (4 * (i & 1))) & 15
            e = ((meta >> (8 + i // 8)) & 1) + ((meta >> (16 + i // 4)) & 1)
            u = s * 2.0 ** e
            d = [abs(abs(xb[i]) - k / 4.0 * u) for k in range(8)]
            best = min(d)
            ks = [k for k in range(8) if d[k] == best]
            k_want = ks[0] if len(ks) == 1 else [k for k in ks if k % 2 == 0][0]
            assert c & 7 == k_want, (r, i, xb[i], c, k_want)
            assert bool(c & 8) == bool(np.signbit(xb[i])), (r, i)


def pin_hif4_residual(o):
    """RFQ with HiF4 (Eq. 9-10): the residual x - V is exact in fp32 for fp32
    inputs, and its quantized form never moves an element away from x:
    |x - V - Vr| <= |x - V| (zero is on the grid and rounding is to nearest)."""
    x = _hif4_blocks(47, 120).astype(np.float32).astype(np.float64)
    qc, qm, rc, rm = o.hif4_quantize(x)
    v = hif4_decode_py(qc, qm.reshape(-1, 1))
    vr = hif4_decode_py(rc, rm.reshape(-1, 1))
    r64 = x - v
    r32 = (x.astype(np.float32) - v.astype(np.float32)).astype(np.float64)
    assert np.array_equal(r32, r64)
    assert np.all(np.abs(x - v - vr) <= np.abs(x - v))
    nz = np.abs(x - v).sum(1) > 0
    assert np.all(np.abs(x - v - vr).sum(1)[nz] < np.abs(x - v).sum(1)[nz])
    rq, rmq, _, _ = o.hif4_quantize(r64, residual=False)
    assert np.array_equal(rq, rc) and np.array_equal(rmq, rm)


def pin_hif4_gemm_brute_force(o):
    """The HiF4 RFQ product against numpy on values decoded here (Eq. 6, 11)."""
    rng = np.random.default_rng(53)
    for M, N, K in ((3, 5, 64), (7, 4, 192), (2, 9, 128)):
        x = rng.standard_normal((M, K)) * np.exp(rng.uniform(-3, 3, (M, 1)))
        w = rng.normal(0, 0.02, (N, K))
        qc, qm, rc, rm = o.hif4_quantize(x)
        wc, wm, _, _ = o.hif4_quantize(w, residual=False)
        z, bound = o.hif4_gemm(qc, qm, rc, rm, wc, wm)
        dq, dr, dw = hif4_decode_py(qc, qm), hif4_decode_py(rc, rm), hif4_decode_py(wc, wm)
        want = dq @ dw.T + dr @ dw.T
        assert np.all(np.abs(z - want) <= 1e-12 * bound + 1e-300), (M, N, K)
        assert np.allclose(bound, np.abs(dq) @ np.abs(dw).T + np.abs(dr) @ np.abs(dw).T,
                           rtol=1e-12, atol=0)
        z0, _ = o.hif4_gemm(qc, qm, None, None, wc, wm)
        assert np.all(np.abs(z0 - dq @ dw.T) <= 1e-12 * bound + 1e-300)


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
