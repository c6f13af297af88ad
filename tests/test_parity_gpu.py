"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Quantizer codes and scales: bit-exact.  Dequantization: exact.  RFQ product:
within the tolerance derived in gpu_util.  The small cases span several
tiles and ragged tails; the full-size cases use the shapes of the synthetic
workloads, with every output checked for the quantizers and sampled outputs
(plus whole rows) for the products.
"""
import numpy as np
import pytest
import torch

import paper_2608_26581_amd as rfq
from paper_2608_26581_amd import workloads as wl
from gpu_util import (assert_gemm_close, dev, dev_bf16, host, host_bf16_as_f32,
                      x_device)
from oracle_pins import (SWEEP_SCALE_BYTES, padded_floats, padded_bytes, read_golden,
                         scale_sweep_blocks)

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def _quant_both(o, data, residual=True, rows=None):
    """GPU and oracle quantization of a workload's activations."""
    x = x_device(data)
    g = [None if t is None else host(t) for t in rfq.rfq_quantize_act(x, residual=residual)]
    torch.cuda.synchronize()
    xr = data["x"] if rows is None else data["x"][rows]
    if rows is not None:
        g = [None if a is None else a[rows] for a in g]
    r = o.quantize(xr, residual=residual)
    return g, r


def _assert_codes_equal(g, r, what):
    names = ("q_codes", "q_scales", "r_codes", "r_scales")
    for n, a, b in zip(names, g, r):
        if b is None:
            assert a is None
            continue
        if not np.array_equal(a, b):
            i = np.argwhere(a != b)[0]
            raise AssertionError("%s %s differ at %s: gpu %#x oracle %#x" %
                                 (what, n, tuple(i), a[tuple(i)], b[tuple(i)]))


# ----------------------------------------------------------------- golden
@pytest.mark.parametrize("name", ["h1_mixed_block.txt", "h2_outlier_block.txt",
                                  "h3_representable_block.txt", "h4_zero_blocks.txt",
                                  "h4_negative_zero_block.txt"])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_golden_blocks(name, dtype):
    g = read_golden(name)
    x = padded_floats(g["x"])
    if len(g["x"]) == 1:
        x = np.full(32, float(g["x"][0]))
    xt = torch.tensor(x, dtype=torch.float32).reshape(1, 32).to(dtype).cuda()
    qc, qs, rc, rs = [host(t) for t in rfq.rfq_quantize_act(xt)]
    assert qs[0, 0] == int(g["q_scale"][0], 16)
    assert bytes(qc[0]) == bytes(padded_bytes(g["q_codes"]))
    assert rs[0, 0] == int(g["r_scale"][0], 16)
    assert bytes(rc[0]) == bytes(padded_bytes(g["r_codes"]))


def test_golden_identity_gemm():
    g = read_golden("h5_identity_weight.txt")
    x = torch.tensor(padded_floats(g["x"]), dtype=torch.float32).reshape(1, 32).cuda()
    q = rfq.rfq_quantize_act(x)
    w = rfq.rfq_quantize_weight(torch.eye(32, dtype=torch.float32).cuda())
    assert np.all(host(w[1]) == int(g["w_scale"][0], 16))
    z = host(rfq.rfq_gemm(*q, *w))
    assert np.array_equal(z[0], padded_floats(g["z_rfq"]).astype(np.float32))
    z0 = host(rfq.rfq_gemm(q[0], q[1], None, None, *w))
    assert np.array_equal(z0[0], padded_floats(g["z_plain"]).astype(np.float32))


# -------------------------------------------------------------- quantizer
QUANT_SMALL = [
    ("tiny", None, None),             # 64 x 256 fp32, full size
    ("quant", 300, 4096),             # ragged row count
    ("qwen", 7, 96),                  # odd number of blocks per row
    ("wan", 129, 5120),
    ("quant", 1, 32),                 # single block
]


@pytest.mark.parametrize("name,M,K", QUANT_SMALL)
@pytest.mark.parametrize("residual", [True, False])
def test_quantize_small(orc, name, M, K, residual):
    w = wl.WORKLOADS[name]
    if M is not None:
        w = w.scaled(M=M, K=K, weights=())
    data = wl.generate(w, seed=11)
    _say("quantize %s M=%d K=%d residual=%s" % (name, w.M, w.K, residual))
    g, r = _quant_both(orc, data, residual)
    _assert_codes_equal(g, r, name)


@pytest.mark.parametrize("name", ["quant", "qwen", "wan"])
def test_quantize_full_size(orc, name):
    data = wl.generate(wl.WORKLOADS[name], seed=0)
    M = data["x"].shape[0]
    rows = None if M <= 8192 else np.arange(0, M, 8)      # wan: every 8th row
    _say("quantize full %s %s" % (name, data["x"].shape))
    g, r = _quant_both(orc, data, True, rows)
    _assert_codes_equal(g, r, name)


def test_quantize_weight_full_size(orc):
    data = wl.generate(wl.WORKLOADS["qwen"], seed=0)
    w = data["w"]
    _say("quantize weight %s" % (w.shape,))
    wc, ws = [host(t) for t in rfq.rfq_quantize_weight(dev(w))]
    rows = np.arange(0, w.shape[0], 3)
    oc, os_, _, _ = orc.quantize(w[rows], residual=False)
    _assert_codes_equal((wc[rows], ws[rows]), (oc, os_), "weight")


def test_quantize_special_values(orc):
    """Subnormal, huge and mixed-sign blocks, fp32 and bf16."""
    rng = np.random.default_rng(5)
    x = rng.standard_normal((16, 128)).astype(np.float32)
    x[0] = 0.0
    x[1] = -0.0
    x[2, :32] = np.float32(1e-39)                          # subnormal block
    x[2, 32:64] = rng.standard_normal(32).astype(np.float32) * np.float32(1e-40)
    x[3, :32] = np.float32(3e38)
    x[3, 32:64] = rng.standard_normal(32).astype(np.float32) * np.float32(1e37)
    x[4] *= np.float32(2.0 ** -120)
    x[5] *= np.float32(2.0 ** 120)
    x[6, 5] = 6.0e4
    for arr in (x, wl.bf16_bits_to_f32(wl.f32_to_bf16_bits(x))):
        for dt in (torch.float32, torch.bfloat16):
            if dt == torch.bfloat16 and arr is x:
                continue
            xt = torch.from_numpy(arr).cuda().to(dt)
            g = [host(t) for t in rfq.rfq_quantize_act(xt)]
            _assert_codes_equal(g, orc.quantize(arr.astype(np.float64)), "special %s" % dt)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_scale_byte_sweep_through_the_converters(orc, dtype):
    """Pins the conventions of the gfx950 scaled FP4 conversions that
    bit-exactness rests on (round to nearest even, saturation at 6, sign of
    zero, the scale operand of every byte) at scale bytes 0, 1, 2, 3, 127,
    200 and 252: every E2M1 grid point, midpoint and fp32 (bf16) neighbour
    of a midpoint, both signs, in blocks whose maximum sets that byte, plus
    clamped blocks at byte 0 (maximum below 2^-125, subnormal elements, and
    nonzero codes in both the primary and the residual stage).  Sec. 3.2
    Eq. 3-4 and Sec. 4.3 Eq. 9-10 through the oracle (itself pinned against
    brute force on the same blocks), bit-exact; dequantization exact; the
    products of these codes within tolerance (byte 0 reaching the scaled
    MFMA as 2^-127), on the general, few-row and large-tile kernels."""
    bf16 = dtype == torch.bfloat16
    x = scale_sweep_blocks(bf16)
    _say("scale byte sweep %s rows %d" % (dtype, x.shape[0]))
    xt = torch.from_numpy(x.astype(np.float32)).cuda().to(dtype)
    g = [host(t) for t in rfq.rfq_quantize_act(xt)]
    ref = orc.quantize(x)
    _assert_codes_equal(g, ref, "sweep %s" % dtype)
    assert g[1][-1].max() == 0 and g[0][-1].any() and g[3][-1].max() == 0 and g[2][-1].any()
    w = [host(t) for t in rfq.rfq_quantize_weight(xt)]
    _assert_codes_equal(w, ref[:2], "sweep weight %s" % dtype)
    for c, sc in ((g[0], g[1]), (g[2], g[3])):
        d = host(rfq.rfq_dequant(dev(c), dev(sc)))
        assert np.array_equal(d.astype(np.float64), orc.dequant(c, sc))

    row_bytes = np.array(list(SWEEP_SCALE_BYTES) + [0])
    rng = np.random.default_rng(31)
    # K = 128: general kernel; 8 rows, K = 512: few-row kernel; 320 rows,
    # K = 512: large-tile kernel.
    for reps, kreps in ((1, 1), (1, 4), (40, 4)):
        xs = np.tile(x, (reps, kreps))
        xst = torch.from_numpy(xs.astype(np.float32)).cuda().to(dtype)
        q = rfq.rfq_quantize_act(xst)
        qh = [host(t) for t in q]
        K = xs.shape[1]
        for j in (100, 0, -100):
            # Weights scaled by 2^j; only rows whose products stay far from
            # fp32 underflow and overflow are compared.
            wv = (rng.standard_normal((96, K)) * 2.0 ** j).astype(np.float32)
            wq = rfq.rfq_quantize_weight(dev(wv))
            _say("sweep product rows=%d K=%d j=%d" % (xs.shape[0], K, j))
            for out_dtype in (torch.float32, torch.bfloat16):
                z = rfq.rfq_gemm(*q, *wq, out_dtype=out_dtype)
                zh = host_bf16_as_f32(z) if out_dtype == torch.bfloat16 else host(z)
                zr, bound = orc.gemm(*qh, host(wq[0]), host(wq[1]))
                ok = np.abs(np.tile(row_bytes, reps) - 127 + j) <= 100
                assert_gemm_close(zh[ok], zr[ok], bound[ok], out_dtype == torch.bfloat16,
                                  "sweep product K=%d j=%d" % (K, j))


@pytest.mark.parametrize("M,K", [(64, 4096), (5, 96), (3, 2080)])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_quantize_unaligned_scale_pointers(orc, M, K, dtype):
    """Scale tensors may start at any byte (only code tensors must be 16-byte
    aligned): outputs at an odd offset equal the oracle's."""
    data = wl.generate(wl.WORKLOADS["quant"].scaled(M=M, K=K, weights=()), seed=21)
    x = torch.from_numpy(data["x"]).cuda().to(dtype)
    xr = data["x"] if dtype == torch.float32 else \
        wl.bf16_bits_to_f32(wl.f32_to_bf16_bits(data["x"]))
    _say("unaligned scales M=%d K=%d %s" % (M, K, dtype))
    raw = [torch.empty(M * K // 32 + 1, dtype=torch.uint8, device="cuda") for _ in range(2)]
    qs, rs = [r[1:].view(M, K // 32) for r in raw]
    qc = torch.empty((M, K // 2), dtype=torch.uint8, device="cuda")
    rc = torch.empty((M, K // 2), dtype=torch.uint8, device="cuda")
    rfq.rfq_quantize_act(x, out=[qc, qs, rc, rs])
    _assert_codes_equal([host(t) for t in (qc, qs, rc, rs)], orc.quantize(xr), "unaligned act")
    wc = torch.empty((M, K // 2), dtype=torch.uint8, device="cuda")
    rfq.rfq_quantize_weight(x, out=[wc, qs])
    o = orc.quantize(xr, residual=False)
    _assert_codes_equal([host(wc), host(qs)], o[:2], "unaligned weight")


def test_power_of_two_equivariance():
    """Metamorphic: scaling X by 2^j keeps every code and shifts every scale
    byte by j; the product scales by exactly 2^j (no oracle involved)."""
    data = wl.generate(wl.WORKLOADS["qwen"].scaled(M=256, K=1024,
                                                  weights=(("w", 1024, 384),)), seed=3)
    x = dev(data["x"])
    w = rfq.rfq_quantize_weight(dev(data["w"]))
    base = rfq.rfq_quantize_act(x)
    z = host(rfq.rfq_gemm(*base, *w))
    for j in (-5, 3):
        sc = rfq.rfq_quantize_act(x * 2.0 ** j)
        assert torch.equal(sc[0], base[0]) and torch.equal(sc[2], base[2])
        assert torch.equal(sc[1].int(), base[1].int() + j)
        assert torch.equal(sc[3].int(), base[3].int() + j)
        zj = host(rfq.rfq_gemm(*sc, *w))
        assert np.array_equal(zj, z * np.float32(2.0 ** j))


def test_determinism():
    data = wl.generate(wl.WORKLOADS["qwen"].scaled(M=512, K=2048,
                                                  weights=(("w", 2048, 1024),)), seed=4)
    x = x_device(data)
    w = rfq.rfq_quantize_weight(dev(data["w"]))
    a = rfq.rfq_quantize_act(x)
    b = rfq.rfq_quantize_act(x)
    for s, t in zip(a, b):
        assert torch.equal(s, t)
    assert torch.equal(rfq.rfq_gemm(*a, *w), rfq.rfq_gemm(*b, *w))


# ---------------------------------------------------------------- dequant
def test_dequant_exact(orc):
    data = wl.generate(wl.WORKLOADS["qwen"].scaled(M=130, K=2080, weights=()), seed=6)
    q = rfq.rfq_quantize_act(x_device(data))
    for c, s in ((q[0], q[1]), (q[2], q[3])):
        d = host(rfq.rfq_dequant(c, s)).astype(np.float64)
        assert np.array_equal(d, orc.dequant(host(c), host(s)))


def test_dequant_all_codes_and_scales(orc):
    codes = np.arange(256, dtype=np.uint8).reshape(16, 16)
    scales = np.array([[0], [1], [2], [60], [120], [126], [127], [128], [129], [130],
                       [200], [250], [252], [253], [254], [127]], np.uint8)
    d = host(rfq.rfq_dequant(dev(codes), dev(scales))).astype(np.float64)
    # fp32 output: values beyond the fp32 range (6 * 2^127) become infinite.
    with np.errstate(over="ignore"):
        want = orc.dequant(codes, scales).astype(np.float32).astype(np.float64)
    assert np.array_equal(d, want)


def test_dequant_beyond_one_grid_pass(orc):
    """More 8-element chunks than one pass of the dequantization grid covers
    (65536 workgroups of 256 lanes): every element is written, exactly."""
    rows, K = 4160, 40960                          # 21.3 M chunks
    gen = torch.Generator(device="cuda").manual_seed(7)
    codes = torch.randint(0, 256, (rows, K // 2), dtype=torch.uint8, device="cuda", generator=gen)
    scales = torch.randint(100, 150, (rows, K // 32), dtype=torch.uint8, device="cuda",
                           generator=gen)
    out = torch.full((rows, K), float("nan"), device="cuda")
    _say("dequant %dx%d (several grid passes)" % (rows, K))
    rfq.rfq_dequant(codes, scales, out=out)
    assert not torch.isnan(out).any()
    wrap_row = 65536 * 256 // (K // 8)             # first row of the second pass
    sel = [0, 1, wrap_row - 1, wrap_row, wrap_row + 1, rows - 1]
    got = host(out[sel]).astype(np.float64)
    assert np.array_equal(got, orc.dequant(host(codes[sel]), host(scales[sel])))


# ---------------------------------------------------------------- product
GEMM_SMALL = [
    ("tiny", 64, 256, 256),
    ("qwen", 200, 328, 1056),       # ragged M and N, K not a multiple of 256
    ("qwen", 129, 257, 512),
    ("qwen", 513, 769, 2048),       # several 256-wide tiles, ragged both ways
    ("wan", 256, 384, 5120),
    ("qwen", 70, 300, 640),         # K a multiple of 128 but not of 512
    ("qwen", 1, 1, 32),
    ("qwen", 3, 130, 96),
    # few activation rows, K a multiple of 512: the skinny kernel
    ("qwen", 1, 300, 512),
    ("qwen", 16, 256, 1024),
    ("qwen", 37, 130, 2048),          # three row slices, ragged
    ("qwen", 65, 33, 1536),           # five row slices in one workgroup row
    ("qwen", 100, 300, 1024),         # two workgroup rows of up to 64 rows
    ("qwen", 128, 260, 512),          # the few-row kernel's largest M
    ("wan", 64, 200, 5120),           # K range split unevenly over the waves
    ("qwen", 5, 1, 512),
    # enough weight rows for 32 per workgroup (16 elsewhere), ragged
    ("qwen", 16, 8200, 512),
    ("qwen", 40, 8200, 512),
    # 64 weight rows per workgroup (5-64 rows at 11264 <= N < 16384, 33-64
    # from N = 16384), one, two and four row slices, ragged
    ("qwen", 9, 12300, 1024),
    ("qwen", 24, 12300, 512),
    ("qwen", 50, 11300, 1024),
    ("qwen", 40, 16400, 512),
    # 32 weight rows per workgroup at up to 4 rows from N = 16384, ragged
    ("qwen", 3, 16400, 512),
    # 65-128 rows with 96 or more 128-wide column tiles: the large-tile kernel
    ("qwen", 100, 12300, 512),
    # long K at a narrow grid (at most one workgroup per CU), ragged N; 4-5
    # groups of 512 per wave at K = 9216
    ("qwen", 3, 1000, 8192),
    ("qwen", 16, 4000, 9216),
]


def _gemm_case(name, M, N, K, seed):
    w = wl.WORKLOADS[name]
    w = w.scaled(M=M, K=K, weights=(("w", K, N),))
    return wl.generate(w, seed=seed)


@pytest.mark.parametrize("name,M,N,K", GEMM_SMALL)
@pytest.mark.parametrize("residual", [True, False])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_gemm_small(orc, name, M, N, K, residual, out_dtype):
    data = _gemm_case(name, M, N, K, seed=M + N + K)
    _say("gemm %s M=%d N=%d K=%d residual=%s out=%s" % (name, M, N, K, residual, out_dtype))
    q = rfq.rfq_quantize_act(x_device(data), residual=residual)
    w = rfq.rfq_quantize_weight(dev(data["w"]))
    z = rfq.rfq_gemm(*q, *w, out_dtype=out_dtype)
    zh = host(z) if out_dtype == torch.float32 else host_bf16_as_f32(z)
    hq = [None if t is None else host(t) for t in q]
    zr, bound = orc.gemm(*hq, host(w[0]), host(w[1]))
    assert_gemm_close(zh, zr, bound, out_dtype == torch.bfloat16, "gemm %s" % name)


def _tile_samples(M, N, T, rng):
    """One output at a random position inside every T x T tile of an M x N
    product (tiles cut at the edges), so that every output tile of the
    product kernels (256 x 256 and 128 x 128) holds a sampled output."""
    tm, tn = np.meshgrid(np.arange(0, M, T), np.arange(0, N, T), indexing="ij")
    tm, tn = tm.ravel(), tn.ravel()
    rows = tm + (rng.random(tm.size) * np.minimum(T, M - tm)).astype(np.int64)
    cols = tn + (rng.random(tn.size) * np.minimum(T, N - tn)).astype(np.int64)
    return rows, cols


@pytest.mark.parametrize("name", ["qwen", "wan"])
def test_gemm_full_size_sampled(orc, name):
    data = wl.generate(wl.WORKLOADS[name], seed=0)
    M, K = data["x"].shape
    N = data["w"].shape[0]
    _say("gemm full %s M=%d N=%d K=%d" % (name, M, N, K))
    q = rfq.rfq_quantize_act(x_device(data))
    w = rfq.rfq_quantize_weight(dev(data["w"]))
    z32 = host(rfq.rfq_gemm(*q, *w))
    zbf = host_bf16_as_f32(rfq.rfq_gemm(*q, *w, out_dtype=torch.bfloat16))
    hq = [host(t) for t in q]
    hw = [host(t) for t in w]
    rng = np.random.default_rng(1)
    tr, tc = _tile_samples(M, N, 128, rng)
    rows = np.concatenate([rng.integers(0, M, 4000), np.repeat([0, M - 1], N), tr])
    cols = np.concatenate([rng.integers(0, N, 4000), np.tile(np.arange(N), 2), tc])
    zr, bound = orc.gemm_sampled(*hq, *hw, rows, cols)
    assert_gemm_close(z32[rows, cols], zr, bound, False, "full fp32")
    assert_gemm_close(zbf[rows, cols], zr, bound, True, "full bf16")


def _gemm_bits(z):
    return z.view(torch.int16) if z.dtype == torch.bfloat16 else z.view(torch.int32)


@pytest.mark.parametrize("residual", [True, False])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_gemm_tile_shapes_agree(orc, residual, out_dtype):
    """The large-tile product runs 256 x 256 tiles, or 128 x 128 ones while
    those number fewer than 512.  1300 x 6500 (ragged both ways, 8 stages,
    two scale groups) takes the 256-wide tiles: sampled against the oracle in
    every 64 x 64 tile, the last row and the last column in full.  Row and
    column slices of the same operands take the 128-wide tiles and must give
    the same bits (rows and columns are independent; both tile shapes
    accumulate each output in the same order)."""
    M, N, K = 1300, 6500, 1024
    data = _gemm_case("qwen", M, N, K, seed=77)
    _say("gemm tile shapes M=%d N=%d K=%d residual=%s out=%s" % (M, N, K, residual, out_dtype))
    q = rfq.rfq_quantize_act(x_device(data), residual=residual)
    w = rfq.rfq_quantize_weight(dev(data["w"]))
    z = rfq.rfq_gemm(*q, *w, out_dtype=out_dtype)
    zh = host(z) if out_dtype == torch.float32 else host_bf16_as_f32(z)
    rng = np.random.default_rng(5)
    tr, tc = _tile_samples(M, N, 64, rng)
    rows = np.concatenate([tr, np.full(N, M - 1), np.arange(M)])
    cols = np.concatenate([tc, np.arange(N), np.full(M, N - 1)])
    hq = [None if t is None else host(t) for t in q]
    zr, bound = orc.gemm_sampled(*hq, host(w[0]), host(w[1]), rows, cols)
    assert_gemm_close(zh[rows, cols], zr, bound, out_dtype == torch.bfloat16, "256-wide tiles")
    for a, b in ((0, 300), (1000, 1300), (129, 387)):
        qs = [None if t is None else t[a:b] for t in q]
        zs = rfq.rfq_gemm(*qs, *w, out_dtype=out_dtype)
        assert torch.equal(_gemm_bits(zs), _gemm_bits(z[a:b])), "rows %d:%d" % (a, b)
    for a, b in ((0, 1000), (5500, 6500)):
        zs = rfq.rfq_gemm(*q, w[0][a:b], w[1][a:b], out_dtype=out_dtype)
        assert torch.equal(_gemm_bits(zs), _gemm_bits(z[:, a:b].contiguous())), "cols %d:%d" % (a, b)


@pytest.mark.parametrize("residual", [True, False])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_gemm_last_round_peeled(orc, residual, out_dtype):
    """1400 x 11000 has 6 x 43 = 258 tiles of 256 x 256, two past a round of
    256: the tile rows of that last round (rows 1280-1399) run 128 x 128
    tiles in a second launch.  Sampled against the oracle in every 64 x 64
    tile, the last row and the last column; the 256-wide rows and the peeled
    rows give the bits of products of those rows alone (256-wide tiles for
    rows 0-1279, 128-wide ones for rows 1152-1399)."""
    M, N, K = 1400, 11000, 512
    data = _gemm_case("qwen", M, N, K, seed=78)
    _say("gemm peeled last round M=%d N=%d K=%d residual=%s out=%s" % (M, N, K, residual, out_dtype))
    q = rfq.rfq_quantize_act(x_device(data), residual=residual)
    w = rfq.rfq_quantize_weight(dev(data["w"]))
    z = rfq.rfq_gemm(*q, *w, out_dtype=out_dtype)
    zh = host(z) if out_dtype == torch.float32 else host_bf16_as_f32(z)
    rng = np.random.default_rng(6)
    tr, tc = _tile_samples(M, N, 64, rng)
    rows = np.concatenate([tr, np.full(N, M - 1), np.arange(M)])
    cols = np.concatenate([tc, np.arange(N), np.full(M, N - 1)])
    hq = [None if t is None else host(t) for t in q]
    zr, bound = orc.gemm_sampled(*hq, host(w[0]), host(w[1]), rows, cols)
    assert_gemm_close(zh[rows, cols], zr, bound, out_dtype == torch.bfloat16, "peeled product")
    for a, b in ((0, 1280), (1152, 1400)):
        qs = [None if t is None else t[a:b] for t in q]
        zs = rfq.rfq_gemm(*qs, *w, out_dtype=out_dtype)
        assert torch.equal(_gemm_bits(zs), _gemm_bits(z[a:b])), "rows %d:%d" % (a, b)


@pytest.mark.parametrize("M,N,K", [(256, 12288, 4096), (300, 4096, 12288), (129, 12288, 4096)])
def test_gemm_mid_rows_full_width(orc, M, N, K):
    """Between 129 and a few hundred activation rows at the workloads' weight
    shapes (128 x 128 tiles), sampled in every 64 x 64 output tile, plus the
    first and last rows in full."""
    data = _gemm_case("qwen", M, N, K, seed=M + 3)
    _say("gemm mid rows M=%d N=%d K=%d" % (M, N, K))
    q = rfq.rfq_quantize_act(x_device(data))
    w = rfq.rfq_quantize_weight(dev(data["w"]))
    z32 = host(rfq.rfq_gemm(*q, *w))
    zbf = host_bf16_as_f32(rfq.rfq_gemm(*q, *w, out_dtype=torch.bfloat16))
    rng = np.random.default_rng(M)
    tr, tc = _tile_samples(M, N, 64, rng)
    rows = np.concatenate([tr, np.repeat([0, M - 1], N)])
    cols = np.concatenate([tc, np.tile(np.arange(N), 2)])
    zr, bound = orc.gemm_sampled(*[host(t) for t in q], *[host(t) for t in w], rows, cols)
    assert_gemm_close(z32[rows, cols], zr, bound, False, "mid rows fp32")
    assert_gemm_close(zbf[rows, cols], zr, bound, True, "mid rows bf16")


# 6 tiles of 128 x 128 or fewer: 8 parts; K = 8192 (8 parts of 1024), 8704
# (parts of 1536 and a last one of 1024), 9216 at a ragged shape, 2560 (5
# parts of 512) with 40 rows (past the few-row kernel's range in the split
# product); M x N not a multiple of 4 for the scalar sum.
SPLIT = [(130, 300, 8192), (131, 301, 8704), (200, 257, 9216), (40, 300, 2560),
         (5, 5000, 12288), (16, 4900, 12800)]    # few-row kernel, K in 3 parts


@pytest.mark.parametrize("M,N,K", SPLIT)
@pytest.mark.parametrize("residual", [True, False])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_gemm_split_matches_oracle(orc, M, N, K, residual, out_dtype):
    """K split over workgroups: every output against the oracle; with a
    workspace one byte short of the plan's it runs unsplit and gives
    rfq_gemm's bits."""
    data = _gemm_case("qwen", M, N, K, seed=K + M)
    _say("gemm split M=%d N=%d K=%d residual=%s out=%s" % (M, N, K, residual, out_dtype))
    q = rfq.rfq_quantize_act(x_device(data), residual=residual)
    w = rfq.rfq_quantize_weight(dev(data["w"]))
    nbytes = rfq.rfq_gemm_workspace_bytes(M, N, K)
    assert nbytes > 0
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    z = rfq.rfq_gemm_split(*q, *w, ws, out_dtype=out_dtype)
    zh = host(z) if out_dtype == torch.float32 else host_bf16_as_f32(z)
    hq = [None if t is None else host(t) for t in q]
    zr, bound = orc.gemm(*hq, host(w[0]), host(w[1]))
    assert_gemm_close(zh, zr, bound, out_dtype == torch.bfloat16, "gemm split")
    short = rfq.rfq_gemm_split(*q, *w, ws[:nbytes - 16], out_dtype=out_dtype)
    assert torch.equal(_gemm_bits(short), _gemm_bits(rfq.rfq_gemm(*q, *w, out_dtype=out_dtype)))


@pytest.mark.parametrize("M,N,K", [(256, 4096, 12288), (129, 5120, 13824), (100, 12288, 12288),
                                   (64, 4096, 12288), (100, 12288, 4096), (24, 4096, 12288),
                                   (20, 5120, 13824), (16, 5120, 13824), (1, 5120, 13824)])
def test_gemm_split_full_width(orc, M, N, K):
    """Down-projection and wide shapes with few activation rows (K split in
    4, 3, 2, 8, 2, 8 and 6 parts over 128-wide tiles, and in 3 parts by the
    few-row kernel at 16 and 1 rows x 5120), sampled in every 64 x 64 output
    tile plus the last row and column in full."""
    data = _gemm_case("qwen", M, N, K, seed=M + 5)
    _say("gemm split full M=%d N=%d K=%d" % (M, N, K))
    q = rfq.rfq_quantize_act(x_device(data))
    w = rfq.rfq_quantize_weight(dev(data["w"]))
    assert rfq.rfq_gemm_workspace_bytes(M, N, K) > 0
    z32 = host(rfq.rfq_gemm(*q, *w, split=True))
    zbf = host_bf16_as_f32(rfq.rfq_gemm(*q, *w, out_dtype=torch.bfloat16, split=True))
    rng = np.random.default_rng(M)
    tr, tc = _tile_samples(M, N, 64, rng)
    rows = np.concatenate([tr, np.full(N, M - 1), np.arange(M)])
    cols = np.concatenate([tc, np.arange(N), np.full(M, N - 1)])
    zr, bound = orc.gemm_sampled(*[host(t) for t in q], *[host(t) for t in w], rows, cols)
    assert_gemm_close(z32[rows, cols], zr, bound, False, "split fp32")
    assert_gemm_close(zbf[rows, cols], zr, bound, True, "split bf16")


# ---------------------------------------------------- streaming form
STREAM = [
    ("qwen", 1, 300, 512),
    ("qwen", 16, 256, 1024),
    ("qwen", 37, 130, 2048),
    ("wan", 64, 200, 5120),
    ("qwen", 100, 97, 512),           # two workgroup rows, the second ragged
    ("qwen", 150, 97, 1024),          # more rows than the codes path's few-row kernel
    ("qwen", 24, 12300, 512),         # 64 weight rows per workgroup, ragged
]


@pytest.mark.parametrize("name,M,N,K", STREAM)
@pytest.mark.parametrize("xdt", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("residual", [True, False])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_gemm_stream_matches_oracle(orc, name, M, N, K, xdt, residual, out_dtype):
    """The activations quantized inside the product give the oracle's product
    of the oracle's codes of X, within the product's tolerance."""
    data = _gemm_case(name, M, N, K, seed=3 * M + N + K)
    xr = data["x"] if xdt == torch.float32 else wl.bf16_bits_to_f32(data["x_bf16"])
    x = dev(data["x"]) if xdt == torch.float32 else dev_bf16(data["x_bf16"])
    _say("gemm_stream %s M=%d N=%d K=%d x=%s residual=%s out=%s" %
         (name, M, N, K, xdt, residual, out_dtype))
    w = rfq.rfq_quantize_weight(dev(data["w"]))
    z = rfq.rfq_gemm_stream(x, *w, residual=residual, out_dtype=out_dtype)
    zh = host(z) if out_dtype == torch.float32 else host_bf16_as_f32(z)
    oq = orc.quantize(xr, residual=residual)
    zr, bound = orc.gemm(*oq, host(w[0]), host(w[1]))
    assert_gemm_close(zh, zr, bound, out_dtype == torch.bfloat16, "gemm_stream %s" % name)


@pytest.mark.parametrize("M,N,K", [(1, 300, 512), (16, 256, 1024), (64, 200, 5120), (23, 515, 2048),
                                   (65, 97, 1536), (128, 300, 512), (100, 33, 2048),
                                   (12, 12300, 1024), (2, 16400, 512), (40, 12300, 1024),
                                   (3, 1000, 8192), (16, 4000, 9216)])
@pytest.mark.parametrize("residual", [True, False])
def test_gemm_stream_bit_identical_to_quantize_then_gemm(M, N, K, residual):
    """Where rfq_gemm runs its few-row kernel (up to 64 rows, and up to 128
    where N <= 12160) both forms accumulate every output in the same order
    (groups, k-steps, primary then residual, the same four-wave sum) on the
    same codes: the streaming form must reproduce quantize + product bit for
    bit."""
    data = _gemm_case("qwen", M, N, K, seed=M * N + K)
    x = dev_bf16(data["x_bf16"])
    w = rfq.rfq_quantize_weight(dev(data["w"]))
    _say("gemm_stream vs codes M=%d N=%d K=%d residual=%s" % (M, N, K, residual))
    for dt in (torch.float32, torch.bfloat16):
        zs = rfq.rfq_gemm_stream(x, *w, residual=residual, out_dtype=dt)
        q = rfq.rfq_quantize_act(x, residual=residual)
        zc = rfq.rfq_gemm(*q, *w, out_dtype=dt)
        assert torch.equal(zs.view(torch.int16) if dt == torch.bfloat16 else zs.view(torch.int32),
                           zc.view(torch.int16) if dt == torch.bfloat16 else zc.view(torch.int32))


@pytest.mark.parametrize("M,N,K", [(1, 12288, 4096), (16, 12288, 4096), (8, 4096, 12288),
                                   (100, 4096, 4096), (64, 4096, 12288)])
def test_decode_shapes_full(orc, M, N, K):
    """Decode-sized products at the workloads' weight shapes, every output
    checked, in both forms (codes in and streaming)."""
    data = _gemm_case("qwen", M, N, K, seed=N + M)
    x = dev_bf16(data["x_bf16"])
    w = rfq.rfq_quantize_weight(dev(data["w"]))
    _say("decode M=%d N=%d K=%d" % (M, N, K))
    q = rfq.rfq_quantize_act(x)
    zc = host(rfq.rfq_gemm(*q, *w))
    zs = host(rfq.rfq_gemm_stream(x, *w))
    hq = [host(t) for t in q]
    _assert_codes_equal(hq, orc.quantize(wl.bf16_bits_to_f32(data["x_bf16"])), "decode x")
    zr, bound = orc.gemm(*hq, host(w[0]), host(w[1]))
    assert_gemm_close(zc, zr, bound, False, "decode codes")
    assert_gemm_close(zs, zr, bound, False, "decode stream")


def test_gemm_identity_weight_matches_dequant():
    """I7 on GPU outputs: with W = I the product returns deq(q) + deq(r)
    (exact here because the sum of the two fp32 terms is exact)."""
    g = read_golden("h1_mixed_block.txt")
    x = torch.tensor(np.tile(padded_floats(g["x"]), (40, 4)), dtype=torch.float32).cuda()
    q = rfq.rfq_quantize_act(x)
    w = rfq.rfq_quantize_weight(torch.eye(128, dtype=torch.float32).cuda())
    z = rfq.rfq_gemm(*q, *w)
    assert torch.equal(z, rfq.rfq_dequant(q[0], q[1]) + rfq.rfq_dequant(q[2], q[3]))


# ---------------------------------------------------------------- SwiGLU
@pytest.mark.parametrize("M,Nh", [(3, 96), (64, 12288), (257, 640)])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_swiglu_quantize(orc, M, Nh, dtype):
    rng = np.random.default_rng(M * Nh)
    gf = (rng.standard_normal((M, Nh)) * 2).astype(np.float32)
    uf = rng.standard_normal((M, Nh)).astype(np.float32)
    if dtype == torch.bfloat16:
        gb, ub = wl.f32_to_bf16_bits(gf), wl.f32_to_bf16_bits(uf)
        g, u = dev_bf16(gb), dev_bf16(ub)
        gf, uf = wl.bf16_bits_to_f32(gb), wl.bf16_bits_to_f32(ub)
    else:
        g, u = dev(gf), dev(uf)
    _say("swiglu quantize M=%d Nh=%d %s" % (M, Nh, dtype))
    qc, qs, rc, rs, h = rfq.rfq_swiglu_quantize_act(g, u, return_h=True)
    hg = host_bf16_as_f32(h).astype(np.float64)
    href = orc.swiglu(gf, uf)
    ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(href), 2.0 ** -126))) - 7)
    assert np.all(np.abs(hg - href) <= ulp)
    _assert_codes_equal([host(t) for t in (qc, qs, rc, rs)], orc.quantize(hg), "swiglu")


def test_swiglu_mlp_block_stagewise(orc):
    """The chained MLP block at reduced width: quantize -> gate/up product ->
    SwiGLU + quantize -> down product, each stage against the oracle on the
    GPU's own input to that stage."""
    w = wl.WORKLOADS["swiglu"].scaled(M=192, K=512, weights=(
        ("w_gate", 512, 640), ("w_up", 512, 640), ("w_down", 640, 512)))
    data = wl.generate(w, seed=2)
    q = rfq.rfq_quantize_act(x_device(data))
    wgu = rfq.rfq_quantize_weight(dev(np.concatenate([data["w_gate"], data["w_up"]], 0)))
    gu = rfq.rfq_gemm(*q, *wgu, out_dtype=torch.bfloat16)
    gu_h = host_bf16_as_f32(gu)
    zr, bound = orc.gemm(*[host(t) for t in q], host(wgu[0]), host(wgu[1]))
    assert_gemm_close(gu_h, zr, bound, True, "gate/up")
    gate, up = gu[:, :640].contiguous(), gu[:, 640:].contiguous()
    hq = rfq.rfq_swiglu_quantize_act(gate, up, return_h=True)
    hg = host_bf16_as_f32(hq[4]).astype(np.float64)
    href = orc.swiglu(gu_h[:, :640], gu_h[:, 640:])
    ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(href), 2.0 ** -126))) - 7)
    assert np.all(np.abs(hg - href) <= ulp)
    _assert_codes_equal([host(t) for t in hq[:4]], orc.quantize(hg), "h")
    wd = rfq.rfq_quantize_weight(dev(data["w_down"]))
    z = host(rfq.rfq_gemm(*hq[:4], *wd))
    zr, bound = orc.gemm(*[host(t) for t in hq[:4]], host(wd[0]), host(wd[1]))
    assert_gemm_close(z, zr, bound, False, "down")


def test_plain_mxfp4_agrees_with_hipblaslt(orc):
    """Independent cross-check of the MXFP4 encoding (nibble order, E8M0
    scales, block layout): the vendor's block-scaled FP4 product on the very
    same codes and scales agrees with the oracle to within one bf16 ulp of
    its output (its own accumulation and rounding are not ours: observed up
    to one ulp off), far below what a wrong nibble order or scale would
    give."""
    if not hasattr(torch, "float4_e2m1fn_x2"):
        pytest.skip("this torch has no FP4 dtype")
    w = wl.WORKLOADS["qwen"].scaled(M=256, K=1024, weights=(("w", 1024, 512),))
    data = wl.generate(w, seed=1)
    q = rfq.rfq_quantize_act(x_device(data))
    wq = rfq.rfq_quantize_weight(dev(data["w"]))
    try:
        zv = torch._scaled_mm(q[0].view(torch.float4_e2m1fn_x2),
                              wq[0].view(torch.float4_e2m1fn_x2).t(),
                              q[1].view(torch.float8_e8m0fnu), wq[1].view(torch.float8_e8m0fnu),
                              out_dtype=torch.bfloat16)
    except (RuntimeError, ValueError, NotImplementedError) as e:
        pytest.skip("block-scaled FP4 product unavailable: %s" % e)
    z = host(rfq.rfq_gemm(q[0], q[1], None, None, *wq))
    zr, bound = orc.gemm(host(q[0]), host(q[1]), None, None, host(wq[0]), host(wq[1]))
    assert_gemm_close(z, zr, bound, False, "phi=0")
    zv = host_bf16_as_f32(zv).astype(np.float64)
    err = np.abs(zv - zr)
    tol = 2.0 ** -10 * bound + 2.0 ** -7 * np.abs(zr)
    assert np.all(err <= tol), "vendor: %d outputs differ by more than one bf16 ulp" % int(
        (err > tol).sum())


# ------------------------------------------------- fallback indicator phi
PHI_SHAPES = [
    ("qwen", 200, 328, 1024),       # large-tile kernel, ragged M and N
    ("qwen", 129, 257, 2560),       # large-tile kernel, ragged indicator rows
    ("qwen", 512, 300, 2048),       # large-tile kernel, two full workgroup rows
    ("qwen", 200, 328, 1056),       # general kernel, K not a multiple of 256
    ("wan", 64, 96, 640),           # general kernel
]


def _phi_case(name, M, N, K, seed):
    w = wl.WORKLOADS[name].scaled(M=M, K=K, weights=(("w", K, N),))
    data = wl.generate(w, seed=seed)
    q = rfq.rfq_quantize_act(x_device(data))
    wq = rfq.rfq_quantize_weight(dev(data["w"]))
    return q, wq


@pytest.mark.parametrize("name,M,N,K", PHI_SHAPES)
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_gemm_phi_random_maps(orc, name, M, N, K, out_dtype):
    """Eq. 11 with a given phi map against the oracle: random maps at three
    densities, maps constant along rows or along columns (whole residual row
    blocks of a stage skipped, or whole stages), and arbitrary nonzero bytes
    (any nonzero byte means on); phi = 1 and phi = 0 give exactly the RFQ
    and the plain products."""
    q, wq = _phi_case(name, M, N, K, 21)
    hq = [host(t) for t in q] + [host(t) for t in wq]
    rng = np.random.default_rng(M + K)
    shape = ((M + 63) // 64, (K + 255) // 256)
    _say("phi %s M=%d N=%d K=%d %s" % (name, M, N, K, out_dtype))
    maps = [rng.random(shape) < p for p in (0.25, 0.5, 0.75)]
    maps.append(np.repeat(rng.integers(0, 2, (1, shape[1])), shape[0], 0))
    maps.append(np.repeat(rng.integers(0, 2, (shape[0], 1)), shape[1], 1))
    maps.append(rng.integers(0, 256, shape))
    for trial, phi in enumerate(maps):
        phi = np.ascontiguousarray(phi).astype(np.uint8)
        z = rfq.rfq_gemm_phi(*q, *wq, torch.from_numpy(phi).cuda(), out_dtype=out_dtype)
        zr, bound = orc.gemm_phi(*hq, phi)
        zg = host_bf16_as_f32(z) if out_dtype == torch.bfloat16 else host(z)
        assert_gemm_close(zg, zr, bound, out_dtype == torch.bfloat16, "phi trial %d" % trial)
    ones = torch.ones(shape, dtype=torch.uint8, device="cuda")
    zeros = torch.zeros(shape, dtype=torch.uint8, device="cuda")
    assert torch.equal(rfq.rfq_gemm_phi(*q, *wq, ones, out_dtype=out_dtype),
                       rfq.rfq_gemm(*q, *wq, out_dtype=out_dtype))
    assert torch.equal(rfq.rfq_gemm_phi(*q, *wq, zeros, out_dtype=out_dtype),
                       rfq.rfq_gemm(q[0], q[1], None, None, *wq, out_dtype=out_dtype))


@pytest.mark.parametrize("M,K", [(150, 800), (64, 4096), (257, 5120)])
def test_fallback_map_rules(orc, M, K):
    """Both map rules bit-exact against the oracle; the residual-nonzero map
    leaves the product unchanged (tiles it switches off carry zero codes)."""
    rng = np.random.default_rng(K)
    x = rng.standard_normal((M, K)).astype(np.float32)
    grid = np.array([0, 0.5, 1, 1.5, 2, 3, 4, 6], np.float32)
    x[64:128] = rng.choice(grid, x[64:128].shape) * rng.choice(np.float32([-1, 1]),
                                                                 x[64:128].shape)
    x[:64, K // 3] *= 80
    q = rfq.rfq_quantize_act(torch.from_numpy(x).cuda())
    hq = [host(t) for t in q]
    _say("fallback map M=%d K=%d" % (M, K))
    phi0 = rfq.rfq_fallback_map(q[2], q[1], rfq.RFQ_PHI_RESIDUAL_NONZERO)
    assert np.array_equal(host(phi0), orc.fallback_map(hq[2], hq[1], 0))
    thr = int(np.median(hq[1])) + 2
    phi1 = rfq.rfq_fallback_map(None, q[1], rfq.RFQ_PHI_SCALE_AT_LEAST, thr)
    assert np.array_equal(host(phi1), orc.fallback_map(None, hq[1], 1, thr))
    if M >= 128:
        assert not host(phi0)[1].any()
    w = rng.normal(0, 0.02, (192, K)).astype(np.float32)
    wq = rfq.rfq_quantize_weight(torch.from_numpy(w).cuda())
    z1 = rfq.rfq_gemm(*q, *wq)
    zphi = rfq.rfq_gemm_phi(*q, *wq, phi0)
    assert torch.equal(zphi.abs(), z1.abs()) and torch.equal(zphi == 0, z1 == 0)
    assert np.array_equal(host(zphi)[host(zphi) != 0], host(z1)[host(z1) != 0])


def test_fallback_map_beyond_one_grid_pass():
    """More tiles than one pass of the map's grid (65536 workgroups): every
    tile is decided.  Codes and scales are zero except for chosen bytes, so
    the expected maps follow from the construction: rule 0 marks a tile where
    a residual code has a nonzero magnitude (negative zero, code 0x8, does not
    count); rule 1 where a primary scale byte reaches the threshold."""
    M, K = 64 * 257 + 5, 256 * 256                 # 258 x 256 = 66048 tiles
    pr, pc = (M + 63) // 64, K // 256
    rng = np.random.default_rng(11)
    tiles = np.unique(np.concatenate([rng.integers(0, pr * pc, 3000),
                                      [0, 65535, 65536, 65537, pr * pc - 1]]))
    p, c = tiles // pc, tiles % pc
    m = np.minimum(64 * p + rng.integers(0, 64, tiles.size), M - 1)
    # Residual codes: one byte per chosen tile; 0x80, 0x88 and 0x08 hold only
    # zero magnitudes.
    byte = 128 * c + rng.integers(0, 128, tiles.size)
    val = rng.choice(np.uint8([0x01, 0x70, 0x80, 0x88, 0x08, 0x3B]), tiles.size)
    rc = torch.zeros((M, K // 2), dtype=torch.uint8, device="cuda")
    rc[torch.from_numpy(m).cuda(), torch.from_numpy(byte).cuda()] = torch.from_numpy(val).cuda()
    want0 = np.zeros((pr, pc), np.uint8)
    want0[p[(val & 0x77) != 0], c[(val & 0x77) != 0]] = 1
    # Primary scale bytes: one per chosen tile, below, at or above the threshold.
    thr = 131
    kb = 8 * c + rng.integers(0, 8, tiles.size)
    sv = rng.choice(np.uint8([thr - 1, thr, 255, 1]), tiles.size)
    qs = torch.zeros((M, K // 32), dtype=torch.uint8, device="cuda")
    qs[torch.from_numpy(m).cuda(), torch.from_numpy(kb).cuda()] = torch.from_numpy(sv).cuda()
    want1 = np.zeros((pr, pc), np.uint8)
    want1[p[sv >= thr], c[sv >= thr]] = 1
    _say("fallback map M=%d K=%d (%d tiles)" % (M, K, pr * pc))
    assert np.array_equal(host(rfq.rfq_fallback_map(rc, qs, rfq.RFQ_PHI_RESIDUAL_NONZERO)), want0)
    assert np.array_equal(host(rfq.rfq_fallback_map(None, qs, rfq.RFQ_PHI_SCALE_AT_LEAST, thr)),
                          want1)


# --------------------------------------------------- fused SwiGLU epilogue
def _fused_and_unfused(data, K, Nh, res_in, res_out, stages=None):
    """The chained path (gate and up products with bf16 Z, then the SwiGLU
    quantizer) and the fused one on the same codes.  With a dict `stages`,
    the chained path's intermediates are returned in it as host arrays:
    q (activation codes), wg and wu (weight codes), g and u (fp32 values of
    the bf16 products)."""
    q = rfq.rfq_quantize_act(x_device(data), residual=res_in)
    wg = rfq.rfq_quantize_weight(dev(data["w_gate"]))
    wu = rfq.rfq_quantize_weight(dev(data["w_up"]))
    # The fused path runs the large-tile product; rfq_gemm does so above 128
    # rows (and from 65 where N > 12160).  With up to 128 rows the reference
    # runs on codes zero-padded to 129 rows (rows are independent: padding
    # changes no output of the real rows).
    M = q[0].shape[0]
    qg = q
    if M <= 128:
        qg = [None if t is None else torch.cat([t, torch.zeros((129 - M, t.shape[1]),
                                                               dtype=t.dtype, device=t.device)])
              for t in q]
    g = rfq.rfq_gemm(*qg, *wg, out_dtype=torch.bfloat16)[:M].contiguous()
    u = rfq.rfq_gemm(*qg, *wu, out_dtype=torch.bfloat16)[:M].contiguous()
    ref = rfq.rfq_swiglu_quantize_act(g, u, residual=res_out, return_h=True)
    if stages is not None:
        stages.update(q=[None if t is None else host(t) for t in q],
                      wg=[host(t) for t in wg], wu=[host(t) for t in wu],
                      g=host_bf16_as_f32(g), u=host_bf16_as_f32(u))
    wgu = (rfq.interleave_gate_up(wg[0], wu[0]), rfq.interleave_gate_up(wg[1], wu[1]))
    got = rfq.rfq_gemm_swiglu_quantize(*q, *wgu, residual=res_out, return_h=True)
    return got, ref


# (1300, 3296, 512): the fused product (N = 6592) runs 256 x 256 tiles, the
# chained gate and up products (N = 3296) 128 x 128 ones.
FUSED = [(200, 640, 512), (64, 96, 1024), (300, 1280, 1536), (1, 32, 512), (1300, 3296, 512)]


@pytest.mark.parametrize("M,Nh,K", FUSED)
@pytest.mark.parametrize("res_in,res_out", [(True, True), (False, True), (True, False)])
def test_gemm_swiglu_fused_matches_chained(M, Nh, K, res_in, res_out):
    """The fused epilogue is bit-identical to the chained path (whose stages
    are pinned to the oracle in test_swiglu_mlp_block_stagewise): codes,
    scales and h."""
    w = wl.WORKLOADS["swiglu"].scaled(M=M, K=K, weights=(
        ("w_gate", K, Nh), ("w_up", K, Nh), ("w_down", Nh, K)))
    data = wl.generate(w, seed=8)
    _say("fused swiglu M=%d Nh=%d K=%d res_in=%s res_out=%s" % (M, Nh, K, res_in, res_out))
    got, ref = _fused_and_unfused(data, K, Nh, res_in, res_out)
    for n, a, b in zip(("hq_codes", "hq_scales", "hr_codes", "hr_scales", "h"), got, ref):
        if b is None:
            assert a is None
            continue
        assert torch.equal(a, b), n


def test_gemm_swiglu_fused_full_size_and_down_product(orc):
    """Config-5 shape (4096 x 4096 -> 2 x 12288 -> 4096), every stage of the
    chained path against the oracle on the GPU's own input to that stage
    (Sec. 4.3 Eq. 8-11 applied twice): the gate and up products sampled in
    every 128 x 128 output tile, all 4096 x 12288 elements of h within one
    bf16 ulp of the oracle's SwiGLU of the GPU's g and u, all codes and
    scales of h (primary and residual) bit-exact against the oracle's
    quantizer; the fused gate/up epilogue equals the chained path bit for
    bit; the down product on the fused codes is checked against the oracle
    on sampled rows and in every output tile."""
    data = wl.generate(wl.WORKLOADS["swiglu"], seed=0)
    _say("fused swiglu full size")
    st = {}
    got, ref = _fused_and_unfused(data, 4096, 12288, True, True, stages=st)
    for n, a, b in zip(("hq_codes", "hq_scales", "hr_codes", "hr_scales", "h"), got, ref):
        assert torch.equal(a, b), n
    # Stages of the chained path, each on the GPU's own input to it.
    M, K, Nh = 4096, 4096, 12288
    rng = np.random.default_rng(12)
    for zname, wname in (("g", "wg"), ("u", "wu")):
        rows, cols = _tile_samples(M, Nh, 128, rng)
        zr, bound = orc.gemm_sampled(*st["q"], *st[wname], rows, cols)
        assert_gemm_close(st[zname][rows, cols], zr, bound, True, "full-size %s product" % zname)
    _say("swiglu stage full size")
    hg = host_bf16_as_f32(ref[4])
    href = orc.swiglu(st["g"], st["u"])
    del st
    ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(href), 2.0 ** -126))) - 7)
    assert np.all(np.abs(hg - href) <= ulp)
    del href, ulp
    _assert_codes_equal([host(t) for t in ref[:4]], orc.quantize(hg), "h full size")
    del hg
    wd = rfq.rfq_quantize_weight(dev(data["w_down"]))
    z = host(rfq.rfq_gemm(*got[:4], *wd))
    rows = np.arange(0, 4096, 97)
    hq = [host(t)[rows] for t in got[:4]]
    zr, bound = orc.gemm(*hq, host(wd[0]), host(wd[1]))
    assert_gemm_close(z[rows], zr, bound, False, "down on fused codes")
    tr, tc = _tile_samples(M, K, 128, rng)
    zr, bound = orc.gemm_sampled(*[host(t) for t in got[:4]], host(wd[0]), host(wd[1]), tr, tc)
    assert_gemm_close(z[tr, tc], zr, bound, False, "down on fused codes, every tile")


# ---------------------------------------------------------------- edges
def test_codes_beyond_4gib(orc):
    """Maximum sizes: an activation tensor whose code tensors pass 2^32
    bytes (the product then runs on the kernel with 64-bit offsets).  Codes
    are checked bit-exactly and the product within tolerance on rows around
    the 4 GiB byte boundary, the last row and random rows."""
    M, K, N = (1 << 21) + 48, 4096, 64
    assert M * K // 2 > 1 << 32
    _say("beyond 4 GiB: M=%d K=%d N=%d" % (M, K, N))
    gen = torch.Generator(device="cuda").manual_seed(7)
    x = torch.randn((M, K), generator=gen, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    q = rfq.rfq_quantize_act(x)
    data = _gemm_case("qwen", 8, N, K, seed=99)
    w = rfq.rfq_quantize_weight(dev(data["w"]))
    z = rfq.rfq_gemm(*q, *w)
    boundary = (1 << 32) // (K // 2)               # first row whose codes start at 2^32
    rows = np.unique(np.concatenate([
        [0, boundary - 2, boundary - 1, boundary, boundary + 1, M - 2, M - 1],
        np.random.default_rng(3).integers(0, M, 24)]))
    idx = torch.from_numpy(rows).cuda()
    xr = host_bf16_as_f32(x.index_select(0, idx).contiguous())
    g = [host(t.index_select(0, idx)) for t in q]
    zr_rows = host(z.index_select(0, idx))
    del x, q, z
    torch.cuda.empty_cache()
    ref = orc.quantize(xr)
    _assert_codes_equal(g, ref, "beyond 4 GiB")
    zr, bound = orc.gemm(*ref, host(w[0]), host(w[1]))
    assert_gemm_close(zr_rows, zr, bound, False, "beyond 4 GiB product")


def test_gemm_split_long_k(orc):
    """The split product over a long reduction: K = 2^20 in 8 parts of 2^17
    (1024 stages each), every output against the oracle, and against the
    unsplit product within the same tolerance."""
    M, N, K = 33, 40, 1 << 20
    gen = torch.Generator(device="cuda").manual_seed(21)
    x = torch.randn((M, K), generator=gen, device="cuda").to(torch.bfloat16)
    wt = torch.randn((N, K), generator=gen, device="cuda") * 0.02
    q = rfq.rfq_quantize_act(x)
    w = rfq.rfq_quantize_weight(wt)
    nbytes = rfq.rfq_gemm_workspace_bytes(M, N, K)
    assert nbytes == 8 * M * N * 4
    _say("gemm split long K: M=%d N=%d K=%d" % (M, N, K))
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    z = host(rfq.rfq_gemm_split(*q, *w, ws))
    zu = host(rfq.rfq_gemm(*q, *w))
    zr, bound = orc.gemm(*[host(t) for t in q], host(w[0]), host(w[1]))
    assert_gemm_close(z, zr, bound, False, "split long K")
    assert_gemm_close(zu, zr, bound, False, "unsplit long K")


def test_empty_inputs_are_noops():
    x = torch.empty((0, 64), dtype=torch.bfloat16, device="cuda")
    q = rfq.rfq_quantize_act(x)
    assert q[0].shape == (0, 32)
    w = rfq.rfq_quantize_weight(torch.randn(16, 64, device="cuda"))
    z = rfq.rfq_gemm(*q, *w)
    assert z.shape == (0, 16)
    w0 = rfq.rfq_quantize_weight(torch.empty((0, 64), device="cuda"))
    q1 = rfq.rfq_quantize_act(torch.randn(4, 64, device="cuda"))
    assert rfq.rfq_gemm(*q1, *w0).shape == (4, 0)
    torch.cuda.synchronize()


def test_stream_argument_is_honoured(orc):
    data = _gemm_case("qwen", 256, 256, 512, seed=9)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        q = rfq.rfq_quantize_act(x_device(data), stream=s)
        w = rfq.rfq_quantize_weight(dev(data["w"]), stream=s)
        z = rfq.rfq_gemm(*q, *w, stream=s)
    s.synchronize()
    zr, bound = orc.gemm(*[host(t) for t in q], host(w[0]), host(w[1]))
    assert_gemm_close(host(z), zr, bound, False, "stream")


# ------------------------------------------------------------- HIP graphs
@pytest.mark.parametrize("M,N,K", [(16, 1024, 2048), (300, 512, 1024)])
def test_path_replays_from_a_hip_graph(M, N, K):
    """The quantizer, the product and its streaming form capture into a HIP
    graph (no allocation, memset or host synchronisation inside the calls);
    every replay, with eager work between replays, reproduces the eager
    results, and new input values flow through the captured graph."""
    gen = torch.Generator(device="cuda").manual_seed(M + N + K)
    x = torch.randn((M, K), generator=gen, device="cuda").to(torch.bfloat16)
    w = rfq.rfq_quantize_weight(torch.randn((N, K), generator=gen, device="cuda") * 0.02)
    q = [torch.empty((M, K // 2), dtype=torch.uint8, device="cuda"),
         torch.empty((M, K // 32), dtype=torch.uint8, device="cuda"),
         torch.empty((M, K // 2), dtype=torch.uint8, device="cuda"),
         torch.empty((M, K // 32), dtype=torch.uint8, device="cuda")]
    z = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    zs = torch.empty((M, N), dtype=torch.float32, device="cuda")

    def path():
        rfq.rfq_quantize_act(x, out=q)
        rfq.rfq_gemm(*q, *w, out=z)
        rfq.rfq_gemm_stream(x, *w, out=zs)

    def eager_results():
        path()
        torch.cuda.synchronize()
        return [t.clone() for t in q] + [z.clone(), zs.clone()]

    want = eager_results()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        path()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        path()
    _say("graph replay M=%d N=%d K=%d" % (M, N, K))
    for i in range(4):
        for t in q + [z, zs]:
            t.zero_()
        torch.randn((1024, 1024), generator=gen, device="cuda").sum()   # eager work between
        graph.replay()
        torch.cuda.synchronize()
        for a, b in zip(q + [z, zs], want):
            assert torch.equal(a, b), "replay %d differs from the eager result" % i
    x.copy_(torch.randn((M, K), generator=gen, device="cuda").to(torch.bfloat16))
    want = eager_results()
    for t in q + [z, zs]:
        t.zero_()
    graph.replay()
    torch.cuda.synchronize()
    for a, b in zip(q + [z, zs], want):
        assert torch.equal(a, b), "replay with new inputs differs from the eager result"


@pytest.mark.parametrize("M,N,K", [(130, 300, 8192), (16, 5120, 13824)])
def test_split_products_replay_from_a_hip_graph(M, N, K):
    """The split product with a caller-owned workspace and the allocation-free
    one on the static scratch array capture into one HIP graph (two kernels
    each, nothing allocated or cleared inside the calls; 128-wide tiles, and
    the few-row kernel's own split at 16 rows x 5120); every replay
    reproduces the eager results, and both give the same bits."""
    gen = torch.Generator(device="cuda").manual_seed(5)
    x = torch.randn((M, K), generator=gen, device="cuda").to(torch.bfloat16)
    w = rfq.rfq_quantize_weight(torch.randn((N, K), generator=gen, device="cuda") * 0.02)
    q = rfq.rfq_quantize_act(x)
    ws = torch.empty(rfq.rfq_gemm_workspace_bytes(M, N, K), dtype=torch.uint8, device="cuda")
    assert ws.numel() > 0
    za = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    zb = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")

    def path():
        rfq.rfq_quantize_act(x, out=q)
        rfq.rfq_gemm_split(*q, *w, ws, out=za)
        rfq.rfq_gemm_split_noalloc(*q, *w, out=zb)

    path()
    torch.cuda.synchronize()
    want = [za.clone(), zb.clone()]
    assert torch.equal(want[0].view(torch.int16), want[1].view(torch.int16))
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        path()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        path()
    _say("graph replay split M=%d N=%d K=%d" % (M, N, K))
    for i in range(4):
        za.zero_()
        zb.zero_()
        rfq.rfq_gemm(*q, *w, out=torch.empty_like(za))     # eager work between replays
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(za, want[0]) and torch.equal(zb, want[1]), "replay %d" % i


@pytest.mark.parametrize("M,N,K", [(300, 700, 640), (3, 5000, 8192)])
def test_hif4_path_replays_from_a_hip_graph(M, N, K):
    """The HiF4 quantizer, product, bf16-weight product and split product
    (128-wide tiles in 2 parts; the few-row kernel in 4 at 3 rows x 5000)
    capture into a HIP graph; every replay (eager work between) reproduces
    the eager results."""
    gen = torch.Generator(device="cuda").manual_seed(5)
    x = torch.randn((M, K), generator=gen, device="cuda").to(torch.bfloat16)
    hw = rfq.rfq_hif4_quantize(torch.randn((N, K), generator=gen, device="cuda") * 0.02,
                               residual=False)
    wv = rfq.rfq_hif4_dequant(hw[0], hw[1], out_dtype=torch.bfloat16)
    q = [torch.empty((M, K // 2), dtype=torch.uint8, device="cuda"),
         torch.empty((M, K // 64), dtype=torch.int32, device="cuda"),
         torch.empty((M, K // 2), dtype=torch.uint8, device="cuda"),
         torch.empty((M, K // 64), dtype=torch.int32, device="cuda")]
    z = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    z2 = torch.empty((M, N), dtype=torch.float32, device="cuda")
    z3 = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(rfq.rfq_hif4_gemm_workspace_bytes(M, N, K), dtype=torch.uint8,
                     device="cuda")
    assert ws.numel() > 0

    def path():
        rfq.rfq_hif4_quantize(x, out=q)
        rfq.rfq_hif4_gemm(*q, hw[0], hw[1], out=z)
        rfq.rfq_hif4_gemm_wbf16(*q, wv, out=z2)
        rfq.rfq_hif4_gemm_split(*q, hw[0], hw[1], ws, out=z3)

    path()
    torch.cuda.synchronize()
    want = [t.clone() for t in q + [z, z2, z3]]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        path()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        path()
    _say("hif4 graph replay M=%d N=%d K=%d" % (M, N, K))
    for i in range(4):
        for t in q + [z, z2, z3]:
            t.zero_()
        torch.randn((1024, 1024), generator=gen, device="cuda").sum()
        graph.replay()
        torch.cuda.synchronize()
        for a, b in zip(q + [z, z2, z3], want):
            assert torch.equal(a, b), "replay %d differs from the eager result" % i
