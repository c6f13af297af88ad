"""Parity of the HiF4 path (Sec. 3.3, Eq. 5-6, with RFQ's residual) with
the CPU oracle, through the C ABI.

Quantizer codes and metadata words: bit-exact (the encoder reading is the
same on both sides; parity of that reading with the paper is unpinned, since
the paper defines only the decode).  Dequantization: exact.  Product: within
the tolerance of gpu_util (every product of two HiF4 values is exact in
fp32, so only the fp32 sums round).  The small cases span several 128 x 256
tiles with ragged edges; the full-size case uses the shapes of the Qwen-like
workload with sampled rows and columns.
"""
import numpy as np
import pytest
import torch

import paper_2608_26581_amd as rfq
from paper_2608_26581_amd import workloads as wl
from gpu_util import assert_gemm_close, dev, dev_bf16, host, host_bf16_as_f32
from oracle_pins import padded_bytes, padded_floats, read_golden

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def _meta_u32(t):
    return host(t).view(np.uint32)


def _x_dev(x32, bf16):
    if bf16:
        return dev_bf16(wl.f32_to_bf16_bits(x32))
    return dev(np.ascontiguousarray(x32, np.float32))


def _gpu_quant(x32, bf16, residual=True):
    q = rfq.rfq_hif4_quantize(_x_dev(x32, bf16), residual=residual)
    torch.cuda.synchronize()
    qc, qm, rc, rm = q
    return (host(qc), _meta_u32(qm), None if rc is None else host(rc),
            None if rm is None else _meta_u32(rm)), q


def _assert_same(g, r, what):
    for n, a, b in zip(("q_codes", "q_meta", "r_codes", "r_meta"), g, r):
        if b is None:
            assert a is None, (what, n)
            continue
        if not np.array_equal(a, b):
            i = tuple(np.argwhere(a != b)[0])
            raise AssertionError("%s %s differ at %s: gpu %#x oracle %#x (%d differ)" %
                                 (what, n, i, int(a[i]), int(b[i]), int((a != b).sum())))


def _values_bf16_exact(x):
    return wl.bf16_bits_to_f32(wl.f32_to_bf16_bits(x))


def _hard_blocks(rng, rows, K, near_ties):
    """Blocks built around the format's grid: each 4-element group has one
    element at 1.75 2^e S (forcing its exponent) and the others at exact
    rounding ties (2j+1)/8 S 2^e, optionally one fp32 step off; plus zeros,
    negative zeros, tiny blocks (byte 0) and huge ones (saturating byte 255)."""
    x = np.zeros((rows, K), np.float64)
    for r in range(rows):
        for b0 in range(0, K, 64):
            kind = rng.integers(0, 8)
            blk = np.zeros(64)
            if kind == 0:
                blk[:] = 0.0
                blk[rng.integers(0, 64, 5)] = -0.0
            elif kind == 1:
                blk[:] = rng.standard_normal(64) * 1e-20
            elif kind == 2:
                blk[:] = rng.standard_normal(64) * 1e7
            else:
                byte = int(rng.integers(60, 230))
                S = (4 + (byte & 3)) * 2.0 ** ((byte >> 2) - 50)
                for j in range(16):
                    e = int(rng.integers(0, 3))
                    g = np.array([(2 * int(rng.integers(0, 7)) + 1) / 8.0 * S * 2.0 ** e
                                  for _ in range(4)])
                    g[int(rng.integers(0, 4))] = 1.75 * S * 2.0 ** e
                    blk[4 * j:4 * j + 4] = g * np.where(rng.random(4) < 0.5, -1.0, 1.0)
            x[r, b0:b0 + 64] = blk
    x = x.astype(np.float32)
    if near_ties:
        sel = rng.random(x.shape) < 0.3
        up = rng.random(x.shape) < 0.5
        x = np.where(sel, np.where(up, np.nextafter(x, np.float32(np.inf)),
                                   np.nextafter(x, np.float32(-np.inf))), x).astype(np.float32)
    return x


# ---------------------------------------------------------------- golden
def test_golden_encode_block():
    g = read_golden("h7_hif4_encode.txt")
    x = padded_floats(g["x"], 64).reshape(1, 64).astype(np.float32)
    for bf16 in (False, True):
        (qc, qm, _, _), _ = _gpu_quant(x, bf16, residual=False)
        assert int(qm[0, 0]) == int(g["meta"][0], 16)
        assert np.array_equal(qc[0], padded_bytes(g["codes"], 32))


def test_golden_decode_block():
    g = read_golden("h6_hif4_decode.txt")
    codes = dev(padded_bytes(g["codes"], 32).reshape(1, 32))
    meta = dev(np.array([[int(g["meta"][0], 16)]], np.uint32).view(np.int32))
    out = host(rfq.rfq_hif4_dequant(codes, meta))
    want = padded_floats(g["values"], 64)
    assert np.array_equal(out[0].astype(np.float64), want)
    assert np.array_equal(np.signbit(out[0]), np.signbit(want))


# ---------------------------------------------------------------- quantizer
QUANT_SHAPES = [(1, 64), (3, 192), (37, 640), (130, 1088), (257, 2048)]


@pytest.mark.parametrize("rows,K", QUANT_SHAPES)
@pytest.mark.parametrize("bf16", [False, True])
def test_quantize_random_matches_oracle(orc, rows, K, bf16):
    _say("hif4 quantize random %dx%d bf16=%s" % (rows, K, bf16))
    x = wl.generate(wl.WORKLOADS["tiny"].scaled(M=rows, K=K, weights=()), seed=rows + K)["x"]
    if bf16:
        x = _values_bf16_exact(x)
    g, _ = _gpu_quant(x, bf16)
    _assert_same(g, orc.hif4_quantize(x.astype(np.float64)), "random")
    gw, _ = _gpu_quant(x, bf16, residual=False)
    _assert_same(gw, orc.hif4_quantize(x.astype(np.float64), residual=False), "weights")


@pytest.mark.parametrize("bf16,near", [(False, False), (False, True), (True, False)])
def test_quantize_ties_and_edges_match_oracle(orc, bf16, near):
    _say("hif4 quantize ties bf16=%s near=%s" % (bf16, near))
    rng = np.random.default_rng(11 + near)
    x = _hard_blocks(rng, 24, 512, near)
    if bf16:
        x = _values_bf16_exact(x)
    g, _ = _gpu_quant(x, bf16)
    _assert_same(g, orc.hif4_quantize(x.astype(np.float64)), "ties")


def test_quantize_full_size_matches_oracle(orc):
    _say("hif4 quantize qwen 4096x4096 bf16")
    data = wl.generate("qwen")
    g, _ = _gpu_quant(data["x"], True)
    _assert_same(g, orc.hif4_quantize(data["x"].astype(np.float64)), "qwen")


def test_dequant_matches_oracle(orc):
    rng = np.random.default_rng(5)
    x = _hard_blocks(rng, 9, 320, True)
    _, (qc, qm, rc, rm) = _gpu_quant(x, False)
    for c, m in ((qc, qm), (rc, rm)):
        out = host(rfq.rfq_hif4_dequant(c, m)).astype(np.float64)
        want = orc.hif4_dequant(host(c), host(m).view(np.uint32))
        assert np.array_equal(out, want)
        assert np.array_equal(np.signbit(out), np.signbit(want))


# ---------------------------------------------------------------- product
GEMM_SHAPES = [(1, 1, 64), (37, 300, 192), (128, 256, 64), (130, 257, 640),
               (256, 512, 1024), (300, 700, 320)]


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
@pytest.mark.parametrize("residual", [True, False])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_gemm_matches_oracle(orc, M, N, K, residual, out_dtype):
    _say("hif4 gemm %dx%dx%d residual=%s %s" % (M, N, K, residual, out_dtype))
    w = wl.WORKLOADS["tiny"].scaled(M=M, K=K, weights=(("w", K, N),))
    data = wl.generate(w, seed=M * 7 + N + K)
    _, q = _gpu_quant(data["x"], False, residual)
    _, wq = _gpu_quant(data["w"], False, residual=False)
    z = rfq.rfq_hif4_gemm(q[0], q[1], q[2], q[3], wq[0], wq[1], out_dtype=out_dtype)
    zh = host(z.float())
    oq = orc.hif4_quantize(data["x"].astype(np.float64), residual)
    ow = orc.hif4_quantize(data["w"].astype(np.float64), residual=False)
    zr, bound = orc.hif4_gemm(oq[0], oq[1], oq[2], oq[3], ow[0], ow[1])
    assert_gemm_close(zh, zr, bound, out_dtype == torch.bfloat16, "hif4 gemm")


def test_gemm_full_size_sampled(orc):
    """Qwen-like shapes (M 4096, K 4096, N 12288), bf16 activations, in the
    configuration the benchmark times; 48 sampled rows x 96 sampled columns."""
    _say("hif4 gemm full size sampled")
    data = wl.generate("qwen")
    x, w = data["x"], data["w"]
    _, q = _gpu_quant(x, True)
    _, wq = _gpu_quant(w, False, residual=False)
    z = host(rfq.rfq_hif4_gemm(*q, wq[0], wq[1]))
    rng = np.random.default_rng(3)
    rows = np.sort(np.concatenate([[0, 4095], rng.choice(4096, 46, replace=False)]))
    cols = np.sort(np.concatenate([[0, 12287], rng.choice(12288, 94, replace=False)]))
    oq = orc.hif4_quantize(x[rows].astype(np.float64))
    ow = orc.hif4_quantize(w[cols].astype(np.float64), residual=False)
    zr, bound = orc.hif4_gemm(oq[0], oq[1], oq[2], oq[3], ow[0], ow[1])
    assert_gemm_close(z[np.ix_(rows, cols)], zr, bound, False, "hif4 full")


def test_gemm_hif4_residual_reduces_error(orc):
    """RFQ's point (Sec. 4.3): with the residual term the product is closer
    to the unquantized one than with the primary code alone."""
    data = wl.generate(wl.WORKLOADS["tiny"].scaled(M=128, K=1024, weights=(("w", 1024, 256),)),
                       seed=9)
    _, q = _gpu_quant(data["x"], False)
    _, wq = _gpu_quant(data["w"], False, residual=False)
    z1 = host(rfq.rfq_hif4_gemm(*q, wq[0], wq[1])).astype(np.float64)
    z0 = host(rfq.rfq_hif4_gemm(q[0], q[1], None, None, wq[0], wq[1])).astype(np.float64)
    wd = orc.hif4_dequant(host(wq[0]), _meta_u32(wq[1]))
    exact = data["x"].astype(np.float64) @ wd.T
    e1 = np.linalg.norm(z1 - exact) / np.linalg.norm(exact)
    e0 = np.linalg.norm(z0 - exact) / np.linalg.norm(exact)
    assert e1 < 0.25 * e0, (e1, e0)


def test_dequant_bf16_is_exact(orc):
    rng = np.random.default_rng(6)
    x = _hard_blocks(rng, 7, 384, False)
    _, (qc, qm, rc, rm) = _gpu_quant(x, False)
    for c, m in ((qc, qm), (rc, rm)):
        ob = rfq.rfq_hif4_dequant(c, m, out_dtype=torch.bfloat16)
        got = host(ob.float()).astype(np.float64)
        want = orc.hif4_dequant(host(c), host(m).view(np.uint32))
        assert np.array_equal(got, want)
        assert np.array_equal(np.signbit(got), np.signbit(want))


@pytest.mark.parametrize("M,N,K", [(37, 300, 192), (130, 257, 640), (256, 512, 1024),
                                   (1, 5, 64)])
@pytest.mark.parametrize("residual", [True, False])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_gemm_wbf16_bit_identical_to_codes(M, N, K, residual, out_dtype):
    """Weights decoded once to bf16 give the same LDS tiles, hence the same
    bits, as the product that decodes the weight codes itself."""
    _say("hif4 gemm wbf16 %dx%dx%d residual=%s %s" % (M, N, K, residual, out_dtype))
    w = wl.WORKLOADS["tiny"].scaled(M=M, K=K, weights=(("w", K, N),))
    data = wl.generate(w, seed=M + 3 * N + K)
    _, q = _gpu_quant(data["x"], False, residual)
    _, wq = _gpu_quant(data["w"], False, residual=False)
    wv = rfq.rfq_hif4_dequant(wq[0], wq[1], out_dtype=torch.bfloat16)
    z1 = rfq.rfq_hif4_gemm(*q, wq[0], wq[1], out_dtype=out_dtype)
    z2 = rfq.rfq_hif4_gemm_wbf16(*q, wv, out_dtype=out_dtype)
    torch.cuda.synchronize()
    assert torch.equal(z1.view(torch.int16) if out_dtype == torch.bfloat16 else z1.view(torch.int32),
                       z2.view(torch.int16) if out_dtype == torch.bfloat16 else z2.view(torch.int32))


def test_gemm_wbf16_any_bf16_weight(orc):
    """Arbitrary bf16 weights (not HiF4 values): exact products, fp32 sums;
    the reference multiplies the oracle's decoded activations with the bf16
    weights in fp64."""
    M, N, K = 150, 300, 448
    data = wl.generate(wl.WORKLOADS["tiny"].scaled(M=M, K=K, weights=(("w", K, N),)), seed=8)
    wb = wl.f32_to_bf16_bits(data["w"] * 10.0)
    _, q = _gpu_quant(data["x"], False)
    z = host(rfq.rfq_hif4_gemm_wbf16(*q, dev_bf16(wb))).astype(np.float64)
    oq = orc.hif4_quantize(data["x"].astype(np.float64))
    vq = orc.hif4_dequant(oq[0], oq[1])
    vr = orc.hif4_dequant(oq[2], oq[3])
    wf = wl.bf16_bits_to_f32(wb).astype(np.float64)
    zr = vq @ wf.T + vr @ wf.T
    bound = np.abs(vq) @ np.abs(wf).T + np.abs(vr) @ np.abs(wf).T
    assert_gemm_close(z, zr, bound, False, "hif4 wbf16")


# Up to 4 and up to 8 rows (16 weight rows and 8 waves per workgroup), 9-16
# rows with 8 waves (few workgroups) and with 4 (N above 12256); K ending in
# half a chunk of 128 (64, 192, 576, 4160) and fewer chunks than waves.
# Workgroup shapes of the few-row kernel (weight rows, activation rows,
# waves): 16 x 4 up to 4 rows; 16 x 8, 32 x 8 or 64 x 8 up to 8 and 16 x 16,
# 32 x 16 or 64 x 16 up to 16, by N (at most 4096, below 11264, from 11264;
# the bf16-weight form stays at 32 rows there); sixteen waves up to 8 rows
# where N <= 4096, eight elsewhere; 17-64 rows in two or four slices of 16
# rows per workgroup; each with a ragged last workgroup.
FEW_SHAPES = [(1, 1, 64), (2, 33, 192), (5, 300, 640), (16, 700, 1024), (3, 64, 128),
              (8, 257, 4160), (9, 12300, 576), (6, 5000, 320), (7, 11300, 192),
              (12, 4200, 256), (3, 16400, 256), (4, 4096, 8192),
              # 17-64 rows: two or four slices of 16 rows per workgroup
              (17, 300, 640), (24, 12300, 320), (33, 5000, 256), (50, 4096, 1024),
              (64, 11300, 128),
              # 65-128 rows at N <= 4096: two launches on 64-row halves
              (100, 300, 640)]


@pytest.mark.parametrize("M,N,K", FEW_SHAPES)
@pytest.mark.parametrize("residual", [True, False])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_gemm_few_rows_matches_oracle(orc, M, N, K, residual, out_dtype):
    """At most 64 activation rows run the few-row kernel (K split over eight
    or sixteen waves, partial sums added in wave order; above 16 rows in
    slices of 16); fewer K chunks than waves included.  The bf16-weight form
    is bit-identical to it."""
    _say("hif4 few rows %dx%dx%d residual=%s %s" % (M, N, K, residual, out_dtype))
    w = wl.WORKLOADS["tiny"].scaled(M=M, K=K, weights=(("w", K, N),))
    data = wl.generate(w, seed=M * 13 + N + K)
    _, q = _gpu_quant(data["x"], False, residual)
    _, wq = _gpu_quant(data["w"], False, residual=False)
    z = rfq.rfq_hif4_gemm(*q, wq[0], wq[1], out_dtype=out_dtype)
    wv = rfq.rfq_hif4_dequant(wq[0], wq[1], out_dtype=torch.bfloat16)
    z2 = rfq.rfq_hif4_gemm_wbf16(*q, wv, out_dtype=out_dtype)
    torch.cuda.synchronize()
    assert torch.equal(z.view(torch.int16) if out_dtype == torch.bfloat16 else z.view(torch.int32),
                       z2.view(torch.int16) if out_dtype == torch.bfloat16 else z2.view(torch.int32))
    oq = orc.hif4_quantize(data["x"].astype(np.float64), residual)
    ow = orc.hif4_quantize(data["w"].astype(np.float64), residual=False)
    zr, bound = orc.hif4_gemm(oq[0], oq[1], oq[2], oq[3], ow[0], ow[1])
    assert_gemm_close(host(z.float()), zr, bound, out_dtype == torch.bfloat16, "hif4 few")


def test_gemm_few_rows_decode_shape(orc):
    """Decode shape of the Qwen-like layer: 1 and 16 rows x 12288 x 4096."""
    data = wl.generate("qwen")
    _, wq = _gpu_quant(data["w"], False, residual=False)
    ow = orc.hif4_quantize(data["w"].astype(np.float64), residual=False)
    for M in (1, 16):
        _say("hif4 few rows decode M=%d" % M)
        x = data["x"][:M]
        _, q = _gpu_quant(x, True)
        z = host(rfq.rfq_hif4_gemm(*q, wq[0], wq[1]))
        oq = orc.hif4_quantize(x.astype(np.float64))
        zr, bound = orc.hif4_gemm(oq[0], oq[1], oq[2], oq[3], ow[0], ow[1])
        assert_gemm_close(z, zr, bound, False, "hif4 decode M=%d" % M)


def test_gemm_full_size_k12288_sampled(orc):
    """The down-projection shape of the MLP workload (M 4096, N 4096,
    K 12288): the largest reduction of the configurations, at the edge of
    the product tolerance's derivation; 40 sampled rows x 64 columns."""
    _say("hif4 gemm 4096x4096x12288 sampled")
    w = wl.WORKLOADS["qwen"].scaled(M=4096, K=12288, weights=(("w", 12288, 4096),))
    data = wl.generate(w, seed=4)
    x, wt = data["x"], data["w"]
    _, q = _gpu_quant(x, True)
    _, wq = _gpu_quant(wt, False, residual=False)
    z = host(rfq.rfq_hif4_gemm(*q, wq[0], wq[1]))
    rng = np.random.default_rng(12)
    rows = np.sort(np.concatenate([[0, 4095], rng.choice(4096, 38, replace=False)]))
    cols = np.sort(np.concatenate([[0, 4095], rng.choice(4096, 62, replace=False)]))
    oq = orc.hif4_quantize(x[rows].astype(np.float64))
    ow = orc.hif4_quantize(wt[cols].astype(np.float64), residual=False)
    zr, bound = orc.hif4_gemm(oq[0], oq[1], oq[2], oq[3], ow[0], ow[1])
    assert_gemm_close(z[np.ix_(rows, cols)], zr, bound, False, "hif4 K=12288")


# K split over workgroups: 6 tiles of 128 x 128 -> 8 parts of 5 blocks; 9
# tiles, 16 blocks -> 4 parts of 4; 10 tiles, 64 blocks -> 8 parts of 8.
HIF4_SPLIT = [(200, 300, 2560), (300, 257, 1024), (150, 640, 4096),
              (3, 5000, 8192),      # few-row form, 313 workgroups: K in 4 parts
              (20, 5000, 6208)]     # 157 workgroups: 3 parts, the last chunk half


@pytest.mark.parametrize("M,N,K", HIF4_SPLIT)
@pytest.mark.parametrize("residual", [True, False])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_gemm_split_matches_oracle(orc, M, N, K, residual, out_dtype):
    """rfq_hif4_gemm_split (fp32 partials per part of K, added in order)
    against the oracle, every output; a workspace below the plan's size runs
    the unsplit product, bit for bit."""
    _say("hif4 gemm split %dx%dx%d residual=%s %s" % (M, N, K, residual, out_dtype))
    nbytes = rfq.rfq_hif4_gemm_workspace_bytes(M, N, K)
    assert nbytes > 0
    w = wl.WORKLOADS["tiny"].scaled(M=M, K=K, weights=(("w", K, N),))
    data = wl.generate(w, seed=M + 5 * N + K)
    _, q = _gpu_quant(data["x"], False, residual)
    _, wq = _gpu_quant(data["w"], False, residual=False)
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    z = rfq.rfq_hif4_gemm_split(*q, wq[0], wq[1], ws, out_dtype=out_dtype)
    oq = orc.hif4_quantize(data["x"].astype(np.float64), residual)
    ow = orc.hif4_quantize(data["w"].astype(np.float64), residual=False)
    zr, bound = orc.hif4_gemm(oq[0], oq[1], oq[2], oq[3], ow[0], ow[1])
    assert_gemm_close(host(z.float()), zr, bound, out_dtype == torch.bfloat16, "hif4 split")
    small = torch.empty(nbytes - 16, dtype=torch.uint8, device="cuda")
    z1 = rfq.rfq_hif4_gemm_split(*q, wq[0], wq[1], small, out_dtype=out_dtype)
    z2 = rfq.rfq_hif4_gemm(*q, wq[0], wq[1], out_dtype=out_dtype)
    iv = torch.int32 if out_dtype == torch.float32 else torch.int16
    assert torch.equal(z1.view(iv), z2.view(iv)), "short workspace: not the unsplit product"


@pytest.mark.parametrize("M,N,K", [(1024, 2560, 640), (1100, 4100, 256)])
@pytest.mark.parametrize("residual", [True, False])
def test_gemm_split_decoding_weights_is_the_unsplit_product(M, N, K, residual):
    """From 1024 rows without a split of K, rfq_hif4_gemm_split decodes the
    weights to bf16 in the workspace and runs the bf16-weight product: the
    bits of rfq_hif4_gemm, in both output types (ragged N included); with a
    workspace one byte short it runs rfq_hif4_gemm itself."""
    nbytes = rfq.rfq_hif4_gemm_workspace_bytes(M, N, K)
    assert nbytes == N * K * 2
    _say("hif4 gemm split, W decoded: %dx%dx%d residual=%s" % (M, N, K, residual))
    w = wl.WORKLOADS["tiny"].scaled(M=M, K=K, weights=(("w", K, N),))
    data = wl.generate(w, seed=M + N + K)
    _, q = _gpu_quant(data["x"], False, residual)
    _, wq = _gpu_quant(data["w"], False, residual=False)
    ws = torch.full((nbytes,), 0xFF, dtype=torch.uint8, device="cuda")
    for dt, iv in ((torch.float32, torch.int32), (torch.bfloat16, torch.int16)):
        want = rfq.rfq_hif4_gemm(*q, wq[0], wq[1], out_dtype=dt)
        got = rfq.rfq_hif4_gemm_split(*q, wq[0], wq[1], ws, out_dtype=dt)
        assert torch.equal(got.view(iv), want.view(iv)), dt
        short = rfq.rfq_hif4_gemm_split(*q, wq[0], wq[1], ws[:nbytes - 1], out_dtype=dt)
        assert torch.equal(short.view(iv), want.view(iv)), dt


@pytest.mark.parametrize("M,N,K,nrows", [(256, 4096, 12288, 24), (64, 4096, 12288, 8),
                                         (30, 4000, 12288, 8), (40, 5120, 13824, 8),
                                         (1, 5120, 13824, 1), (40, 12288, 4096, 8)])
def test_gemm_split_down_projection_sampled(orc, M, N, K, nrows):
    """Split products at full width, sampled rows against the oracle in
    every column: 128-wide tiles at the down-projection shape (4096 x 12288
    weights) for 256 rows (64 tiles, 4 parts of 48 blocks), 64 rows and 30
    rows (ragged N; 32 tiles, 8 parts), and the few-row form at 40 and 1 rows
    x 5120 x 13824 (3 and 4 parts) and 40 rows x 12288 x 4096 (2 parts)."""
    assert rfq.rfq_hif4_gemm_workspace_bytes(M, N, K) > 0
    _say("hif4 gemm split %dx%dx%d sampled" % (M, N, K))
    w = wl.WORKLOADS["qwen"].scaled(M=M, K=K, weights=(("w", K, N),))
    data = wl.generate(w, seed=9)
    x, wt = data["x"], data["w"]
    _, q = _gpu_quant(x, True)
    _, wq = _gpu_quant(wt, False, residual=False)
    z = host(rfq.rfq_hif4_gemm(*q, wq[0], wq[1], split=True))
    rng = np.random.default_rng(13)
    inner = rng.choice(np.arange(1, M - 1), max(0, nrows - 2), replace=False) if M > 2 else []
    rows = np.unique(np.concatenate([[0, M - 1], inner]).astype(np.int64))
    oq = orc.hif4_quantize(x[rows].astype(np.float64))
    ow = orc.hif4_quantize(wt.astype(np.float64), residual=False)
    zr, bound = orc.hif4_gemm(oq[0], oq[1], oq[2], oq[3], ow[0], ow[1])
    assert_gemm_close(z[rows], zr, bound, False, "hif4 split sampled")


@pytest.mark.parametrize("residual", [True, False])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_gemm_wide_tiles_ragged(orc, residual, out_dtype):
    """A product with enough 128 x 256 tiles to fill the chip (16 x 16, ragged
    in both directions) runs the 256-wide weight tiles; the smaller shapes
    above run the 128-wide ones.  K = 640 (ten blocks) passes the LDS
    double buffer back and forth.  Checked: against the oracle in fp32 and
    bf16 output, bit-identity of the bf16-weight form with the codes form,
    and guard bytes around both outputs."""
    M, N, K = 2000, 4000, 640
    _say("hif4 gemm wide tiles %dx%dx%d residual=%s %s" % (M, N, K, residual, out_dtype))
    w = wl.WORKLOADS["tiny"].scaled(M=M, K=K, weights=(("w", K, N),))
    data = wl.generate(w, seed=21)
    _, q = _gpu_quant(data["x"], False, residual)
    _, wq = _gpu_quant(data["w"], False, residual=False)
    esize = 4 if out_dtype == torch.float32 else 2
    guard = 4096

    def guarded():
        raw = torch.full((M * N * esize + 2 * guard,), 0xA5, dtype=torch.uint8, device="cuda")
        return raw, raw[guard:guard + M * N * esize].view(out_dtype).view(M, N)

    raw1, z1 = guarded()
    raw2, z2 = guarded()
    rfq.rfq_hif4_gemm(*q, wq[0], wq[1], out=z1)
    wv = rfq.rfq_hif4_dequant(wq[0], wq[1], out_dtype=torch.bfloat16)
    rfq.rfq_hif4_gemm_wbf16(*q, wv, out=z2)
    torch.cuda.synchronize()
    for raw in (raw1, raw2):
        r = host(raw)
        assert np.all(r[:guard] == 0xA5) and np.all(r[-guard:] == 0xA5), "write outside Z"
    iv = torch.int32 if out_dtype == torch.float32 else torch.int16
    assert torch.equal(z1.view(iv), z2.view(iv)), "bf16-weight form differs from codes form"
    z = host(z1) if out_dtype == torch.float32 else host_bf16_as_f32(z1)
    oq = orc.hif4_quantize(data["x"].astype(np.float64), residual)
    ow = orc.hif4_quantize(data["w"].astype(np.float64), residual=False)
    zr, bound = orc.hif4_gemm(oq[0], oq[1], oq[2], oq[3], ow[0], ow[1])
    assert_gemm_close(z, zr, bound, out_dtype == torch.bfloat16, "hif4 wide tiles")
