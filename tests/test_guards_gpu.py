"""Out-of-bounds writes: every output buffer of every entry point sits between
guard regions filled with a known byte pattern; after the call the guards must
be intact.  Ragged shapes exercise the kernels' tail handling on both product
kernels."""
import numpy as np
import pytest
import torch

import paper_2608_26581_amd as rfq
from paper_2608_26581_amd import rfq as binding
from paper_2608_26581_amd import workloads as wl

pytestmark = pytest.mark.gpu

GUARD = 4096          # bytes on each side (keeps 16-byte alignment)
PATTERN = 0xA5


class Guarded:
    """A device tensor of `shape` and `dtype` inside a larger byte buffer."""

    def __init__(self, shape, dtype):
        n = int(np.prod(shape)) * torch.tensor([], dtype=dtype).element_size()
        self.n = n
        self.raw = torch.full((n + 2 * GUARD,), PATTERN, dtype=torch.uint8, device="cuda")
        self.t = self.raw[GUARD:GUARD + n].view(dtype).view(*shape)

    def check(self, what):
        torch.cuda.synchronize()
        head = self.raw[:GUARD].cpu().numpy()
        tail = self.raw[GUARD + self.n:].cpu().numpy()
        assert np.all(head == PATTERN), "%s: write before the buffer" % what
        assert np.all(tail == PATTERN), "%s: write past the buffer" % what


def _codes(rows, K):
    return [Guarded((rows, K // 2), torch.uint8), Guarded((rows, K // 32), torch.uint8)]


def _check_all(bufs, what):
    for i, b in enumerate(bufs):
        b.check("%s[%d]" % (what, i))


@pytest.mark.parametrize("M,N,K", [(131, 97, 512), (131, 97, 96), (1, 1, 1024), (257, 300, 1536),
                                   (37, 77, 1024), (1300, 6500, 512), (131, 301, 8704)])
def test_outputs_stay_in_bounds(M, N, K):
    w = wl.WORKLOADS["qwen"].scaled(M=M, K=K, weights=(("w", K, N),))
    data = wl.generate(w, seed=31)
    x = torch.from_numpy(data["x"]).cuda()
    xb = torch.from_numpy(data["x_bf16"].view(np.int16)).cuda().view(torch.bfloat16)
    for xin, tag in ((x, "fp32"), (xb, "bf16")):
        qb = _codes(M, K) + _codes(M, K)
        rfq.rfq_quantize_act(xin, out=[b.t for b in qb])
        _check_all(qb, "quantize_act %s" % tag)
    q = [b.t for b in qb]
    wb = _codes(N, K)
    rfq.rfq_quantize_weight(torch.from_numpy(data["w"]).cuda(), out=[b.t for b in wb])
    _check_all(wb, "quantize_weight")
    wq = [b.t for b in wb]
    for dt in (torch.float32, torch.bfloat16):
        zb = Guarded((M, N), dt)
        rfq.rfq_gemm(*q, *wq, out=zb.t)
        zb.check("gemm %s" % dt)
        zb = Guarded((M, N), dt)
        rfq.rfq_gemm(q[0], q[1], None, None, *wq, out=zb.t)
        zb.check("gemm plain %s" % dt)
        nbytes = rfq.rfq_gemm_workspace_bytes(M, N, K)
        if nbytes:
            # K split over workgroups: the partials stay inside the workspace.
            wsb = Guarded((nbytes,), torch.uint8)
            zb = Guarded((M, N), dt)
            rfq.rfq_gemm_split(*q, *wq, wsb.t, out=zb.t)
            zb.check("gemm split %s" % dt)
            wsb.check("gemm split workspace %s" % dt)
    phi_shape = ((M + 63) // 64, (K + 255) // 256)
    pb = Guarded(phi_shape, torch.uint8)
    rfq.rfq_fallback_map(None, q[1], rfq.RFQ_PHI_SCALE_AT_LEAST, 128, out=pb.t)
    pb.check("fallback_map scale")
    pb2 = Guarded(phi_shape, torch.uint8)
    rfq.rfq_fallback_map(q[2], q[1], rfq.RFQ_PHI_RESIDUAL_NONZERO, out=pb2.t)
    pb2.check("fallback_map residual")
    zb = Guarded((M, N), torch.bfloat16)
    rfq.rfq_gemm_phi(*q, *wq, pb.t, out=zb.t)
    zb.check("gemm_phi")
    if K % 512 == 0:
        for dt in (torch.float32, torch.bfloat16):
            zb = Guarded((M, N), dt)
            rfq.rfq_gemm_stream(xb, *wq, out=zb.t)
            zb.check("gemm_stream %s" % dt)
    db = Guarded((M, K), torch.float32)
    rfq.rfq_dequant(q[0], q[1], out=db.t)
    db.check("dequant")


@pytest.mark.parametrize("M,Nh,K", [(131, 96, 512), (3, 32, 1024)])
def test_swiglu_outputs_stay_in_bounds(M, Nh, K):
    rng = np.random.default_rng(M)
    g = torch.from_numpy(rng.standard_normal((M, Nh)).astype(np.float32)).cuda()
    u = torch.from_numpy(rng.standard_normal((M, Nh)).astype(np.float32)).cuda()
    hb = _codes(M, Nh) + _codes(M, Nh)
    rfq.rfq_swiglu_quantize_act(g.to(torch.bfloat16), u.to(torch.bfloat16),
                                out=[b.t for b in hb])
    _check_all(hb, "swiglu_quantize")
    for dt in (torch.float32, torch.bfloat16):
        gd, ud = g.to(dt), u.to(dt)
        hb = _codes(M, Nh) + _codes(M, Nh)
        h = Guarded((M, Nh), torch.bfloat16)
        st = binding.load().rfq_swiglu_quantize_act(
            binding._ptr(gd), binding._ptr(ud), binding._dtype_code(gd), M, Nh,
            *[binding._ptr(b.t) for b in hb], binding._ptr(h.t), binding._stream(None))
        assert st == 0
        _check_all(hb, "swiglu_quantize %s" % dt)
        h.check("swiglu_quantize h %s" % dt)
    x = torch.from_numpy(rng.standard_normal((M, K)).astype(np.float32)).cuda()
    q = rfq.rfq_quantize_act(x)
    wgu = rfq.rfq_quantize_weight(torch.from_numpy(
        rng.normal(0, 0.02, (2 * Nh, K)).astype(np.float32)).cuda())
    fb = _codes(M, Nh) + _codes(M, Nh)
    rfq.rfq_gemm_swiglu_quantize(*q, *wgu, out=[b.t for b in fb])
    _check_all(fb, "gemm_swiglu_quantize")


def test_binding_rejects_bad_tensors():
    """The binding refuses tensors whose pointer the kernels could not use
    safely (wrong shape, dtype, layout, or a half-given operand pair) before
    calling the library."""
    M, N, K = 8, 64, 512
    x = torch.randn(M, K, device="cuda")
    w = torch.randn(N, K, device="cuda")
    q = binding.rfq_quantize_act(x)
    wq = binding.rfq_quantize_weight(w)
    bad = [
        # scales with too few rows: the kernel would read past them
        (ValueError, lambda: binding.rfq_gemm(q[0], q[1][:M - 1], q[2], q[3], *wq)),
        (ValueError, lambda: binding.rfq_gemm(q[0], q[1], q[2], q[3], wq[0], wq[1][:, :8])),
        (ValueError, lambda: binding.rfq_gemm(q[0], q[1], q[2], None, *wq)),
        (TypeError, lambda: binding.rfq_gemm(q[0].view(torch.int8), q[1], q[2], q[3], *wq)),
        (ValueError, lambda: binding.rfq_gemm(q[0], q[1], q[2], q[3], *wq,
                                              out=torch.empty(M, N - 1, device="cuda"))),
        (TypeError, lambda: binding.rfq_gemm(q[0], q[1], q[2], q[3], *wq,
                                             out=torch.empty(M, N, device="cuda",
                                                             dtype=torch.float16))),
        (ValueError, lambda: binding.rfq_gemm_phi(*q, *wq, torch.ones(1, 1, dtype=torch.uint8,
                                                                       device="cuda"))),
        (ValueError, lambda: binding.rfq_gemm_stream(x.t(), *wq)),          # not contiguous
        (ValueError, lambda: binding.rfq_gemm_stream(x, wq[0][:, :128], wq[1][:, :8])),
        (TypeError, lambda: binding.rfq_quantize_act(x.to(torch.float16))),
        (ValueError, lambda: binding.rfq_quantize_act(
            x, out=(q[0][:4], q[1], q[2], q[3]))),
        (ValueError, lambda: binding.rfq_dequant(q[0], q[1][:, :4])),
        (ValueError, lambda: binding.rfq_dequant(q[0], q[1], out=torch.empty(M, K - 32,
                                                                             device="cuda"))),
        (ValueError, lambda: binding.rfq_fallback_map(q[2][:4], q[1],
                                                      binding.RFQ_PHI_RESIDUAL_NONZERO)),
        (ValueError, lambda: binding.rfq_gemm_swiglu_quantize(q[0], q[1], q[2], q[3],
                                                              wq[0][:63], wq[1][:63])),
    ]
    for i, (exc, call) in enumerate(bad):
        with pytest.raises(exc):
            call()
    # The valid calls still work after the refused ones.
    z = binding.rfq_gemm(*q, *wq)
    torch.cuda.synchronize()
    assert z.shape == (M, N) and torch.isfinite(z).all()


@pytest.mark.parametrize("M,N,K", [(131, 97, 192), (1, 1, 64), (257, 300, 640), (37, 515, 128),
                                   (12, 11301, 128), (6, 4999, 64), (70, 400, 128)])
def test_hif4_outputs_stay_in_bounds(M, N, K):
    w = wl.WORKLOADS["qwen"].scaled(M=M, K=K, weights=(("w", K, N),))
    data = wl.generate(w, seed=37)
    x = torch.from_numpy(data["x"]).cuda()
    xb = torch.from_numpy(data["x_bf16"].view(np.int16)).cuda().view(torch.bfloat16)

    def hif4(rows):
        return [Guarded((rows, K // 2), torch.uint8), Guarded((rows, K // 64), torch.int32)]

    for xin, tag in ((x, "fp32"), (xb, "bf16")):
        qb = hif4(M) + hif4(M)
        rfq.rfq_hif4_quantize(xin, out=[b.t for b in qb])
        _check_all(qb, "hif4_quantize %s" % tag)
    q = [b.t for b in qb]
    wb = hif4(N)
    rfq.rfq_hif4_quantize(torch.from_numpy(data["w"]).cuda(), residual=False,
                          out=[wb[0].t, wb[1].t, None, None])
    _check_all(wb, "hif4_quantize weight")
    for dt in (torch.float32, torch.bfloat16):
        d = Guarded((M, K), dt)
        rfq.rfq_hif4_dequant(q[0], q[1], out=d.t)
        d.check("hif4_dequant %s" % dt)
    wv = rfq.rfq_hif4_dequant(wb[0].t, wb[1].t, out_dtype=torch.bfloat16)
    for res in (True, False):
        for dt in (torch.float32, torch.bfloat16):
            z = Guarded((M, N), dt)
            rfq.rfq_hif4_gemm(q[0], q[1], q[2] if res else None, q[3] if res else None,
                              wb[0].t, wb[1].t, out=z.t)
            z.check("hif4_gemm res=%s %s" % (res, dt))
            z = Guarded((M, N), dt)
            rfq.rfq_hif4_gemm_wbf16(q[0], q[1], q[2] if res else None, q[3] if res else None,
                                    wv, out=z.t)
            z.check("hif4_gemm_wbf16 res=%s %s" % (res, dt))
    # The split product (where the shape splits): Z and the workspace.
    nb = rfq.rfq_hif4_gemm_workspace_bytes(M, N, K)
    if nb:
        for res in (True, False):
            for dt in (torch.float32, torch.bfloat16):
                z, wsb = Guarded((M, N), dt), Guarded((nb,), torch.uint8)
                rfq.rfq_hif4_gemm_split(q[0], q[1], q[2] if res else None, q[3] if res else None,
                                        wb[0].t, wb[1].t, wsb.t, out=z.t)
                z.check("hif4_gemm_split res=%s %s" % (res, dt))
                wsb.check("hif4_gemm_split workspace res=%s %s" % (res, dt))
