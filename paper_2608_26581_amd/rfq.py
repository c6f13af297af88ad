"""Thin Python binding of librfq (C ABI declared in include/rfq.h).

Argument marshalling only: every step of the RFQ path runs in the HIP
kernels of librfq.so.  torch supplies device memory and the current HIP
stream.  There is no fallback of any kind: if the library is missing, or a
call fails, an exception is raised.

Each function carries the name of the C entry point it calls.  Tensors must be
contiguous device tensors on the current device; outputs are allocated when
not passed in.
"""
import ctypes
import os

import torch

_PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG_DIR, "librfq.so")

RFQ_F32 = 0
RFQ_BF16 = 1

_STATUS_NAMES = {
    0: "RFQ_OK", 1: "RFQ_ERR_NULL", 2: "RFQ_ERR_SHAPE", 3: "RFQ_ERR_DTYPE",
    4: "RFQ_ERR_ALIGN", 5: "RFQ_ERR_DEVICE", 6: "RFQ_ERR_LAUNCH",
}

# Every symbol declared in include/rfq.h.
EXPORTS = (
    "rfq_quantize_act", "rfq_quantize_weight", "rfq_gemm", "rfq_dequant",
    "rfq_swiglu_quantize_act", "rfq_gemm_phi", "rfq_fallback_map", "rfq_gemm_swiglu_quantize",
    "rfq_gemm_stream", "rfq_hif4_quantize", "rfq_hif4_dequant", "rfq_hif4_gemm",
    "rfq_hif4_gemm_wbf16", "rfq_mfma_fp4_loop", "rfq_mfma_bf16_loop", "rfq_gemm_split",
    "rfq_gemm_workspace_bytes",
    "rfq_gemm_split_noalloc", "rfq_hif4_gemm_split", "rfq_hif4_gemm_workspace_bytes",
    "rfq_status_str", "rfq_abi_version",
)

# Work items of rfq_mfma_fp4_loop (256 workgroups of 512) and its flops per
# iteration (each of the 2048 waves issues 8 MFMAs of 32 x 32 x 64).
MFMA_LOOP_ITEMS = 256 * 512
MFMA_LOOP_FLOPS_PER_ITER = 256 * 8 * 8 * 2 * 32 * 32 * 64
# rfq_mfma_bf16_loop: the same grid, 8 MFMAs of 32 x 32 x 16 per wave and iteration.
MFMA_BF16_LOOP_FLOPS_PER_ITER = 256 * 8 * 8 * 2 * 32 * 32 * 16

RFQ_PHI_RESIDUAL_NONZERO = 0
RFQ_PHI_SCALE_AT_LEAST = 1

_lib = None


class RfqError(RuntimeError):
    """A librfq call returned a status other than RFQ_OK."""

    def __init__(self, func, status):
        self.status = status
        super().__init__("%s failed: %s (%s)" % (
            func, _STATUS_NAMES.get(status, status), rfq_status_str(status)))


def load():
    """Loads librfq.so once; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            "librfq.so is not built (expected at %s); run __graft_entry__.build()" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    P, I64, I32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    lib.rfq_quantize_act.argtypes = [P, I32, I64, I64, P, P, P, P, P]
    lib.rfq_quantize_weight.argtypes = [P, I32, I64, I64, P, P, P]
    lib.rfq_gemm.argtypes = [P, P, P, P, P, P, I64, I64, I64, P, I32, P]
    lib.rfq_dequant.argtypes = [P, P, I64, I64, P, P]
    lib.rfq_swiglu_quantize_act.argtypes = [P, P, I32, I64, I64, P, P, P, P, P, P]
    lib.rfq_gemm_swiglu_quantize.argtypes = [P, P, P, P, P, P, I64, I64, I64, P, P, P, P, P, P]
    lib.rfq_gemm_phi.argtypes = [P, P, P, P, P, P, P, I64, I64, I64, P, I32, P]
    lib.rfq_fallback_map.argtypes = [P, P, I64, I64, I32, I32, P, P]
    lib.rfq_gemm_stream.argtypes = [P, I32, I32, P, P, I64, I64, I64, P, I32, P]
    lib.rfq_hif4_quantize.argtypes = [P, I32, I64, I64, P, P, P, P, P]
    lib.rfq_hif4_dequant.argtypes = [P, P, I64, I64, P, I32, P]
    lib.rfq_hif4_gemm.argtypes = [P, P, P, P, P, P, I64, I64, I64, P, I32, P]
    lib.rfq_hif4_gemm_wbf16.argtypes = [P, P, P, P, P, I64, I64, I64, P, I32, P]
    lib.rfq_mfma_fp4_loop.argtypes = [I64, I32, P, P]
    lib.rfq_mfma_bf16_loop.argtypes = [I64, I32, P, P]
    lib.rfq_gemm_split.argtypes = [P, P, P, P, P, P, I64, I64, I64, P, I32, P, I64, P]
    lib.rfq_gemm_split_noalloc.argtypes = [P, P, P, P, P, P, I64, I64, I64, P, I32, P]
    lib.rfq_gemm_workspace_bytes.argtypes = [I64, I64, I64]
    lib.rfq_gemm_workspace_bytes.restype = I64
    lib.rfq_hif4_gemm_split.argtypes = [P, P, P, P, P, P, I64, I64, I64, P, I32, P, I64, P]
    lib.rfq_hif4_gemm_workspace_bytes.argtypes = [I64, I64, I64]
    lib.rfq_hif4_gemm_workspace_bytes.restype = I64
    for f in ("rfq_quantize_act", "rfq_quantize_weight", "rfq_gemm", "rfq_dequant",
              "rfq_swiglu_quantize_act", "rfq_gemm_swiglu_quantize", "rfq_gemm_phi",
              "rfq_fallback_map", "rfq_gemm_stream", "rfq_hif4_quantize", "rfq_hif4_dequant",
              "rfq_hif4_gemm", "rfq_hif4_gemm_wbf16", "rfq_mfma_fp4_loop", "rfq_mfma_bf16_loop",
              "rfq_gemm_split", "rfq_hif4_gemm_split",
              "rfq_gemm_split_noalloc"):
        getattr(lib, f).restype = I32
    lib.rfq_status_str.argtypes = [I32]
    lib.rfq_status_str.restype = ctypes.c_char_p
    lib.rfq_abi_version.argtypes = []
    lib.rfq_abi_version.restype = I32
    _lib = lib
    return lib


def rfq_status_str(status):
    return load().rfq_status_str(int(status)).decode()


def rfq_abi_version():
    return int(load().rfq_abi_version())


def _ptr(t):
    return None if t is None else t.data_ptr()


# The current stream's raw handle: torch's direct accessor when it has one
# (a fraction of a microsecond), else the public Stream object (a few).
_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)


def _stream(stream, dev=None):
    if stream is not None:
        return stream.cuda_stream
    if _raw_stream is not None:
        return _raw_stream(torch.cuda.current_device() if dev is None else dev)
    return torch.cuda.current_stream().cuda_stream


def _check(func, status):
    if status != 0:
        raise RfqError(func, status)


def _dtype_code(t):
    if t.dtype == torch.bfloat16:
        return RFQ_BF16
    if t.dtype == torch.float32:
        return RFQ_F32
    raise TypeError("unsupported dtype %s (bf16 or fp32)" % t.dtype)


# Argument checks.  The C ABI takes raw pointers and cannot see how large a
# buffer is or where it lives, so every tensor is checked here before its
# pointer is passed on: a device tensor of the current device, contiguous,
# of the stated dtype and exact shape.

def _need(t, name, dtypes=None, shape=None, dev=None):
    """Raises unless t is a contiguous tensor of device dev (default: the
    current device) with a dtype in dtypes and the given shape.  One combined
    test on the common path: the binding runs once per call of small
    decode-sized products, where host time counts."""
    try:
        if (t.is_cuda and t.is_contiguous() and (dtypes is None or t.dtype in dtypes)
                and (shape is None or t.shape == shape)
                and t.get_device() == (torch.cuda.current_device() if dev is None else dev)):
            return
    except AttributeError:
        pass
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    cur = torch.cuda.current_device() if dev is None else dev
    if t.get_device() != cur:
        raise ValueError("%s is on %s, not on the current device cuda:%d" % (name, t.device, cur))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if dtypes is not None and t.dtype not in dtypes:
        raise TypeError("%s must be %s, not %s" % (name, " or ".join(map(str, dtypes)), t.dtype))
    raise ValueError("%s must have shape %s, not %s" % (name, tuple(shape), tuple(t.shape)))


_U8 = (torch.uint8,)
_FLOAT = (torch.float32, torch.bfloat16)


def _ok(t, dtypes, shape, dev):
    """The common case of _need in one expression (no message to build)."""
    try:
        return (t.is_cuda and t.is_contiguous() and t.dtype in dtypes and t.shape == shape
                and t.get_device() == dev)
    except AttributeError:
        return False


def _need_codes(codes, scales, rows, K, name, dev=None):
    """An MXFP4 operand: codes [rows][K/2] and scales [rows][K/32], uint8."""
    if (dev is not None and _ok(codes, _U8, (rows, K // 2), dev)
            and _ok(scales, _U8, (rows, K // 32), dev)):
        return
    _need(codes, name + " codes", _U8, (rows, K // 2), dev)
    _need(scales, name + " scales", _U8, (rows, K // 32), dev)


def _need_pair(codes, scales, rows, K, name, dev=None):
    """An optional operand: both tensors or neither."""
    if (codes is None) != (scales is None):
        raise ValueError("%s codes and scales must both be given or both be None" % name)
    if codes is not None:
        _need_codes(codes, scales, rows, K, name, dev)


def _shape_of_codes(codes, name):
    """(rows, K) of a codes tensor [rows][K/2]."""
    if not isinstance(codes, torch.Tensor) or codes.dim() != 2:
        raise ValueError("%s must be a 2-D tensor [rows][K/2]" % name)
    return codes.shape[0], codes.shape[1] * 2


def _codes_out(rows, K, device):
    return (torch.empty((rows, K // 2), dtype=torch.uint8, device=device),
            torch.empty((rows, K // 32), dtype=torch.uint8, device=device))


def _outputs(out, rows, K, device, residual, name, dev=None):
    """Codes outputs (qc, qs, rc, rs): allocated, or the caller's checked."""
    if out is None:
        qc, qs = _codes_out(rows, K, device)
        rc, rs = _codes_out(rows, K, device) if residual else (None, None)
        return qc, qs, rc, rs
    qc, qs, rc, rs = out
    _need_codes(qc, qs, rows, K, name + " primary", dev)
    _need_pair(rc, rs, rows, K, name + " residual", dev)
    return qc, qs, rc, rs


def _z_out(out, out_dtype, M, N, device, dev=None):
    if out is None:
        if out_dtype not in _FLOAT:
            raise TypeError("out_dtype must be torch.float32 or torch.bfloat16")
        return torch.empty((M, N), dtype=out_dtype, device=device)
    if dev is None or not _ok(out, _FLOAT, (M, N), dev):
        _need(out, "out", _FLOAT, (M, N), dev)
    return out


def rfq_quantize_act(x, residual=True, out=None, stream=None):
    """X[M][K] -> (q_codes, q_scales, r_codes, r_scales); r_* are None when
    residual is False.  out may supply the four (or two) output tensors."""
    _need(x, "x", _FLOAT)
    dev = x.get_device()
    if x.dim() != 2:
        raise ValueError("x must be 2-D [M][K]")
    M, K = x.shape
    qc, qs, rc, rs = _outputs(out, M, K, x.device, residual, "out", dev)
    st = load().rfq_quantize_act(_ptr(x), _dtype_code(x), M, K, _ptr(qc), _ptr(qs),
                                 _ptr(rc), _ptr(rs), _stream(stream, dev))
    _check("rfq_quantize_act", st)
    return qc, qs, rc, rs


def rfq_quantize_weight(w, out=None, stream=None):
    """W[N][K] -> (w_codes, w_scales)."""
    _need(w, "w", _FLOAT)
    if w.dim() != 2:
        raise ValueError("w must be 2-D [N][K]")
    N, K = w.shape
    if out is None:
        wc, ws = _codes_out(N, K, w.device)
    else:
        wc, ws = out
        _need_codes(wc, ws, N, K, "out")
    st = load().rfq_quantize_weight(_ptr(w), _dtype_code(w), N, K, _ptr(wc), _ptr(ws),
                                    _stream(stream))
    _check("rfq_quantize_weight", st)
    return wc, ws


def rfq_gemm_workspace_bytes(M, N, K):
    """Workspace rfq_gemm_split splits K with for this shape (0: no split)."""
    return int(load().rfq_gemm_workspace_bytes(int(M), int(N), int(K)))


def rfq_gemm(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales,
             out_dtype=torch.float32, out=None, stream=None, split=False):
    """Z[M][N] = (deq q + deq r) deq(w)^T; r_* None gives plain MXFP4.
    split=True: rfq_gemm_split with a workspace from torch's allocator where
    the shape splits K (a different fp32 summation order)."""
    M, K = _shape_of_codes(q_codes, "q codes")
    N, Kw = _shape_of_codes(w_codes, "w codes")
    if Kw != K:
        raise ValueError("K mismatch between activation and weight codes")
    _need(q_codes, "q codes", _U8, (M, K // 2))
    dev = q_codes.get_device()
    _need_codes(q_codes, q_scales, M, K, "q", dev)
    _need_pair(r_codes, r_scales, M, K, "r", dev)
    _need_codes(w_codes, w_scales, N, K, "w", dev)
    z = _z_out(out, out_dtype, M, N, q_codes.device, dev)
    if split:
        nbytes = load().rfq_gemm_workspace_bytes(M, N, K)
        if nbytes > 0:
            ws = torch.empty(nbytes, dtype=torch.uint8, device=q_codes.device)
            st = load().rfq_gemm_split(_ptr(q_codes), _ptr(q_scales), _ptr(r_codes),
                                       _ptr(r_scales), _ptr(w_codes), _ptr(w_scales), M, N, K,
                                       _ptr(z), _dtype_code(z), _ptr(ws), nbytes,
                                       _stream(stream, dev))
            _check("rfq_gemm_split", st)
            return z
    st = load().rfq_gemm(_ptr(q_codes), _ptr(q_scales), _ptr(r_codes), _ptr(r_scales),
                         _ptr(w_codes), _ptr(w_scales), M, N, K, _ptr(z), _dtype_code(z),
                         _stream(stream, dev))
    _check("rfq_gemm", st)
    return z


def rfq_gemm_split_noalloc(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales,
                           out=None, out_dtype=torch.float32, stream=None):
    """rfq_gemm_split on the library's static device scratch array (no
    device allocation in the library; pass `out` to allocate nothing here
    either)."""
    M, K = _shape_of_codes(q_codes, "q codes")
    N, Kw = _shape_of_codes(w_codes, "w codes")
    if Kw != K:
        raise ValueError("K mismatch between activation and weight codes")
    _need(q_codes, "q codes", _U8, (M, K // 2))
    dev = q_codes.get_device()
    _need_codes(q_codes, q_scales, M, K, "q", dev)
    _need_pair(r_codes, r_scales, M, K, "r", dev)
    _need_codes(w_codes, w_scales, N, K, "w", dev)
    z = _z_out(out, out_dtype, M, N, q_codes.device, dev)
    st = load().rfq_gemm_split_noalloc(_ptr(q_codes), _ptr(q_scales), _ptr(r_codes),
                                       _ptr(r_scales), _ptr(w_codes), _ptr(w_scales), M, N, K,
                                       _ptr(z), _dtype_code(z), _stream(stream, dev))
    _check("rfq_gemm_split_noalloc", st)
    return z


def rfq_gemm_split(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, workspace,
                   out_dtype=torch.float32, out=None, stream=None):
    """rfq_gemm with K split over workgroups where the shape calls for it;
    workspace: a contiguous device uint8 tensor (rfq_gemm_workspace_bytes
    long, or shorter to run unsplit) or None."""
    M, K = _shape_of_codes(q_codes, "q codes")
    N, Kw = _shape_of_codes(w_codes, "w codes")
    if Kw != K:
        raise ValueError("K mismatch between activation and weight codes")
    _need(q_codes, "q codes", _U8, (M, K // 2))
    dev = q_codes.get_device()
    _need_codes(q_codes, q_scales, M, K, "q", dev)
    _need_pair(r_codes, r_scales, M, K, "r", dev)
    _need_codes(w_codes, w_scales, N, K, "w", dev)
    nbytes = 0
    if workspace is not None:
        _need(workspace, "workspace", _U8, None, dev)
        nbytes = workspace.numel()
    z = _z_out(out, out_dtype, M, N, q_codes.device, dev)
    st = load().rfq_gemm_split(_ptr(q_codes), _ptr(q_scales), _ptr(r_codes), _ptr(r_scales),
                               _ptr(w_codes), _ptr(w_scales), M, N, K, _ptr(z), _dtype_code(z),
                               _ptr(workspace), nbytes, _stream(stream, dev))
    _check("rfq_gemm_split", st)
    return z


def rfq_gemm_stream(x, w_codes, w_scales, residual=True, out_dtype=torch.float32, out=None,
                    stream=None):
    """Streaming form: Z[M][N] from X[M][K] (bf16 or fp32) quantized inside the
    product's K loop (primary and, with residual, the quantized residual)."""
    _need(x, "x", _FLOAT)
    dev = x.get_device()
    if x.dim() != 2:
        raise ValueError("x must be 2-D [M][K]")
    M, K = x.shape
    N, Kw = _shape_of_codes(w_codes, "w codes")
    if Kw != K:
        raise ValueError("K mismatch between activations and weight codes")
    _need_codes(w_codes, w_scales, N, K, "w", dev)
    z = _z_out(out, out_dtype, M, N, x.device, dev)
    st = load().rfq_gemm_stream(_ptr(x), _dtype_code(x), int(bool(residual)), _ptr(w_codes),
                                _ptr(w_scales), M, N, K, _ptr(z), _dtype_code(z),
                                _stream(stream, dev))
    _check("rfq_gemm_stream", st)
    return z


def rfq_gemm_phi(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, phi,
                 out_dtype=torch.float32, out=None, stream=None):
    """RFQ product with a fallback-indicator map phi[ceil(M/64)][ceil(K/256)]
    (uint8; None: phi = 1)."""
    M, K = _shape_of_codes(q_codes, "q codes")
    N, Kw = _shape_of_codes(w_codes, "w codes")
    if Kw != K:
        raise ValueError("K mismatch between activation and weight codes")
    _need_codes(q_codes, q_scales, M, K, "q")
    _need_pair(r_codes, r_scales, M, K, "r")
    _need_codes(w_codes, w_scales, N, K, "w")
    if phi is not None:
        _need(phi, "phi", _U8, ((M + 63) // 64, (K + 255) // 256))
    z = _z_out(out, out_dtype, M, N, q_codes.device)
    st = load().rfq_gemm_phi(_ptr(q_codes), _ptr(q_scales), _ptr(r_codes), _ptr(r_scales),
                             _ptr(w_codes), _ptr(w_scales), _ptr(phi), M, N, K, _ptr(z),
                             _dtype_code(z), _stream(stream))
    _check("rfq_gemm_phi", st)
    return z


def rfq_fallback_map(r_codes, q_scales, rule, threshold=0, out=None, stream=None):
    """phi[ceil(M/64)][ceil(K/256)] by RFQ_PHI_RESIDUAL_NONZERO (reads r_codes)
    or RFQ_PHI_SCALE_AT_LEAST (reads q_scales; phi = 1 where a scale byte >=
    threshold)."""
    if not isinstance(q_scales, torch.Tensor) or q_scales.dim() != 2:
        raise ValueError("q_scales must be a 2-D tensor [M][K/32] (it gives M and K)")
    M, K = q_scales.shape[0], q_scales.shape[1] * 32
    if rule == RFQ_PHI_RESIDUAL_NONZERO:
        _need(r_codes, "r codes", _U8, (M, K // 2))
    else:
        _need(q_scales, "q scales", _U8, (M, K // 32))
    shape = ((M + 63) // 64, (K + 255) // 256)
    if out is None:
        phi = torch.empty(shape, dtype=torch.uint8, device=q_scales.device)
    else:
        phi = out
        _need(phi, "out", _U8, shape)
    st = load().rfq_fallback_map(_ptr(r_codes), _ptr(q_scales), M, K, int(rule), int(threshold),
                                 _ptr(phi), _stream(stream))
    _check("rfq_fallback_map", st)
    return phi


def rfq_mfma_fp4_loop(iters, random_operands=True, sink=None, stream=None):
    """Measurement support: a register-only loop of FP4 scaled MFMAs on every
    CU (MFMA_LOOP_FLOPS_PER_ITER flops per iteration); returns the sink of
    one fp32 checksum per work item."""
    if sink is None:
        sink = torch.empty(MFMA_LOOP_ITEMS, dtype=torch.float32, device="cuda")
    else:
        _need(sink, "sink", (torch.float32,), (MFMA_LOOP_ITEMS,))
    st = load().rfq_mfma_fp4_loop(int(iters), 1 if random_operands else 0, _ptr(sink),
                                  _stream(stream, sink.get_device()))
    _check("rfq_mfma_fp4_loop", st)
    return sink


def rfq_mfma_bf16_loop(iters, random_operands=True, sink=None, stream=None):
    """Measurement support: rfq_mfma_fp4_loop on the bf16 matrix cores
    (MFMA_BF16_LOOP_FLOPS_PER_ITER flops per iteration)."""
    if sink is None:
        sink = torch.empty(MFMA_LOOP_ITEMS, dtype=torch.float32, device="cuda")
    else:
        _need(sink, "sink", (torch.float32,), (MFMA_LOOP_ITEMS,))
    st = load().rfq_mfma_bf16_loop(int(iters), 1 if random_operands else 0, _ptr(sink),
                                   _stream(stream, sink.get_device()))
    _check("rfq_mfma_bf16_loop", st)
    return sink


def rfq_dequant(codes, scales, out=None, stream=None):
    """codes[rows][K/2], scales[rows][K/32] -> fp32 [rows][K]."""
    rows, K = _shape_of_codes(codes, "codes")
    _need_codes(codes, scales, rows, K, "dequantization input")
    if out is None:
        o = torch.empty((rows, K), dtype=torch.float32, device=codes.device)
    else:
        o = out
        _need(o, "out", (torch.float32,), (rows, K))
    st = load().rfq_dequant(_ptr(codes), _ptr(scales), rows, K, _ptr(o), _stream(stream))
    _check("rfq_dequant", st)
    return o


def rfq_swiglu_quantize_act(g, u, residual=True, return_h=False, out=None, stream=None):
    """h = bf16(silu(g) * u) -> RFQ codes; returns (qc, qs, rc, rs, h or None)."""
    _need(g, "g", _FLOAT)
    _need(u, "u", _FLOAT)
    if g.shape != u.shape or g.dtype != u.dtype or g.dim() != 2:
        raise ValueError("g and u must be 2-D with the same shape and dtype")
    M, Nh = g.shape
    qc, qs, rc, rs = _outputs(out, M, Nh, g.device, residual, "out")
    h = torch.empty((M, Nh), dtype=torch.bfloat16, device=g.device) if return_h else None
    st = load().rfq_swiglu_quantize_act(_ptr(g), _ptr(u), _dtype_code(g), M, Nh, _ptr(qc),
                                        _ptr(qs), _ptr(rc), _ptr(rs), _ptr(h), _stream(stream))
    _check("rfq_swiglu_quantize_act", st)
    return qc, qs, rc, rs, h


def rfq_gemm_swiglu_quantize(q_codes, q_scales, r_codes, r_scales, wgu_codes, wgu_scales,
                             residual=True, return_h=False, out=None, stream=None):
    """Gate/up product with SwiGLU + RFQ quantization of h in its epilogue.
    wgu_* are the quantized interleaved gate/up weights [2 Nh][K]
    (interleave_gate_up).  Returns (hq_codes, hq_scales, hr_codes, hr_scales,
    h or None); hr_* are None when residual is False."""
    M, K = _shape_of_codes(q_codes, "q codes")
    N2, Kw = _shape_of_codes(wgu_codes, "gate/up codes")
    if Kw != K:
        raise ValueError("K mismatch between activation and weight codes")
    if N2 % 2:
        raise ValueError("gate/up codes must have an even number of rows [2 Nh][K/2]")
    Nh = N2 // 2
    _need_codes(q_codes, q_scales, M, K, "q")
    _need_pair(r_codes, r_scales, M, K, "r")
    _need_codes(wgu_codes, wgu_scales, N2, K, "gate/up")
    hqc, hqs, hrc, hrs = _outputs(out, M, Nh, q_codes.device, residual, "out")
    h = (torch.empty((M, Nh), dtype=torch.bfloat16, device=q_codes.device)
         if return_h else None)
    st = load().rfq_gemm_swiglu_quantize(
        _ptr(q_codes), _ptr(q_scales), _ptr(r_codes), _ptr(r_scales), _ptr(wgu_codes),
        _ptr(wgu_scales), M, Nh, K, _ptr(hqc), _ptr(hqs), _ptr(hrc), _ptr(hrs), _ptr(h),
        _stream(stream))
    _check("rfq_gemm_swiglu_quantize", st)
    return hqc, hqs, hrc, hrs, h


# ---- HiF4 (64-element blocks; codes [rows][K/2] uint8, meta [rows][K/64]
# int32 holding the uint32 metadata words bit for bit).

_I32 = (torch.int32,)


def _need_hif4(codes, meta, rows, K, name, dev=None):
    if (dev is not None and _ok(codes, _U8, (rows, K // 2), dev)
            and _ok(meta, _I32, (rows, K // 64), dev)):
        return
    _need(codes, name + " codes", _U8, (rows, K // 2), dev)
    _need(meta, name + " meta", _I32, (rows, K // 64), dev)


def _hif4_out(rows, K, device):
    return (torch.empty((rows, K // 2), dtype=torch.uint8, device=device),
            torch.empty((rows, K // 64), dtype=torch.int32, device=device))


def rfq_hif4_quantize(x, residual=True, out=None, stream=None):
    """X[rows][K] (K a multiple of 64) -> (q_codes, q_meta, r_codes, r_meta)
    in HiF4; r_* are None when residual is False (the weight quantizer)."""
    _need(x, "x", _FLOAT)
    dev = x.get_device()
    if x.dim() != 2:
        raise ValueError("x must be 2-D [rows][K]")
    rows, K = x.shape
    if out is None:
        qc, qm = _hif4_out(rows, K, x.device)
        rc, rm = _hif4_out(rows, K, x.device) if residual else (None, None)
    else:
        qc, qm, rc, rm = out
        _need_hif4(qc, qm, rows, K, "out primary", dev)
        if (rc is None) != (rm is None):
            raise ValueError("residual codes and meta must both be given or both be None")
        if rc is not None:
            _need_hif4(rc, rm, rows, K, "out residual", dev)
    st = load().rfq_hif4_quantize(_ptr(x), _dtype_code(x), rows, K, _ptr(qc), _ptr(qm),
                                  _ptr(rc), _ptr(rm), _stream(stream, dev))
    _check("rfq_hif4_quantize", st)
    return qc, qm, rc, rm


def rfq_hif4_dequant(codes, meta, out_dtype=torch.float32, out=None, stream=None):
    """HiF4 codes[rows][K/2], meta[rows][K/64] -> [rows][K] fp32 or bf16
    (exact either way)."""
    rows, K = _shape_of_codes(codes, "codes")
    _need_hif4(codes, meta, rows, K, "dequantization input")
    dev = codes.get_device()
    if out is None:
        if out_dtype not in _FLOAT:
            raise TypeError("out_dtype must be torch.float32 or torch.bfloat16")
        o = torch.empty((rows, K), dtype=out_dtype, device=codes.device)
    else:
        o = out
        _need(o, "out", _FLOAT, (rows, K), dev)
    st = load().rfq_hif4_dequant(_ptr(codes), _ptr(meta), rows, K, _ptr(o), _dtype_code(o),
                                 _stream(stream, dev))
    _check("rfq_hif4_dequant", st)
    return o


def _hif4_operands(q_codes, q_meta, r_codes, r_meta, w_codes, w_meta):
    """(M, N, K, device) of a HiF4 product's checked operands."""
    M, K = _shape_of_codes(q_codes, "q codes")
    N, Kw = _shape_of_codes(w_codes, "w codes")
    if Kw != K:
        raise ValueError("K mismatch between activation and weight codes")
    _need(q_codes, "q codes", _U8, (M, K // 2))
    dev = q_codes.get_device()
    _need_hif4(q_codes, q_meta, M, K, "q", dev)
    if (r_codes is None) != (r_meta is None):
        raise ValueError("r codes and meta must both be given or both be None")
    if r_codes is not None:
        _need_hif4(r_codes, r_meta, M, K, "r", dev)
    _need_hif4(w_codes, w_meta, N, K, "w", dev)
    return M, N, K, dev


def rfq_hif4_gemm(q_codes, q_meta, r_codes, r_meta, w_codes, w_meta,
                  out_dtype=torch.float32, out=None, stream=None, split=False):
    """HiF4 RFQ product Z[M][N] = (V_q + V_r) V_w^T; r_* None: primary only.
    split=True: rfq_hif4_gemm_split with a workspace from torch's allocator
    where the shape splits K (a different fp32 summation order) or decodes
    the weights into it (the same bits)."""
    M, N, K, dev = _hif4_operands(q_codes, q_meta, r_codes, r_meta, w_codes, w_meta)
    z = _z_out(out, out_dtype, M, N, q_codes.device, dev)
    if split:
        nbytes = load().rfq_hif4_gemm_workspace_bytes(M, N, K)
        if nbytes > 0:
            ws = torch.empty(nbytes, dtype=torch.uint8, device=q_codes.device)
            st = load().rfq_hif4_gemm_split(_ptr(q_codes), _ptr(q_meta), _ptr(r_codes),
                                            _ptr(r_meta), _ptr(w_codes), _ptr(w_meta), M, N, K,
                                            _ptr(z), _dtype_code(z), _ptr(ws), nbytes,
                                            _stream(stream, dev))
            _check("rfq_hif4_gemm_split", st)
            return z
    st = load().rfq_hif4_gemm(_ptr(q_codes), _ptr(q_meta), _ptr(r_codes), _ptr(r_meta),
                              _ptr(w_codes), _ptr(w_meta), M, N, K, _ptr(z), _dtype_code(z),
                              _stream(stream, dev))
    _check("rfq_hif4_gemm", st)
    return z


def rfq_hif4_gemm_workspace_bytes(M, N, K):
    """Workspace rfq_hif4_gemm_split splits K with for this shape (0: no split)."""
    return int(load().rfq_hif4_gemm_workspace_bytes(int(M), int(N), int(K)))


def rfq_hif4_gemm_split(q_codes, q_meta, r_codes, r_meta, w_codes, w_meta, workspace,
                        out_dtype=torch.float32, out=None, stream=None):
    """rfq_hif4_gemm with K split over workgroups where the shape calls for
    it, or (from 1024 rows) with the weights decoded to bf16 in the workspace
    first (the same bits); workspace: a contiguous device uint8 tensor
    (rfq_hif4_gemm_workspace_bytes long, or shorter to run rfq_hif4_gemm) or
    None."""
    M, N, K, dev = _hif4_operands(q_codes, q_meta, r_codes, r_meta, w_codes, w_meta)
    nbytes = 0
    if workspace is not None:
        _need(workspace, "workspace", _U8, None, dev)
        nbytes = workspace.numel()
    z = _z_out(out, out_dtype, M, N, q_codes.device, dev)
    st = load().rfq_hif4_gemm_split(_ptr(q_codes), _ptr(q_meta), _ptr(r_codes), _ptr(r_meta),
                                    _ptr(w_codes), _ptr(w_meta), M, N, K, _ptr(z),
                                    _dtype_code(z), _ptr(workspace), nbytes,
                                    _stream(stream, dev))
    _check("rfq_hif4_gemm_split", st)
    return z


def rfq_hif4_gemm_wbf16(q_codes, q_meta, r_codes, r_meta, w_bf16, out_dtype=torch.float32,
                        out=None, stream=None):
    """HiF4 RFQ product with bf16 weights w[N][K] (e.g. rfq_hif4_dequant of
    HiF4 weight codes with out_dtype=torch.bfloat16, decoded once)."""
    M, K = _shape_of_codes(q_codes, "q codes")
    _need(q_codes, "q codes", _U8, (M, K // 2))
    dev = q_codes.get_device()
    _need_hif4(q_codes, q_meta, M, K, "q", dev)
    if (r_codes is None) != (r_meta is None):
        raise ValueError("r codes and meta must both be given or both be None")
    if r_codes is not None:
        _need_hif4(r_codes, r_meta, M, K, "r", dev)
    if not isinstance(w_bf16, torch.Tensor) or w_bf16.dim() != 2 or w_bf16.shape[1] != K:
        raise ValueError("w_bf16 must be a 2-D tensor [N][K] with the activations' K")
    N = w_bf16.shape[0]
    _need(w_bf16, "w_bf16", (torch.bfloat16,), (N, K), dev)
    z = _z_out(out, out_dtype, M, N, q_codes.device, dev)
    st = load().rfq_hif4_gemm_wbf16(_ptr(q_codes), _ptr(q_meta), _ptr(r_codes), _ptr(r_meta),
                                    _ptr(w_bf16), M, N, K, _ptr(z), _dtype_code(z),
                                    _stream(stream, dev))
    _check("rfq_hif4_gemm_wbf16", st)
    return z


def interleave_gate_up(gate, up):
    """Rows of gate [Nh][...] and up [Nh][...] interleaved in groups of 32
    (the weight layout rfq_gemm_swiglu_quantize takes).  Works on fp32
    weights and, equivalently, on their codes or scales, since weights are
    quantized row by row.  A one-off layout step, not part of the path."""
    if gate.shape != up.shape or gate.shape[0] % 32:
        raise ValueError("gate and up must have the same shape, rows a multiple of 32")
    nh = gate.shape[0]
    g = gate.reshape(nh // 32, 32, *gate.shape[1:])
    u = up.reshape(nh // 32, 32, *up.shape[1:])
    return torch.stack((g, u), dim=1).reshape(2 * nh, *gate.shape[1:]).contiguous()
