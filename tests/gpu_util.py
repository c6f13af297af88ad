"""Helpers for the GPU parity tests: host/device transfer and the tolerance
of the RFQ product.

Tolerance of the product (written from the arithmetic): every product of two
codes is exact, so the only error of an fp32 evaluation is the rounding of
its sums.  With at most 2K terms in any order the worst case is gamma_2K <
2^-10 for K <= 8192 (and about 2^-9.4 at K = 12288, where random-sign sums
stay far below it), relative to the bound B = sum_k |q w| + |r w|:

    |Z_gpu - Z_ref| <= 2^-10 * B                      (fp32 output)
    |Z_gpu - Z_ref| <= 2^-10 * B + 2^-8 * |Z_ref|     (bf16 output: plus half
                                                       a bf16 ulp <= 2^-9 |Z|)
"""
import numpy as np
import torch

TOL_SUM = 2.0 ** -10
TOL_BF16 = 2.0 ** -8


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def dev_bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def host(t):
    return t.cpu().numpy()


def host_bf16_as_f32(t):
    b = t.view(torch.int16).cpu().numpy().view(np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def x_device(data):
    """Device tensor of a workload's activations in its own dtype."""
    if data["x_bf16"] is not None:
        return dev_bf16(data["x_bf16"])
    return dev(data["x"])


def assert_gemm_close(z_gpu, z_ref, bound, bf16_out=False, what=""):
    z_gpu = np.asarray(z_gpu, np.float64)
    tol = TOL_SUM * bound + (TOL_BF16 * np.abs(z_ref) if bf16_out else 0.0)
    err = np.abs(z_gpu - z_ref)
    bad = err > tol
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError("%s: %d outputs out of tolerance; first at %s: gpu %r ref %r "
                             "bound %r" % (what, int(bad.sum()), tuple(i), z_gpu[tuple(i)],
                                           z_ref[tuple(i)], bound[tuple(i)]))
