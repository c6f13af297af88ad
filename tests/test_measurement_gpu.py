"""The measurement-support loops of FP4 scaled MFMAs (rfq_mfma_fp4_loop)
and of bf16 MFMAs (rfq_mfma_bf16_loop), through the C ABI: they compute
what they state, so the rates they are timed at count the stated flops."""
import numpy as np
import pytest
import torch

import paper_2608_26581_amd as rfq
from gpu_util import host

pytestmark = pytest.mark.gpu


def test_mfma_loop_constant_operands_sum_exactly():
    """Code 0x2 is 1.0 and the scales are 1.0: every 32x32x64 MFMA adds 64 to
    each of a lane's 16 accumulator elements, eight accumulators per lane,
    so each work item's checksum is 8 * 16 * 64 * iters."""
    for iters in (1, 5, 2048):
        print("mfma loop constant iters=%d" % iters, flush=True)
        s = host(rfq.rfq_mfma_fp4_loop(iters, random_operands=False))
        assert s.shape == (rfq.MFMA_LOOP_ITEMS,)
        assert np.all(s == 8192.0 * iters), (iters, s[:4])


def test_mfma_loop_random_operands_are_deterministic():
    print("mfma loop random iters=3", flush=True)
    a = host(rfq.rfq_mfma_fp4_loop(3, random_operands=True))
    b = host(rfq.rfq_mfma_fp4_loop(3, random_operands=True))
    assert np.all(np.isfinite(a))
    assert np.array_equal(a, b)
    # Random codes differ from lane to lane: the checksums are not all equal.
    assert np.unique(a).size > 1000


def test_mfma_bf16_loop_constant_operands_sum_exactly():
    """bf16 1.0 operands: every 32x32x16 MFMA adds 16 to each of a lane's 16
    accumulator elements, eight accumulators per lane, so each work item's
    checksum is 8 * 16 * 16 * iters."""
    for iters in (1, 5, 8192):
        print("mfma bf16 loop constant iters=%d" % iters, flush=True)
        s = host(rfq.rfq_mfma_bf16_loop(iters, random_operands=False))
        assert s.shape == (rfq.MFMA_LOOP_ITEMS,)
        assert np.all(s == 2048.0 * iters), (iters, s[:4])


def test_mfma_bf16_loop_random_operands_are_finite_and_deterministic():
    print("mfma bf16 loop random iters=3", flush=True)
    a = host(rfq.rfq_mfma_bf16_loop(3, random_operands=True))
    b = host(rfq.rfq_mfma_bf16_loop(3, random_operands=True))
    assert np.all(np.isfinite(a))
    assert np.array_equal(a, b)
    assert np.unique(a).size > 1000
