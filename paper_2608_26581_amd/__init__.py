"""RFQ (Residual Fallback Quantization) with MXFP4 and HiF4 codes on MI355X (gfx950).

The compute path is librfq.so (HIP kernels behind the C ABI in include/rfq.h);
this package holds its Python binding and the seeded synthetic workloads.
"""
from .rfq import (  # noqa: F401
    EXPORTS, LIB_PATH, MFMA_BF16_LOOP_FLOPS_PER_ITER, MFMA_LOOP_FLOPS_PER_ITER, MFMA_LOOP_ITEMS, RFQ_PHI_RESIDUAL_NONZERO, RFQ_PHI_SCALE_AT_LEAST, RfqError,
    interleave_gate_up, load, rfq_abi_version, rfq_dequant, rfq_fallback_map, rfq_gemm,
    rfq_gemm_phi, rfq_gemm_stream, rfq_gemm_swiglu_quantize, rfq_quantize_act, rfq_quantize_weight,
    rfq_hif4_dequant, rfq_hif4_gemm, rfq_hif4_gemm_split, rfq_hif4_gemm_wbf16,
    rfq_hif4_gemm_workspace_bytes, rfq_hif4_quantize, rfq_status_str,
    rfq_gemm_split, rfq_gemm_split_noalloc, rfq_gemm_workspace_bytes, rfq_mfma_bf16_loop, rfq_mfma_fp4_loop,
    rfq_swiglu_quantize_act,
)
