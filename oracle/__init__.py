"""Python access to the CPU oracle (oracle/rfq_oracle.c for MXFP4,
oracle/hif4_oracle.c for HiF4) through ctypes.

TEST INFRASTRUCTURE ONLY: imported by the test suite, by the smoke check and
by the CPU-baseline leg of the benchmark, never by the product path.  It shares
no code with the GPU library; inputs arrive as numpy arrays.
"""
import ctypes
import os
import subprocess

import numpy as np

ORACLE_DIR = os.path.dirname(os.path.abspath(__file__))
SRCS = [os.path.join(ORACLE_DIR, "rfq_oracle.c"), os.path.join(ORACLE_DIR, "hif4_oracle.c")]
LIB = os.path.join(ORACLE_DIR, "liboracle.so")
CFLAGS = ["-O2", "-std=c99", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra"]

_lib = None


def build(extra_flags=(), out=LIB):
    """Compile the oracle with gcc (plain -O2, no fast-math)."""
    cmd = ["gcc", *CFLAGS, *extra_flags, *SRCS, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def _load(path=LIB):
    D = ctypes.POINTER(ctypes.c_double)
    U8 = ctypes.POINTER(ctypes.c_uint8)
    I64 = ctypes.c_int64
    lib = ctypes.CDLL(path)
    lib.oracle_e2m1_value.argtypes = [ctypes.c_int]
    lib.oracle_e2m1_value.restype = ctypes.c_double
    lib.oracle_e2m1_encode.argtypes = [ctypes.c_double]
    lib.oracle_e2m1_encode.restype = ctypes.c_int
    lib.oracle_block_exponent.argtypes = [ctypes.c_double]
    lib.oracle_block_exponent.restype = ctypes.c_int
    lib.oracle_round_bf16.argtypes = [ctypes.c_double]
    lib.oracle_round_bf16.restype = ctypes.c_double
    lib.oracle_rfq_quantize.argtypes = [D, I64, I64, U8, U8, U8, U8]
    lib.oracle_dequant.argtypes = [U8, U8, I64, I64, D]
    lib.oracle_gemm.argtypes = [U8, U8, U8, U8, U8, U8, I64, I64, I64, D, D]
    lib.oracle_gemm_phi.argtypes = [U8, U8, U8, U8, U8, U8, U8, I64, I64, I64, D, D]
    lib.oracle_fallback_map.argtypes = [U8, U8, I64, I64, ctypes.c_int, ctypes.c_int, U8]
    lib.oracle_gemm_sampled.argtypes = [U8, U8, U8, U8, U8, U8, I64,
                                        ctypes.POINTER(ctypes.c_int64),
                                        ctypes.POINTER(ctypes.c_int64), I64, D, D]
    lib.oracle_swiglu.argtypes = [D, D, I64, D]
    lib.oracle_residual.argtypes = [D, I64, I64, D]
    U32 = ctypes.POINTER(ctypes.c_uint32)
    lib.oracle_hif4_macro_value.argtypes = [ctypes.c_int]
    lib.oracle_hif4_macro_value.restype = ctypes.c_double
    lib.oracle_hif4_macro_byte.argtypes = [ctypes.c_double]
    lib.oracle_hif4_macro_byte.restype = ctypes.c_int
    lib.oracle_hif4_value.argtypes = [ctypes.c_uint32, ctypes.c_int, ctypes.c_int]
    lib.oracle_hif4_value.restype = ctypes.c_double
    lib.oracle_hif4_quantize.argtypes = [D, I64, I64, U8, U32, U8, U32]
    lib.oracle_hif4_dequant.argtypes = [U8, U32, I64, I64, D]
    lib.oracle_hif4_gemm.argtypes = [U8, U32, U8, U32, U8, U32, I64, I64, I64, D, D]
    for f in ("oracle_hif4_quantize", "oracle_hif4_dequant", "oracle_hif4_gemm"):
        getattr(lib, f).restype = None
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = ctypes.c_int
    lib.oracle_set_num_threads.argtypes = [ctypes.c_int]
    lib.oracle_set_num_threads.restype = None
    for f in ("oracle_rfq_quantize", "oracle_dequant", "oracle_gemm", "oracle_gemm_phi",
              "oracle_fallback_map",
              "oracle_gemm_sampled", "oracle_swiglu", "oracle_residual"):
        getattr(lib, f).restype = None
    return lib


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        _lib = _load()
    return _lib


class Oracle:
    """Binds the numpy wrappers to one compiled oracle library (the default
    one, or a variant built with extra flags by a test)."""

    def __init__(self, handle):
        self.h = handle

    @staticmethod
    def _d(a):
        return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))

    @staticmethod
    def _u8(a):
        if a is None:
            return None
        return a.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8))

    def num_threads(self):
        return int(self.h.oracle_num_threads())

    def set_num_threads(self, n):
        self.h.oracle_set_num_threads(int(n))

    def e2m1_value(self, code):
        return self.h.oracle_e2m1_value(int(code))

    def e2m1_encode(self, y):
        return self.h.oracle_e2m1_encode(float(y))

    def block_exponent(self, amax):
        return self.h.oracle_block_exponent(float(amax))

    def round_bf16(self, v):
        return self.h.oracle_round_bf16(float(v))

    def quantize(self, x, residual=True):
        """x [rows][K] -> (q_codes, q_scales, r_codes, r_scales) uint8; the
        residual pair is None when residual is False."""
        x = np.ascontiguousarray(x, dtype=np.float64)
        rows, K = x.shape
        assert K % 32 == 0
        qc = np.zeros((rows, K // 2), np.uint8)
        qs = np.zeros((rows, K // 32), np.uint8)
        rc = np.zeros((rows, K // 2), np.uint8) if residual else None
        rs = np.zeros((rows, K // 32), np.uint8) if residual else None
        self.h.oracle_rfq_quantize(self._d(x), rows, K, self._u8(qc), self._u8(qs),
                                   self._u8(rc), self._u8(rs))
        return qc, qs, rc, rs

    def dequant(self, codes, scales):
        codes = np.ascontiguousarray(codes, np.uint8)
        scales = np.ascontiguousarray(scales, np.uint8)
        rows, K = codes.shape[0], codes.shape[1] * 2
        out = np.empty((rows, K), np.float64)
        self.h.oracle_dequant(self._u8(codes), self._u8(scales), rows, K, self._d(out))
        return out

    def residual(self, x):
        x = np.ascontiguousarray(x, dtype=np.float64)
        out = np.empty_like(x)
        self.h.oracle_residual(self._d(x), x.shape[0], x.shape[1], self._d(out))
        return out

    def gemm(self, qc, qs, rc, rs, wc, ws):
        """Z[M][N] and bound[M][N] in fp64 (rc, rs None: plain MXFP4)."""
        arrs = [np.ascontiguousarray(a, np.uint8) if a is not None else None
                for a in (qc, qs, rc, rs, wc, ws)]
        M, K, N = arrs[0].shape[0], arrs[0].shape[1] * 2, arrs[4].shape[0]
        z = np.empty((M, N), np.float64)
        b = np.empty((M, N), np.float64)
        self.h.oracle_gemm(*[self._u8(a) for a in arrs], M, N, K, self._d(z), self._d(b))
        return z, b

    def gemm_phi(self, qc, qs, rc, rs, wc, ws, phi):
        """Z and bound with the phi map phi[ceil(M/64)][ceil(K/256)]."""
        arrs = [np.ascontiguousarray(a, np.uint8) if a is not None else None
                for a in (qc, qs, rc, rs, wc, ws, phi)]
        M, K, N = arrs[0].shape[0], arrs[0].shape[1] * 2, arrs[4].shape[0]
        z = np.empty((M, N), np.float64)
        b = np.empty((M, N), np.float64)
        self.h.oracle_gemm_phi(*[self._u8(a) for a in arrs], M, N, K, self._d(z), self._d(b))
        return z, b

    def fallback_map(self, rc, qs, rule, threshold=0):
        """phi[ceil(M/64)][ceil(K/256)] by rule 0 (nonzero residual codes) or
        rule 1 (a primary scale byte >= threshold)."""
        qs = np.ascontiguousarray(qs, np.uint8)
        M, K = qs.shape[0], qs.shape[1] * 32
        rc = np.ascontiguousarray(rc if rc is not None else np.zeros((M, K // 2)), np.uint8)
        phi = np.empty(((M + 63) // 64, (K + 255) // 256), np.uint8)
        self.h.oracle_fallback_map(self._u8(rc), self._u8(qs), M, K, int(rule), int(threshold),
                                   self._u8(phi))
        return phi

    def gemm_sampled(self, qc, qs, rc, rs, wc, ws, rows, cols):
        arrs = [np.ascontiguousarray(a, np.uint8) if a is not None else None
                for a in (qc, qs, rc, rs, wc, ws)]
        K = arrs[0].shape[1] * 2
        rows = np.ascontiguousarray(rows, np.int64)
        cols = np.ascontiguousarray(cols, np.int64)
        z = np.empty(len(rows), np.float64)
        b = np.empty(len(rows), np.float64)
        P = ctypes.POINTER(ctypes.c_int64)
        self.h.oracle_gemm_sampled(*[self._u8(a) for a in arrs], K,
                                   rows.ctypes.data_as(P), cols.ctypes.data_as(P),
                                   len(rows), self._d(z), self._d(b))
        return z, b

    # ---- HiF4 (oracle/hif4_oracle.c)
    @staticmethod
    def _u32(a):
        if a is None:
            return None
        return a.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32))

    def hif4_macro_value(self, byte):
        return self.h.oracle_hif4_macro_value(int(byte))

    def hif4_macro_byte(self, amax):
        return self.h.oracle_hif4_macro_byte(float(amax))

    def hif4_value(self, meta, i, code):
        return self.h.oracle_hif4_value(int(meta), int(i), int(code))

    def hif4_quantize(self, x, residual=True):
        """x [rows][K] (K a multiple of 64) -> (q_codes, q_meta, r_codes,
        r_meta): codes uint8 [rows][K/2], metadata uint32 [rows][K/64]; the
        residual pair is None when residual is False."""
        x = np.ascontiguousarray(x, dtype=np.float64)
        rows, K = x.shape
        assert K % 64 == 0
        qc = np.zeros((rows, K // 2), np.uint8)
        qm = np.zeros((rows, K // 64), np.uint32)
        rc = np.zeros((rows, K // 2), np.uint8) if residual else None
        rm = np.zeros((rows, K // 64), np.uint32) if residual else None
        self.h.oracle_hif4_quantize(self._d(x), rows, K, self._u8(qc), self._u32(qm),
                                    self._u8(rc), self._u32(rm))
        return qc, qm, rc, rm

    def hif4_dequant(self, codes, meta):
        codes = np.ascontiguousarray(codes, np.uint8)
        meta = np.ascontiguousarray(meta, np.uint32)
        rows, K = codes.shape[0], codes.shape[1] * 2
        out = np.empty((rows, K), np.float64)
        self.h.oracle_hif4_dequant(self._u8(codes), self._u32(meta), rows, K, self._d(out))
        return out

    def hif4_gemm(self, qc, qm, rc, rm, wc, wm):
        """Z[M][N] and bound[M][N] in fp64 of the HiF4 RFQ product (rc, rm
        None: primary only)."""
        qc, rc, wc = [np.ascontiguousarray(a, np.uint8) if a is not None else None
                      for a in (qc, rc, wc)]
        qm, rm, wm = [np.ascontiguousarray(a, np.uint32) if a is not None else None
                      for a in (qm, rm, wm)]
        M, K, N = qc.shape[0], qc.shape[1] * 2, wc.shape[0]
        z = np.empty((M, N), np.float64)
        b = np.empty((M, N), np.float64)
        self.h.oracle_hif4_gemm(self._u8(qc), self._u32(qm), self._u8(rc), self._u32(rm),
                                self._u8(wc), self._u32(wm), M, N, K, self._d(z), self._d(b))
        return z, b

    def swiglu(self, g, u):
        g = np.ascontiguousarray(g, np.float64)
        u = np.ascontiguousarray(u, np.float64)
        h = np.empty_like(g)
        self.h.oracle_swiglu(self._d(g), self._d(u), g.size, self._d(h))
        return h


def default():
    return Oracle(lib())


def variant(extra_flags, tag):
    """An oracle built with extra compiler flags into its own library (used
    by tests that plant a mistake in the oracle to show a pin catches it)."""
    out = os.path.join(ORACLE_DIR, "liboracle_%s.so" % tag)
    build(extra_flags, out=out)
    return Oracle(_load(out))
