"""C-ABI contract of librfq, checked on the CPU: the library loads, exports
every symbol include/rfq.h declares, and rejects bad arguments on the host
before any HIP call.  No call here reaches a kernel launch."""
import ctypes
import os
import re

import pytest

import paper_2608_26581_amd as rfq
from paper_2608_26581_amd import rfq as binding

REPO = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(REPO, "include", "rfq.h")

OK, ENULL, ESHAPE, EDTYPE, EALIGN, EDEVICE, ELAUNCH = range(7)
A = 0x10000          # a fake, 16-byte aligned address: never dereferenced here
MIS = 0x10008        # misaligned by 8


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rfq_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_boundary():
    assert declared_functions() == sorted(binding.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(rfq.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_library_resolves_every_symbol_at_load():
    """Loading with immediate binding fails on any undefined symbol: a kernel
    whose host-side launch handle the compiler dropped would otherwise show
    up only when that kernel is first launched."""
    import subprocess
    import sys
    code = ("import ctypes, os, sys; ctypes.CDLL(sys.argv[1], mode=os.RTLD_NOW); "
            "print('resolved')")
    res = subprocess.run([sys.executable, "-c", code, binding.LIB_PATH],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 0 and "resolved" in res.stdout, res.stderr


def test_binding_names_match_the_c_names():
    for name in declared_functions():
        assert callable(getattr(rfq, name)), name


def test_version_and_status_strings():
    assert rfq.rfq_abi_version() == 1
    seen = set()
    for s in range(7):
        txt = rfq.rfq_status_str(s)
        assert txt and txt not in seen
        seen.add(txt)
    assert rfq.rfq_status_str(99) == "unknown status"


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(binding, "_lib", None)
    monkeypatch.setattr(binding, "LIB_PATH", str(tmp_path / "nope.so"))
    with pytest.raises(RuntimeError, match="not built"):
        binding.load()


def _lib():
    return binding.load()


def test_quantize_act_validation():
    q = _lib().rfq_quantize_act
    assert q(None, 1, 4, 64, A, A, A, A, None) == ENULL
    assert q(A, 1, 4, 64, None, A, A, A, None) == ENULL
    assert q(A, 1, 4, 64, A, None, A, A, None) == ENULL
    assert q(A, 1, 4, 64, A, A, A, None, None) == ENULL      # half residual pair
    assert q(A, 1, 4, 64, A, A, None, A, None) == ENULL
    assert q(A, 2, 4, 64, A, A, A, A, None) == EDTYPE
    assert q(A, -1, 4, 64, A, A, A, A, None) == EDTYPE
    assert q(A, 1, -1, 64, A, A, A, A, None) == ESHAPE
    assert q(A, 1, 4, 48, A, A, A, A, None) == ESHAPE
    assert q(A, 1, 4, 0, A, A, A, A, None) == ESHAPE
    assert q(A, 1, 4, 16, A, A, A, A, None) == ESHAPE
    assert q(MIS, 1, 4, 64, A, A, A, A, None) == EALIGN
    assert q(A, 1, 4, 64, MIS, A, A, A, None) == EALIGN
    assert q(A, 1, 4, 64, A, A, MIS, A, None) == EALIGN
    assert q(A, 1, 0, 64, A, A, A, A, None) == OK              # empty: no-op
    assert q(None, 1, 0, 64, None, None, None, None, None) == OK
    assert q(A, 0, 0, 64, A, A, None, None, None) == OK


def test_hif4_validation():
    lib = _lib()
    q = lib.rfq_hif4_quantize
    assert q(None, 1, 4, 128, A, A, A, A, None) == ENULL
    assert q(A, 1, 4, 128, A, A, A, None, None) == ENULL      # half residual pair
    assert q(A, 7, 4, 128, A, A, A, A, None) == EDTYPE
    assert q(A, 1, 4, 96, A, A, A, A, None) == ESHAPE         # K not a multiple of 64
    assert q(A, 1, 4, 32, A, A, A, A, None) == ESHAPE
    assert q(A, 1, -1, 64, A, A, A, A, None) == ESHAPE
    assert q(A, 1, 1 << 40, 1 << 20, A, A, A, A, None) == ESHAPE
    assert q(MIS, 1, 4, 64, A, A, A, A, None) == EALIGN
    assert q(A, 1, 4, 64, A, A + 2, A, A, None) == EALIGN     # meta word alignment
    assert q(None, 1, 0, 64, None, None, None, None, None) == OK
    d = lib.rfq_hif4_dequant
    assert d(A, A, 4, 96, A, 0, None) == ESHAPE
    assert d(A, A, 4, 64, A, 5, None) == EDTYPE
    assert d(None, A, 4, 64, A, 1, None) == ENULL
    assert d(A, A, 4, 64, MIS, 0, None) == EALIGN
    assert d(None, None, 0, 64, None, 1, None) == OK
    gw = lib.rfq_hif4_gemm_wbf16
    assert gw(A, A, A, A, None, 8, 8, 128, A, 0, None) == ENULL
    assert gw(A, A, A, None, A, 8, 8, 128, A, 0, None) == ENULL
    assert gw(A, A, A, A, A, 8, 8, 96, A, 0, None) == ESHAPE
    assert gw(A, A, A, A, A, 8, 8, 128, A, 4, None) == EDTYPE
    assert gw(A, A, A, A, MIS, 8, 8, 128, A, 0, None) == EALIGN
    assert gw(A, A, A, A, A, 0, 8, 128, A, 0, None) == OK
    g = lib.rfq_hif4_gemm
    args = [A, A, A, A, A, A, 8, 8, 128, A, 0, None]

    def call(**kw):
        a = list(args)
        for k, v in kw.items():
            a[int(k[1:])] = v
        return g(*a)

    assert call(a0=None) == ENULL
    assert call(a3=None) == ENULL                     # half residual pair
    assert call(a10=2) == EDTYPE
    assert call(a8=96) == ESHAPE
    assert call(a7=-1) == ESHAPE
    assert call(a6=1 << 40) == ESHAPE
    assert call(a4=MIS) == EALIGN
    assert call(a1=A + 2) == EALIGN
    assert call(a9=MIS) == EALIGN
    assert call(a6=0) == OK
    assert call(a0=None, a1=None, a2=None, a3=None, a9=None, a6=0) == OK


def test_quantize_weight_validation():
    q = _lib().rfq_quantize_weight
    assert q(None, 0, 4, 64, A, A, None) == ENULL
    assert q(A, 0, 4, 64, None, A, None) == ENULL
    assert q(A, 5, 4, 64, A, A, None) == EDTYPE
    assert q(A, 0, 4, 33, A, A, None) == ESHAPE
    assert q(A, 0, -2, 64, A, A, None) == ESHAPE
    assert q(MIS, 0, 4, 64, A, A, None) == EALIGN
    assert q(A, 0, 0, 64, A, A, None) == OK


def test_gemm_validation():
    g = _lib().rfq_gemm
    args = [A, A, A, A, A, A, 8, 8, 64, A, 0, None]

    def call(**kw):
        a = list(args)
        for k, v in kw.items():
            a[int(k[1:])] = v
        return g(*a)

    assert call(a0=None) == ENULL
    assert call(a1=None) == ENULL
    assert call(a4=None) == ENULL
    assert call(a5=None) == ENULL
    assert call(a9=None) == ENULL
    assert call(a2=None) == ENULL                     # half residual pair
    assert call(a3=None) == ENULL
    assert call(a10=3) == EDTYPE
    assert call(a8=40) == ESHAPE
    assert call(a8=0) == ESHAPE
    assert call(a6=-1) == ESHAPE
    assert call(a7=-1) == ESHAPE
    assert call(a6=1 << 40) == ESHAPE
    assert call(a0=MIS) == EALIGN
    assert call(a4=MIS) == EALIGN
    assert call(a2=MIS) == EALIGN
    assert call(a9=MIS) == EALIGN
    assert call(a6=0) == OK
    assert call(a7=0) == OK
    assert call(a2=None, a3=None, a6=0) == OK         # plain MXFP4, empty
    assert call(a0=None, a1=None, a2=None, a3=None, a9=None, a6=0) == OK
    assert call(a4=None, a5=None, a9=None, a7=0) == OK


def test_gemm_stream_validation():
    g = _lib().rfq_gemm_stream
    # x, x_dtype, residual, w_codes, w_scales, M, N, K, z, z_dtype, stream
    args = [A, 1, 1, A, A, 8, 8, 512, A, 0, None]

    def call(**kw):
        a = list(args)
        for k, v in kw.items():
            a[int(k[1:])] = v
        return g(*a)

    assert call(a0=None) == ENULL
    assert call(a3=None) == ENULL
    assert call(a4=None) == ENULL
    assert call(a8=None) == ENULL
    assert call(a1=2) == EDTYPE
    assert call(a9=7) == EDTYPE
    assert call(a7=256) == ESHAPE                      # K not a multiple of 512
    assert call(a7=96) == ESHAPE
    assert call(a7=0) == ESHAPE
    assert call(a5=-1) == ESHAPE
    assert call(a6=-1) == ESHAPE
    assert call(a5=1 << 20, a7=1 << 12) == ESHAPE      # X of 8 GiB: above the 2 GiB limit
    assert call(a5=65535 * 16 + 1, a6=1) == ESHAPE   # more than 65535 row slices
    assert call(a0=MIS) == EALIGN
    assert call(a3=MIS) == EALIGN
    assert call(a4=MIS) == EALIGN
    assert call(a8=MIS) == EALIGN
    assert call(a5=0) == OK
    assert call(a6=0) == OK
    assert call(a0=None, a8=None, a5=0) == OK
    assert call(a3=None, a4=None, a8=None, a6=0) == OK


def test_dequant_and_swiglu_validation():
    d = _lib().rfq_dequant
    assert d(None, A, 4, 64, A, None) == ENULL
    assert d(A, A, 4, 63, A, None) == ESHAPE
    assert d(A, A, 4, 64, MIS, None) == EALIGN
    assert d(A, A, 0, 64, A, None) == OK
    s = _lib().rfq_swiglu_quantize_act
    assert s(A, None, 1, 4, 64, A, A, A, A, None, None) == ENULL
    assert s(A, A, 1, 4, 64, A, A, A, None, None, None) == ENULL
    assert s(A, A, 9, 4, 64, A, A, A, A, None, None) == EDTYPE
    assert s(A, A, 1, 4, 100, A, A, A, A, None, None) == ESHAPE
    assert s(A, MIS, 1, 4, 64, A, A, A, A, None, None) == EALIGN
    assert s(A, A, 1, 4, 64, A, A, A, A, MIS, None) == EALIGN
    assert s(A, A, 1, 0, 64, A, A, A, A, None, None) == OK


def test_gemm_swiglu_validation():
    f = _lib().rfq_gemm_swiglu_quantize
    #       q  qs r  rs w  ws  M   Nh   K    hq hs hr hrs h
    ok = (A, A, A, A, A, A, 64, 128, 512, A, A, A, A, None, None)

    def call(**kw):
        args = list(ok)
        names = ["q", "qs", "r", "rs", "w", "ws", "M", "Nh", "K", "hq", "hs", "hr", "hrs",
                 "h", "st"]
        for k, v in kw.items():
            args[names.index(k)] = v
        return f(*args)

    assert call(K=480) == ESHAPE             # not a multiple of 32
    assert call(K=256) == ESHAPE             # multiple of 32, not of 512
    assert call(Nh=100) == ESHAPE            # hidden width not a multiple of 32
    assert call(Nh=-32) == ESHAPE
    assert call(M=-1) == ESHAPE
    assert call(M=0) == OK and call(Nh=0) == OK
    assert call(M=1 << 23, K=1024) == ESHAPE     # activation codes of 4 GiB
    assert call(q=None) == ENULL
    assert call(hq=None) == ENULL
    assert call(r=None) == ENULL             # half of the residual input pair
    assert call(hrs=None) == ENULL           # half of the residual output pair
    assert call(qs=MIS) == EALIGN            # scale tensors must be 16-byte aligned
    assert call(ws=MIS) == EALIGN
    assert call(hq=MIS) == EALIGN
    assert call(h=MIS) == EALIGN


def test_gemm_phi_and_fallback_map_validation():
    f = _lib().rfq_gemm_phi
    #       q  qs r  rs w  ws phi  M  N   K    z  dt st
    assert f(A, A, A, A, A, A, A, 4, 8, 64, A, 9, None) == EDTYPE
    assert f(A, A, A, A, A, A, A, 4, 8, 100, A, 0, None) == ESHAPE
    assert f(A, A, A, A, A, A, A, 4, 8, (1 << 20) + 32, A, 0, None) == ESHAPE
    assert f(A, A, A, None, A, A, A, 4, 8, 64, A, 0, None) == ENULL
    assert f(A, A, MIS, A, A, A, A, 4, 8, 64, A, 0, None) == EALIGN
    assert f(A, A, A, A, A, A, A, 0, 8, 64, A, 0, None) == OK
    # Without a map (or without the residual) the call is rfq_gemm's.
    assert f(A, A, A, A, A, A, None, 4, 8, 100, A, 0, None) == ESHAPE
    m = _lib().rfq_fallback_map
    #       rc qs  M  K   rule thr phi st
    assert m(A, A, 4, 64, 2, 0, A, None) == ESHAPE
    assert m(A, A, 4, 96 + 1, 0, 0, A, None) == ESHAPE
    assert m(None, A, 4, 64, 0, 0, A, None) == ENULL
    assert m(A, None, 4, 64, 1, 9, A, None) == ENULL
    assert m(A, A, 4, 64, 0, 0, None, None) == ENULL
    assert m(MIS, A, 4, 64, 0, 0, A, None) == EALIGN
    assert m(A, A, 0, 64, 0, 0, A, None) == OK


def test_size_limits():
    """Sizes past the stated limits are shape errors, reported before any
    device call (one launch covers at most 2^32 - 1 work items; products of
    sizes never overflow)."""
    lib = _lib()
    q = lib.rfq_quantize_act
    assert q(A, 1, 4, (1 << 31) + 32, A, A, A, A, None) == ESHAPE      # K above 2^31
    assert q(A, 1, 1 << 32, 64, A, A, A, A, None) == ESHAPE            # 2^33 MX blocks
    assert q(A, 1, 1 << 62, 1 << 20, A, A, A, A, None) == ESHAPE       # M * K overflows int64
    assert q(A, 1, (1 << 32) - 63, 32, A, A, A, A, None) == ESHAPE     # one block too many
    assert lib.rfq_quantize_weight(A, 0, 1 << 40, 1 << 10, A, A, None) == ESHAPE
    assert lib.rfq_swiglu_quantize_act(A, A, 1, 1 << 33, 64, A, A, A, A, None, None) == ESHAPE
    g = lib.rfq_gemm
    assert g(A, A, A, A, A, A, 1 << 21, 1 << 21, 64, A, 0, None) == ESHAPE   # tile grid > 2^32
    assert g(A, A, A, A, A, A, 1 << 31, 1, 64, A, 0, None) == ESHAPE         # M not below 2^31
    assert g(A, A, A, A, A, A, 8, 8, 1 << 40, A, 0, None) == ESHAPE          # K above 2^31
    f = lib.rfq_gemm_phi
    assert f(A, A, A, A, A, A, A, 1 << 21, 1 << 21, 64, A, 0, None) == ESHAPE
    d = lib.rfq_dequant
    assert d(A, A, 1 << 40, 1 << 20, A, None) == ESHAPE                 # 2^60 elements
    assert d(A, A, 1 << 62, 64, A, None) == ESHAPE                      # rows * K overflows int64
    m = lib.rfq_fallback_map
    assert m(A, A, 1 << 40, 1 << 20, 0, 0, A, None) == ESHAPE
    s = lib.rfq_gemm_stream
    assert s(A, 1, 1, A, A, 8, 1 << 28, 512, A, 0, None) == ESHAPE     # 2^24 column slices
    assert s(A, 1, 1, A, A, 8, 8, 1 << 40, A, 0, None) == ESHAPE       # K above 2^31
    sw = lib.rfq_gemm_swiglu_quantize
    assert sw(A, A, A, A, A, A, 64, 1 << 31, 512, A, A, A, A, None, None) == ESHAPE


def test_gemm_split_validation_and_workspace_sizes():
    """rfq_gemm_split checks what rfq_gemm checks plus its workspace; the
    workspace query is host-only: parts x M x N x 4 bytes where K splits."""
    f = _lib().rfq_gemm_split
    assert f(A, A, A, A, A, A, 8, 8, 512, A, 7, A, 64, None) == EDTYPE
    assert f(A, A, A, A, A, A, 8, 8, 100, A, 0, A, 64, None) == ESHAPE
    assert f(A, A, A, A, A, A, 8, 8, 512, A, 0, A, -1, None) == ESHAPE
    assert f(A, A, A, A, A, A, 8, 8, 512, A, 0, None, 64, None) == ENULL
    assert f(A, A, A, A, A, A, 8, 8, 512, A, 0, MIS, 64, None) == EALIGN
    assert f(A, A, A, A, A, A, 0, 8, 512, None, 0, None, 0, None) == OK
    w = _lib().rfq_gemm_workspace_bytes
    assert w(129, 4096, 12288) == 4 * 129 * 4096 * 4       # 64 tiles: 4 parts
    assert w(512, 4096, 12288) == 2 * 512 * 4096 * 4       # 128 tiles: 2 parts
    assert w(512, 5120, 13824) == 3 * 512 * 5120 * 4       # 160 tiles, K >= 8192: 3 parts
    assert w(64, 4096, 12288) == 8 * 64 * 4096 * 4         # 32 tiles: 8 parts
    assert w(100, 12288, 4096) == 2 * 100 * 12288 * 4      # 96 tiles: 2 parts
    assert w(1024, 4096, 12288) == 0                       # 256 tiles
    assert w(129, 12288, 4096) == 0                        # 192 tiles, K below 8192
    assert w(20, 4096, 12288) == 0                         # few-row kernel
    assert w(24, 4096, 12288) == 8 * 24 * 4096 * 4         # from 24 rows at K >= 12288: split
    assert w(32, 4096, 8192) == 0                          # few-row kernel up to 32 rows
    assert w(16, 5120, 13824) == 3 * 16 * 5120 * 4         # uneven few-row grid: K in 3 parts
    assert w(1, 5000, 12288) == 3 * 1 * 5000 * 4           # the same (313 workgroups)
    assert w(1, 6000, 12288) == 0                          # 375: last round over a quarter full
    assert w(20, 9216, 4096) == 0                          # uneven, but K below 8192: from 33 rows
    assert w(16, 5120, 8192) == 0                          # too short for 3 parts of 8 groups
    assert w(16, 4096, 13824) == 0                         # 256 workgroups: even
    assert w(17, 5120, 13824) == 6 * 17 * 5120 * 4         # uneven few-row grid: split from 17
    assert w(64, 12288, 4096) == 0                         # few-row kernel, 64 weight rows
    assert w(48, 13824, 5120) == 0                         # the same
    assert w(64, 16384, 12288) == 2 * 64 * 16384 * 4       # 128 tiles, from N = 16384: split
    assert w(129, 4096, 12300) == 0                        # K not a multiple of 512
    assert w(-1, 4096, 12288) == 0 and w(129, 4096, 100) == 0


def test_hif4_gemm_split_validation_and_workspace_sizes():
    """rfq_hif4_gemm_split checks what rfq_hif4_gemm checks plus its
    workspace; the workspace query is host-only: parts x M x N x 4 bytes where
    K splits (128-wide tiles, at most 128 of them, more rows than the
    few-row form takes)."""
    f = _lib().rfq_hif4_gemm_split
    assert f(A, A, A, A, A, A, 8, 8, 512, A, 7, A, 64, None) == EDTYPE
    assert f(A, A, A, A, A, A, 8, 8, 96, A, 0, A, 64, None) == ESHAPE
    assert f(A, A, A, A, A, A, 8, 8, 512, A, 0, A, -1, None) == ESHAPE
    assert f(A, A, A, A, A, A, 8, 8, 512, A, 0, None, 64, None) == ENULL
    assert f(None, A, A, A, A, A, 8, 8, 512, A, 0, A, 64, None) == ENULL
    assert f(A, A, A, None, A, A, 8, 8, 512, A, 0, A, 64, None) == ENULL
    assert f(A, A, A, A, A, A, 8, 8, 512, A, 0, MIS, 64, None) == EALIGN
    assert f(A, A, A, A, A, A, 0, 8, 512, None, 0, None, 0, None) == OK
    w = _lib().rfq_hif4_gemm_workspace_bytes
    assert w(256, 4096, 12288) == 4 * 256 * 4096 * 4       # 64 tiles: 4 parts
    assert w(512, 4096, 12288) == 2 * 512 * 4096 * 4       # 128 tiles: 2 parts
    assert w(200, 300, 2560) == 8 * 200 * 300 * 4          # 6 tiles: 8 parts of 5 blocks
    assert w(129, 12288, 4096) == 0                        # 192 tiles
    assert w(1023, 4096, 12288) == 0                       # 256 tiles: no split
    assert w(1024, 4096, 12288) == 4096 * 12288 * 2        # from 1024 rows: W decoded into it
    assert w(4096, 12288, 4096) == 12288 * 4096 * 2
    assert w(1024, 32768, 32768) == 0                      # the decoded W would pass 1 GiB
    assert w(20, 4096, 12288) == 0                         # few-row form, 256 workgroups
    assert w(24, 4096, 12288) == 8 * 24 * 4096 * 4         # tiles from 24 rows (N <= 4096, long K)
    assert w(64, 4096, 12288) == 8 * 64 * 4096 * 4         # the same
    assert w(128, 4096, 12288) == 8 * 128 * 4096 * 4       # instead of two few-row halves
    assert w(39, 4096, 4096) == 0                          # few-row form up to 39 rows at K = 4096
    assert w(40, 4096, 4096) == 8 * 40 * 4096 * 4          # then tiles
    assert w(1, 5120, 13824) == 4 * 1 * 5120 * 4           # few-row form, 320 workgroups: 4 parts
    assert w(16, 5120, 13824) == 3 * 16 * 5120 * 4         # 160 workgroups: 3 parts
    assert w(48, 5120, 13824) == 3 * 48 * 5120 * 4         # the same up to 48 rows
    assert w(49, 5120, 13824) == 6 * 49 * 5120 * 4         # then tiles (40 of them: 6 parts)
    assert w(40, 12288, 4096) == 2 * 40 * 12288 * 4        # few-row form, 384 workgroups: 2 parts
    assert w(64, 12288, 4096) == 2 * 64 * 12288 * 4        # tiles (96: 2 parts)
    assert w(16, 12288, 4096) == 0                         # 192 workgroups, one chunk a wave at 4
    assert w(1, 9216, 4096) == 0                           # 576 workgroups: a gain of 0.15 only
    assert w(8, 3072, 16384) == 0                          # 16 waves a workgroup: no split
    assert w(1, 13824, 5120) == 0                          # 864 workgroups: filled enough
    assert w(16, 5120, 1024) == 0                          # 8 chunks: under two a wave
    assert w(200, 300, 448) == 0                           # 7 blocks: under 2 parts of 4
    assert w(200, 300, 100) == 0 and w(-1, 300, 2560) == 0


def test_gemm_split_noalloc_validation():
    """The allocation-free split product checks what rfq_gemm checks."""
    f = _lib().rfq_gemm_split_noalloc
    assert f(A, A, A, A, A, A, 8, 8, 512, A, 7, None) == EDTYPE
    assert f(A, A, A, A, A, A, 8, 8, 100, A, 0, None) == ESHAPE
    assert f(A, A, A, A, A, A, 1 << 21, 1 << 21, 64, A, 0, None) == ESHAPE
    assert f(A, A, A, A, A, A, 0, 8, 512, None, 0, None) == OK
    assert f(None, A, A, A, A, A, 8, 8, 512, A, 0, None) == ENULL
    assert f(A, A, A, None, A, A, 8, 8, 512, A, 0, None) == ENULL
    assert f(A, A, A, A, A, A, 8, 8, 512, MIS, 0, None) == EALIGN


def test_mfma_loop_validation():
    """The measurement loop: iteration count 1 .. 2^24, a 16-byte aligned
    sink."""
    for f in (_lib().rfq_mfma_fp4_loop, _lib().rfq_mfma_bf16_loop):
        assert f(0, 1, A, None) == ESHAPE
        assert f(-5, 1, A, None) == ESHAPE
        assert f((1 << 24) + 1, 0, A, None) == ESHAPE
        assert f(4, 1, None, None) == ENULL
        assert f(4, 1, MIS, None) == EALIGN


def test_binding_rejects_host_tensors():
    """The binding passes only device pointers on: host tensors are refused
    before any library call (a host pointer would fault in a kernel)."""
    import torch
    x = torch.zeros(4, 64)
    c = torch.zeros(4, 32, dtype=torch.uint8)
    s = torch.zeros(4, 2, dtype=torch.uint8)
    m = torch.zeros(4, 1, dtype=torch.int32)
    xb = torch.zeros(4, 64, dtype=torch.bfloat16)
    calls = [
        lambda: binding.rfq_quantize_act(x),
        lambda: binding.rfq_quantize_weight(x),
        lambda: binding.rfq_gemm(c, s, None, None, c, s),
        lambda: binding.rfq_gemm_phi(c, s, c, s, c, s, None),
        lambda: binding.rfq_gemm_stream(x, c, s),
        lambda: binding.rfq_dequant(c, s),
        lambda: binding.rfq_fallback_map(c, s, binding.RFQ_PHI_RESIDUAL_NONZERO),
        lambda: binding.rfq_swiglu_quantize_act(x, x),
        lambda: binding.rfq_gemm_swiglu_quantize(c, s, None, None, c, s),
        lambda: binding.rfq_hif4_quantize(x),
        lambda: binding.rfq_hif4_dequant(c, m),
        lambda: binding.rfq_hif4_gemm(c, m, None, None, c, m),
        lambda: binding.rfq_hif4_gemm_wbf16(c, m, None, None, xb),
        lambda: binding.rfq_mfma_fp4_loop(4, sink=torch.zeros(binding.MFMA_LOOP_ITEMS)),
        lambda: binding.rfq_mfma_bf16_loop(4, sink=torch.zeros(binding.MFMA_LOOP_ITEMS)),
        lambda: binding.rfq_gemm_split(c, s, None, None, c, s, None),
        lambda: binding.rfq_gemm_split_noalloc(c, s, None, None, c, s),
    ]
    for call in calls:
        with pytest.raises(ValueError, match="device tensor"):
            call()


def test_valid_arguments_without_a_gpu_report_device_error():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present; fake pointers must not reach a launch")
    assert _lib().rfq_quantize_act(A, 1, 4, 64, A, A, A, A, None) == EDEVICE
    assert _lib().rfq_gemm(A, A, A, A, A, A, 8, 8, 64, A, 0, None) == EDEVICE
    assert _lib().rfq_gemm_stream(A, 1, 1, A, A, 8, 8, 512, A, 0, None) == EDEVICE
    assert _lib().rfq_hif4_quantize(A, 1, 4, 64, A, A, A, A, None) == EDEVICE
    assert _lib().rfq_hif4_gemm(A, A, A, A, A, A, 8, 8, 64, A, 0, None) == EDEVICE
    assert _lib().rfq_mfma_fp4_loop(4, 1, A, None) == EDEVICE
    assert _lib().rfq_mfma_bf16_loop(4, 1, A, None) == EDEVICE
    assert _lib().rfq_gemm_split(A, A, A, A, A, A, 8, 8, 512, A, 0, A, 64, None) == EDEVICE
    assert _lib().rfq_gemm_split_noalloc(A, A, A, A, A, A, 8, 8, 512, A, 0, None) == EDEVICE
    # The HiF4 product's launch-size limit sits at the largest grid it may
    # launch: 128-row tiles of 256 weight rows with 768 work items or of 128
    # weight rows with 640, whichever the dispatch picks (N = 256: two
    # 128-wide tiles, 1280 work items per 128 activation rows).
    tile_rows = 0xFFFFFFFF // 1280
    g = _lib().rfq_hif4_gemm
    assert g(A, A, A, A, A, A, tile_rows * 128, 256, 64, A, 0, None) == EDEVICE
    assert g(A, A, A, A, A, A, (tile_rows + 1) * 128, 256, 64, A, 0, None) == ESHAPE
