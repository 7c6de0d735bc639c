"""The C ABI without a GPU: the library loads, exports every function that
include/w8a8.h declares, and rejects bad arguments with the documented status
before touching HIP (the fake device addresses below are never dereferenced).
Also the host-side routing rule of the protected layers."""
from __future__ import annotations

import ctypes
import os
import re

import pytest
import torch

import paper_2606_12280_amd as pkg
from paper_2606_12280_amd import _lib, layer, ops

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "w8a8.h")

OK, NULL, SHAPE, ALIGN, ALIAS, UNSUP = 0, 1, 2, 3, 4, 5
A = 0x7F0000000000          # fake, 256-byte aligned device addresses
B = 0x7F0100000000
C = 0x7F0200000000
D = 0x7F0300000000
E = 0x7F0400000000
F = 0x7F0500000000
G = 0x7F0600000000


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return re.findall(r"^[A-Za-z_][\w \*]*?\b(\w+)\s*\(", text, flags=re.M)


@pytest.fixture(scope="module")
def lib():
    return pkg.load()


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert len(names) >= 10
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(_lib.SIGNATURES), "binding and header disagree"


def test_version_and_status_strings(lib):
    assert lib.w8a8_abi_version() == 2
    for s in range(7):
        assert lib.w8a8_status_string(s)
    assert lib.w8a8_status_string(99) == b"unknown status"
    assert lib.w8a8_last_hip_error() == b""


def test_quant_act_validation(lib):
    f = lib.w8a8_quant_act
    assert f(None, B, 4, 64, C, D, None) == NULL
    assert f(A, B, -1, 64, C, D, None) == SHAPE
    assert f(A, B, (1 << 22) + 1, 64, C, D, None) == SHAPE
    assert f(A, B, 4, 0, C, D, None) == SHAPE
    assert f(A, B, 4, 100, C, D, None) == UNSUP
    assert f(A, B, 4, 65536 + 64, C, D, None) == UNSUP
    assert f(A, B, 1 << 22, 32768 + 64, C, D, None) == SHAPE  # a 2^32 work-item grid
    assert f(A + 8, B, 4, 64, C, D, None) == ALIGN
    assert f(A, B + 4, 4, 64, C, D, None) == ALIGN
    assert f(A, B, 4, 64, C + 1, D, None) == ALIGN
    assert f(A, B, 4, 64, A, D, None) == ALIAS               # Xq over X
    assert f(A, B, 4, 64, C, C + 64, None) == ALIAS          # x_scale inside Xq


def test_prepare_weight_validation(lib):
    f = lib.w8a8_prepare_weight
    assert f(A, B, 8, 64, C, D, None, None) == NULL
    assert f(A, B, -1, 64, C, D, E, None) == SHAPE
    assert f(A, B, 8, 64, C, D, B, None) == ALIAS            # inv_lambda over lambda
    assert f(A, B + 8, 8, 64, C, D, E, None) == ALIGN


def test_linear_validation(lib):
    f = lib.w8a8_linear
    assert f(A, B, C, D, None, 4, 8, 64, None, None) == NULL
    assert f(A, B, C, D, None, 4, (1 << 20) + 1, 64, E, None) == SHAPE
    assert f(A, B, C, D, None, 1 << 22, 1 << 20, 64, E, None) == SHAPE   # M*N > 2^38
    assert f(A, B, C, D, None, 4, 8, 96, E, None) == UNSUP
    assert f(A, B, C, D, E + 1, 4, 8, 64, E + 4096, None) == ALIGN       # odd bias
    assert f(A, B, C, D, None, 4, 8, 64, C, None) == ALIAS               # Y over Wq
    assert f(A, B, C, D, E, 4, 8, 64, E, None) == ALIAS                  # Y over bias
    g = lib.w8a8_gemm_i32
    assert g(A, B, 4, 8, 64, None, None) == NULL
    assert g(A, B, 4, 8, 64, A + 16, None) == ALIAS
    h = lib.bf16_linear
    assert h(A, None, None, 4, 8, 64, C, None) == NULL
    assert h(A, B, None, 4, 8, 64, A, None) == ALIAS
    assert h(A, B, None, 4, 8, 0, C, None) == SHAPE


def test_empty_token_batch_is_a_no_op(lib):
    """M = 0 returns OK without touching the GPU (this process has none), with
    NULL for every buffer sized by M; the other arguments are still checked,
    and the moments of no entries stay an error."""
    assert lib.w8a8_act_absmax(None, 0, 64, B, None) == OK
    assert lib.w8a8_act_absmax(None, 0, 64, None, None) == NULL
    assert lib.w8a8_act_absmax(None, 0, 96, B, None) == UNSUP
    assert lib.w8a8_act_moments(A, 0, 64, B, C, None) == SHAPE
    assert lib.w8a8_quant_act(None, B, 0, 64, None, None, None) == OK
    assert lib.w8a8_quant_act(None, None, 0, 64, None, None, None) == NULL
    assert lib.w8a8_quant_act(None, B + 4, 0, 64, None, None, None) == ALIGN
    assert lib.w8a8_adaln_quant_act(None, B, C, D, 0, 64, 1e-6, None, None, None) == OK
    assert lib.w8a8_adaln_quant_act(None, B, C, D, 0, 64, -1.0, None, None, None) == UNSUP
    assert lib.w8a8_linear(None, None, C, D, None, 0, 8, 64, None, None) == OK
    assert lib.w8a8_linear(None, None, None, D, None, 0, 8, 64, None, None) == NULL
    assert lib.w8a8_linear(None, None, C, D, None, 0, 0, 64, None, None) == SHAPE
    assert lib.w8a8_linear(None, None, C, D, None, 0, 8, 96, None, None) == UNSUP
    assert lib.w8a8_linear(None, None, C, D, E, 0, 8, 64, None, None) == OK
    assert lib.w8a8_gemm_i32(None, B, 0, 8, 64, None, None) == OK
    assert lib.bf16_linear(None, B, None, 0, 8, 64, None, None) == OK
    assert lib.bf16_linear(None, B, None, 0, 8, 0, None, None) == SHAPE
    assert lib.q8_0_linear(None, B, C, None, 0, 8, 64, D, None, None) == OK
    assert lib.q8_0_linear(None, B, C, None, 0, 8, 64, None, None, None) == NULL
    assert lib.q4_k_linear(None, B, C, D, E, None, 0, 8, 256, G, None, None) == OK
    assert lib.q4_k_linear(None, B, C, D, E, None, 0, 8, 128, G, None, None) == UNSUP
    assert lib.w8a8_gemm_config(0, 8, 64, 0, None, None, None) == NULL


def test_gemm_config_picks_tiles_by_rounds(lib):
    """The host-side tile choice: the estimated time (rounds of the 256 CUs x
    tile area / measured rate) of each candidate, computed here by hand."""
    cfg = ops.w8a8_gemm_config
    T288, T192, S192, S256, U = (288, 256, 768), (192, 256, 512), (192, 128, 512), \
        (256, 128, 512), (192, 256, 256)
    # every DiT linear at M = 4608 = 16 x 288 fills whole rounds of 288 x 256
    for N, K in [(16384, 4096), (4096, 16384), (12288, 4096), (4096, 4096)]:
        assert cfg(4608, N, K) == T288 and cfg(4608, N, K, bf16=True) == T288
    # N = 4350: 272 large tiles take 2 rounds, 408 of 192 x 256 take 2 too
    # (2 x 49152 / 0.82 < 2 x 73728); at N = 12290 (784 tiles, 4 rounds,
    # against 1176, 5 rounds) the large tiles win (5 x 49152 / 0.82 > 4 x 73728)
    assert cfg(4545, 4350, 384) == T192
    assert cfg(4545, 12290, 384) == T288
    # fewer than a round of tiles: the smallest tile
    assert cfg(64, 512, 256) == S192 and cfg(200, 4096, 512) == S192
    # M = 1000: 384 tiles of 192 x 128 take 2 rounds, 256 of 256 x 128 one
    assert cfg(1000, 8190, 256) == S256
    # K not a multiple of 128 bytes: the uniform 64-byte K tile kernel ...
    assert cfg(513, 384, 4160) == U and cfg(1, 1, 64) == U
    # ... unless bf16 doubles the bytes per row
    assert cfg(513, 384, 4160, bf16=True) == S192
    # at the size limit (M N <= 2^38) every grid stays below 2^32 work-items
    for M, N in [(1 << 22, 1 << 16), (1 << 18, 1 << 20), ((1 << 22) - 1, 65535), (1, 1 << 20),
                 (1 << 22, 1), (300000, 916000)]:
        for bf16 in (False, True):
            for K in (64, 128):
                tm, tn, nt = cfg(M, N, K, bf16=bf16)
                assert -(-M // tm) * -(-N // tn) * nt < 1 << 32, (M, N, K, bf16)
    out = ctypes.c_int32()
    f = lib.w8a8_gemm_config
    assert f(4, 8, 64, 0, None, ctypes.byref(out), ctypes.byref(out)) == NULL
    assert f(0, 8, 64, 0, ctypes.byref(out), ctypes.byref(out), ctypes.byref(out)) == SHAPE
    assert f(4, 8, 96, 0, ctypes.byref(out), ctypes.byref(out), ctypes.byref(out)) == UNSUP


def test_calibration_validation(lib):
    f = lib.w8a8_smooth_factors
    assert f(A, B, 8, 64, 0.5, None, None) == NULL
    assert f(A, B, 8, 64, 0.0, C, None) == UNSUP
    assert f(A, B, 8, 64, 1.0, C, None) == UNSUP
    assert f(A, B, 8, 64, float("nan"), C, None) == UNSUP
    assert f(A, B, 8, 64, 0.5, A, None) == ALIAS
    g = lib.w8a8_act_absmax
    assert g(A, 8, 64, None, None) == NULL
    assert g(A, 8, 64, A + 64, None) == ALIAS
    assert g(A + 2, 8, 64, C, None) == ALIGN


def test_moments_noalloc_validation(lib):
    f = lib.w8a8_act_moments_noalloc
    assert f(None, 8, 64, C, None) == NULL
    assert f(A, 8, 64, None, None) == NULL
    assert f(A, 0, 64, C, None) == SHAPE
    assert f(A, (1 << 22) + 1, 64, C, None) == SHAPE
    assert f(A, 8, 0, C, None) == SHAPE
    assert f(A, 8, 96, C, None) == UNSUP
    assert f(A, 8, 65536 + 64, C, None) == UNSUP
    assert f(A + 2, 8, 64, C, None) == ALIGN
    assert f(A, 8, 64, C + 4, None) == ALIGN
    assert f(A, 8, 64, A + 64, None) == ALIAS        # stats inside X


def test_moments_validation(lib):
    f = lib.w8a8_act_moments
    assert f(None, 8, 64, B, C, None) == NULL
    assert f(A, 8, 64, None, C, None) == NULL
    assert f(A, 8, 64, B, None, None) == NULL
    assert f(A, 0, 64, B, C, None) == SHAPE
    assert f(A, 8, 0, B, C, None) == SHAPE
    assert f(A, 8, 96, B, C, None) == UNSUP          # K % 64 != 0
    assert f(A + 2, 8, 64, B, C, None) == ALIGN
    assert f(A, 8, 64, B + 4, C, None) == ALIGN
    assert f(A, 8, 64, B, C + 4, None) == ALIGN
    assert f(A, 8, 64, A + 512, C, None) == ALIAS     # workspace inside X (1 KiB)
    assert f(A, 8, 64, B, B + 1024, None) == ALIAS    # stats inside the workspace
    assert f(A, 8, 64, B, A, None) == ALIAS
    expr = re.search(r"#define W8A8_MOMENTS_WORK_BYTES \(([^\n]*)\)\n", open(HEADER).read())
    assert expr and _lib.MOMENTS_WORK_BYTES == eval(expr.group(1), {}) == 6 * 1024 * 8


def test_q8_0_validation(lib):
    q = lib.q8_0_quantize
    assert q(None, 8, 64, B, C, None) == NULL
    assert q(A, 0, 64, B, C, None) == SHAPE
    assert q(A, 8, 32, B, C, None) == UNSUP             # K % 64 != 0
    assert q(A + 2, 8, 64, B, C, None) == ALIGN
    assert q(A, 8, 64, B + 8, C, None) == ALIGN
    assert q(A, 8, 64, B, C + 1, None) == ALIGN
    assert q(A, 8, 64, A + 64, C, None) == ALIAS        # codes inside W
    assert q(A, 8, 64, B, B + 256, None) == ALIAS       # scales inside the codes
    dq = lib.q8_0_dequantize
    assert dq(A, B, 8, 64, None, None) == NULL
    assert dq(A, B, 8, 64, A, None) == ALIAS
    assert dq(A, B, 8, 64, C + 8, None) == ALIGN
    f = lib.q8_0_linear
    assert f(A, B, C, None, 4, 8, 64, D, None, None) == NULL
    assert f(A, B, C, None, 4, 8, 64, None, E, None) == NULL
    assert f(A, B, C, None, 4, 8, 64, D, D, None) == ALIAS          # Y inside work
    assert f(A, B, C, None, 4, 8, 64, B, E, None) == ALIAS          # work over the codes
    assert f(A, B, C, None, 4, 8, 64, D + 8, E, None) == ALIGN
    assert f(A, B, C, None, 4, 8, 96, D, E, None) == UNSUP


def test_q4_k_validation(lib):
    q = lib.q4_k_quantize
    assert q(None, 8, 256, B, C, D, E, None) == NULL
    assert q(A, 8, 256, B, C, D, None, None) == NULL
    assert q(A, 8, 256, B, None, D, E, None) == NULL
    assert q(A, 0, 256, B, C, D, E, None) == SHAPE
    assert q(A, 8, 128, B, C, D, E, None) == UNSUP          # K % 256 != 0
    assert q(A, 8, 96, B, C, D, E, None) == UNSUP
    assert q(A + 2, 8, 256, B, C, D, E, None) == ALIGN
    assert q(A, 8, 256, B + 8, C, D, E, None) == ALIGN       # codes
    assert q(A, 8, 256, B, C + 2, D, E, None) == ALIGN       # packed scales
    assert q(A, 8, 256, B, C, D + 1, E, None) == ALIGN       # d
    assert q(A, 8, 256, A + 64, C, D, E, None) == ALIAS      # codes inside W
    assert q(A, 8, 256, B, B + 1020, D, E, None) == ALIAS    # scales overlap the codes (1 KiB)
    assert q(A, 8, 256, B, C, C + 92, E, None) == ALIAS      # d overlaps the scales (96 B)
    assert q(A, 8, 256, B, C, D, D + 8, None) == ALIAS       # dmin inside d (16 B)
    assert q(A, 8, 256, B, C, D, D + 16, None) != ALIAS      # dmin right after d
    dq = lib.q4_k_dequantize
    assert dq(A, B, C, D, 8, 256, None, None) == NULL
    assert dq(A, B, C, D, 8, 256, A + 16, None) == ALIAS
    assert dq(A, B, C, D, 8, 256, F + 8, None) == ALIGN
    f = lib.q4_k_linear
    assert f(A, B, C, D, E, None, 4, 8, 256, G, None, None) == NULL
    assert f(A, B, C, D, E, None, 4, 8, 256, None, G, None) == NULL
    assert f(A, B, C, D, E, None, 4, 8, 256, G, G, None) == ALIAS     # Y inside work
    assert f(A, B, C, D, E, None, 4, 8, 256, B, G, None) == ALIAS     # work over the codes
    assert f(A, B, C, D, E, None, 4, 8, 512 + 64, G, 0x7F0700000000, None) == UNSUP
    assert f(A, B, C, D, E, None, -1, 8, 256, G, 0x7F0700000000, None) == SHAPE


def test_adaln_validation(lib):
    f = lib.w8a8_adaln_quant_act
    assert f(None, B, C, D, 4, 64, 1e-6, E, E + 4096, None) == NULL
    assert f(A, B, None, D, 4, 64, 1e-6, E, E + 4096, None) == NULL
    assert f(A, B, C, D, -1, 64, 1e-6, E, E + 4096, None) == SHAPE
    assert f(A, B, C, D, 4, 96, 1e-6, E, E + 4096, None) == UNSUP          # K % 64 != 0
    assert f(A, B, C, D, 4, 8256, 1e-6, E, E + 65536, None) == UNSUP       # K > 8192
    assert f(A, B, C, D, 4, 64, -1e-6, E, E + 4096, None) == UNSUP
    assert f(A, B, C, D, 4, 64, float("nan"), E, E + 4096, None) == UNSUP
    assert f(A, B, C, D, 4, 64, float("inf"), E, E + 4096, None) == UNSUP
    assert f(A, B + 2, C, D, 4, 64, 1e-6, E, E + 4096, None) == ALIGN      # shift
    assert f(A, B, C, D, 4, 64, 1e-6, E, E + 2, None) == ALIGN             # x_scale
    assert f(A, B, C, D, 4, 64, 1e-6, A, E + 4096, None) == ALIAS          # Xq over X
    assert f(A, B, C, D, 4, 64, 1e-6, E, C + 64, None) == ALIAS            # x_scale in scale


def test_binding_rejects_host_tensors():
    X = torch.zeros(4, 64, dtype=torch.bfloat16)
    il = torch.ones(64)
    with pytest.raises(ValueError, match="GPU"):
        ops.w8a8_quant_act(X, il)
    with pytest.raises(TypeError):
        ops.w8a8_quant_act(X.float(), il)


def test_binding_fails_loudly_without_library(monkeypatch):
    monkeypatch.setattr(_lib, "_lib", None)
    monkeypatch.setattr(_lib, "LIB_PATH", "/nonexistent/libw8a8.so")
    with pytest.raises(RuntimeError, match="no CPU fallback"):
        _lib.load()


def test_status_error_carries_name():
    err = _lib.W8A8Error("w8a8_linear", 4, "overlap")
    assert "W8A8_ERR_ALIAS" in str(err) and err.status == 4


def test_protection_rule_first_17_down_projections():
    flags = layer.protected_layers(211, 17)
    idx = [i for i, f in enumerate(flags) if f]
    assert len(idx) == 17
    assert all(i % 4 == 3 for i in idx)
    assert idx == [4 * j + 3 for j in range(17)]
    assert sum(1 for i in range(211) if i % 4 == 3) == 52
