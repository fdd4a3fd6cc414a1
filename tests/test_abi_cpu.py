"""The C-ABI library without a GPU: symbols, plan table, argument checks.

Nothing here launches a kernel; every call either is host-only (plan
queries) or returns before any device work (argument validation), or, on a
host without a gfx950 device, must report KERNELARC_ERR_UNSUPPORTED.  The
calls that pass validation with host buffers run only where no device is
visible (on a GPU host they would launch on host memory).
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kernelarc.h")


@pytest.fixture(scope="module")
def ka():
    from paper_2608_17071_amd import kernelarc
    return kernelarc


def _device_present():
    """True where a GPU is visible: there, a call that passes validation
    launches a kernel, so the calls below that would pass it with host
    buffers are made only where no device exists (they then report
    KERNELARC_ERR_UNSUPPORTED)."""
    import torch
    return torch.cuda.device_count() > 0


def header_functions():
    with open(HEADER) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kernelarc_\w+)\s*\(", text)))


def test_every_declared_symbol_is_exported(ka):
    names = header_functions()
    assert len(names) >= 10
    lib = ctypes.CDLL(ka.LIBRARY)
    for n in names:
        assert hasattr(lib, n), f"{n} declared in kernelarc.h but not exported"
    assert set(names) == set(ka.EXPORTED), "binding and header disagree"


def test_status_strings(ka):
    for st in (ka.OK, ka.ERR_INVALID_ARG, ka.ERR_UNSUPPORTED, ka.ERR_LAUNCH):
        assert ka.kernelarc_status_string(st)
    assert ka.kernelarc_status_string(99) == b"unknown status"


def test_plan_table(ka):
    names = ka.plan_names()
    assert len(names) == ka.plan_count() >= 6
    assert len(set(names)) == len(names)
    assert ka.plan_name(-1) is None and ka.plan_name(ka.plan_count()) is None
    gen = names.index("generic_64x64_scalar")
    # K not a multiple of 8 -> generic; few rows -> GEMV or streaming; more -> a tile plan
    assert ka.select_plan(128, 256, 250) == gen
    for M in (1, 4):
        assert names[ka.select_plan(M, 4096, 4096)].startswith("gemv")
    for M in (16, 32):
        assert names[ka.select_plan(M, 4096, 4096)].startswith("stream")
    for M in (33, 64, 65, 512, 4096, 8192):
        assert names[ka.select_plan(M, 4096, 4096)].startswith("tile")
    assert ka.select_plan(-1, 4, 4) == -1
    # every selected plan supports its shape; the generic plan supports everything
    for (M, N, K) in [(1, 2048, 2048), (64, 8192, 8192), (512, 5120, 5120), (4096, 8192, 8192),
                      (7, 9, 24), (300, 77, 1000), (0, 5, 8)]:
        p = ka.select_plan(M, N, K)
        assert ka.plan_supports(p, M, N, K), (M, N, K, names[p])
        assert ka.plan_supports(gen, M, N, K)


def test_plan_limits(ka):
    names = ka.plan_names()
    tile = names.index("tile_256x256_k64_w8")
    assert not ka.plan_supports(tile, 512, 512, 12)            # K % 8
    assert ka.kernelarc_plan_supports(99, 1, 1, 1, 1) == -1
    assert ka.kernelarc_plan_supports(tile, -1, 1, 1, 1) == -1
    assert ka.kernelarc_plan_uses_workspace(tile, 4096, 4096, 4096) == 0
    assert ka.kernelarc_plan_uses_workspace(names.index("tile_128x128_k64_w4_splitk"), 512, 1024, 2048) == 1
    stream_split = names.index("stream_mfma16_k64_splitk")
    assert ka.plan_supports(stream_split, 64, 8192, 8192) and ka.plan_supports(stream_split, 1, 8, 8)
    assert not ka.plan_supports(stream_split, 65, 512, 512)    # M > 64
    assert not ka.plan_supports(stream_split, 0, 512, 512)
    assert not ka.plan_supports(stream_split, 16, 512, 516)    # K % 8
    assert ka.kernelarc_plan_uses_workspace(stream_split, 16, 4096, 4096) == 1


def test_plan_name_for_a_shape(ka):
    """kernelarc_plan_name(M, N, K, residual, buf, len): the chosen plan's
    name, the same as the id query, with its buffer and size checks."""
    for (M, N, K, r) in [(16, 4096, 4096, 1), (4096, 4096, 4096, 1), (8192, 8192, 8192, 0), (1, 2048, 2048, 1),
                         (128, 256, 250, 1), (0, 5, 8, 0)]:
        assert ka.plan_name_for(M, N, K, bool(r)) == ka.plan_name(ka.select_plan(M, N, K, bool(r)))
    buf = ctypes.create_string_buffer(64)
    f = ka.kernelarc_plan_name
    assert f(16, 4096, 4096, 1, buf, 64) == ka.OK and buf.value == b"stream_mfma16_r16_k128s2"
    need = len(buf.value) + 1
    small = ctypes.create_string_buffer(b"x" * 8, need - 1)
    assert f(16, 4096, 4096, 1, small, need - 1) == ka.ERR_INVALID_ARG    # too small: nothing written
    assert small.raw[:8] == b"x" * 8
    assert ka.kernelarc_last_error().startswith(b"buf holds")
    assert f(16, 4096, 4096, 1, buf, need) == ka.OK
    assert f(-1, 4, 4, 1, buf, 64) == ka.ERR_INVALID_ARG
    assert f(4, 4, 4, 1, None, 64) == ka.ERR_INVALID_ARG


def test_row_block_stream_plans(ka):
    """16-row streaming blocks: no K split once the blocks fill the CUs
    (N = 4096 gives 256 workgroups), the rule's split below that; chosen for
    few rows up to N = 4096, and for up to 64 rows while N <= 2048 and
    K <= 4096."""
    names = ka.plan_names()
    r16 = names.index("stream_mfma16_r16_k128s2")
    r32 = names.index("stream_mfma16_r32_k64s4")
    assert ka.plan_supports(r16, 1, 8, 8) and ka.plan_supports(r16, 64, 4096, 14336)
    assert not ka.plan_supports(r16, 65, 512, 512)
    assert not ka.plan_supports(r16, 16, 512, 516)              # K % 8
    assert ka.kernelarc_plan_uses_workspace(r16, 16, 4096, 4096) == 0
    assert ka.kernelarc_plan_uses_workspace(r16, 16, 1024, 4096) == 1
    assert ka.kernelarc_plan_uses_workspace(r32, 16, 4096, 4096) == 1
    assert ka.kernelarc_plan_uses_workspace(r16, 16, 4096, 256) == 0   # too shallow to split
    # the kernel addresses whole 16-row token blocks: a wide output whose
    # 16-row block passes 2^31 bytes is refused even for one row
    assert ka.plan_supports(r16, 1, 1 << 25, 8) and not ka.plan_supports(r16, 1, 1 << 26, 8)
    sel = lambda m, n, k: names[ka.select_plan(m, n, k, True)]
    assert sel(16, 4096, 4096) == "stream_mfma16_r16_k128s2"
    assert sel(8, 2048, 2048) == "stream_mfma16_r16_k128s2"
    assert sel(32, 4096, 14336) == "stream_mfma16_r16_k128s2"
    assert sel(16, 8192, 8192) == "stream_mfma16_k64_splitk"
    assert sel(64, 2048, 2048) == "stream_mfma16_r16_k128s2"
    assert sel(48, 1024, 4096) == "stream_mfma16_r16_k128s2"
    assert sel(64, 2048, 8192).startswith("tile_")
    assert sel(64, 4096, 4096).startswith("tile_")
    assert sel(3, 4096, 4096) == "gemv_valu_w4"
    # wide outputs between 512 and 1024 rows take the big tiles
    assert sel(1024, 13824, 5120) == "tile_256x256_k64_w4_m16a"       # one partial round of 256x256 tiles
    assert sel(1024, 20480, 4096) == "tile_256x256_k64_w4_m16a_bands"  # the rest fits one 128x128 round
    assert sel(1024, 28672, 4096) == "tile_256x256_k64_w4_m16a"
    assert sel(768, 24576, 4096) == "tile_256x256_k64_w8_tailsplit"    # one round and an eighth, no bands
    assert sel(2048, 8448, 1024) == "tile_256x256_k64_w4_m16a_bands"  # whole rounds plus a partial one
    assert sel(8192, 8192, 8192) == "tile_256x256_k64_w4_m16a"
    assert sel(1024, 8192, 8192) == "tile_256x128_k64s3_w8_lag"
    assert sel(512, 8192, 8192) == "tile_256x128_k64s3_w8_lag_splitk"  # the measured table entry
    # a partial last round of 256x256 tiles: two column bands when the rest
    # fits one round of 128x128 tiles, else the 4-wave tile over every tile,
    # or the tail split after one full round when the last holds at most a
    # quarter of the CUs
    assert sel(4096, 5120, 5120) == "tile_256x256_k64_w4_m16a_bands"  # the measured table entry
    assert sel(4096, 4352, 4096) == "tile_256x256_k64_w4_m16a_bands"
    for (M, N, K) in [(8192, 5120, 5120), (4096, 14336, 4096), (2048, 14336, 4096), (4096, 11008, 4096)]:
        assert sel(M, N, K) == "tile_256x256_k64_w4_m16a", (M, N, K)
    assert sel(6144, 6144, 6144) == "tile_256x256_k64_w4_m16a"         # two full rounds and a quarter
    assert sel(6144, 2816, 4096) == "tile_256x256_k64_w8_tailsplit"    # one full round and 8 tiles, no bands
    bands = names.index("tile_256x256_k64_w4_m16a_bands")
    for (M, N, K) in [(65, 8, 8), (4000, 4360, 200), (4096, 5120, 5120)]:
        assert ka.plan_supports(bands, M, N, K)
        assert ka.kernelarc_plan_uses_workspace(bands, M, N, K) == 0


def test_validation_before_any_device_work(ka):
    f = ka.kernelarc_gemm_bf16_residual
    buf = (ctypes.c_uint16 * 4096)()
    base = ctypes.addressof(buf)
    # negative sizes
    assert f(-1, 4, 4, base, base, base, base, None) == ka.ERR_INVALID_ARG
    assert ka.kernelarc_last_error().startswith(b"negative size")
    # empty output: nothing to do
    assert f(0, 4, 4, None, None, None, None, None) == ka.OK
    assert f(4, 0, 4, None, None, None, None, None) == ka.OK
    # NULL operands
    assert f(4, 4, 4, base, base, base, None, None) == ka.ERR_INVALID_ARG
    assert f(4, 4, 4, None, base, base, base + 4096, None) == ka.ERR_INVALID_ARG
    assert f(4, 4, 4, base, base, None, base + 4096, None) == ka.ERR_INVALID_ARG
    # Y overlapping X, or partially overlapping R
    X, W, R, Y = base, base + 64, base + 128, base + 256
    assert f(4, 4, 4, X, W, R, X + 16, None) == ka.ERR_INVALID_ARG
    assert f(4, 4, 4, X, W, R, R + 2, None) == ka.ERR_INVALID_ARG
    assert ka.kernelarc_gemm_bf16(4, 4, 4, X, W, W + 8, None) == ka.ERR_INVALID_ARG
    # a forced plan id out of range
    assert ka.kernelarc_gemm_bf16_with_plan(-3, 4, 4, 4, X, W, R, Y, None) == ka.ERR_UNSUPPORTED
    assert ka.kernelarc_gemm_bf16_with_plan(99, 4, 4, 4, X, W, R, Y, None) == ka.ERR_UNSUPPORTED


def test_no_device_is_unsupported(ka):
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    buf = (ctypes.c_uint16 * 4096)()
    base = ctypes.addressof(buf)
    st = ka.kernelarc_gemm_bf16_residual(4, 4, 4, base, base + 64, base + 128, base + 256, None)
    assert st == ka.ERR_UNSUPPORTED
    assert ka.kernelarc_last_error()


def test_python_side_checks(ka):
    import torch
    x = torch.zeros(4, 8, dtype=torch.bfloat16)
    w = torch.zeros(4, 8, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        ka.gemm_bf16(x, w)                       # CPU tensors are rejected before the ABI
    with pytest.raises(TypeError):
        ka.gemm_bf16(x.float(), w)
    with pytest.raises(ValueError):
        ka.gemm_bf16(torch.zeros(4, 7, dtype=torch.bfloat16), w)


def test_general_form_validation(ka):
    f = ka.kernelarc_gemm_bf16_ex
    buf = (ctypes.c_uint16 * 8192)()
    base = ctypes.addressof(buf)
    X, W, C, B, Y = base, base + 2048, base + 4096, base + 6144, base + 8192
    # (M, N, K, alpha, X, ldx, W, ldw, beta, C, ldc, bias, Y, ldy, stream)
    assert f(4, 4, 8, 1.0, X, 7, W, 8, 1.0, C, 4, None, Y, 4, None) == ka.ERR_INVALID_ARG   # ldx < K
    assert ka.kernelarc_last_error().startswith(b"a leading dimension is smaller")
    assert f(4, 4, 8, 1.0, X, 8, W, 8, 1.0, C, 3, None, Y, 4, None) == ka.ERR_INVALID_ARG   # ldc < N
    assert f(4, 4, 8, 1.0, X, 8, W, 8, 1.0, C, 4, None, Y, -1, None) == ka.ERR_INVALID_ARG  # negative ld
    if not _device_present():
        assert f(4, 4, 8, 1.0, X, 8, W, 8, 0.0, C, 3, None, Y, 4, None) != ka.ERR_INVALID_ARG   # beta 0: C unused
    # Y overlapping the bias, or C in part (only Y == C with ldy == ldc is allowed)
    assert f(4, 4, 8, 1.0, X, 8, W, 8, 1.0, C, 4, Y + 4, Y, 4, None) == ka.ERR_INVALID_ARG
    assert f(4, 4, 8, 1.0, X, 8, W, 8, 1.0, Y + 2, 4, None, Y, 4, None) == ka.ERR_INVALID_ARG
    assert f(4, 4, 8, 1.0, X, 8, W, 8, 1.0, Y, 6, None, Y, 4, None) == ka.ERR_INVALID_ARG
    # strided extents count: row 3 of a ldy = 512 Y reaches W
    assert f(4, 4, 8, 1.0, X, 8, W, 8, 1.0, None, 4, None, X - 3 * 1024 + 2048 + 16, 512, None) == ka.ERR_INVALID_ARG
    assert f(0, 4, 8, 1.0, None, 8, None, 8, 1.0, None, 4, None, None, 4, None) == ka.OK


def test_general_form_plan_selection(ka):
    names = ka.plan_names()
    # decode shapes stream in both forms, strided ones too
    dense = names[ka.select_plan_ex(16, 4096, 4096, 1, 4096, 4096, 4096, 4096, 1.0, 1.0, 0)]
    general = names[ka.select_plan_ex(16, 4096, 4096, 1, 4096, 4096, 4096, 4096, 2.0, 1.0, 0)]
    strided = names[ka.select_plan_ex(16, 4096, 4096, 1, 4104, 4112, 4100, 4096, 1.0, 0.5, 1)]
    assert dense == names[ka.select_plan(16, 4096, 4096, True)]
    assert dense == general == strided == "stream_mfma16_r16_k128s2"
    assert names[ka.select_plan_ex(16, 8192, 8192, 1, 8192, 8192, 8192, 8192, 2.0, 1.0, 1)] == \
        "stream_mfma16_k64_splitk"
    assert names[ka.select_plan_ex(2, 4096, 4096, 1, 4104, 4096, 4096, 4096, 1.0, 1.0, 1)] == "gemv_valu_w4"
    assert names[ka.select_plan_ex(4096, 4096, 14336, 1, 14336, 14336, 4096, 4096, 1.0, 1.0, 1)].startswith("tile")


def test_swiglu_validation(ka):
    f = ka.kernelarc_swiglu_bf16
    buf = (ctypes.c_uint16 * 8192)()
    base = ctypes.addressof(buf)
    X, G, U, H = base, base + 2048, base + 4096, base + 8192
    # (M, N, K, X, Wg, Wu, H, stream)
    assert f(-1, 4, 8, X, G, U, H, None) == ka.ERR_INVALID_ARG
    assert f(0, 4, 8, None, None, None, None, None) == ka.OK
    assert f(4, 4, 8, X, G, U, None, None) == ka.ERR_INVALID_ARG            # H NULL
    assert f(4, 4, 8, X, G, None, H, None) == ka.ERR_INVALID_ARG            # Wu NULL
    assert f(4, 4, 8, X, G, U, U + 16, None) == ka.ERR_INVALID_ARG          # H overlaps Wu
    assert ka.kernelarc_last_error().startswith(b"H overlaps")
    assert f(4, 4, 8, X, G, U, X, None) == ka.ERR_INVALID_ARG               # H overlaps X
    assert f(4, 1 << 30, 8, X, G, U, H, None) == ka.ERR_INVALID_ARG         # N too large
    if not _device_present():
        assert f(4, 4, 8, X, G, G, H, None) != ka.ERR_INVALID_ARG           # Wg == Wu is allowed
    assert ka.kernelarc_swiglu_bf16_with_plan(-1, 4, 4, 8, X, G, U, H, None) == ka.ERR_UNSUPPORTED


def test_swiglu_plans(ka):
    names = ka.plan_names()
    gen = names.index("generic_64x64_scalar")
    assert ka.select_plan_swiglu(64, 100, 250) == gen                        # K % 8
    assert ka.select_plan_swiglu(-1, 4, 8) == -1
    for (M, N, K) in [(1, 14336, 4096), (16, 14336, 4096), (64, 4096, 4096), (512, 13824, 5120),
                      (4096, 14336, 4096), (300, 77, 1000), (7, 9, 24), (0, 5, 8)]:
        p = ka.select_plan_swiglu(M, N, K)
        assert ka.plan_supports_swiglu(p, M, N, K), (M, N, K, names[p])
        assert names[p].startswith("tile") or p == gen
    # partial last rounds of 256x256 gate/up tiles run on the 4-wave AGPR tile
    for (M, N, K) in [(2048, 14336, 4096), (1024, 14336, 4096), (4096, 11008, 4096)]:
        assert names[ka.select_plan_swiglu(M, N, K)] == "tile_256x256_k64_w4_m16a", (M, N, K)
    # plans whose waves cannot hold gate/up block pairs, or that are not tiles
    for n in ("tile_64x64_k64s4_w4", "tile_64x64_k128s3_w4_splitk", "stream_mfma16_k64_splitk", "gemv_valu_w4",
              "stream_mfma16_r16_k128s2"):
        assert not ka.plan_supports_swiglu(names.index(n), 64, 1024, 1024), n
    for n in ("tile_256x256_k64_w8", "tile_128x128_k64_w4", "tile_64x128_k64s4_w4_splitk", "generic_64x64_scalar"):
        assert ka.plan_supports_swiglu(names.index(n), 64, 1024, 1024), n
    assert not ka.plan_supports_swiglu(names.index("tile_256x256_k64_w8"), 64, 1024, 1020)   # K % 8
    assert ka.kernelarc_plan_supports_swiglu(999, 1, 1, 1) == -1


def test_i8_validation_and_plans(ka):
    f = ka.kernelarc_gemm_i8
    buf = (ctypes.c_uint8 * 16384)()
    base = ctypes.addressof(buf)
    X, W, SX, SW, Y = base, base + 2048, base + 4096, base + 4608, base + 8192
    # (M, N, K, qX, sx, qW, sw, R, Y, stream)
    assert f(-1, 4, 16, X, SX, W, SW, None, Y, None) == ka.ERR_INVALID_ARG
    assert f(4, 4, 65536 + 16, X, SX, W, SW, None, Y, None) == ka.ERR_INVALID_ARG      # int32 range
    assert ka.kernelarc_last_error().startswith(b"K=")
    assert f(4, 4, 16, X, None, W, SW, None, Y, None) == ka.ERR_INVALID_ARG            # NULL scale
    assert f(4, 4, 16, X, SX + 2, W, SW, None, Y, None) == ka.ERR_INVALID_ARG          # misaligned scale
    assert f(4, 4, 16, X, SX, W, SW, None, X + 8, None) == ka.ERR_INVALID_ARG          # Y overlaps qX
    assert f(4, 4, 16, X, SX, W, SW, None, SW, None) == ka.ERR_INVALID_ARG             # Y overlaps sw
    assert f(4, 4, 16, X, SX, W, SW, Y + 2, Y, None) == ka.ERR_INVALID_ARG             # partial Y/R overlap
    assert f(0, 4, 16, None, None, None, None, None, None, None) == ka.OK
    g = ka.kernelarc_swiglu_i8
    assert g(4, 4, 16, X, SX, W, SW, W, None, Y, None) == ka.ERR_INVALID_ARG           # NULL up scales
    names = ka.plan_names()
    gen = names.index("generic_64x64_scalar")
    assert ka.select_plan_i8(64, 128, 40) == gen                                        # K % 16
    for (M, N, K, glu) in [(4096, 4096, 4096, 0), (8192, 8192, 8192, 0), (1024, 13824, 5120, 1),
                           (4096, 14336, 4096, 1), (300, 77, 1024, 1), (16, 4096, 4096, 1), (64, 16384, 1024, 0)]:
        p = ka.select_plan_i8(M, N, K, glu)
        assert ka.plan_supports_i8(p, M, N, K, glu), (M, N, K, glu, names[p])
        assert names[p].startswith("tile"), (M, N, K, glu, names[p])
    # plain INT8 GEMMs up to 64 rows stream: 16-row blocks up to N = 4096,
    # 32-row blocks up to N = 8192
    for (M, N, K, plan) in [(16, 4096, 4096, "stream_mfma16_r16_k128s2"), (1, 64, 16, "stream_mfma16_r16_k128s2"),
                            (64, 2048, 2048, "stream_mfma16_r16_k128s2"), (16, 8192, 8192, "stream_mfma16_r32_k64s4")]:
        assert names[ka.select_plan_i8(M, N, K, False)] == plan, (M, N, K)
    # the 4-wave AGPR tile takes plain INT8 with K from 8192 up
    for (M, N, K, glu, plan) in [(8192, 8192, 8192, 0, "tile_256x256_k64_w4_m16a"),
                                 (4096, 5120, 10240, 0, "tile_256x256_k64_w4_m16a"),
                                 (4096, 4096, 4096, 0, "tile_256x256_k64_w8"),
                                 (4096, 14336, 4096, 0, "tile_256x256_k64_w8"),
                                 (8192, 8192, 8192, 1, "tile_256x256_k64_w8")]:
        assert names[ka.select_plan_i8(M, N, K, glu)] == plan, (M, N, K, glu)
    assert names[ka.select_plan_f8(8192, 8192, 8192, False)] == "tile_256x256_k64_w8"
    for n in ("stream_mfma16_k64_splitk", "gemv_valu_w4"):
        assert not ka.plan_supports_i8(names.index(n), 16, 1024, 1024)
    r16 = names.index("stream_mfma16_r16_k128s2")
    assert ka.plan_supports_i8(r16, 16, 1024, 1024) and not ka.plan_supports_i8(r16, 16, 1024, 1024, True)
    assert not ka.plan_supports_i8(r16, 65, 1024, 1024) and not ka.plan_supports_i8(r16, 16, 1024, 1032)
    assert not ka.plan_supports_f8(r16, 16, 1024, 1024)
    assert not ka.plan_supports_i8(names.index("tile_64x64_k64s4_w4"), 64, 1024, 1024, True)
    assert ka.plan_supports_i8(names.index("tile_64x64_k64s4_w4"), 64, 1024, 1024, False)
    assert not ka.plan_supports_i8(names.index("tile_256x256_k64_w8"), 64, 1024, 1032)  # K % 16


def test_grouped_validation_and_plans(ka):
    f = ka.kernelarc_gemm_bf16_grouped
    buf = (ctypes.c_uint16 * 16384)()
    base = ctypes.addressof(buf)
    X, W, C, Y = base, base + 4096, base + 8192, base + 12288
    # (G, M_pad, N, K, X, W, counts, Y, stream)
    assert f(-1, 4, 4, 8, X, W, C, Y, None) == ka.ERR_INVALID_ARG
    assert f(2, 4, 4, 8, X, W, C, None, None) == ka.ERR_INVALID_ARG              # NULL output
    assert f(2, 4, 4, 8, X, W, C + 2, Y, None) == ka.ERR_INVALID_ARG             # misaligned counts
    assert f(2, 4, 4, 8, X, W, C, X + 16, None) == ka.ERR_INVALID_ARG            # output overlaps X
    assert f(2, 4, 4, 8, X, W, C, C - 16, None) == ka.ERR_INVALID_ARG            # output overlaps counts
    assert f(1 << 20, 1 << 12, 4, 8, X, W, C, Y, None) == ka.ERR_INVALID_ARG     # G * M_pad too large
    assert f(0, 4, 4, 8, None, None, None, None, None) == ka.OK
    assert ka.kernelarc_swiglu_bf16_grouped(2, 4, 4, 8, X, W, None, C, Y, None) == ka.ERR_INVALID_ARG
    names = ka.plan_names()
    assert ka.select_plan_grouped(4, 64, 100, 250) == names.index("generic_64x64_scalar")
    for (G, Mpad, N, K, glu) in [(256, 96, 2048, 4096, 1), (256, 256, 4096, 2048, 0), (8, 33, 77, 136, 0)]:
        p = ka.select_plan_grouped(G, Mpad, N, K, glu)
        assert ka.plan_supports_grouped(p, G, Mpad, N, K, glu) and names[p].startswith("tile"), names[p]
    # the case study's shapes: 128x128 tiles below 128 padded rows, else 256x256 (4 waves for SwiGLU)
    assert names[ka.select_plan_grouped(256, 96, 2048, 4096, True)] == "tile_128x128_k64_w4"
    assert names[ka.select_plan_grouped(256, 256, 2048, 4096, True)] == "tile_256x256_k64_w4_m16a"
    assert names[ka.select_plan_grouped(256, 256, 4096, 2048, False)] == "tile_256x256_k64_w8"
    for n in ("tile_128x128_k64_w4_splitk", "tile_256x256_k64_w8_tailsplit", "stream_mfma16_k64_splitk"):
        assert not ka.plan_supports_grouped(names.index(n), 4, 64, 256, 256)
    assert not ka.plan_supports_grouped(names.index("tile_64x64_k64s4_w4"), 4, 64, 256, 256, True)


def test_f8_plans(ka):
    names = ka.plan_names()
    for (M, N, K, glu) in [(16, 4096, 4096, 0), (4096, 4096, 4096, 0), (8192, 8192, 8192, 0),
                           (4096, 14336, 4096, 1), (300, 77, 1024, 1)]:
        p = ka.select_plan_f8(M, N, K, glu)
        assert ka.plan_supports_f8(p, M, N, K, glu) and names[p].startswith("tile"), (M, N, K, glu, names[p])
    assert not ka.plan_supports_f8(names.index("tile_256x256_k64_w4_m16a"), 64, 1024, 1024)  # 16x16 MFMA tile
    assert ka.plan_supports_i8(names.index("tile_256x256_k64_w4_m16a"), 64, 1024, 1024)      # plain INT8
    assert not ka.plan_supports_i8(names.index("tile_256x256_k64_w4_m16a"), 64, 1024, 1024, True)  # no SwiGLU
    assert ka.plan_supports_f8(names.index("tile_256x256_k64_w8"), 64, 1024, 1 << 17)      # no int32 limit
    assert ka.select_plan_f8(64, 128, 40) == names.index("generic_64x64_scalar")
