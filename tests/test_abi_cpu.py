"""The C ABI loads, exports every declared symbol, and rejects bad arguments
before touching the GPU (no device needed: validation precedes any HIP call)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "masq.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(masq_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    from paper_2603_04800_amd import ops
    return ops.raw()


def test_header_declares_the_four_layer_calls():
    names = _declared_functions()
    for required in ("masq_smooth_quant", "masq_w8a8_gemm", "masq_lowrank_comp",
                     "masq_linear_fused", "masq_linear_fused_workspace_bytes",
                     "masq_status_str"):
        assert required in names


def test_every_declared_symbol_is_exported(lib):
    for name in _declared_functions():
        assert hasattr(lib, name), name
    from paper_2603_04800_amd import ops
    assert set(_declared_functions()) == set(ops.EXPORTED)


def test_header_is_plain_c():
    import shutil
    import subprocess
    import tempfile
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    with tempfile.TemporaryDirectory() as d:
        src = os.path.join(d, "t.c")
        with open(src, "w") as f:
            f.write('#include "masq.h"\nint main(void){return masq_abi_version();}\n')
        r = subprocess.run([gcc, "-std=c99", "-Wall", "-Werror", "-fsyntax-only", "-I",
                            os.path.join(ROOT, "include"), src], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr


def test_status_strings(lib):
    for code in range(9):
        assert lib.masq_status_str(code).startswith(b"MASQ_")
    assert lib.masq_abi_version() == 1


P = 1 << 20          # a fake, 256-byte aligned "device" address; never dereferenced


def _fused(lib, **kw):
    a = dict(x=P, x_dt=1, mod=P, inv=P, wq=P, ws=P, ld=P, ru=P, lr_dt=1, T=16, K=64, N=64,
             rank=16, n_mod=2, y=P, y_dt=1, work=P, work_bytes=1 << 30, stream=None)
    a.update(kw)
    return lib.masq_linear_fused(a["x"], a["x_dt"], a["mod"], a["inv"], a["wq"], a["ws"],
                                 a["ld"], a["ru"], a["lr_dt"], a["T"], a["K"], a["N"],
                                 a["rank"], a["n_mod"], a["y"], a["y_dt"], a["work"],
                                 a["work_bytes"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(x=None), 1), (dict(wq=None), 1), (dict(y=None), 1), (dict(ld=None), 1),
    (dict(work=None), 1),
    (dict(K=40), 2), (dict(N=24), 2), (dict(K=0), 2), (dict(T=-1), 2), (dict(rank=8), 2),
    (dict(rank=272), 2), (dict(n_mod=0), 2), (dict(n_mod=5), 2),
    (dict(x_dt=7), 3), (dict(y_dt=2), 3), (dict(lr_dt=-1), 3),
    (dict(x=P + 8), 4), (dict(ru=P + 4), 4), (dict(work=P + 16), 4),
    (dict(work_bytes=100), 5),
])
def test_fused_rejects_bad_arguments(lib, kw, code):
    assert _fused(lib, **kw) == code


def test_fused_accepts_empty_batch_and_text_only_without_factors(lib):
    assert _fused(lib, T=0, work=None, work_bytes=0) == 0
    # rank 0 (or a single modality) needs no factor pointers; T = 0 is a no-op
    assert _fused(lib, T=0, rank=0, ld=None, ru=None) == 0
    assert _fused(lib, T=0, n_mod=1, ld=None, ru=None) == 0


def test_workspace_query_monotone(lib):
    f = lib.masq_linear_fused_workspace_bytes
    base = f(256, 512, 512, 16, 2)
    assert base >= 256 * 512 + 256 * 4
    assert f(512, 512, 512, 16, 2) > base
    assert f(256, 512, 512, 0, 2) < base
    assert f(0, 512, 512, 16, 2) <= 256 * 2
    assert f(-1, 512, 512, 16, 2) == 0


def test_unfused_calls_validate(lib):
    # smooth_quant: K not a multiple of 16, null output, misaligned input
    assert lib.masq_smooth_quant(P, 1, P, P, 8, 40, 2, P, P, None) == 2
    assert lib.masq_smooth_quant(P, 1, P, P, 8, 64, 2, None, P, None) == 1
    assert lib.masq_smooth_quant(P + 2, 1, P, P, 8, 64, 2, P, P, None) == 4
    assert lib.masq_smooth_quant(P, 1, P, P, 0, 64, 2, P, P, None) == 0
    assert lib.masq_smooth_quant(None, 1, None, None, 0, 64, 2, None, None, None) == 0
    # w8a8_gemm: both outputs null, bad dtype, empty batch
    assert lib.masq_w8a8_gemm(P, P, P, P, 8, 64, 64, None, None, 0, None) == 1
    assert lib.masq_w8a8_gemm(P, P, P, P, 8, 64, 64, None, P, 9, None) == 3
    assert lib.masq_w8a8_gemm(P, P, P, P, 0, 64, 64, P, None, 0, None) == 0
    # lowrank_comp: rank not a multiple of 16; rank 0 is a no-op
    assert lib.masq_lowrank_comp(P, 1, P, P, P, P, 1, 8, 64, 64, 24, 2, P, 1, None) == 2
    assert lib.masq_lowrank_comp(P, 1, P, P, None, None, 1, 8, 64, 64, 0, 2, P, 1, None) == 0


def test_accumulating_calls_refuse_rows_too_long_for_exact_int32(lib):
    """|acc| <= 127 * 127 * c_in (int8) or 127 * 112 * c_in (4-bit codes taken
    as 16 x code) must stay below 2^31: the longest accepted rows are 133136
    and 150976 columns."""
    w8, w4 = 133136, 150976
    assert 127 * 127 * w8 < 2 ** 31 <= 127 * 127 * (w8 + 16)
    assert 127 * 112 * w4 < 2 ** 31 <= 127 * 112 * (w4 + 64)
    g8, g4 = lib.masq_w8a8_gemm, lib.masq_w4a8_gemm
    assert g8(P, P, P, P, 0, w8, 64, P, None, 0, None) == 0
    assert g8(P, P, P, P, 0, w8 + 16, 64, P, None, 0, None) == 2
    assert g4(P, P, P, P, 0, w4, 64, P, None, 0, None) == 0
    assert g4(P, P, P, P, 0, w4 + 64, 64, P, None, 0, None) == 2
    assert _fused(lib, T=0, K=w8, work=None, work_bytes=0) == 0
    assert _fused(lib, T=0, K=w8 + 16, work=None, work_bytes=0) == 2
    assert _fused(lib, K=w8 + 16) == 2
    assert _fused_w4(lib, T=0, K=w4, work=None, work_bytes=0) == 0
    assert _fused_w4(lib, T=0, K=w4 + 64, work=None, work_bytes=0) == 2
    # quantisation alone does not accumulate
    assert lib.masq_smooth_quant(P, 1, P, P, 0, w8 + 16, 2, P, P, None) == 0


def _noalloc(lib, **kw):
    a = dict(x=P, x_dt=1, mod=P, inv=P, wq=P, ws=P, ld=P, ru=P, lr_dt=1, T=0, K=64, N=64,
             rank=16, n_mod=2, y=P, y_dt=1, stream=None)
    a.update(kw)
    return lib.masq_linear_fused_noalloc(a["x"], a["x_dt"], a["mod"], a["inv"], a["wq"],
                                         a["ws"], a["ld"], a["ru"], a["lr_dt"], a["T"], a["K"],
                                         a["N"], a["rank"], a["n_mod"], a["y"], a["y_dt"],
                                         a["stream"])


def test_noalloc_entry_point_validates_before_touching_the_device(lib):
    """masq_linear_fused_noalloc checks its arguments as masq_linear_fused does
    and refuses problems whose workspace exceeds the static scratch
    (64 MiB) with MASQ_ERR_SCRATCH, all before any HIP call."""
    limit = 64 << 20
    f = lib.masq_linear_fused_workspace_bytes
    T_big = 20000                       # 20000 x 3584 codes alone exceed 64 MiB
    assert f(T_big, 3584, 512, 64, 3) > limit
    assert _noalloc(lib, T=T_big, K=3584, N=512, rank=64, n_mod=3) == 8
    assert b"MASQ_ERR_SCRATCH" in lib.masq_status_str(8)
    assert _noalloc(lib, T=0) == 0
    assert _noalloc(lib, T=0, x=None, y=None, wq=None) == 0
    assert _noalloc(lib, T=16, K=40) == 2
    assert _noalloc(lib, T=16, x=None) == 1
    assert _noalloc(lib, T=16, y_dt=5) == 3
    assert _noalloc(lib, T=16, x=P + 8) == 4
    assert _noalloc(lib, T=16, rank=8) == 2
    assert _noalloc(lib, T=0, K=133136 + 16) == 2


def test_mas_only_entry_point_validates(lib):
    """masq_mas_only_linear checks sizes, dtypes, pointers, alignment and the
    workspace before enqueueing anything; c_in must be a multiple of 64."""
    f, wsb = lib.masq_mas_only_linear, lib.masq_mas_only_workspace_bytes
    big = 1 << 30

    def call(**kw):
        a = dict(x=P, x_dt=1, mod=P, inv=P, wq=P, ws=P, T=16, K=128, N=64, M=3, y=P, y_dt=1,
                 work=P, wb=big)
        a.update(kw)
        return f(a["x"], a["x_dt"], a["mod"], a["inv"], a["wq"], a["ws"], a["T"], a["K"], a["N"],
                 a["M"], a["y"], a["y_dt"], a["work"], a["wb"], None)
    assert call(K=96) == 7                       # c_in % 64 != 0: not supported
    assert call(K=40) == 2
    assert call(N=24) == 2
    assert call(M=0) == 2 and call(M=5) == 2
    assert call(x_dt=4) == 3
    assert call(wq=None) == 1 and call(work=None) == 1
    assert call(ws=P + 4) == 4 and call(work=P + 128) == 4
    assert call(wb=16) == 5
    assert call(T=0, x=None, y=None, work=None, wb=0) == 0
    assert call(T=0, K=133136 + 64) == 2          # exact int32 accumulation bound
    assert wsb(16, 128, 64, 3) >= 16 * 128 + 16 * 4 * 2
    assert wsb(4096, 128, 64, 3) > wsb(16, 128, 64, 3)
    assert wsb(-1, 128, 64, 3) == 0 and wsb(16, 128, 64, 5) == 0


def test_validation_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    """tests/sanitized_validation.c, linked against the library whose
    entry-point host code is built with ASan and UBSan, calls every entry
    point with invalid arguments (and empty batches) and checks the status
    codes; any sanitizer report fails the run."""
    import shutil
    import subprocess
    clang = "/opt/rocm/llvm/bin/clang"
    if not os.path.exists(clang) or shutil.which("hipcc") is None and not os.path.exists(
            "/opt/rocm/bin/hipcc"):
        pytest.skip("ROCm clang/hipcc not available")
    from paper_2603_04800_amd import build
    lib = build.build_sanitized()
    exe = str(tmp_path / "sanitized_validation")
    r = subprocess.run([clang, "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
                        "-fno-sanitize-recover=all", "-I", os.path.join(ROOT, "include"),
                        os.path.join(ROOT, "tests", "sanitized_validation.c"),
                        "-L", os.path.dirname(lib), "-lmasq_sanitized",
                        "-Wl,-rpath," + os.path.dirname(lib), "-o", exe],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout + r.stderr


def test_binding_refuses_host_tensors():
    import torch
    from paper_2603_04800_amd import ops
    x = torch.zeros(4, 64)
    with pytest.raises(ValueError):
        ops.smooth_quant(x, torch.zeros(4, dtype=torch.int32), torch.ones(1, 64))


def _fused_w4(lib, fn="masq_linear_fused_w4a8", **kw):
    a = dict(x=P, x_dt=1, mod=P, inv=P, wq=P, ws=P, ld=P, ru=P, lr_dt=1, T=16, K=128, N=64,
             rank=16, n_mod=2, y=P, y_dt=1, work=P, work_bytes=1 << 30, stream=None)
    a.update(kw)
    return getattr(lib, fn)(a["x"], a["x_dt"], a["mod"], a["inv"], a["wq"], a["ws"],
                            a["ld"], a["ru"], a["lr_dt"], a["T"], a["K"], a["N"], a["rank"],
                            a["n_mod"], a["y"], a["y_dt"], a["work"], a["work_bytes"],
                            a["stream"])


@pytest.mark.parametrize("fn", ["masq_linear_fused_w4a8", "masq_linear_stage1_w4a8",
                                "masq_linear_stage2_w4a8"])
@pytest.mark.parametrize("kw,code", [
    # the packed weight needs c_in % 64 == 0 (16-column multiples are not enough)
    (dict(K=48), 2), (dict(K=96), 2), (dict(K=200), 2),
    (dict(wq=None), 1), (dict(wq=P + 8), 4), (dict(work_bytes=100), 5),
    (dict(T=0, work=None, work_bytes=0), 0), (dict(K=64, T=0), 0),
])
def test_w4a8_fused_validates(lib, fn, kw, code):
    assert _fused_w4(lib, fn, **kw) == code


def test_w4a8_gemm_validates(lib):
    f = lib.masq_w4a8_gemm
    assert f(P, P, P, P, 8, 96, 64, P, None, 0, None) == 2         # c_in % 64 != 0
    assert f(P, P, P, P, 8, 64, 40, P, None, 0, None) == 2         # c_out % 16 != 0
    assert f(P, P, P, P, 8, 64, 64, None, None, 0, None) == 1      # no output
    assert f(P, P, P + 4, P, 8, 64, 64, P, None, 0, None) == 4     # misaligned wq4
    assert f(P, P, P, P, 8, 64, 64, None, P, 9, None) == 3
    assert f(P, P, P, P, 0, 64, 64, P, None, 0, None) == 0         # empty batch


def test_w4_linear_refuses_mismatched_packed_width():
    import torch
    from paper_2603_04800_amd import ops
    with pytest.raises(ValueError):
        ops.Linear(torch.ones(2, 128), torch.zeros(16, 128, dtype=torch.uint8), torch.ones(16))


def test_calibration_calls_validate(lib):
    """The GPU calibration entry points check sizes, dtypes, pointers and
    alignment before enqueueing anything."""
    P = 1 << 20
    cr, sf, qw = lib.masq_channel_range, lib.masq_smoothing_factors, lib.masq_quantize_weight
    assert cr(P, 2, P, 8, 64, 2, P, None) == 3              # unknown activation dtype
    assert cr(P, 1, P, 8, 40, 2, P, None) == 2              # c_in % 16 != 0
    assert cr(P, 1, P, 8, 64, 5, P, None) == 2              # n_mod > 4
    assert cr(P, 1, P, -1, 64, 2, P, None) == 2             # T < 0
    assert cr(P, 1, None, 8, 64, 2, P, None) == 1           # no modality ids
    assert cr(P, 1, P, 8, 64, 2, P + 8, None) == 4          # misaligned output
    assert sf(P, P, 64, 40, 2, P, P, None) == 2             # c_out % 16 != 0
    assert sf(P, None, 64, 64, 2, P, P, None) == 1          # no weight
    assert sf(P, P, 64, 64, 0, P, P, None) == 2             # n_mod < 1
    assert qw(P, P, 64, 64, 6, P, P, None) == 2             # bits must be 8 or 4
    assert qw(P, P, 48, 64, 8, P + 4, P, None) == 4         # misaligned codes
    assert qw(P, P, 64, 64, 8, P, None, None) == 1          # no step output


def test_cmc_calibration_calls_validate(lib):
    """masq_gather_smoothed, masq_weight_difference and masq_dgemm check
    sizes, dtypes, pointers and alignment before enqueueing anything."""
    import ctypes
    P = 1 << 20
    gs, wd, dg = lib.masq_gather_smoothed, lib.masq_weight_difference, lib.masq_dgemm
    assert gs(P, 2, 8, 64, P, 4, P, P, None) == 3            # unknown activation dtype
    assert gs(P, 1, 8, 40, P, 4, P, P, None) == 2            # c_in % 16 != 0
    assert gs(P, 1, 8, 64, P, -1, P, P, None) == 2           # n_rows < 0
    assert gs(P, 1, 8, 64, None, 4, P, P, None) == 1         # no row list
    assert gs(P, 1, 8, 64, P, 4, P, P + 8, None) == 4        # misaligned output
    assert gs(None, 1, 0, 64, None, 0, None, None, None) == 0   # nothing to gather
    assert wd(P, P, P, P, 64, 40, P, None) == 2              # c_out % 16 != 0
    assert wd(P, P, None, P, 64, 64, P, None) == 1           # no codes
    assert wd(P, P, P, P, 64, 64, P + 8, None) == 4          # misaligned output
    one = ctypes.c_double(0.0)
    assert dg(-1, 4, 4, P, 4, 1, P, 4, 1, one, P, 4, None) == 2       # m < 0
    assert dg(4, 4, 4, P, -4, 1, P, 4, 1, one, P, 4, None) == 2       # negative stride
    assert dg(4, 8, 4, P, 4, 1, P, 8, 1, one, P, 4, None) == 2        # ldc < n
    assert dg(65535 * 128 + 1, 4, 4, P, 4, 1, P, 4, 1, one, P, 4, None) == 2
    assert dg(4, 4, 4, None, 4, 1, P, 4, 1, one, P, 4, None) == 1     # no A
    assert dg(4, 4, 0, None, 0, 0, None, 0, 0, one, None, 4, None) == 1   # k = 0 still writes c
    assert dg(4, 4, 4, P + 4, 4, 1, P, 4, 1, one, P, 4, None) == 4    # misaligned A
    assert dg(0, 4, 4, None, 4, 1, None, 4, 1, one, None, 4, None) == 0   # empty output


def test_factorisation_calls_validate(lib):
    """masq_cholesky, masq_trsm_right and masq_jacobi_svd check sizes,
    pointers and alignment before enqueueing anything; empty problems
    enqueue nothing."""
    import ctypes
    P = 1 << 20
    ch, tr, jb = lib.masq_cholesky, lib.masq_trsm_right, lib.masq_jacobi_svd
    z = ctypes.c_double(0.0)
    assert ch(-1, P, 4, z, P, None, None) == 2                   # n < 0
    assert ch(8, P, 4, z, P, None, None) == 2                    # lda < n
    assert ch(65536, P, 65536, z, P, None, None) == 2            # n too large
    assert ch(8, P, 8, ctypes.c_double(-1.0), P, None, None) == 2    # negative ridge
    assert ch(8, P, 8, ctypes.c_double(float("nan")), P, None, None) == 2
    assert ch(8, P, 8, ctypes.c_double(float("inf")), P, None, None) == 2
    assert ch(8, P, 8, z, None, None, None) == 1                 # no info word
    assert ch(8, None, 8, z, P, None, None) == 1                 # no matrix
    assert ch(8, P + 4, 8, z, P, None, None) == 4                # misaligned matrix
    assert ch(8, P, 8, z, P + 2, None, None) == 4                # misaligned info
    assert ch(8, P, 8, z, P, P + 4, None) == 4                   # misaligned trace
    assert ch(0, None, 0, z, P, None, None) == 0                 # empty
    assert tr(-1, 4, P, 4, 1, P, 4, None) == 2                   # m < 0
    assert tr(4, 8, P, 4, 1, P, 8, None) == 2                    # ldl < n
    assert tr(4, 8, P, 8, 1, P, 4, None) == 2                    # ldy < n
    assert tr(4, 8, P, 8, 2, P, 8, None) == 2                    # trans not 0 or 1
    assert tr(4, 8, None, 8, 1, P, 8, None) == 1                 # no factor
    assert tr(4, 8, P, 8, 0, P + 4, 8, None) == 4                # misaligned Y
    assert tr(0, 8, None, 8, 1, None, 8, None) == 0              # no rows
    assert jb(4, 0, P, P, P, P, P, 0, 10, None, None) == 2       # n < 1
    assert jb(4, 1025, P, P, P, P, P, 0, 10, None, None) == 2    # n > 1024
    assert jb(0, 4, P, P, P, P, P, 0, 10, None, None) == 2       # m < 1
    assert jb(4, 4, P, P, P, P, P, 4, 10, None, None) == 2       # unknown flag
    assert jb(4, 4, P, P, P, P, P, 0, 0, None, None) == 2        # no sweeps allowed
    assert jb(4, 4, P, P, None, P, P, 0, 10, P, None) == 1       # no sigma
    assert jb(4, 4, P, P, P, P, P, 0, 10, None, None) == 1       # no sweep counter
    assert jb(4, 4, P, P, P, P + 4, P, 0, 10, P, None) == 4      # misaligned u
    assert jb(4, 4, P, P, P, P, P, 0, 10, P + 2, None) == 4      # misaligned sweeps


def test_mas_optimisation_calls_validate(lib):
    """masq_dequantize_rows, masq_mae_sign, masq_mas_gradient, masq_mae_loss
    and masq_adam_log_step check their arguments before enqueueing anything;
    masq_mae_partials is plain host arithmetic."""
    import ctypes
    P = 1 << 20
    dq, ms, mg = lib.masq_dequantize_rows, lib.masq_mae_sign, lib.masq_mas_gradient
    assert dq(P, P, -1, 4, P, None) == 2                         # rows < 0
    assert dq(None, P, 4, 4, P, None) == 1                       # no codes
    assert dq(P, P, 4, 4, P + 8, None) == 4                      # misaligned output
    assert dq(None, None, 0, 4, None, None) == 0                 # empty
    assert lib.masq_mae_partials(0) == 0
    assert lib.masq_mae_partials(1) == 1
    assert lib.masq_mae_partials(4096) == 1
    assert lib.masq_mae_partials(4097) == 2
    assert ms(P, P, -1, P, P, None) == 2
    assert ms(P, None, 8, P, P, None) == 1
    assert ms(P, P, 8, P + 4, P, None) == 4
    assert ms(None, None, 0, None, None, None) == 0
    assert mg(P, P, P, P, P, 4, 0, 16, P, P, None) == 2          # c_in = 0
    assert mg(P, P, P, None, P, 4, 16, 16, P, P, None) == 1      # no B
    assert mg(P, P, P, P, P, 4, 16, 16, P, P + 4, None) == 4     # misaligned grad
    ml, ad = lib.masq_mae_loss, lib.masq_adam_log_step
    assert ml(P, -1, P, None) == 2                               # count < 0
    assert ml(None, 8, P, None) == 1                             # no block sums
    assert ml(P, 8, None, None) == 1                             # no loss output
    assert ml(P, 8, P + 4, None) == 4                            # misaligned loss
    d = ctypes.c_double
    ok = (d(1.0), d(1e-2), d(0.9), d(0.999), d(1e-8))
    assert ad(P, P, P, P, P, P, -1, *ok, 1, None) == 2           # c_in < 0
    assert ad(P, P, P, P, P, P, 8, *ok, -1, None) == 2           # step < 0
    assert ad(P, P, P, P, P, P, 8, d(1.0), d(1e-2), d(1.0), d(0.999), d(1e-8), 1, None) == 2
    assert ad(P, P, P, P, P, P, 8, d(1.0), d(1e-2), d(0.9), d(0.999), d(0.0), 1, None) == 2
    assert ad(P, P, P, P, P, P, 8, d(float("nan")), d(1e-2), d(0.9), d(0.999), d(1e-8), 1,
              None) == 2
    assert ad(P, P, P, None, P, P, 8, *ok, 1, None) == 1         # step 1 needs a gradient
    assert ad(P, P, P, P, P, P + 2, 8, *ok, 1, None) == 4        # misaligned inverse factors
    assert ad(None, None, None, None, None, None, 0, *ok, 1, None) == 0   # empty


def test_dgemm_binding_refuses_an_output_aliasing_an_input():
    import torch
    from paper_2603_04800_amd import ops
    a = torch.zeros((4, 4), dtype=torch.float64)
    with pytest.raises(ValueError, match="share memory"):
        ops.dgemm(a, a, c=a)
    b = torch.zeros((4, 4), dtype=torch.float64)
    with pytest.raises(ValueError, match="share memory"):
        ops.dgemm(b.T, a, c=b)
