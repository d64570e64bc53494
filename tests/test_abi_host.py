"""Host-side checks of the C ABI: the library loads, exports every symbol the
header declares, and rejects bad arguments before touching a device."""
import math
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2505_17701_amd import binding as cd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "countdown.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(cd.LIB_PATH):
        from paper_2505_17701_amd import build

        build.build()
    return cd.load_library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(countdown_\w+)\s*\(", text)))


def test_header_declarations_match_binding_list():
    assert declared_functions() == sorted(cd.EXPORTS)


def test_every_declared_symbol_is_exported(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", cd.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (countdown_\w+)", out))
    for name in declared_functions():
        assert name in exported, name
        assert getattr(lib, name) is not None


def test_header_compiles_as_c():
    src = f'#include "{HEADER}"\nint main(void) {{ return countdown_abi_version() == 0; }}\n'
    res = subprocess.run(["gcc", "-x", "c", "-std=c99", "-Wall", "-Werror", "-fsyntax-only", "-"],
                         input=src, text=True, capture_output=True)
    assert res.returncode == 0, res.stderr


def test_abi_version_and_status_strings(lib):
    assert cd.countdown_abi_version() == 9
    for st in (cd.CD_OK, cd.CD_EINVAL, cd.CD_EUNSUPPORTED, cd.CD_EHIP, cd.CD_ENOMEM):
        assert cd.status_string(st).startswith(("CD_OK", "CD_E"))
    assert "unknown" in cd.status_string(12345)


@pytest.mark.parametrize("shape,expect", [
    ((4096, 11008, 1, 0), cd.CD_OK),
    ((8192, 28672, 4, 0), cd.CD_OK),
    ((256, 688, 1, 0), cd.CD_OK),
    ((4096, 14336, 8, 256), cd.CD_OK),
    ((4100, 11008, 1, 0), cd.CD_EINVAL),        # d_model % 8
    ((4096, 11004, 1, 0), cd.CD_EINVAL),        # d_ff % 8
    ((0, 11008, 1, 0), cd.CD_EINVAL),
    ((16384, 11008, 1, 0), cd.CD_EUNSUPPORTED),  # d_model > 8192
    ((4096, 11008, 0, 0), cd.CD_EINVAL),
    ((4096, 11008, 9, 0), cd.CD_EUNSUPPORTED),
    ((8192, 28672, 8, 0), cd.CD_EUNSUPPORTED),   # batch x d_model > 32768
    ((4160, 1024, 4, 0), cd.CD_OK),              # 4 tokens x 16 chunks of 512
    ((4160, 1024, 5, 0), cd.CD_EUNSUPPORTED),    # tile of 8 tokens x 16 chunks
    ((4160, 1024, 7, 0), cd.CD_EUNSUPPORTED),
    ((2056, 4104, 8, 0), cd.CD_OK),              # 8 tokens x 8 chunks
    ((4096, 14336, 1, 200), cd.CD_EUNSUPPORTED), # rank not a power of two
    ((4096, 14336, 1, -8), cd.CD_EINVAL),
])
def test_check_shape(lib, shape, expect):
    assert cd.countdown_check_shape(*shape) == expect


GOOD = dict(x=0x1000, W_gate=0x2000, W_up=0x3000, W_down=0x4000, y=0x5000)


def check(variant=cd.CD_VARIANT_MONO, B=1, thld=1.0, A_t=None, B_t=None, d_rank=0, **kw):
    p = dict(GOOD)
    p.update(kw)
    return cd.countdown_check_args(variant, 4096, 11008, 4, d_rank, p["x"], B, p["W_gate"],
                                   p["W_up"], p["W_down"], A_t, B_t, thld, p["y"])


def test_check_args_accepts_good_calls(lib):
    assert check() == cd.CD_OK
    assert check(B=4, thld=-math.inf) == cd.CD_OK
    assert check(thld=math.inf) == cd.CD_OK
    assert check(cd.CD_VARIANT_DUAL_IDEAL) == cd.CD_OK
    assert check(cd.CD_VARIANT_DENSE) == cd.CD_OK
    assert check(cd.CD_VARIANT_DUAL_PRED, A_t=0x6000, B_t=0x7000, d_rank=256) == cd.CD_OK


@pytest.mark.parametrize("bad", [
    dict(x=None), dict(W_gate=None), dict(W_up=None), dict(W_down=None), dict(y=None),
    dict(x=0x1002), dict(W_up=0x3008), dict(y=0x5004),            # not 16-byte aligned
    dict(B=0), dict(B=5), dict(thld=math.nan),
])
def test_check_args_rejects(lib, bad):
    assert check(**bad) == cd.CD_EINVAL


def test_predictor_pointer_rules(lib):
    pred = cd.CD_VARIANT_DUAL_PRED
    assert check(pred, A_t=0x6000, B_t=None, d_rank=256) == cd.CD_EINVAL
    assert check(pred, A_t=None, B_t=0x7000, d_rank=256) == cd.CD_EINVAL
    assert check(pred, A_t=0x6000, B_t=0x7000, d_rank=0) == cd.CD_EINVAL
    assert check(pred, A_t=0x6004, B_t=0x7000, d_rank=256) == cd.CD_EINVAL
    assert check(cd.CD_VARIANT_MONO, A_t=0x6000, B_t=0x7000, d_rank=256) == cd.CD_EINVAL


def test_null_plan_is_rejected_without_device(lib):
    assert lib.countdown_ffn_mono(None, 0x1000, 1, 0x2000, 0x3000, 0x4000, 1.0, 0x5000,
                                  None) == cd.CD_EINVAL
    assert lib.countdown_ffn_dual(None, 0x1000, 1, 0x2000, 0x3000, 0x4000, None, None, 1.0,
                                  0x5000, None) == cd.CD_EINVAL
    assert lib.countdown_plan_destroy(None) == cd.CD_OK
    assert lib.countdown_plan_set_phases(None, cd.CD_PHASE_ALL) == cd.CD_EINVAL
    assert lib.countdown_export_active(None, None, None, None, None, None) == cd.CD_EINVAL


def test_plan_create_rejects_bad_sizes_before_any_hip_call(lib):
    import ctypes as C

    h = C.c_void_p()
    assert lib.countdown_plan_create(4100, 11008, 1, 0, 0, C.byref(h)) == cd.CD_EINVAL
    assert lib.countdown_plan_create(4096, 11008, 1, 0, 0x80, C.byref(h)) == cd.CD_EINVAL
    assert lib.countdown_plan_create(4096, 11008, 1, 0, 4, C.byref(h)) == cd.CD_EINVAL
    assert h.value is None


def test_ternary_pointer_rules(lib):
    tern = cd.CD_VARIANT_DUAL_TERN
    assert check(tern, A_t=0x6000) == cd.CD_OK               # A_t carries the packed theta
    assert check(tern, A_t=0x6000, d_rank=256) == cd.CD_OK   # the rank is not used
    assert check(tern) == cd.CD_EINVAL
    assert check(tern, A_t=0x6008) == cd.CD_EINVAL
    assert check(tern, A_t=0x6000, B_t=0x7000) == cd.CD_EINVAL
    assert check(6, A_t=0x6000) == cd.CD_EINVAL
    assert lib.countdown_ffn_tern(None, 0x1000, 1, 0x2000, 0x3000, 0x4000, 0x6000, 1.0, 0x5000,
                                  None) == cd.CD_EINVAL
    assert lib.countdown_calibrate(None, tern, 0x1000, 4, 0x2000, 0x3000, None, None, 0.5,
                                   0x5000, None, None) == cd.CD_EINVAL


def _unpack_reference(packed, d_model, d_ff):
    """The packed layout as the header states it, decoded by plain loops."""
    C = 1
    while 512 * C < d_model:
        C *= 2
    W = max(1, C // 2)
    row_words = 64 * W
    assert packed.size == d_ff * row_words
    value = {0: 0, 1: 1, 2: -1}
    out = np.zeros((d_ff, d_model), dtype=np.int8)
    for i in range(d_ff):
        for l in range(64):
            for j in range(C):
                word = int(packed[i * row_words + l * W + j // 2])
                for e in range(8):
                    m = e // 2
                    byte = (1 if j % 2 == 0 else 0) + (2 if e % 2 else 0)
                    code = (word >> (8 * byte + 2 * m)) & 3
                    col = j * 512 + 8 * l + e
                    assert code != 3
                    if col < d_model:
                        out[i, col] = value[code]
                    else:
                        assert code == 0
    return out


@pytest.mark.parametrize("d_model,d_ff", [(8, 16), (512, 24), (520, 8), (1032, 16), (4096, 8),
                                          (8192, 8)])
def test_ternary_pack_layout(lib, d_model, d_ff):
    from workloads import make_ternary

    T = make_ternary(990, d_model, d_ff)
    packed = cd.countdown_ternary_pack(T)
    assert packed.dtype == np.uint32
    np.testing.assert_array_equal(_unpack_reference(packed, d_model, d_ff), T)


def test_ternary_pack_rejects(lib):
    assert cd.countdown_ternary_words(4100, 8) == 0
    assert cd.countdown_ternary_words(4096, 11008) == 11008 * 256
    assert cd.countdown_ternary_words(8192, 8) == 8 * 512
    assert cd.countdown_ternary_words(256, 8) == 8 * 64
    bad = np.zeros((8, 16), dtype=np.int8)
    bad[3, 5] = 2
    with pytest.raises(cd.CountdownError):
        cd.countdown_ternary_pack(bad)


def test_missing_library_fails_loudly(tmp_path):
    """No fallback: loading a library that is not there raises, naming the build step."""
    import subprocess
    import sys

    code = (
        "import sys; sys.path.insert(0, %r)\n"
        "from paper_2505_17701_amd import binding as cd\n"
        "cd.LIB_PATH = %r\n"
        "try:\n"
        "    cd.load_library(cd.LIB_PATH)\n"
        "except RuntimeError as e:\n"
        "    print('raised:', e)\n"
        "    sys.exit(0)\n"
        "sys.exit(1)\n" % (ROOT, str(tmp_path / "absent.so")))
    res = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "build" in res.stdout


def test_binding_checks_shapes_before_pointers():
    """The C ABI sees only pointers, so the binding checks every tensor's shape against
    the plan first: an undersized x, weight, predictor, packed theta or y raises
    ValueError before any pointer is taken (CPU tensors suffice to show it)."""
    import types

    import torch

    plan = types.SimpleNamespace(d_model=64, d_ff=128, d_rank=8, max_batch=2)
    x = torch.zeros(2, 64, dtype=torch.bfloat16)
    W = torch.zeros(128, 64, dtype=torch.bfloat16)
    A = torch.zeros(8, 64, dtype=torch.bfloat16)
    Bt = torch.zeros(128, 8, dtype=torch.bfloat16)
    cd._layer_shapes(plan, x, W, W, W, A, Bt)  # the right shapes pass
    bad = [dict(x=torch.zeros(2, 32, dtype=torch.bfloat16)),
           dict(x=torch.zeros(128, dtype=torch.bfloat16)),
           dict(W_gate=W[:64]), dict(W_up=W[:, :32]), dict(W_down=W.reshape(64, 128)),
           dict(A_t=A[:4]), dict(B_t=Bt[:, :4])]
    for b in bad:
        kw = dict(x=x, W_gate=W, W_up=W, W_down=W, A_t=A, B_t=Bt)
        kw.update(b)
        with pytest.raises(ValueError):
            cd._layer_shapes(plan, **kw)
    words = cd.countdown_ternary_words(64, 128)
    cd._layer_shapes(plan, x, W, W, W, theta_packed=torch.zeros(words, dtype=torch.int32))
    with pytest.raises(ValueError):
        cd._layer_shapes(plan, x, W, W, W, theta_packed=torch.zeros(words - 1, dtype=torch.int32))
    B, y = cd._out(plan, x, None)
    assert B == 2 and tuple(y.shape) == (2, 64)
    with pytest.raises(ValueError):
        cd._out(plan, x, torch.zeros(1, 64))
    with pytest.raises(TypeError):
        cd._out(plan, x, torch.zeros(2, 64, dtype=torch.float64))


def test_bench_refuses_more_than_one_gpu():
    """bench.py times one GPU: --gpus N > 1 exits with status 2 and says why,
    before it touches a device."""
    import sys

    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"], cwd=root,
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr and r.stdout == ""


@pytest.mark.parametrize("d_model,expect", [(4096, 8), (4160, 4), (8192, 4), (256, 8), (2056, 8)])
def test_max_batch_for(lib, d_model, expect):
    """The widest batch a plan accepts: the batch tile (1, 2, 4 or 8 tokens) times
    d_model rounded up to a power-of-two number of 512-column chunks stays within
    32768 token columns."""
    assert cd.max_batch_for(d_model) == expect


def test_plan_create_refuses_unsupported_tile_before_hip(lib):
    """d_model 4160 at 5 tokens would need an 8-token tile of 16 chunks; plan creation
    refuses it on the host, before any HIP call."""
    with pytest.raises(cd.CountdownError) as e:
        cd.Plan(4160, 1024, max_batch=5)
    assert e.value.status == cd.CD_EUNSUPPORTED


def _hip_devices():
    import ctypes as C

    try:
        hip = C.CDLL("libamdhip64.so")
    except OSError:
        return 0
    n = C.c_int(0)
    return n.value if hip.hipGetDeviceCount(C.byref(n)) == 0 else 0


def test_hip_failures_map_to_cd_ehip(lib):
    """Where the HIP runtime has no device, the first HIP call after the host checks
    fails, and plan creation, the entry point without allocation and the streaming
    read aid each return CD_EHIP (the hipError_t mapping), writing no plan handle."""
    import ctypes as C

    if _hip_devices() > 0:
        pytest.skip("a GPU is visible: these calls would reach it with placeholder pointers")
    h = C.c_void_p()
    assert lib.countdown_plan_create(4096, 11008, 1, 0, 0, C.byref(h)) == cd.CD_EHIP
    assert h.value is None
    vp = C.c_void_p
    assert lib.countdown_ffn_mono_noalloc(vp(0x1000), 1, vp(0x2000), vp(0x3000), vp(0x4000), 256,
                                          688, 1.0, vp(0x5000), None) == cd.CD_EHIP
    assert lib.countdown_stream_read(vp(0x1000), 16, vp(0x2000), None) == cd.CD_EHIP


def test_bench_traffic_gated_by_kernel_source(tmp_path, monkeypatch):
    """bench.py reports a committed FETCH_SIZE + WRITE_SIZE figure only while the
    kernel source it was taken on is unchanged: the digest ignores comments and
    whitespace, a code change invalidates the figure (traffic null)."""
    import bench

    a = tmp_path / "a.hip"
    b = tmp_path / "b.hip"
    a.write_text("int f(int x) { return x + 1; } // one\n/* block */\n")
    b.write_text("int f(int x)  {\n  return x + 1;  }  // two\n")
    monkeypatch.setattr(bench, "KERNEL_SRCS", [str(a)])
    d_a = bench.kernel_source_digest()
    monkeypatch.setattr(bench, "KERNEL_SRCS", [str(b)])
    assert bench.kernel_source_digest() == d_a  # comments and spacing only
    b.write_text("int f(int x) { return x + 2; }\n")
    assert bench.kernel_source_digest() != d_a

    monkeypatch.setattr(bench, "KERNEL_SRCS", [str(a)])
    (tmp_path / "profiles").mkdir()
    summary = tmp_path / "profiles" / "line_traffic.md"
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "TRAFFIC_SUMMARIES", {("w", "v", 0.9, 1): "line_traffic.md"})
    summary.write_text(f"# x\n\n- kernel_source_digest: `{d_a}`\n- hbm_bytes_per_launch: `1234.0`\n")
    assert bench.measured_traffic(("w", "v", 0.9, 1)) == 1234.0
    assert bench.measured_traffic(("w", "v", 0.7, 1)) is None  # no summary for the line
    summary.write_text("# x\n\n- kernel_source_digest: `stale`\n- hbm_bytes_per_launch: `1234.0`\n")
    assert bench.measured_traffic(("w", "v", 0.9, 1)) is None
