"""The C ABI without a GPU: the library loads, exports every entry point that
include/mpq.h declares, and rejects invalid arguments before touching the
device (argument checks never call HIP)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mpq.h")
LIB = os.path.join(ROOT, "paper_2002_09049_amd", "libmpq.so")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mpq_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        from paper_2002_09049_amd import build
        build.build()
    from paper_2002_09049_amd import mpq
    return mpq.load(LIB)


def test_header_declares_the_three_calls():
    names = _declared()
    for n in ("mpq_fit_layer", "mpq_output_error", "mpq_reconstruct", "mpq_last_error"):
        assert n in names


def test_exports_every_declared_symbol(lib):
    from paper_2002_09049_amd import mpq
    for name in _declared():
        assert hasattr(lib, name), name
    assert sorted(mpq.EXPORTS) == _declared()


def _fit(lib, **kw):
    args = dict(W=1, c_out=4, d=16, bits=4, max_points=4, grid=None, n_grid=8, tol=1e-3,
                codes=1, scales=1, counts=1, err=None)
    args.update(kw)
    g = args["grid"]
    garr = None if g is None else (ctypes.c_float * len(g))(*g)
    return lib.mpq_fit_layer(args["W"], args["c_out"], args["d"], args["bits"],
                             args["max_points"], garr, args["n_grid"], args["tol"],
                             args["codes"], args["scales"], args["counts"], args["err"], None)


@pytest.mark.parametrize("kw", [
    dict(c_out=-1), dict(d=0), dict(bits=1), dict(bits=9), dict(max_points=0),
    dict(max_points=65), dict(n_grid=0), dict(n_grid=4097), dict(tol=-1.0),
    dict(tol=float("inf")), dict(tol=float("nan")), dict(W=None), dict(codes=None),
    dict(scales=None), dict(counts=None),
    dict(grid=[0.5, 0.25], n_grid=2), dict(grid=[0.0, 1.0], n_grid=2),
    dict(grid=[0.5, 1.5], n_grid=2), dict(grid=[0.5, 0.5], n_grid=2),
])
def test_fit_rejects_invalid_arguments(lib, kw):
    from paper_2002_09049_amd import mpq
    assert _fit(lib, **kw) == mpq.MPQ_ERR_INVALID_ARG
    assert lib.mpq_last_error()


def test_fit_with_no_channels_is_a_no_op(lib):
    # c_out = 0 with otherwise valid arguments returns before any device call
    assert _fit(lib, c_out=0, W=None, codes=None, scales=None, counts=None) == 0


def test_output_error_and_reconstruct_reject_invalid_arguments(lib):
    from paper_2002_09049_amd import mpq
    E = mpq.MPQ_ERR_INVALID_ARG
    oe = lib.mpq_output_error
    assert oe(1, 1, 1, 1, -1, 4, 2, 1, 8, 1, None, None) == E
    assert oe(1, 1, 1, 1, 4, 0, 2, 1, 8, 1, None, None) == E
    assert oe(1, 1, 1, 1, 4, 4, 2, 1, 0, 1, None, None) == E
    assert oe(1, 1, 1, 1, 4, 4, 0, 1, 8, 1, None, None) == E
    assert oe(1, 1, 1, 1, 4, 4, 2, None, 8, 1, None, None) == E
    assert oe(1, 1, 1, 1, 4, 4, 2, 1, 8, None, None, None) == E
    assert oe(None, None, None, None, 0, 4, 2, None, 8, None, None, None) == 0
    rc = lib.mpq_reconstruct
    assert rc(1, 1, 1, -1, 4, 2, 1, None) == E
    assert rc(1, 1, 1, 4, 0, 2, 1, None) == E
    assert rc(1, 1, 1, 4, 4, 65, 1, None) == E
    assert b"max_points" in lib.mpq_last_error()
    assert rc(None, 1, 1, 4, 4, 2, 1, None) == E
    assert b"NULL" in lib.mpq_last_error()
    assert rc(None, None, None, 0, 4, 2, None, None) == 0


def test_output_error_noalloc_rejects_invalid_arguments(lib):
    """The no-allocation output error checks its arguments as mpq_output_error
    does, before its workspace lookup (a HIP call) and before any launch."""
    from paper_2002_09049_amd import mpq
    E = mpq.MPQ_ERR_INVALID_ARG
    oe = lib.mpq_output_error_noalloc
    assert oe(1, 1, 1, 1, -1, 4, 2, 1, 8, 1, None, None) == E
    assert oe(1, 1, 1, 1, 4, 0, 2, 1, 8, 1, None, None) == E
    assert oe(1, 1, 1, 1, 4, 4, 2, 1, 0, 1, None, None) == E
    assert oe(1, 1, 1, 1, 4, 4, 0, 1, 8, 1, None, None) == E
    assert oe(1, 1, 1, 1, 4, 4, 2, None, 8, 1, None, None) == E
    assert oe(1, 1, 1, 1, 4, 4, 2, 1, 8, None, None, None) == E
    assert oe(1, 1, 1, 1, (1 << 24) + 1, 4, 2, 1, 8, 1, None, None) == E
    assert oe(None, None, None, None, 0, 4, 2, None, 8, None, None, None) == 0
    assert re.search(r"#define MPQ_NOALLOC_BYTES \(64 << 20\)", open(HEADER).read())


def test_fit_max_dim_rejects_bad_grid(lib):
    from paper_2002_09049_amd import mpq
    assert lib.mpq_fit_max_dim(0) == mpq.MPQ_ERR_INVALID_ARG


def test_layer_struct_matches_header(tmp_path):
    """The binding's mpq_layer has the header's size and field offsets
    (checked by compiling the header with gcc)."""
    import subprocess
    from paper_2002_09049_amd import mpq
    fields = [f for f, _ in mpq.Layer._fields_]
    src = tmp_path / "off.c"
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "mpq.h"\nint main(void){\n'
                   '  printf("%zu\\n", sizeof(mpq_layer));\n' +
                   "".join(f'  printf("%zu\\n", offsetof(mpq_layer, {f}));\n' for f in fields) +
                   "  return 0;\n}\n")
    exe = tmp_path / "off"
    subprocess.check_call(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)])
    out = [int(x) for x in subprocess.check_output([str(exe)]).split()]
    assert out[0] == ctypes.sizeof(mpq.Layer)
    assert out[1:] == [getattr(mpq.Layer, f).offset for f in fields]


def test_batched_calls_reject_invalid_arguments(lib):
    from paper_2002_09049_amd import mpq
    E = mpq.MPQ_ERR_INVALID_ARG
    arr = (mpq.Layer * 2)()
    for L in arr:
        L.W, L.c_out, L.d, L.codes, L.scales, L.counts = 1, 4, 16, 1, 1, 1
        L.X, L.n, L.out_err, L.W_hat = 1, 8, 1, 1
    p = ctypes.addressof(arr)
    assert lib.mpq_fit_layers(p, -1, 4, 4, None, 8, 1e-3, None) == E
    assert lib.mpq_fit_layers(None, 2, 4, 4, None, 8, 1e-3, None) == E
    assert lib.mpq_fit_layers(p, 2, 9, 4, None, 8, 1e-3, None) == E
    arr[1].d = 0
    assert lib.mpq_fit_layers(p, 2, 4, 4, None, 8, 1e-3, None) == E
    assert b"layer 1" in lib.mpq_last_error()
    arr[1].d = 16
    arr[0].codes = None
    assert lib.mpq_fit_layers(p, 2, 4, 4, None, 8, 1e-3, None) == E
    assert b"layer 0" in lib.mpq_last_error()
    arr[0].codes = 1
    arr[1].n = 0
    assert lib.mpq_output_error_layers(p, 2, 4, None) == E
    arr[1].n = 8
    arr[0].W_hat = None
    assert lib.mpq_reconstruct_layers(p, 2, 4, None) == E
    # no channels at all: nothing to do, no device call
    for L in arr:
        L.c_out = 0
    assert lib.mpq_fit_layers(p, 2, 4, 4, None, 8, 1e-3, None) == 0
    assert lib.mpq_output_error_layers(p, 2, 4, None) == 0
    assert lib.mpq_reconstruct_layers(p, 2, 4, None) == 0
    assert lib.mpq_fit_layers(p, 0, 4, 4, None, 8, 1e-3, None) == 0


def test_output_error_rejects_oversized_dims(lib):
    from paper_2002_09049_amd import mpq
    E = mpq.MPQ_ERR_INVALID_ARG
    big = (1 << 24) + 1
    assert lib.mpq_output_error(1, 1, 1, 1, 4, 4, 2, 1, big, 1, None, None) == E
    assert lib.mpq_output_error(1, 1, 1, 1, big, 4, 2, 1, 8, 1, None, None) == E
    # d: a tile of 128 rows of D stays below 2 GiB
    max_d = int(re.search(r"#define MPQ_MAX_ERR_D (\d+)", open(HEADER).read()).group(1))
    assert (max_d + 31) // 32 * 32 * 128 * 4 < 2 ** 31
    assert lib.mpq_output_error(1, 1, 1, 1, 4, max_d + 1, 2, 1, 8, 1, None, None) == E
    assert "d must be <=" in mpq.last_error()


def test_timing_records_nothing_until_a_launch(lib):
    """Turning the per-launch timing on and off, and reading it with no launch
    recorded, touch no device."""
    from paper_2002_09049_amd import mpq
    assert lib.mpq_timing_enable(1) == 0
    assert lib.mpq_timing_read(None, 0) == 0
    assert lib.mpq_timing_read(None, -1) == mpq.MPQ_ERR_INVALID_ARG
    assert lib.mpq_timing_enable(0) == 0
    assert mpq.timing_read() == []
    assert lib.mpq_timing_only(b"x" * 64) == mpq.MPQ_ERR_INVALID_ARG
    assert lib.mpq_timing_only(b"gemm_err_kernel") == 0
    assert lib.mpq_timing_only(None) == 0
    assert lib.mpq_fit_kernel_of(0, 4, 8, 1, ctypes.create_string_buffer(64), 64) == mpq.MPQ_ERR_INVALID_ARG


def test_kernel_time_struct_matches_header(tmp_path):
    import subprocess
    from paper_2002_09049_amd import mpq
    src = tmp_path / "kt.c"
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "mpq.h"\nint main(void){\n'
                   '  printf("%zu %zu %zu\\n", sizeof(mpq_kernel_time), offsetof(mpq_kernel_time, name),'
                   ' offsetof(mpq_kernel_time, ms));\n  return 0;\n}\n')
    exe = tmp_path / "kt"
    subprocess.check_call(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)])
    out = [int(x) for x in subprocess.check_output([str(exe)]).split()]
    assert out == [ctypes.sizeof(mpq.KernelTime), mpq.KernelTime.name.offset, mpq.KernelTime.ms.offset]


def test_quantize_layers_checks_every_layer_first(lib):
    from paper_2002_09049_amd import mpq
    E = mpq.MPQ_ERR_INVALID_ARG
    arr = (mpq.Layer * 2)()
    for L in arr:
        L.W, L.c_out, L.d, L.codes, L.scales, L.counts = 1, 4, 16, 1, 1, 1
        L.X, L.n, L.out_err, L.W_hat = 1, 8, 1, 1
    p = ctypes.addressof(arr)
    q = lib.mpq_quantize_layers
    assert q(p, 2, 9, 4, None, 8, 1e-3, None) == E
    arr[1].n = 0            # an output-error layer without calibration columns
    assert q(p, 2, 4, 4, None, 8, 1e-3, None) == E
    assert b"layer 1" in lib.mpq_last_error()
    arr[1].out_err = None   # ... is fine once it asks for no output error
    arr[0].W_hat = None     # and a layer may skip the reconstruction
    arr[0].codes = None
    assert q(p, 2, 4, 4, None, 8, 1e-3, None) == E
    assert b"layer 0" in lib.mpq_last_error()
    for L in arr:
        L.c_out = 0
    assert q(p, 2, 4, 4, None, 8, 1e-3, None) == 0


def _calib(lib, **kw):
    args = dict(W=1, c_out=4, d=16, bits=4, max_points=4, grid=None, n_grid=8, X=1, n=8, eps=1e-3,
                relative=1, codes=1, scales=1, counts=1, err=None, xerr=1)
    args.update(kw)
    g = args["grid"]
    garr = None if g is None else (ctypes.c_float * len(g))(*g)
    return lib.mpq_fit_layer_calib(args["W"], args["c_out"], args["d"], args["bits"],
                                   args["max_points"], garr, args["n_grid"], args["X"], args["n"],
                                   args["eps"], args["relative"], args["codes"], args["scales"],
                                   args["counts"], args["err"], args["xerr"], None)


@pytest.mark.parametrize("kw", [
    dict(c_out=-1), dict(d=0), dict(bits=1), dict(max_points=0), dict(max_points=65),
    dict(n_grid=0), dict(eps=-1.0), dict(eps=float("inf")), dict(eps=float("nan")),
    dict(W=None), dict(codes=None), dict(X=None), dict(xerr=None), dict(n=0),
    dict(n=16777217), dict(c_out=16777217), dict(grid=[0.5, 0.25], n_grid=2),
])
def test_calib_fit_rejects_invalid_arguments(lib, kw):
    from paper_2002_09049_amd import mpq
    assert _calib(lib, **kw) == mpq.MPQ_ERR_INVALID_ARG
    assert lib.mpq_last_error()


def test_calib_fit_with_no_channels_is_a_no_op(lib):
    assert _calib(lib, c_out=0, W=None, codes=None, scales=None, counts=None, X=None, xerr=None) == 0


def test_calib_layers_check_every_layer_first(lib):
    from paper_2002_09049_amd import mpq
    E = mpq.MPQ_ERR_INVALID_ARG
    arr = (mpq.Layer * 2)()
    for L in arr:
        L.W, L.c_out, L.d, L.codes, L.scales, L.counts = 1, 4, 16, 1, 1, 1
        L.X, L.n, L.fit_xerr = 1, 8, 1
    p = ctypes.addressof(arr)
    f = lib.mpq_fit_layers_calib
    arr[1].fit_xerr = None
    assert f(p, 2, 4, 4, None, 8, 1e-3, 1, None) == E
    assert b"layer 1" in lib.mpq_last_error()
    arr[1].fit_xerr = 1
    assert f(p, 2, 4, 4, None, 8, -1.0, 1, None) == E
    assert f(p, 2, 9, 4, None, 8, 1e-3, 1, None) == E
    for L in arr:
        L.c_out = 0
    assert f(p, 2, 4, 4, None, 8, 1e-3, 0, None) == 0


def test_integer_calls_reject_invalid_arguments(lib):
    from paper_2002_09049_amd import mpq
    E = mpq.MPQ_ERR_INVALID_ARG
    sc = lib.mpq_integer_scales
    assert sc(1, 1, 4, 4, -1, 1, None, None) == E
    assert sc(1, 1, 4, 4, 63, 1, None, None) == E
    assert sc(1, 1, 4, 0, 8, 1, None, None) == E
    assert sc(None, 1, 4, 4, 8, 1, None, None) == E
    assert sc(1, 1, -1, 4, 8, 1, None, None) == E
    assert sc(None, None, 0, 4, 8, None, None, None) == 0
    fw = lib.mpq_integer_forward
    ok = dict(codes=1, A=1, counts=1, c=4, d=16, P=4, X=1, n=8, p=8, Y=1)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return fw(a["codes"], a["A"], a["counts"], a["c"], a["d"], a["P"], a["X"], a["n"], a["p"],
                  a["Y"], None)
    for kw in (dict(p=-1), dict(p=63), dict(d=0), dict(d=131073), dict(P=0), dict(P=65),
               dict(c=-1), dict(n=-1), dict(codes=None), dict(A=None), dict(counts=None),
               dict(X=None), dict(Y=None), dict(c=1 << 20, d=4096, P=4),
               dict(n=1 << 20, d=4096)):
        assert call(**kw) == E, kw
    assert call(c=0, codes=None, A=None, counts=None, Y=None) == 0
    assert call(n=0, X=None, Y=None) == 0


def test_int_layer_struct_matches_header(tmp_path):
    import subprocess
    from paper_2002_09049_amd import mpq
    fields = [f for f, _ in mpq.IntLayer._fields_]
    src = tmp_path / "off.c"
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "mpq.h"\nint main(void){\n'
                   '  printf("%zu\\n", sizeof(mpq_int_layer));\n' +
                   "".join(f'  printf("%zu\\n", offsetof(mpq_int_layer, {f}));\n' for f in fields) +
                   "  return 0;\n}\n")
    exe = tmp_path / "off"
    subprocess.check_call(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)])
    out = [int(x) for x in subprocess.check_output([str(exe)]).split()]
    assert out[0] == ctypes.sizeof(mpq.IntLayer)
    assert out[1:] == [getattr(mpq.IntLayer, f).offset for f in fields]


def test_fit_options_struct_matches_header(tmp_path):
    import subprocess
    from paper_2002_09049_amd import mpq
    fields = [f for f, _ in mpq.FitOptions._fields_]
    src = tmp_path / "off.c"
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "mpq.h"\nint main(void){\n'
                   '  printf("%zu\\n", sizeof(mpq_fit_options));\n' +
                   "".join(f'  printf("%zu\\n", offsetof(mpq_fit_options, {f}));\n' for f in fields) +
                   "  return 0;\n}\n")
    exe = tmp_path / "off"
    subprocess.check_call(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)])
    out = [int(x) for x in subprocess.check_output([str(exe)]).split()]
    assert out[0] == ctypes.sizeof(mpq.FitOptions)
    assert out[1:] == [getattr(mpq.FitOptions, f).offset for f in fields]


def test_fit_layers_ex_checks_arguments(lib):
    from paper_2002_09049_amd import mpq
    E = mpq.MPQ_ERR_INVALID_ARG
    arr = (mpq.Layer * 1)()
    L = arr[0]
    L.W, L.c_out, L.d, L.codes, L.scales, L.counts = 1, 4, 16, 1, 1, 1
    p = ctypes.addressof(arr)
    for opt in (None, mpq.FitOptions(1, 0, 0.0, 0), mpq.FitOptions(1, 1, 1e-3, 1)):
        o = None if opt is None else ctypes.addressof(opt)
        assert lib.mpq_fit_layers_ex(p, 1, 9, 4, None, 8, 1e-3, o, None) == E
        assert lib.mpq_fit_layers_ex(p, 1, 4, 0, None, 8, 1e-3, o, None) == E
    opt = mpq.FitOptions(0, 1, 1e-3, 1)          # calib needs X and fit_xerr
    assert lib.mpq_fit_layers_ex(p, 1, 4, 4, None, 8, 1e-3, ctypes.addressof(opt), None) == E
    L.c_out = 0
    assert lib.mpq_fit_layers_ex(p, 1, 4, 4, None, 8, 1e-3, ctypes.addressof(opt), None) == 0


def test_workspace_cap_gives_nomem(lib):
    """MPQ_WORKSPACE_LIMIT caps each scratch allocation before any HIP call:
    the output error's request fails with MPQ_ERR_NOMEM (no device needed)."""
    from paper_2002_09049_amd import mpq
    os.environ["MPQ_WORKSPACE_LIMIT"] = "64"
    try:
        rc = lib.mpq_output_error(1, 1, 1, 1, 4, 16, 2, 1, 8, 1, None, None)
        assert rc == mpq.MPQ_ERR_NOMEM, rc
        assert "scratch" in mpq.last_error()
    finally:
        del os.environ["MPQ_WORKSPACE_LIMIT"]
