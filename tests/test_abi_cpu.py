"""CPU checks of the C-ABI library: it loads, exports every function that
include/curvadion.h declares, and rejects invalid arguments before touching
the GPU (no compute call is made here)."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2512_13728_amd as cdl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "curvadion.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(cdl.library_path):
        from paper_2512_13728_amd import build
        build.build()
    return cdl.lib()


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cd_[a-z_]+)\s*\(", text)))


def test_header_matches_binding_list():
    assert header_functions() == sorted(cdl.EXPORTED_SYMBOLS)


def test_library_exports_every_declared_symbol(L):
    out = subprocess.run(["nm", "-D", "--defined-only", cdl.library_path],
                         capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\sT\s(cd_[a-z_]+)$", out, flags=re.M))
    for name in header_functions():
        assert name in exported, name
        assert hasattr(L, name)
    hdr = open(os.path.join(ROOT, "include", "curvadion.h")).read()
    assert L.cd_abi_version() == int(re.search(r"#define CD_ABI_VERSION (\d+)", hdr).group(1))


def _desc(**kw):
    d = dict(m=64, n=32, r_max=8, grad_dtype=cdl.F32, tau=0.5, eps=1e-8, eta_local_scale=1.0,
             policy=cdl.POLICY_RMMC, H=1)
    d.update(kw)
    return cdl.LayerDesc(**d)


@pytest.mark.parametrize("kw,msg", [
    (dict(m=0), "m and n"), (dict(n=-3), "m and n"), (dict(r_max=0), "r_max"),
    (dict(r_max=33), "r_max"), (dict(m=4000, n=4000, r_max=2000), "1024"),
    (dict(grad_dtype=7), "dtype"), (dict(policy=9), "policy"),
    (dict(tau=float("nan")), "tau"), (dict(eps=-1.0), "eps"), (dict(eps=float("inf")), "eps"),
    (dict(eta_local_scale=-0.5), "eta_local_scale"), (dict(policy=cdl.POLICY_EVERY_H, H=0), "H"),
    (dict(weight_decay=-0.01), "weight_decay"), (dict(weight_decay=float("nan")), "weight_decay"),
])
def test_layer_create_rejects_bad_descriptors(L, kw, msg):
    h = ctypes.c_void_p(123)
    d = _desc(**kw)
    assert L.cd_layer_create(ctypes.byref(d), ctypes.byref(h)) == cdl.CD_EINVAL
    assert h.value is None
    assert msg in L.cd_last_error().decode()


def test_null_arguments_are_einval(L):
    h = ctypes.c_void_p()
    assert L.cd_layer_create(None, ctypes.byref(h)) == cdl.CD_EINVAL
    d = _desc()
    assert L.cd_layer_create(ctypes.byref(d), None) == cdl.CD_EINVAL
    res = cdl.Result()
    assert L.cd_step(None, 1, 2, 3, 4, 0.9, 0.01, 4, None, ctypes.byref(res)) == cdl.CD_EINVAL
    assert L.cd_group_create(None, 1, ctypes.byref(h)) == cdl.CD_EINVAL
    arr = (ctypes.c_void_p * 1)(None)
    assert L.cd_group_create(arr, 0, ctypes.byref(h)) == cdl.CD_EINVAL
    assert L.cd_group_create(arr, 1, ctypes.byref(h)) == cdl.CD_EINVAL
    assert L.cd_group_step(None, None, None, None, None, 0.9, 0.01, 4, None, None, None) == cdl.CD_EINVAL
    p, s = ctypes.c_double(), ctypes.c_longlong()
    assert L.cd_layer_get_state(None, ctypes.byref(p), ctypes.byref(s)) == cdl.CD_EINVAL
    assert L.cd_layer_set_state(None, 1.0, 0) == cdl.CD_EINVAL
    P, R = ctypes.c_void_p(), ctypes.c_void_p()
    assert L.cd_layer_last_factors(None, ctypes.byref(P), ctypes.byref(R)) == cdl.CD_EINVAL
    f = ctypes.c_int()
    assert L.cd_layer_rank_deficient(None, ctypes.byref(f)) == cdl.CD_EINVAL
    assert L.cd_group_set_timing(None, 1) == cdl.CD_EINVAL
    assert L.cd_group_set_timing_kinds(None, b"gate") == cdl.CD_EINVAL
    assert L.cd_destroy(None) == cdl.CD_OK
    assert L.cd_group_destroy(None) == cdl.CD_OK


def test_product_path_has_no_fallback():
    """The binding refuses to run without the library: no CPU path exists."""
    import importlib
    import paper_2512_13728_amd as mod
    saved_path, saved_lib = mod.library_path, mod._lib
    try:
        mod.library_path = os.path.join(ROOT, "does_not_exist.so")
        mod._lib = None
        with pytest.raises(mod.LibraryNotBuilt):
            mod.Layer(8, 8, 2)
    finally:
        mod.library_path, mod._lib = saved_path, saved_lib


def test_package_does_not_import_oracle():
    src_dir = os.path.join(ROOT, "paper_2512_13728_amd")
    for dirpath, _, files in os.walk(src_dir):
        for f in files:
            if f.endswith((".py", ".cpp", ".hip", ".hpp", ".h")):
                text = open(os.path.join(dirpath, f), errors="replace").read()
                assert "oracle" not in text.lower().replace("oracles", ""), f


def test_operand_check_refuses_what_the_kernels_would_misread():
    """The binding's operand check: the kernels index G, M, X (m x n) and Q
    (n x r) by the sizes alone, so a wrong shape, dtype or layout is refused
    before the library sees the pointer."""
    import torch
    m, n, r = 48, 40, 8
    ok = dict(G=torch.zeros(m, n), M=torch.zeros(m, n), X=torch.zeros(m, n), Q=torch.zeros(n, r))
    bad = [
        ("M", torch.zeros(n, m), "shape"),                    # transposed shape
        ("Q", torch.zeros(n, r + 1), "shape"),                # Q wider than the step's rank
        ("X", torch.zeros(m, n, dtype=torch.float64), "float32"),
        ("G", torch.zeros(m, n, dtype=torch.bfloat16), "float32"),   # fp32-gradient layer
        ("M", torch.zeros(n, m).t(), "contiguous"),           # right shape, column-major
        ("Q", torch.zeros(n, 2 * r)[:, :r], "contiguous"),    # a column slice
        ("G", torch.zeros(m, n), "GPU"),                      # host memory
    ]
    for role, t, msg in bad:
        with pytest.raises(ValueError, match=msg):
            cdl.check_operand(t, role, m, n, r, "f32")
    # raw addresses pass through unchecked (the C ABI's contract)
    cdl.check_operand(0x1000, "M", m, n, r, "f32")
    # every check before the device check passes for well-formed host tensors
    for role, t in ok.items():
        with pytest.raises(ValueError, match="GPU"):
            cdl.check_operand(t, role, m, n, r, "f32")
    with pytest.raises(ValueError, match="GPU"):
        cdl.check_operand(torch.zeros(m, n, dtype=torch.bfloat16), "G", m, n, r, "bf16")


def test_plain_c_client_check():
    """A C99 program that includes only include/curvadion.h (and the HIP
    runtime's C API) compiles with gcc -Werror, links against the library and
    sees CD_EINVAL with a message for invalid descriptors and NULL arguments."""
    from paper_2512_13728_amd import build
    exe = build.C_CLIENT
    if not os.path.exists(exe):
        build.build_c_client()
    out = subprocess.run([exe, "check"], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stderr
    assert "check ok" in out.stdout
    assert out.stdout.count("CD_EINVAL") == 8


def _stream_plan(shapes, tmp_path):
    """Streaming-pass launches the library plans for `shapes`: the planning
    header compiled with g++ (it has no HIP dependency) and run on the CPU."""
    exe = tmp_path / "plan_check"
    subprocess.run(["g++", "-std=c++17", "-O1", "-Wall", "-Werror", "-I",
                    os.path.join(ROOT, "paper_2512_13728_amd", "csrc"),
                    os.path.join(ROOT, "tests", "c", "plan_check.cpp"), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], input="".join(f"{m} {n}\n" for m, n in shapes),
                         capture_output=True, text=True, check=True).stdout
    return [tuple(int(x) for x in line.split()) for line in out.splitlines()]


def test_streaming_launch_plan_of_the_workloads(tmp_path):
    """The buffer pass and the local update launch whole layers in group order,
    at most 48 layers and 98304 blocks of 4096 elements per launch: the
    1.3B-shaped set (96 matrices, 24 blocks of 2048x6144, 2048x2048,
    2048x8192, 8192x2048) runs as 3 launches of 32 layers (8 transformer
    blocks, 402.7M elements each), the 160M-shaped set (48 matrices) as one
    launch, and a layer beyond the block cap as a launch of its own."""
    import synthetic as S
    assert _stream_plan(S.WORKLOADS["gpt1p3b"].shapes, tmp_path) == [(32, 98304)] * 3
    assert _stream_plan(S.WORKLOADS["gpt160m"].shapes, tmp_path) == [(48, 20736)]
    assert _stream_plan([(256, 256)], tmp_path) == [(1, 16)]
    # 46341^2 elements (2^31 + 4633): 524290 blocks, alone; the next layer starts a launch
    assert _stream_plan([(13, 7), (46341, 46341), (300, 1000)], tmp_path) == [(1, 1), (1, 524290), (1, 74)]
    # 49 small layers: the layer cap splits them 48 + 1
    assert _stream_plan([(64, 64)] * 49, tmp_path) == [(48, 48), (1, 1)]


def test_static_step_refuses_before_touching_the_gpu(L):
    """cd_step_static checks the descriptor, its state arguments and the
    workspace size against the fixed array before anything else (so these
    errors need no GPU)."""
    st = ctypes.c_longlong(0)
    res = cdl.Result()
    big = _desc(m=8192, n=8192, r_max=1024)
    rc = L.cd_step_static(ctypes.byref(big), 4096, ctypes.byref(st), 16, 16, 16, 16, 0.95, 0.01, 1024, None,
                          ctypes.byref(res))
    assert rc == cdl.CD_EINVAL and b"CD_STATIC_SCRATCH_BYTES" in L.cd_last_error()
    small = _desc()
    assert L.cd_step_static(ctypes.byref(small), None, ctypes.byref(st), 16, 16, 16, 16, 0.95, 0.01, 4, None,
                            ctypes.byref(res)) == cdl.CD_EINVAL
    assert L.cd_step_static(ctypes.byref(small), 4096, None, 16, 16, 16, 16, 0.95, 0.01, 4, None,
                            ctypes.byref(res)) == cdl.CD_EINVAL
    assert L.cd_step_static(ctypes.byref(small), 4100, ctypes.byref(st), 16, 16, 16, 16, 0.95, 0.01, 4, None,
                            ctypes.byref(res)) == cdl.CD_EINVAL     # misaligned prev_norm
    assert L.cd_step_static(ctypes.byref(small), 4096, ctypes.byref(st), 16, 16, 16, 16, 0.95, 0.01, 9, None,
                            ctypes.byref(res)) == cdl.CD_EINVAL     # r > r_max
    assert L.cd_step_static(None, 4096, ctypes.byref(st), 16, 16, 16, 16, 0.95, 0.01, 4, None,
                            ctypes.byref(res)) == cdl.CD_EINVAL
    assert st.value == 0
