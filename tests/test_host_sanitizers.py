"""The engine's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

engine.cpp (admission, paged blocks, chunked prefill, step plans and their
model-stream shares, retire/collect, the inspection hooks and every
documented error return) is compiled with both sanitizers on its host side
and linked, with the normally built kernel objects, into a small C program
that drives MOA_FLAG_PLAN_ONLY engines through the C ABI
(tests/sanitize/plan_driver.c). A plan-only engine makes no HIP call, so this
runs without a GPU. The grouped-GEMM planner, which only runs when a step is
enqueued on a GPU, is checked on its own by tests/sanitize/gemm_plan_check.cpp
(it includes engine.cpp): random ragged row mixes on the 8B, 1B and a small
model's projections, every plan replayed through the kernels' item decode for
exact coverage, launchability and partial-buffer bounds, under the same two
sanitizers. tests/sanitize/step_plan_check.cpp checks every step's attention,
combine, prefill-block and LM-row lists of plan-only engines against the
request bookkeeping (keys covered once per row, partial slots, block-list
offsets, tokens read only once written, share order). The oracle is Python
(numpy) and has no native code to sanitize.
"""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_03014_amd", "csrc")
BUILD = os.path.join(CSRC, "_build")
LLVM = "/opt/rocm/llvm/bin"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN = ["address", "undefined"]


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, " ".join(cmd) + "\n" + r.stdout[-4000:] + r.stderr[-4000:]
    return r


def _kernel_objs():
    if not (os.path.exists(HIPCC) and os.path.exists(os.path.join(LLVM, "clang"))):
        pytest.skip("ROCm toolchain not found")
    from paper_2606_03014_amd.build import build
    objs = [os.path.join(BUILD, s + ".o") for s in ("kernels.hip", "peaks.hip")]
    if not all(os.path.exists(o) for o in objs):
        build()
    return objs


def _hipcc_san(src, obj):
    """Compile one host translation unit with both sanitizers on its host side."""
    from paper_2606_03014_amd.build import FLAGS
    host_san = []
    for s in SAN:          # sanitizers on the host side only
        host_san += ["-Xarch_host", f"-fsanitize={s}"]
    flags = [f for f in FLAGS if f != "-O3"]
    _run([HIPCC] + flags + ["-O1", "-g", "-Xarch_host", "-fno-omit-frame-pointer",
                            "-Xarch_host", "-fno-sanitize-recover=all"] + host_san + ["-c", src, "-o", obj])


def _san_env():
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = "detect_leaks=1:abort_on_error=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    supp = os.path.join(ROOT, "tests", "sanitize", "lsan.supp")
    env["LSAN_OPTIONS"] = f"suppressions={supp}"
    return env


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    objs = _kernel_objs()
    out = tmp_path_factory.mktemp("san")
    eng_o = str(out / "engine_san.o")
    _hipcc_san(os.path.join(CSRC, "engine.cpp"), eng_o)
    drv_o = str(out / "plan_driver.o")
    san = ",".join(SAN)
    _run([os.path.join(LLVM, "clang"), "-std=c11", "-O1", "-g", "-Wall", f"-fsanitize={san}",
          "-fno-sanitize-recover=all", "-I", os.path.join(ROOT, "include"),
          "-c", os.path.join(ROOT, "tests", "sanitize", "plan_driver.c"), "-o", drv_o])
    exe = str(out / "plan_driver")
    _run([os.path.join(LLVM, "clang++"), f"-fsanitize={san}", drv_o, eng_o] + objs +
         ["-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-o", exe])
    return exe


def test_plan_only_engine_is_clean_under_asan_and_ubsan(driver):
    r = subprocess.run([driver], capture_output=True, text=True, env=_san_env(), timeout=300)
    log = r.stdout + r.stderr
    assert r.returncode == 0, log[-6000:]
    assert "ERROR: AddressSanitizer" not in log and "runtime error" not in log, log[-6000:]
    assert "plan_driver: ok" in r.stdout


def _check_program(tmp_path_factory, name):
    """Build tests/sanitize/<name>.cpp (it includes engine.cpp) with both sanitizers."""
    objs = _kernel_objs()
    out = tmp_path_factory.mktemp(name)
    obj = str(out / (name + ".o"))
    _hipcc_san(os.path.join(ROOT, "tests", "sanitize", name + ".cpp"), obj)
    san = ",".join(SAN)
    exe = str(out / name)
    _run([os.path.join(LLVM, "clang++"), f"-fsanitize={san}", obj] + objs +
         ["-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-o", exe])
    return exe


def _run_check(exe, arg, name):
    r = subprocess.run([exe, arg], capture_output=True, text=True, env=_san_env(), timeout=300)
    log = r.stdout + r.stderr
    assert r.returncode == 0, log[-6000:]
    assert "ERROR: AddressSanitizer" not in log and "runtime error" not in log, log[-6000:]
    assert f"{name}: ok" in r.stdout
    return r.stdout


@pytest.fixture(scope="module")
def plan_check(tmp_path_factory):
    return _check_program(tmp_path_factory, "gemm_plan_check")


@pytest.fixture(scope="module")
def step_check(tmp_path_factory):
    return _check_program(tmp_path_factory, "step_plan_check")


def test_gemm_plans_cover_every_output_once_and_launch(plan_check):
    # 120 random steps per (dtype, model shape): about 3,500 plans, every
    # share launch replayed item by item
    _run_check(plan_check, "120", "gemm_plan_check")


def test_step_work_lists_cover_every_key_once_in_causal_order(step_check):
    # four plan-only engines (f32; bf16 at head_dim 64 and 128 on model
    # streams; bf16 on one stream), 300 requests each with histories up to
    # 33k positions: every step's attention, combine, prefill and LM lists
    out = _run_check(step_check, "300", "step_plan_check")
    assert out.count("split rows") == 4
