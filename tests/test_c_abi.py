"""The C ABI from plain C: tests/c_abi_host.c is compiled as C99 with gcc
against include/fiona.h and linked to the built library, then run (no GPU:
it exercises the entry points that need none, through the header's own
declarations rather than the Python binding's)."""
import os
import shutil
import subprocess

import pytest

import synth
import paper_2609_35352_amd as fiona

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM_INCLUDE = "/opt/rocm/include"


def test_header_compiles_as_c_and_host_entry_points_run(tmp_path):
    if shutil.which("gcc") is None or not os.path.isdir(ROCM_INCLUDE):
        pytest.skip("gcc or the ROCm headers are missing")
    if not os.path.exists(fiona.LIB_PATH):
        pytest.fail("libfiona.so is not built (run __graft_entry__.build())")
    exe = str(tmp_path / "c_abi_host")
    lib_dir = os.path.dirname(fiona.LIB_PATH)
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__", "-I" + os.path.join(ROOT, "include"),
           "-I" + ROCM_INCLUDE, os.path.join(ROOT, "tests", "c_abi_host.c"), "-L" + lib_dir, "-lfiona",
           "-Wl,-rpath," + lib_dir, "-o", exe]
    cc = subprocess.run(cmd, capture_output=True, text=True)
    assert cc.returncode == 0, cc.stderr
    # no diagnostic in the library's own header (the ROCm headers' are theirs)
    assert "fiona.h" not in cc.stderr, cc.stderr
    q = [str(v) for v in synth.ntt_primes(256, 4)]
    run = subprocess.run([exe] + q, capture_output=True, text=True, timeout=120)
    assert run.returncode == 0 and run.stdout.strip().endswith("ok"), run.stdout + run.stderr


@pytest.mark.gpu
@pytest.mark.parametrize("seed", [1, 2, 3])
def test_hot_path_from_c_matches_oracle(tmp_path, seed):
    """tests/c_abi_gpu.c: a C program allocates with hipMalloc, runs
    fiona_hybrid_linear and fiona_hybrid_linear_static on its own stream and
    compares both with oracle_weighted_sum word for word."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import oracle
    if shutil.which("gcc") is None:
        pytest.skip("gcc is missing")
    oracle.lib()   # built if missing
    exe = str(tmp_path / "c_abi_gpu")
    lib_dir, oracle_dir = os.path.dirname(fiona.LIB_PATH), os.path.join(ROOT, "oracle")
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__", "-I" + os.path.join(ROOT, "include"),
           "-I" + ROCM_INCLUDE, os.path.join(ROOT, "tests", "c_abi_gpu.c"), "-L" + lib_dir, "-lfiona",
           "-L" + oracle_dir, "-loracle", "-L/opt/rocm/lib", "-lamdhip64",
           "-Wl,-rpath," + lib_dir + ":" + oracle_dir + ":/opt/rocm/lib", "-o", exe]
    cc = subprocess.run(cmd, capture_output=True, text=True)
    assert cc.returncode == 0, cc.stderr
    q = [str(v) for v in synth.ntt_primes(512, 3)]
    print("[c-abi] seed %d" % seed, flush=True)
    run = subprocess.run([exe] + q + [str(seed)], capture_output=True, text=True, timeout=120)
    print(run.stdout.strip(), flush=True)
    assert run.returncode == 0 and run.stdout.startswith("ok"), run.stdout + run.stderr
