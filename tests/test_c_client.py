"""The C ABI from a plain C program: include/ws_attn.h compiles with a C
compiler (no HIP or torch headers) and the program links libwsattn.so and
gets the documented answers to version, status and validation queries (no
device is touched: every attention call fails validation)."""
import os
import shutil
import subprocess

import pytest
import torch

from paper_2606_25041_amd import build as wsbuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

if torch.cuda.device_count() > 0:
    pytest.skip("CPU-only module (the C program's calls must fail validation)", allow_module_level=True)


def test_c_client_compiles_links_and_runs(tmp_path):
    if not os.path.exists(wsbuild.LIB):
        wsbuild.build()
    gcc = shutil.which("gcc")
    assert gcc, "gcc is needed for this test"
    exe = os.path.join(tmp_path, "abi_smoke")
    libdir = os.path.dirname(wsbuild.LIB)
    subprocess.run([gcc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "c", "abi_smoke.c"), "-o", exe,
                    os.path.join(libdir, "libwsattn.so"), f"-Wl,-rpath,{libdir}"], check=True)
    res = subprocess.run([exe], capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    assert "c abi ok" in res.stdout
