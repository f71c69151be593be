"""Compile the gfx950 library libwsattn.so in-tree with hipcc.

Usage: python -m paper_2606_25041_amd.build   (or call build()).
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libwsattn.so")
# device sources (built with KERNEL_FLAGS) and the host-only C ABI
DEVICE_SOURCES = [os.path.join(CSRC, "ws_kernels.hip"), os.path.join(CSRC, "ws_bwd.hip"),
                  os.path.join(CSRC, "ws_device.hip")]
HOST_SOURCES = [os.path.join(CSRC, "ws_api.cpp")]
SOURCES = DEVICE_SOURCES + HOST_SOURCES
HEADERS = [os.path.join(CSRC, "ws_kernels.h"), os.path.join(CSRC, "ws_device_util.h"),
           os.path.join(os.path.dirname(HERE), "include", "ws_attn.h")]
# the device code whose hash tags measured counter summaries: the forward
# kernels (attention, merge, append) and, separately, the gradient kernels
KERNEL_SOURCES = [os.path.join(CSRC, "ws_kernels.hip"), os.path.join(CSRC, "ws_kernels.h"),
                  os.path.join(CSRC, "ws_device_util.h")]
BWD_KERNEL_SOURCES = [os.path.join(CSRC, "ws_bwd.hip"), os.path.join(CSRC, "ws_kernels.h"),
                      os.path.join(CSRC, "ws_device_util.h")]
ARCH = "gfx950"


def hipcc():
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


KERNEL_FLAGS = [
    # packed fp32 VALU ops stay off in every kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA results in VGPRs: the softmax reads every score with VALU
    # instructions, which cannot address accumulation registers
    "-mllvm", "-amdgpu-mfma-vgpr-form=1",
]


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    msgs = [ln for ln in (res.stdout + res.stderr).splitlines()
            if "packed-fp32-ops" not in ln and "--hip-link" not in ln]
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + " ".join(cmd) + "\n" + "\n".join(msgs))
    return msgs


def build(verbose=False):
    """Kernels (with their device code-generation flags) and the host-only
    C ABI are compiled separately, then linked into one shared library."""
    common = [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
              "-Wall", "-Wno-unused-function"]
    objs, msgs = [], []
    for src in SOURCES:
        obj = LIB + "." + os.path.splitext(os.path.basename(src))[0] + ".o"
        flags = KERNEL_FLAGS if src in DEVICE_SOURCES else []
        msgs += _run(common + flags + ["-c", src, "-o", obj])
        objs.append(obj)
    msgs += _run([hipcc(), f"--offload-arch={ARCH}", "-shared"] + objs + ["-o", LIB + ".tmp"])
    for f in objs:
        os.remove(f)
    if verbose and msgs:
        print("\n".join(msgs))
    os.replace(LIB + ".tmp", LIB)
    return LIB


CEIL_SRC = os.path.join(CSRC, "ws_ceilings.hip")
CEIL_LIB = os.path.join(HERE, "libwsceil.so")


def build_ceilings(verbose=False):
    """The ceiling microbenchmarks (MFMA loop, streaming read) that the
    benchmark runs beside the attention kernels, as libwsceil.so."""
    msgs = _run([hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared", "-Wall"]
                + KERNEL_FLAGS + [CEIL_SRC, "-o", CEIL_LIB + ".tmp"])
    if verbose and msgs:
        print("\n".join(msgs))
    os.replace(CEIL_LIB + ".tmp", CEIL_LIB)
    return CEIL_LIB


def is_stale():
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(p) > t for p in SOURCES + HEADERS)


if __name__ == "__main__":
    print(build(verbose=True))
    print(build_ceilings(verbose=True))
