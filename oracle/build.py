"""Build the fp64 CPU oracle (test infrastructure only).

``build()`` compiles ``ws_oracle.c`` with gcc -O2 (no fast-math) into
``libwsoracle.so`` next to this file.  ``build_variant(defines, out)`` builds
the same source with extra preprocessor definitions; the test suite uses it
to build deliberately broken variants and show that its pins reject them.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "ws_oracle.c")
LIB = os.path.join(HERE, "libwsoracle.so")


def build_variant(defines, out):
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread",
           "-Wall", "-Wextra", "-Wno-unused-parameter"]
    for key, val in (defines or {}).items():
        cmd.append(f"-D{key}={val}")
    cmd += [SRC, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def build():
    return build_variant({}, LIB)


if __name__ == "__main__":
    print(build())
