"""Build the CPU oracle (test infrastructure) as a shared library with gcc.

Plain C, -O2, no fast-math, single-threaded: floating point is evaluated in
the order the source states it.  Usage: ``python oracle/build.py`` or
``oracle.build.build()``.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SOURCES = ["linattn_oracle.c", "capsule_oracle.c", "fp8_oracle.c", "gdn_oracle.c"]
LIB_PATH = os.path.join(HERE, "_build", "liborc.so")


def build(out_path: str = LIB_PATH, src_dir: str = HERE, extra_flags=()) -> str:
    """Compile the oracle sources in ``src_dir`` into ``out_path``; return the path."""
    os.makedirs(os.path.dirname(out_path), exist_ok=True)
    srcs = [os.path.join(src_dir, s) for s in SOURCES]
    tmp = out_path + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fno-fast-math",
           "-ffp-contract=off", *extra_flags, "-o", tmp, *srcs, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out_path)
    return out_path


if __name__ == "__main__":
    print(build(*(sys.argv[1:2] or [])))
