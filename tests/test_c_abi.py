"""The C ABI from a plain C99 program (no GPU needed: host-only entry
points).  tests/c_abi_check.c includes include/capsule.h, links the built
libcapsule.so and prints its results; they must equal the oracle's."""
import os
import shutil
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB_DIR = os.path.join(ROOT, "paper_2606_20537_amd", "_build")


def test_c_caller_links_and_matches_oracle(orc, tmp_path):
    cc = shutil.which("gcc")
    if cc is None or not os.path.exists(os.path.join(LIB_DIR, "libcapsule.so")):
        pytest.skip("gcc or the built library is missing")
    exe = str(tmp_path / "c_abi_check")
    subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror", "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "c_abi_check.c"), "-o", exe, "-L", LIB_DIR, "-lcapsule",
                    "-Wl,-rpath," + LIB_DIR], check=True)
    out = subprocess.run([exe], check=True, capture_output=True, text=True, timeout=60).stdout
    got = {line.split()[0]: line.split()[1:] for line in out.splitlines()}
    assert got["align"] == [str(orc.align(130, 64)), str(orc.align(64, 64)), "0"]
    want = orc.capsule_bytes([512, 65536, 48], [300, 1, 300], [0, 1, 0], orc.align(200, 64))
    assert got["layout"] == ["0", str(want)]
    assert got["misaligned"] == [str(-5)]          # CAP_E_ALIGN
    assert got["null_set"] == [str(-1)]            # CAP_E_INVAL
    assert " ".join(got["status"]) == "size or layout mismatch"
    ids = np.array([1, -2, 300000, 0, 2147483647], dtype=np.int32)
    assert got["digest"] == [str(orc.digest_tokens(ids))]
