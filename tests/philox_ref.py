"""Philox4x32-10 blocks from rocRAND's engine, for pinning the oracle's
generator to an implementation that is not its own (test infrastructure).

rocRAND's `philox4x32_10_engine` (its header names Random123, the SC'11
authors' library, as the source of its round) is compiled once per session
from `tests/rocrand_philox_ref.cpp` with hipcc as a plain host program; its
ten-round block function is called on given counters and keys.  Where hipcc
or the rocRAND header is missing, `available()` is False and the tests that
need it are skipped.
"""
import atexit
import functools
import os
import shutil
import subprocess
import tempfile

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "rocrand_philox_ref.cpp")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")
HEADER = os.path.join(ROCM, "include", "rocrand", "rocrand_philox4x32_10.h")


def available():
    return os.path.exists(HIPCC) and os.path.exists(HEADER)


@functools.lru_cache(maxsize=1)
def _binary():
    tmp = tempfile.mkdtemp(prefix="philox_ref_")
    atexit.register(shutil.rmtree, tmp, True)
    out = os.path.join(tmp, "philox_ref")
    subprocess.run([HIPCC, "-O1", "-std=c++17", f"-I{os.path.join(ROCM, 'include')}", SRC, "-o", out],
                   check=True, capture_output=True, timeout=300)
    return out


def blocks(counters, keys):
    """counters [n, 4] and keys [n, 2] (uint32) -> rocRAND's output words [n, 4]."""
    counters = np.asarray(counters, dtype=np.uint64).reshape(-1, 4)
    keys = np.asarray(keys, dtype=np.uint64).reshape(-1, 2)
    lines = "\n".join(" ".join(str(int(v)) for v in (*c, *k)) for c, k in zip(counters, keys))
    res = subprocess.run([_binary()], input=lines + "\n", capture_output=True, text=True, check=True, timeout=120)
    return np.array([[int(t) for t in ln.split()] for ln in res.stdout.strip().splitlines()], dtype=np.uint64)
