"""Exhaustive CPU proof of the activation quantize's reciprocal path.

The GPU quantize (stand-alone, fused into the small-M GEMM, and in the
no-allocation and producer paths) forms each int8 code from the token
scale's reciprocal with one Markstein correction and a 1.5 * 2^23 rounding
add instead of an IEEE division per element.  tests/quant_exhaustive.c
replays exactly those binary32 operations for every pair of bf16 values (x,
a) with a >= 2^-96 and |x| <= a (about 1.05e9 pairs) and compares the codes
with round-half-even of the IEEE quotient x / fl(a / 127), the definition the
oracle implements (Sec. 3.4's 8-bit activation cast; the rounding is this
library's reading).  Rows with a < 2^-96 take an IEEE division in the
kernels and need no proof.

Runtime: ~7.5 s on 8 threads of the build container's Xeon (gcc -O2 with
hardware FMA); without hardware FMA glibc's fmaf is exact but slower.
"""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "quant_exhaustive.c")


def _has_fma() -> bool:
    try:
        with open("/proc/cpuinfo") as f:
            return any(" fma " in line + " " for line in f if line.startswith("flags"))
    except OSError:
        return False


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    exe = str(tmp_path_factory.mktemp("qproof") / "quant_exhaustive")
    flags = ["-O2", "-ffp-contract=off", "-pthread"] + (["-mfma"] if _has_fma() else [])
    subprocess.run(["gcc", *flags, "-o", exe, SRC, "-lm"], check=True)
    return exe


def _run(exe, *args):
    r = subprocess.run([exe, *map(str, args)], capture_output=True, text=True, timeout=600)
    fields = dict(kv.split("=") for kv in r.stdout.split()[:2])
    return r.returncode, int(fields["pairs"]), int(fields["mismatches"]), r.stdout


def test_reciprocal_path_is_correctly_rounded_for_every_bf16_pair(checker):
    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    rc, pairs, bad, out = _run(checker, threads)
    assert pairs == 1_049_624_576, out  # every (x, a) with 2^-96 <= a <= max bf16, |x| <= a
    assert bad == 0 and rc == 0, out


def test_checker_rejects_the_uncorrected_product(checker):
    # the same check of fl(x * inv) without the correction finds mismatches
    # (a in [0.5, 1)): the exhaustive run above can fail
    rc, pairs, bad, out = _run(checker, 4, 1, "3F00", "3F7F")
    assert pairs > 0 and bad > 0 and rc == 1, out
