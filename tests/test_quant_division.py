"""The fp16 quantizer computes t = x / s as a product with the row's correctly
rounded reciprocal plus one fma correction (quotient correction with a
correctly rounded reciprocal).  quant_division_check.c proves on the CPU, over
every finite fp16 x and every positive finite fp16 s, that the result equals
the IEEE fp32 quotient the oracle uses; with the correction left out, the same
check fails."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "quant_division_check.c")


def _run(tmp_path, *defs):
    exe = str(tmp_path / "check")
    subprocess.run(["gcc", "-O2", "-mfma", "-fopenmp", "-ffp-contract=off", *defs, "-o", exe, SRC,
                    "-lm"], check=True)
    return subprocess.run([exe], capture_output=True, text=True, timeout=600)


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_division_shortcut_exact_for_all_fp16_pairs(tmp_path):
    r = _run(tmp_path)
    assert r.returncode == 0, r.stdout
    assert "pairs 2015299584 mismatches 0" in r.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_check_catches_missing_correction(tmp_path):
    r = _run(tmp_path, "-DSKIP_CORRECTION")
    assert r.returncode == 1 and "mismatches 0" not in r.stdout
