"""Exhaustive CPU checks of the fp32 identities behind the int8 epilogues' arithmetic.

The row-block and column-block int8 epilogues compute the block scale absmax / 127 as a
product with RN(1/127) plus one fma correction, and turn a scaled moment into its code by
adding 1.5 * 2^23 (the sum's rounding is the round-half-even of App. B's quantiser).
Both are exact only if they agree with IEEE division and rintf on every input they can
meet; kernel_arith.c checks every such input (no GPU involved).
"""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_div127_and_code_rounding_exhaustive(tmp_path):
    exe = str(tmp_path / "kernel_arith")
    subprocess.run(["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-o", exe,
                    os.path.join(HERE, "kernel_arith.c"), "-lm"], check=True)
    env = dict(os.environ)
    env.setdefault("OMP_NUM_THREADS", str(min(8, os.cpu_count() or 1)))
    out = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert out.returncode == 0, out.stdout + out.stderr
    assert out.stdout.strip() == "div127 0 code 0"
