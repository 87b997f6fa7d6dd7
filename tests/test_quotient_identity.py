"""The quantize kernel replaces the per-weight IEEE division w / s by a
reciprocal (one IEEE division per group) and two fused multiply-adds.  This
checks, on the CPU and exhaustively over all binary16 operand pairs, that the
replacement yields the IEEE binary32 quotient exactly, so the codes stay
those of Eq. 1 with true division."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))


def test_reciprocal_fma_quotient_is_ieee(tmp_path):
    exe = str(tmp_path / "fp16_quotient_check")
    subprocess.run(["gcc", "-O2", "-std=c11", "-fno-fast-math", "-ffp-contract=off", "-mfma", "-fopenmp",
                    "-o", exe, os.path.join(HERE, "native", "fp16_quotient_check.c"), "-lm"], check=True)
    out = subprocess.run([exe], check=True, capture_output=True, text=True).stdout.split()
    pairs, bad = int(out[0]), int(out[1])
    assert pairs == 31743 * 63488  # positive finite scales x finite weights
    assert bad == 0
