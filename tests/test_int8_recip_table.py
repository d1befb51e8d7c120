"""The int8 quantiser's single-rounding multipliers (CPU only): the generator re-derives them
by an exhaustive search over every bf16 value under every absmax significand, both signs,
against the correctly rounded code clamp(RNE(fl32(v / gamma))), and the committed header must
hold exactly those ulp adjustments."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_03276_amd", "csrc")


def test_committed_table_matches_exhaustive_derivation(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    exe = str(tmp_path / "gen_int8_recip")
    subprocess.run([gcc, "-O2", "-ffp-contract=off", "-o", exe, os.path.join(CSRC, "gen_int8_recip.c"), "-lm"],
                   check=True, timeout=120)
    r = subprocess.run([exe, "--check", os.path.join(CSRC, "int8_recip_table.h")], stdout=subprocess.PIPE,
                       stderr=subprocess.STDOUT, text=True, timeout=300)
    assert r.returncode == 0, r.stdout
    assert r.stdout.startswith("ok: 128 multipliers")
    # a regenerated header is identical to the committed one
    r = subprocess.run([exe], stdout=subprocess.PIPE, text=True, timeout=300, check=True)
    assert r.stdout == open(os.path.join(CSRC, "int8_recip_table.h")).read()
