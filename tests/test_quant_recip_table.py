"""The quantiser's one-multiply multipliers (CPU only): the generator re-derives them by an
exhaustive search over every bf16 value under every absmax significand, both signs, for
every code format, against the correctly rounded code (clamp(RNE(fl32(v / gamma))) or the
E4M3 code of fl32(v / gamma)), and the committed header must hold exactly those masks."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_03276_amd", "csrc")
HEADER = os.path.join(CSRC, "quant_recip_table.h")


@pytest.fixture(scope="module")
def generator(tmp_path_factory):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    exe = str(tmp_path_factory.mktemp("gen") / "gen_quant_recip")
    subprocess.run([gcc, "-O2", "-ffp-contract=off", "-o", exe, os.path.join(CSRC, "gen_quant_recip.c"), "-lm"],
                   check=True, timeout=120)
    return exe


def test_committed_table_matches_exhaustive_derivation(generator):
    r = subprocess.run([generator, "--check", HEADER], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
                       timeout=600)
    assert r.returncode == 0, r.stdout
    assert r.stdout.rstrip().endswith("ok")
    # int8 has a multiplier for every significand (its kernel instance has no corrected path)
    assert "qmax 127: 51 up, 2 down, 0 without a multiplier" in r.stdout


def test_regenerated_header_is_identical(generator):
    r = subprocess.run([generator], stdout=subprocess.PIPE, text=True, timeout=600, check=True)
    assert r.stdout == open(HEADER).read()
