"""The quantiser's arithmetic on the CPU (no GPU).

The generator re-derives the one-multiply multipliers by an exhaustive search over every
bf16 value under every absmax significand, both signs, for every code format, against the
correctly rounded code (clamp(RNE(fl32(v / gamma))) or the E4M3 code of fl32(v / gamma)),
and the committed header must hold exactly those masks.  Its replay re-runs the exact fp32
arithmetic of every path a row can take in the kernels (one-multiply, corrected quotient,
rescaled row, divided row) over every (bf16 absmax, bf16 value <= absmax) pair, both signs,
for every format (Eq. 2), and no code may differ."""
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
    # -march=native: hardware fma and rounding (the same IEEE results as libm's, much faster);
    # no contraction, no fast-math
    subprocess.run([gcc, "-O2", "-march=native", "-fopenmp", "-ffp-contract=off", "-o", exe,
                    os.path.join(CSRC, "gen_quant_recip.c"), "-lm"], check=True, timeout=120)
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


def test_replay_of_every_quantiser_path(generator):
    """About 2.8e10 codes: every path the kernels can take for a row, for every absmax exponent
    and significand and every bf16 value under it, both signs, for all 8 formats."""
    r = subprocess.run([generator, "--replay"], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
                       timeout=1200)
    assert r.returncode == 0, r.stdout
    lines = r.stdout.strip().splitlines()
    assert lines[-1] == "ok"
    paths = [l for l in lines if "compared" in l]
    assert len(paths) == 8 * 5
    for l in paths:
        assert l.endswith(" 0 differ"), l
        assert int(l.split(": ")[1].split()[0]) > 0, l  # every path ran for every format


def test_replay_catches_a_dropped_correction(tmp_path):
    """The replay has teeth: with the correction step of the quotient planted out (q = v * y
    only), it reports differing codes for the corrected path (one format, int4)."""
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    exe = str(tmp_path / "gen_planted")
    subprocess.run([gcc, "-O2", "-march=native", "-fopenmp", "-ffp-contract=off", "-DREPLAY_PLANT_UNCORRECTED",
                    "-o", exe, os.path.join(CSRC, "gen_quant_recip.c"), "-lm"], check=True, timeout=120)
    r = subprocess.run([exe, "--replay", "7"], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
                       timeout=600)
    assert r.returncode == 1
    corr = [l for l in r.stdout.splitlines() if "corrected quotient" in l]
    assert len(corr) == 1 and not corr[0].endswith(" 0 differ"), r.stdout
