"""Every plausible mistake planted into the oracle fails at least one pin.

For each entry of ``oracle_mistakes.MISTAKES`` a child pytest runs the
oracle's pin tests (``tests/test_oracle_*.py``) with that one mistake
planted (AVITS_PLANT_MISTAKE, applied by ``conftest.py`` before collection)
and must fail; a clean child run must pass, so a failure is the mistake's.
"""
import concurrent.futures as cf
import glob
import os
import subprocess
import sys

import pytest

import oracle_mistakes

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
PINS = sorted(glob.glob(os.path.join(HERE, "test_oracle_*.py")))


def _child(mistake):
    env = dict(os.environ, OMP_NUM_THREADS="1", OPENBLAS_NUM_THREADS="1", MKL_NUM_THREADS="1")
    env.pop("AVITS_PLANT_MISTAKE", None)
    if mistake:
        env["AVITS_PLANT_MISTAKE"] = mistake
    cmd = [sys.executable, "-m", "pytest", "-x", "-q", "-m", "not gpu", "-p", "no:cacheprovider",
           "-p", "no:xdist", "-p", "no:randomly", *PINS]
    r = subprocess.run(cmd, cwd=ROOT, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
                       timeout=600)
    return mistake, r.returncode, r.stdout[-3000:]


@pytest.fixture(scope="module")
def outcomes():
    names = [None] + sorted(oracle_mistakes.MISTAKES)
    with cf.ThreadPoolExecutor(min(8, os.cpu_count() or 2)) as ex:
        return {m: (rc, out) for m, rc, out in ex.map(_child, names)}


def test_clean_pins_pass(outcomes):
    rc, out = outcomes[None]
    assert rc == 0, out


@pytest.mark.parametrize("mistake", sorted(oracle_mistakes.MISTAKES))
def test_planted_mistake_fails_a_pin(outcomes, mistake):
    rc, out = outcomes[mistake]
    # 1: tests failed (not an error in planting, collection or usage).
    assert "planted mistake" not in out or rc == 1, out
    assert rc == 1, f"no pin caught {mistake}:\n{out}"
