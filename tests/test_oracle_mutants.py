"""The oracle's pins catch plausible mistakes: each mistake of
tests/oracle_mutants.py is planted in the oracle (CPU only) and the pin
tests of the op definitions, or of the selection model, must then fail at
least once."""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

from tests.oracle_mutants import MUTANTS, SELECTION_MUTANTS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OP_PINS = ["tests/test_oracle_ops.py", "tests/test_oracle_rope_ext.py"]
SELECTION_PINS = ["tests/test_oracle_selection.py", "tests/test_oracle_tuning.py",
                  "tests/test_oracle_generic.py"]
CASES = [(n, OP_PINS) for n in sorted(MUTANTS)] + [(n, SELECTION_PINS)
                                                   for n in sorted(SELECTION_MUTANTS)]


def _run(case):
    name, pins = case
    env = dict(os.environ, PYTHONPATH=ROOT)
    env.pop("TRI_ORACLE_MUTANT", None)
    if name:
        env["TRI_ORACLE_MUTANT"] = name
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        "-p", "tests.oracle_mutants", *pins],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return name, r.returncode, r.stdout[-1500:]


@pytest.fixture(scope="module")
def outcomes():
    with ThreadPoolExecutor(max_workers=4) as ex:
        return {n: (rc, out) for n, rc, out in ex.map(_run, CASES)}


@pytest.mark.parametrize("name", [n for n, _ in CASES])
def test_pins_catch_the_mistake(outcomes, name):
    rc, out = outcomes[name]
    assert rc == 1, f"{name}: the pins did not fail (exit {rc})\n{out}"


@pytest.mark.parametrize("pins", [OP_PINS, SELECTION_PINS], ids=["ops", "selection"])
def test_pins_pass_without_a_mistake(pins):
    _, rc, out = _run((None, pins))
    assert rc == 0, out
