"""The oracle's pins reject planted mistakes.

Every entry of ``oracle_mutants.MUTANTS`` is applied to a copy of the oracle
source, compiled with the oracle's own flags into a temporary library, and the
pin tests (``tests/test_oracle_*.py``) are run against that library through
``LTO_LIBRARY``.  A mutant counts as rejected when some pin fails (pytest exit
status 1); a crash or a collection error does not count.  The oracle in the
repository is never modified.
"""
import concurrent.futures as cf
import os
import re
import subprocess
import sys

import pytest

from oracle import build as oracle_build
from oracle_mutants import MUTANTS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
# cheap files first: pytest -x stops at the first failing pin
PIN_FILES = ["tests/test_oracle_bf16.py", "tests/test_oracle_clip.py",
             "tests/test_oracle_quantizer.py", "tests/test_oracle_adamw.py",
             "tests/test_oracle_dynamic_map.py", "tests/test_oracle_sqnorm.py"]


def _judge(mutant, src, workdir):
    name, _, old, new = mutant
    if src.count(old) != 1:
        return {"status": "stale", "count": src.count(old)}
    path = os.path.join(workdir, name + ".c")
    with open(path, "w") as f:
        f.write(src.replace(old, new))
    lib = oracle_build.build(src=path, out=os.path.join(workdir, "lib" + name + ".so"))
    env = dict(os.environ, LTO_LIBRARY=lib)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-rf", "-p", "no:cacheprovider",
                        "-m", "not gpu", *PIN_FILES], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=900)
    return {"status": r.returncode, "failed": re.findall(r"^FAILED (\S+)", r.stdout, re.M),
            "tail": r.stdout[-2000:] + r.stderr[-2000:]}


@pytest.fixture(scope="module")
def verdicts(tmp_path_factory):
    with open(oracle_build.SOURCE) as f:
        src = f.read()
    workdir = str(tmp_path_factory.mktemp("oracle_mutants"))
    workers = max(1, min(8, len(os.sched_getaffinity(0))))
    with cf.ThreadPoolExecutor(max_workers=workers) as ex:
        futs = {m[0]: ex.submit(_judge, m, src, workdir) for m in MUTANTS}
        return {name: fut.result() for name, fut in futs.items()}


def test_catalogue_names_are_unique():
    names = [m[0] for m in MUTANTS]
    assert len(names) == len(set(names))


@pytest.mark.parametrize("name", [m[0] for m in MUTANTS])
def test_pins_reject_planted_mistake(name, verdicts):
    v = verdicts[name]
    assert v["status"] != "stale", f"{name}: its text occurs {v['count']} times in the oracle"
    assert v["status"] == 1 and v["failed"], (
        f"{name} was not rejected by any pin (pytest status {v['status']}):\n{v['tail']}")
