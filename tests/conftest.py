import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def _load_oracle_mutant():
    """Test-only: replace the oracle module by a mutated copy (see test_oracle_mutants)."""
    spec = os.environ.get("ADAPLD_ORACLE_MUTANT")
    if not spec:
        return
    import importlib
    import json
    old, new = json.loads(spec)
    import oracle.adapld_oracle as mod
    src = open(mod.__file__).read()
    assert src.count(old) >= 1, old
    src = src.replace(old, new, 1)
    code = compile(src, mod.__file__, "exec")
    exec(code, mod.__dict__)
    import oracle
    importlib.reload(oracle)


_load_oracle_mutant()
