import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


# A copy of the oracle library to test the pins against (tests/test_oracle_mutants.py
# builds copies with planted mistakes and runs the pins in a child process).
_ORACLE_LIB = os.environ.get("ARENA_ORACLE_LIB")
if _ORACLE_LIB:
    from oracle import oracle as _oracle_mod
    _oracle_mod._LIB = _ORACLE_LIB
    _oracle_mod._lib = None
_PROXY_ORACLE_LIB = os.environ.get("ARENA_PROXY_ORACLE_LIB")
if _PROXY_ORACLE_LIB:
    from oracle import proxy as _proxy_mod
    _proxy_mod._LIB = _PROXY_ORACLE_LIB
    _proxy_mod._lib = None


_SCHED_ORACLE_SRC = os.environ.get("ARENA_SCHED_ORACLE_SRC")
if _SCHED_ORACLE_SRC:
    import importlib.util
    import oracle as _oracle_pkg
    _spec = importlib.util.spec_from_file_location("oracle.scheduler_oracle", _SCHED_ORACLE_SRC)
    _sched_mod = importlib.util.module_from_spec(_spec)
    _spec.loader.exec_module(_sched_mod)
    sys.modules["oracle.scheduler_oracle"] = _sched_mod
    _oracle_pkg.scheduler_oracle = _sched_mod


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs the HIP library)")


@pytest.fixture(scope="session")
def oracle():
    from oracle import oracle as o
    o.load()
    return o
