import functools
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs through the C-ABI on the device)")
    config.addinivalue_line("markers", "slow: longer CPU test")


@functools.lru_cache(maxsize=None)
def grammar(name: str):
    from inputs import grammars
    return {"arithmetic": grammars.arithmetic, "json": grammars.json_grammar}[name]()


@functools.lru_cache(maxsize=None)
def host(name: str):
    from inputs.native import HostParser
    return HostParser(grammar(name))


@pytest.fixture(scope="session")
def arith():
    return grammar("arithmetic")


@pytest.fixture(scope="session")
def json_g():
    return grammar("json")


@pytest.fixture(scope="session")
def built():
    """name -> (workload, device-bound Classifier, Oracle), built once per
    session and shared by the GPU modules (the larger builds take minutes)."""
    cache = {}

    def get(name):
        if name not in cache:
            from inputs import configs
            from oracle import Oracle
            from paper_2608_03065_amd.psc import Classifier
            wl = configs.get(name)
            clf = Classifier(wl.grammar, wl.vocab).bind("cuda:0")
            cache[name] = (wl, clf, Oracle(wl.grammar, wl.vocab))
        return cache[name]
    return get
