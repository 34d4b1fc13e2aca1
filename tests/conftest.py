import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:
    sys.path.insert(0, HERE)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


import pytest


@pytest.fixture
def library():
    """Oracle build under test: None means oracle/liboracle.so."""
    return None


@pytest.fixture
def pin_variants(monkeypatch):
    """pin_variants(ev_reg=1, ...): every library Graph created afterwards in
    the test is pinned to those kernel variants (Graph.pin_variant, the
    testing entry point sim_testing_replan), in the order given."""
    def pin(**pins):
        import paper_2002_06790_amd as m
        orig = m.Graph.__init__

        def init(self, *a, **k):
            orig(self, *a, **k)
            for what, value in pins.items():
                self.pin_variant(what, int(value))

        monkeypatch.setattr(m.Graph, "__init__", init)
    return pin
