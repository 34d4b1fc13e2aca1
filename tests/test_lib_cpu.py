"""Host-side checks of the C ABI library that need no GPU."""
import ctypes
import glob
import math
import os
import re

import numpy as np
import pytest

import paper_2002_06790_amd as mlsim

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mlsim.h")


def declared_functions():
    """Every function declared by the headers under include/."""
    names = set()
    for h in sorted(glob.glob(os.path.join(ROOT, "include", "*.h"))):
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(sim_\w+)\s*\(", text))
    return sorted(names)


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(mlsim.LIB_PATH):
        mlsim.build()
    return mlsim.lib()


def test_exports_every_declared_symbol(L):
    names = declared_functions()
    assert set(names) == set(mlsim.EXPORTS)
    for name in names:
        assert hasattr(L, name), name


def test_strerror(L):
    for code in range(0, -7, -1):
        assert L.sim_strerror(code)
    assert L.sim_strerror(-99) == b"unknown error"


def create(L, n, R, ptr, idx, res, prio=None):
    h = ctypes.c_void_p()
    a = [np.ascontiguousarray(x, dt) if x is not None else None
         for x, dt in ((ptr, np.int64), (idx, np.int32), (res, np.int32), (prio, np.int32))]
    rc = L.sim_graph_create(n, R, *[x.ctypes.data if x is not None else None for x in a], ctypes.byref(h))
    return rc, h


def test_graph_errors_without_gpu(L):
    """Malformed graphs are rejected on the host before any HIP call."""
    res = [0, 0]
    assert create(L, 2, 1, [0, 1, 2], [1, 0], res)[0] == mlsim.SIM_E_CYCLE
    assert create(L, 2, 1, [0, 1, 1], [0], res)[0] == mlsim.SIM_E_CYCLE  # self loop
    assert create(L, 2, 1, [0, 1, 1], [2], res)[0] == mlsim.SIM_E_RANGE
    assert create(L, 2, 1, [0, 1, 1], [1], [0, 1])[0] == mlsim.SIM_E_RANGE
    assert create(L, 2, 1, [0, 1, 0], [1], res)[0] == mlsim.SIM_E_INVAL
    assert create(L, 2, 1, [1, 1, 1], [1], res)[0] == mlsim.SIM_E_INVAL
    assert create(L, 2, 0, [0, 1, 1], [1], res)[0] == mlsim.SIM_E_INVAL
    assert create(L, -1, 1, [0], [], [])[0] == mlsim.SIM_E_INVAL
    assert create(L, 2, 5000, [0, 1, 1], [1], res)[0] == mlsim.SIM_E_LIMIT
    rc = L.sim_graph_create(1, 1, None, None, None, None, ctypes.byref(ctypes.c_void_p()))
    assert rc == mlsim.SIM_E_INVAL
    assert L.sim_graph_create(0, 1, None, None, None, None, None) == mlsim.SIM_E_INVAL


def test_run_argument_errors_without_gpu(L):
    assert L.sim_run_batch(None, 1, None, 1, None, 0, None, None, 0, None, 0, None) == mlsim.SIM_E_INVAL
    assert L.sim_critical_path(None, 1, None, 1, None, -1, None, 0, None, None) == mlsim.SIM_E_INVAL


def test_generate_argument_errors_without_gpu(L):
    """Generator parameters are checked on the host before any HIP call."""
    base = ctypes.c_void_p(16)  # never dereferenced: every call below fails its checks first
    out = ctypes.c_void_p(16)
    ok = dict(n_knobs=1, knob_block=1, noise=0, seed=0, scen0=0)

    def gen(n_ops=4, n_scen=8, ld=8, **kw):
        a = dict(ok)
        a.update(kw)
        return L.sim_generate(n_ops, n_scen, base, a["n_knobs"], a["knob_block"], a["noise"], a["seed"],
                              a["scen0"], out, ld, None)

    assert gen(n_knobs=0) == mlsim.SIM_E_INVAL
    assert gen(knob_block=0) == mlsim.SIM_E_INVAL
    assert gen(noise=mlsim.SIM_GEN_NOISE_MAX) == mlsim.SIM_E_INVAL
    assert gen(scen0=-1) == mlsim.SIM_E_INVAL
    assert gen(scen0=2**63 - 4) == mlsim.SIM_E_INVAL  # scen0 + n_scen beyond int64
    assert gen(ld=7) == mlsim.SIM_E_INVAL
    assert gen(n_ops=-1) == mlsim.SIM_E_INVAL
    assert gen(n_scen=0) == mlsim.SIM_OK  # nothing to do
    assert gen(n_ops=0) == mlsim.SIM_OK
    assert L.sim_run_generated(None, 1, base, 1, 1, 0, 0, 0, out, None, 0, None, 0, None) == mlsim.SIM_E_INVAL
    assert L.sim_critical_path_generated(None, 1, base, 1, 1, 0, 0, 0, out, -1, None, 0, None,
                                         None) == mlsim.SIM_E_INVAL


def test_noise_for_sigma():
    assert mlsim.noise_for_sigma(0.0) == 0
    assert mlsim.noise_for_sigma(0.01) == 102739
    with pytest.raises(ValueError):
        mlsim.noise_for_sigma(0.2)


def test_gap_argument_errors_without_gpu(L):
    gap = np.zeros(4, np.int32)
    assert L.sim_run_batch_gap(None, 1, None, 1, None, 0, gap.ctypes.data, None, None, 0, None, 0,
                               None) == mlsim.SIM_E_INVAL


def test_device_model_argument_errors_without_gpu(L):
    gap = np.zeros(4, np.int32)
    delay = np.zeros(4, np.int32)
    assert L.sim_run_batch_dev(None, 1, None, 1, None, 0, gap.ctypes.data, delay.ctypes.data, None, None, 0, None,
                               0, None) == mlsim.SIM_E_INVAL
    assert L.sim_run_batch_dev(None, 1, None, 1, None, 0, None, None, None, None, 0, None, 0,
                               None) == mlsim.SIM_E_INVAL


def test_share_argument_errors_without_gpu(L):
    share = np.ones(4, np.uint8)
    assert L.sim_run_batch_share(None, 1, None, 1, share.ctypes.data, None, None, 0, None, None) == mlsim.SIM_E_INVAL
    hdr = open(os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "mlsim.h")).read()
    assert int(re.search(r"#define SIM_SHARE_MAX (\d+)", hdr).group(1)) == mlsim.SIM_SHARE_MAX
    assert int(re.search(r"#define SIM_SHARE_UNIT (\d+)", hdr).group(1)) == mlsim.SIM_SHARE_UNIT
    assert 4096 * math.lcm(*range(1, 17)) == mlsim.SIM_SHARE_UNIT < 2**32


def test_testing_hook_rejects_bad_arguments_without_gpu(L):
    assert L.sim_testing_replan(None, 0, 0) == mlsim.SIM_E_INVAL
    hdr = open(os.path.join(ROOT, "include", "mlsim_testing.h")).read()
    for name, code in mlsim.TEST_VARIANTS.items():
        assert re.search(r"SIM_TEST_%s = %d\b" % (name.upper(), code), hdr), name


def test_no_environment_variable_selects_library_behaviour():
    """Kernel variants are chosen by the launch plan or pinned through the
    testing entry point, never by the environment (a diagnostic print is the
    one exception)."""
    src = os.path.join(ROOT, "paper_2002_06790_amd", "csrc")
    for f in sorted(os.listdir(src)):
        text = open(os.path.join(src, f)).read()
        for m in re.finditer(r"getenv\(\s*\"(\w+)\"", text):
            assert m.group(1) == "MLSIM_VERBOSE", (f, m.group(1))
        assert "getenv(" not in re.sub(r"getenv\(\s*\"MLSIM_VERBOSE\"\)", "", text), f


def test_algorithm_three_is_invalid(L):
    # the value that once selected a removed algorithm is rejected before any GPU work
    assert L.sim_run_batch(None, 1, None, 1, None, 0, None, None, 0, None, 3, None) == mlsim.SIM_E_INVAL
