"""Every oracle pin again, against a build of oracle.c with AddressSanitizer
and UndefinedBehaviorSanitizer (CPU only).

The pins of tests/test_oracle.py run in a child process that has the
sanitizer runtimes preloaded and sends every oracle call to the checking
build; any out-of-bounds access, use after free or undefined behaviour
(signed overflow, bad shifts, misaligned loads) aborts the child.
"""
import os
import subprocess
import sys

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


def test_oracle_pins_under_sanitizers(tmp_path):
    so = oracle.build(sanitize=True, out=str(tmp_path / "liboracle_san.so"))
    env = oracle.sanitizer_env(so)
    env["PYTHONDONTWRITEBYTECODE"] = "1"
    cmd = [sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-p", "no:xdist",
           os.path.join(HERE, "test_oracle.py"), os.path.join(HERE, "test_workloads.py")]
    p = subprocess.run(cmd, env=env, cwd=os.path.dirname(HERE), capture_output=True, text=True, timeout=1200)
    out = p.stdout + p.stderr
    assert p.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    # the child really used the checking build
    assert " passed" in out


def test_sanitized_build_is_in_use_and_catches_an_overread(tmp_path):
    """The child's oracle calls go to the checking build, and that build
    stops on a planted one-past-the-end read (a mistake planted on the CPU
    in a copy of oracle.c)."""
    so = oracle.build(sanitize=True, out=str(tmp_path / "liboracle_san.so"))
    probe = ("import numpy as np, oracle; L = oracle.lib(); print(L._name); "
             "p = np.array([0, 1, 1], np.int64); i = np.array([1], np.int32); r = np.zeros(2, np.int32); "
             "print(oracle.run_batch(p, i, r, 1, np.ones((2, 3), np.int32))[0].tolist())")
    p = subprocess.run([sys.executable, "-c", probe], env=oracle.sanitizer_env(so), cwd=os.path.dirname(HERE),
                       capture_output=True, text=True, timeout=300)
    assert p.returncode == 0, p.stderr[-3000:]
    assert p.stdout.split("\n")[0] == so and p.stdout.split("\n")[1] == "[2, 2, 2]"
    src = open(os.path.join(os.path.dirname(oracle.__file__), "oracle.c")).read()
    site = "for (int32_t v = 0; v < g->n; ++v) J->finish[(int64_t)v * J->ld_fin + s] = (int32_t)w->fin[v];"
    assert site in src
    bad = tmp_path / "overread.c"
    bad.write_text(src.replace(site, "for (int32_t v = 0; v <= g->n; ++v) (void)*(volatile int64_t *)&w->fin[v];\n"
                                     "    " + site, 1))
    so_bad = str(tmp_path / "liboracle_bad.so")
    subprocess.check_call(["gcc", *oracle.SANITIZE_FLAGS, "-std=c11", "-fPIC", "-shared", "-pthread",
                           "-I", os.path.dirname(oracle.__file__), str(bad), "-o", so_bad])
    p = subprocess.run([sys.executable, "-c", probe], env=oracle.sanitizer_env(so_bad), cwd=os.path.dirname(HERE),
                       capture_output=True, text=True, timeout=300)
    assert p.returncode != 0 and "heap-buffer-overflow" in p.stderr, p.stderr[-3000:]
