"""The package never loads a library built from other sources (CPU).

The build records a digest of every source next to libadpsgd.so; importing
the package compares it with the sources in the tree and rebuilds on a
difference, or refuses with ImportError when ADPSGD_NO_REBUILD is set.  Both
cases run on a copy of the package in a temporary directory.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = "paper_2007_06134_amd"


def _copy_tree(tmp):
    src = os.path.join(ROOT, PKG)
    if not os.path.exists(os.path.join(src, "libadpsgd.so.digest")):
        pytest.skip("the library has not been built here")
    shutil.copytree(src, os.path.join(tmp, PKG), ignore=shutil.ignore_patterns("__pycache__"))
    shutil.copytree(os.path.join(ROOT, "include"), os.path.join(tmp, "include"))


def _import(tmp):
    env = dict(os.environ, ADPSGD_NO_REBUILD="1")
    code = f"import sys; sys.path.insert(0, {tmp!r}); import {PKG} as A; print(A.LIB_PATH)"
    return subprocess.run([sys.executable, "-c", code], cwd=tmp, env=env, capture_output=True, text=True,
                          timeout=300)


def test_current_library_loads(tmp_path):
    _copy_tree(str(tmp_path))
    r = _import(str(tmp_path))
    assert r.returncode == 0, r.stderr[-2000:]
    assert r.stdout.strip() == os.path.join(str(tmp_path), PKG, "libadpsgd.so")


@pytest.mark.parametrize("edited", [os.path.join(PKG, "csrc", "kernels.hip"), os.path.join("include", "adpsgd.h")])
def test_edited_source_is_refused(tmp_path, edited):
    tmp = str(tmp_path)
    _copy_tree(tmp)
    with open(os.path.join(tmp, edited), "a") as f:
        f.write("\n// edited after the build\n")
    r = _import(tmp)
    assert r.returncode != 0
    assert "ImportError" in r.stderr and "built from other sources" in r.stderr, r.stderr[-2000:]


def test_missing_digest_is_refused(tmp_path):
    tmp = str(tmp_path)
    _copy_tree(tmp)
    os.remove(os.path.join(tmp, PKG, "libadpsgd.so.digest"))
    r = _import(tmp)
    assert r.returncode != 0 and "ImportError" in r.stderr
