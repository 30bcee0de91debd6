"""The C ABI: every declared symbol is exported, and the host-side argument
checks answer with status codes (no GPU work is launched by these calls)."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2609_35629_amd as sp
from paper_2609_35629_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "santapp.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(santapp_[a-z_A-Z0-9]+)\s*\(", text)))


def test_header_lists_match_binding():
    assert declared_functions() == sorted(_lib.EXPORTS)


def test_library_exports_every_declared_symbol():
    L = _lib.load()
    out = subprocess.run(["nm", "-D", "--defined-only", _lib.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(line.split()[-1] for line in out.splitlines() if line.strip())
    for name in declared_functions():
        assert name in exported, name
        assert hasattr(L, name)


def test_budget_rule():
    # eq. method-budget: K = min(M, S / (P / R)); P/R = 4 for P = 16, R = 4
    assert sp.budget_to_K(128, 16, 4, 10000) == 32
    assert sp.budget_to_K(124, 16, 4, 10000) == 31
    assert sp.budget_to_K(256, 16, 4, 50) == 50
    assert sp.budget_to_K(2048, 1024, 16, 512) == 32
    with pytest.raises(sp.SantappError) as e:
        sp.budget_to_K(126, 16, 4, 100)  # 126 not divisible by 4
    assert e.value.status == _lib.EINVAL
    with pytest.raises(sp.SantappError):
        sp.budget_to_K(128, 16, 3, 100)  # P not divisible by R


def _status(fn, *args):
    return fn(*args)


def test_host_argument_checks():
    L = _lib.load()
    h = ctypes.c_void_p()
    vp = ctypes.c_void_p
    # NULL K/V
    assert L.santapp_build_teams(None, None, 1, 1, 16, 64, 0, 4, 2, None, ctypes.byref(h)) == _lib.EINVAL
    assert b"K and V" in L.santapp_last_error()
    fake = vp(0x1000)  # never dereferenced: the checks below fail first
    assert L.santapp_build_teams(fake, fake, 1, 1, 16, 64, 0, 0, 2, None, ctypes.byref(h)) == _lib.EINVAL
    assert L.santapp_build_teams(fake, fake, 1, 1, 16, 64, 0, 4, 0, None, ctypes.byref(h)) == _lib.EINVAL
    assert L.santapp_build_teams(fake, fake, 1, 1, 0, 64, 0, 4, 2, None, ctypes.byref(h)) == _lib.EINVAL
    assert L.santapp_build_teams(fake, fake, 1, 1, 16, 64, 7, 4, 2, None, ctypes.byref(h)) == _lib.EDTYPE
    assert L.santapp_build_teams(fake, fake, 1, 1, 16, 96, 0, 4, 2, None, ctypes.byref(h)) == _lib.ELIMIT
    assert L.santapp_build_teams(fake, fake, 1, 1, 16, 64, 0, 4, 2000, None, ctypes.byref(h)) == _lib.ELIMIT
    # misaligned device pointers (16-byte vector accesses)
    odd = vp(0x1008)
    assert L.santapp_build_teams(odd, fake, 1, 1, 16, 64, 0, 4, 2, None, ctypes.byref(h)) == _lib.EINVAL
    assert b"aligned" in L.santapp_last_error()
    assert L.santapp_dense_decode(odd, fake, fake, 1, 4, 100, 128, 0, None, None, 0, 0, 28, 0.0,
                                  fake, fake, 1 << 30, None, None) == _lib.EINVAL
    assert L.santapp_dense_decode(fake, fake, fake, 1, 4, 100, 128, 0, None, None, 0, 0, 28, 0.0,
                                  fake, odd, 1 << 30, None, None) == _lib.EINVAL
    # decode without a table
    assert L.santapp_decode(None, fake, None, None, 0, 0, 1, 1, 0, 0, 0.0, fake, fake, 10, None, None) == _lib.EINVAL
    # dense workspace query is pure host arithmetic
    n = ctypes.c_size_t()
    assert L.santapp_dense_workspace_bytes(1, 28, 4, 32768, 128, 128, ctypes.byref(n)) == _lib.OK
    assert n.value > 0
    assert L.santapp_dense_workspace_bytes(1, 27, 4, 32768, 128, 128, ctypes.byref(n)) == _lib.EINVAL
    # dense decode: bad GQA grouping, too-small workspace, bad scale
    assert L.santapp_dense_decode(fake, fake, fake, 1, 4, 100, 128, 0, None, None, 0, 0, 27, 0.0,
                                  fake, fake, 1 << 30, None, None) == _lib.EINVAL
    assert L.santapp_dense_decode(fake, fake, fake, 1, 4, 100, 128, 0, None, None, 0, 0, 28, 0.0,
                                  fake, fake, 16, None, None) == _lib.EWORKSPACE
    assert L.santapp_dense_decode(fake, fake, fake, 1, 4, 100, 128, 0, None, None, 0, 0, 28, -1.0,
                                  fake, fake, 1 << 30, None, None) == _lib.EINVAL
    assert L.santapp_dense_decode(fake, fake, fake, 1, 4, 100, 128, 0, None, None, 5, 0, 28, 0.0,
                                  fake, fake, 1 << 30, None, None) == _lib.EINVAL  # T > 0, no suffix
    # suffix rows of a pair further apart than the buffer allows
    assert L.santapp_dense_decode(fake, fake, fake, 1, 4, 100, 128, 0, fake, fake, 5, 4, 28, 0.0,
                                  fake, fake, 1 << 30, None, None) == _lib.EINVAL
    assert b"suffix_stride" in L.santapp_last_error()
    # a misaligned suffix buffer
    assert L.santapp_dense_decode(fake, fake, fake, 1, 4, 100, 128, 0, odd, fake, 5, 8, 28, 0.0,
                                  fake, fake, 1 << 30, None, None) == _lib.EINVAL


def test_kmeans_and_label_table_argument_checks():
    """Host-side checks of the k-means and label-table entry points (no GPU
    call is reached)."""
    L = _lib.load()
    fake = ctypes.c_void_p(1 << 20)
    th = _lib.KMeansSettings(4096, 100, 10, 0.01, 0, 0)
    mp = ctypes.c_int()
    args = lambda K, N, d, P, t: (K, 1, 4, N, d, 0, P, ctypes.byref(t), fake, ctypes.byref(mp), None, None)
    assert L.santapp_kmeans_parents(*args(None, 4096, 128, 1024, th)) == _lib.EINVAL
    assert L.santapp_kmeans_parents(*args(fake, 1, 128, 1024, th)) == _lib.EINVAL      # N >= 2
    assert L.santapp_kmeans_parents(*args(fake, 4096, 96, 1024, th)) == _lib.ELIMIT    # head dim
    assert L.santapp_kmeans_parents(*args(fake, 4096, 128, 1, th)) == _lib.ELIMIT      # 4096 centers
    assert b"1024" in L.santapp_last_error()
    bad = _lib.KMeansSettings(4096, 100, 10, 1.0, 0, 0)                                # ratio in [0, 1)
    assert L.santapp_kmeans_parents(*args(fake, 4096, 128, 1024, bad)) == _lib.EINVAL
    bad = _lib.KMeansSettings(0, 100, 10, 0.01, 0, 0)                                  # empty batch
    assert L.santapp_kmeans_parents(*args(fake, 4096, 128, 1024, bad)) == _lib.EINVAL
    h = ctypes.c_void_p()
    assert L.santapp_build_teams_from_labels(fake, fake, 1, 1, 64, 64, 0, None, 4, 2, None,
                                             ctypes.byref(h)) == _lib.EINVAL
    assert L.santapp_build_teams_from_labels(fake, fake, 1, 1, 64, 64, 0, fake, 2000, 2, None,
                                             ctypes.byref(h)) == _lib.ELIMIT
    assert L.santapp_build_teams_from_labels(fake, fake, 1, 1, 64, 64, 0, ctypes.c_void_p((1 << 20) + 4), 4, 2,
                                             None, ctypes.byref(h)) == _lib.EINVAL
    assert b"aligned" in L.santapp_last_error()
    assert L.santapp_build_teams_from_labels(fake, fake, 1, 1, 64, 64, 0, fake, 4, 0, None,
                                             ctypes.byref(h)) == _lib.EINVAL
