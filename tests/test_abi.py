"""The C-ABI library loads and exports every entry point include/wam.h
declares; host-only size queries and argument validation (no GPU needed)."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from paper_2609_34608_amd import _lib as L
from paper_2609_34608_amd import runtime as R
from synth import WORKLOADS, weight_manifest

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "wam.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(wam_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    return L.load()


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert len(names) >= 20
    for n in names:
        assert hasattr(lib, n), n
    # the binding declares exactly the header's functions
    assert sorted(L.EXPORTS) == names


def test_status_strings(lib):
    assert lib.wam_status_string(0) == b"ok"
    for s in range(-6, 0):
        assert lib.wam_status_string(s) != b"unknown status"


@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_host_weight_count_matches_manifest(lib, name):
    w = WORKLOADS[name]
    cfg = R.config_of(w)
    n = sum(int(np.prod(s)) for _, s, _ in weight_manifest(w))
    assert lib.wam_host_weight_count(C.byref(cfg)) == n
    assert lib.wam_traj_elems(C.byref(cfg)) == w.traj
    assert lib.wam_weight_bytes(C.byref(cfg)) > 0
    assert lib.wam_workspace_bytes(C.byref(cfg)) > 0


def test_binding_order_matches_manifest():
    for w in WORKLOADS.values():
        assert R.host_weight_order(w.L) == [n for n, _, _ in weight_manifest(w)]


@pytest.mark.parametrize("bad", [dict(B=0), dict(B=17), dict(D=100), dict(H=5), dict(Nv=0, Na=0), dict(Na=-1),
                                 dict(dtype="bf16", H=4), dict(Cv=17), dict(A=17), dict(Co=65), dict(ln_eps=0.0)])
def test_invalid_configs_rejected(lib, bad):
    """Shape limits of wam_config (include/wam.h); a model needs a trajectory."""
    base = dict(B=1, L=2, D=128, H=4, F=512, Nv=64, Cv=16, Na=16, A=7, No=8, Co=16, dtype="fp32")
    base.update(bad)
    cfg = R.make_config(**base)
    assert lib.wam_host_weight_count(C.byref(cfg)) == 0
    assert lib.wam_workspace_bytes(C.byref(cfg)) == 0
    h = C.c_void_p()
    buf = (C.c_float * 4)()
    st = lib.wam_init(C.byref(cfg), buf, 4, C.c_void_p(1), 1, C.c_void_p(1), 1, None, C.byref(h))
    assert st in (L.WAM_E_SHAPE, L.WAM_E_ARG)
    assert not h.value


def test_init_rejects_short_buffers_without_touching_device(lib):
    w = WORKLOADS["tiny"]
    cfg = R.config_of(w)
    n = lib.wam_host_weight_count(C.byref(cfg))
    host = np.zeros(n, np.float32)
    h = C.c_void_p()
    # wrong host weight count
    assert lib.wam_init(C.byref(cfg), host.ctypes.data_as(C.c_void_p), n - 1, C.c_void_p(8), 1 << 40,
                        C.c_void_p(8), 1 << 40, None, C.byref(h)) == L.WAM_E_SHAPE
    # weight buffer too small
    assert lib.wam_init(C.byref(cfg), host.ctypes.data_as(C.c_void_p), n, C.c_void_p(8), 16,
                        C.c_void_p(8), 1 << 40, None, C.byref(h)) == L.WAM_E_WORKSPACE
    # null handle calls are rejected, not crashed
    assert lib.wam_sync(None) == L.WAM_E_ARG
    assert lib.wam_set_schedule(None, None, 4) == L.WAM_E_ARG
    assert lib.wam_adapt_state(None, L.WAM_ADAPT_RESET_ALL, None) == L.WAM_E_ARG


@pytest.mark.parametrize("one_branch", [dict(Na=0), dict(Nv=0)])
def test_single_branch_configs_accepted(lib, one_branch):
    """A model of an independently executed pair has only video or only action
    tokens (Sec. 3.3, independent execution)."""
    base = dict(B=1, L=2, D=128, H=4, F=512, Nv=64, Cv=16, Na=16, A=7, No=8, Co=16, dtype="fp32")
    base.update(one_branch)
    cfg = R.make_config(**base)
    assert lib.wam_host_weight_count(C.byref(cfg)) > 0
    assert lib.wam_workspace_bytes(C.byref(cfg)) > 0
    assert lib.wam_traj_elems(C.byref(cfg)) == base["Nv"] * 16 + base["Na"] * 7


def test_binding_constants_match_header():
    """Every WAM_* integer constant of include/wam.h has the same value in
    the Python binding."""
    text = open(HEADER).read()
    defs = dict(re.findall(r"#define\s+(WAM_[A-Z0-9_]+)\s+\(?(-?\d+)\)?", text))
    assert len(defs) >= 40
    for name, val in defs.items():
        if hasattr(L, name):
            assert getattr(L, name) == int(val), name
    for name in ("WAM_ADAPT_REBIND", "WAM_E_STATE", "WAM_RR_SINGLE", "WAM_ATTN_PLAIN", "WAM_KC_COUNT"):
        assert getattr(L, name) == int(defs[name])
