"""The C-ABI library loads, exports every symbol include/lst.h declares, and rejects bad
arguments on the host (no GPU call is made by any of these)."""
import ctypes
import os
import re

import pytest

import paper_1606_08061_amd as lst
from paper_1606_08061_amd import build as lst_build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "lst.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(lst_\w+)\s*\(", src)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(lst.LIB_PATH):
        lst_build.build()
    return lst.lib()


def test_header_and_binding_agree():
    assert _declared() == sorted(lst.SIGNATURES)


def test_phase_names_follow_the_header_enum():
    src = open(os.path.join(ROOT, "include", "lst.h")).read()
    vals = {name: int(v) for name, v in re.findall(r"\bLST_PHASE_(\w+)\s*=\s*(\d+)", src)}
    n = int(re.search(r"\bLST_NUM_PHASES\s*=\s*(\d+)", src).group(1))
    assert sorted(vals.values()) == list(range(n)) == list(range(len(lst.PHASES)))
    for name, v in vals.items():
        assert lst.PHASES[v] == name.lower()


def test_every_declared_symbol_is_exported(L):
    for name in _declared():
        assert hasattr(L, name), name
        assert ctypes.cast(getattr(L, name), ctypes.c_void_p).value


def test_status_strings(L):
    for code, name in [(0, "LST_OK"), (-1, "LST_E_ARG"), (-3, "LST_E_INDEX"),
                       (-4, "LST_E_NOT_SPD"), (-5, "LST_E_NONFINITE"), (-8, "LST_E_SYNC"),
                       (7, "LST_E_UNKNOWN")]:
        assert lst.status_string(code) == name


def test_host_argument_errors(L):
    # shape and argument checks run before any device call
    P = 0x1000  # a non-null placeholder; never dereferenced on these paths
    WS = 0x100000  # a 256-byte aligned placeholder workspace
    nb = lst.lst_workspace_bytes(10, 8, 4, 2, 0)
    st, ctx = lst.lst_create(0, 8, 4, 2, 0, 1e-3, P, 8, P, P, P, P, 8, WS, nb, 0)
    assert st == lst.LST_E_SHAPE and ctx == 0
    st, _ = lst.lst_create(10, 8, 4, 2, 5, 1e-3, P, 8, P, P, P, P, 8, WS, nb, 0)
    assert st == lst.LST_E_ARG
    st, _ = lst.lst_create(10, 8, 4, 2, 1, 0.0, P, 8, P, P, P, P, 8, WS, nb, 0)
    assert st == lst.LST_E_ARG
    st, _ = lst.lst_create(10, 8, 4, 2, 0, 1e-3, 0, 8, P, P, P, P, 8, WS, nb, 0)
    assert st == lst.LST_E_ARG
    st, _ = lst.lst_create(10, 8, 4, 2, 0, 1e-3, P, 7, P, P, P, P, 8, WS, nb, 0)
    assert st == lst.LST_E_SHAPE
    st, _ = lst.lst_create(10, 8, 2048, 2, 0, 1e-3, P, 8, P, P, P, P, 8, WS, nb, 0)
    assert st == lst.LST_E_SHAPE
    st, _ = lst.lst_create(10, 8, 512, 64, 0, 1e-3, P, 8, P, P, P, P, 8, WS, nb, 0)
    assert st == lst.LST_E_SHAPE
    # the Taylor softmax keeps w_bar and omega: WO is required
    nt = lst.lst_workspace_bytes(10, 8, 4, 2, lst.LST_LOSS_TAYLOR_SOFTMAX)
    st, _ = lst.lst_create(10, 8, 4, 2, 2, 1e-3, P, 8, P, P, P, 0, 8, WS, nt, 0)
    assert st == lst.LST_E_ARG
    st, _ = lst.lst_create(10, 8, 4, 2, 3, 1e-3, P, 8, P, P, P, P, 8, WS, nt, 0)
    assert st == lst.LST_E_ARG
    st, _ = lst.lst_naive_create(10, 0, 4, 2, 0, 1e-3, P, 8, WS, nb, 0)
    assert st == lst.LST_E_SHAPE
    assert lst.lst_set_option(0, lst.LST_OPT_SPIN_LIMIT, 1) == lst.LST_E_ARG
    assert lst.lst_step(0, P, 1, P, P, 1, 0.1, P, P) == lst.LST_E_ARG
    assert lst.lst_sync_status(0) == lst.LST_E_ARG
    assert lst.lst_materialize_W(0, P, 8) == lst.LST_E_ARG
    # section 5 entry points: a null context is rejected before anything else
    assert lst.lst_restore_pristine(0) == lst.LST_E_ARG
    assert lst.lst_refresh_uinvt(0, 2, 0, 0) == lst.LST_E_ARG
    assert lst.lst_power_iteration(0, 0, 7, P, P, P) == lst.LST_E_ARG
    assert lst.lst_fix_singular_value(0, P, P, 1.0) == lst.LST_E_ARG
    assert lst.lst_singular_stabilize(0, 1e-3, 100.0, 7, P, 8)[0] == lst.LST_E_ARG
    # the sparse input layer: null W1 or status, bad shapes
    assert lst.lst_input_forward(0, 8, 10, 8, P, P, 1, 1, P, P, 0) == lst.LST_E_ARG
    assert lst.lst_input_forward(P, 8, 10, 8, P, P, 1, 1, P, 0, 0) == lst.LST_E_ARG
    assert lst.lst_input_forward(P, 7, 10, 8, P, P, 1, 1, P, P, 0) == lst.LST_E_SHAPE
    assert lst.lst_input_update(P, 8, 10, 8, P, P, 1, 65, P, 0.1, P, 0) == lst.LST_E_SHAPE
    assert lst.lst_input_update(P, 8, 10, 8, P, P, 1, 1, P, -1.0, P, 0) == lst.LST_E_ARG
    lst.lst_destroy(0)


def test_workspace_is_checked_on_the_host(L):
    # the workspace is the caller's: a missing, misaligned or too small one is rejected
    # before anything is enqueued, and its size grows with every dimension it holds
    P = 0x1000
    nb = lst.lst_workspace_bytes(1000, 32, 16, 3, 0)
    assert nb > 0 and nb % 256 == 0
    assert lst.lst_workspace_bytes(0, 32, 16, 3, 0) == 0
    assert lst.lst_workspace_bytes(1000, 32, 16, 3, 9) == 0
    assert lst.lst_workspace_bytes(1000, 32, 32, 3, 0) > nb
    assert lst.lst_workspace_bytes(1000, 64, 16, 3, 0) > nb
    assert lst.lst_workspace_bytes(1000, 32, 16, 6, 0) > nb
    ws = 0x100000
    for args, want in [((0, nb), lst.LST_E_ARG), ((ws + 4, nb), lst.LST_E_ARG),
                       ((ws, nb - 256), lst.LST_E_SHAPE)]:
        st, ctx = lst.lst_create(1000, 32, 16, 3, 0, 1e-3, P, 32, P, P, P, P, 32, *args, 0)
        assert st == want and ctx == 0
    nn = lst.lst_naive_workspace_bytes(1000, 32, 16, 3, 0)
    assert nn >= 1000 * 16 * 4  # holds the D x m output
    st, ctx = lst.lst_naive_create(1000, 32, 16, 3, 0, 1e-3, P, 32, ws, nn - 256, 0)
    assert st == lst.LST_E_SHAPE and ctx == 0


def test_noalloc_step_checks_its_arguments_on_the_host(L):
    # argument and size checks of the allocation-free step run before any device call
    P = 0x1000
    base = [200000, 500, 0, 1e-3, P, 500, P, P, P, 0, 500, P, 128, P, P, 5, 0.1, P, P, P, 0]
    def call(**kw):
        a = list(base)
        for k, v in kw.items():
            a[int(k[1:])] = v
        return lst.lst_step_noalloc(*a)
    assert call(a4=0) == lst.LST_E_ARG         # V
    assert call(a19=0) == lst.LST_E_ARG        # status
    assert call(a17=0) == lst.LST_E_ARG        # loss_dev
    assert call(a16=0.0) == lst.LST_E_ARG      # lr
    assert call(a5=499) == lst.LST_E_SHAPE     # ldv < d
    assert call(a12=-1) == lst.LST_E_SHAPE     # m < 0
    assert call(a2=7) == lst.LST_E_ARG         # loss kind
    assert call(a2=2) == lst.LST_E_ARG         # the Taylor softmax without WO
    # the 16 MiB array holds m = 128 (K = 5) up to d = 2860 and m = 512 up to d = 361 (sizes
    # that fit are not called here: with these stand-in pointers the call would go on to
    # the device)
    assert call(a1=2861, a5=2861, a10=2861) == lst.LST_E_SHAPE
    assert call(a1=362, a5=362, a10=362, a12=512, a15=5) == lst.LST_E_SHAPE


def test_product_path_does_not_import_the_oracle():
    pkg = os.path.join(ROOT, "paper_1606_08061_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"^\s*(from|import)\s+oracle\b", text, re.M), f
                assert "oracle/" not in text, f
