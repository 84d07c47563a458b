"""The C ABI library loads, exports every entry point include/lopa.h declares, and
rejects invalid arguments on the host before any HIP call (no GPU needed)."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lopa.h")


def declared():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w\s\*]+?\b(lopa_\w+)\s*\(", txt, flags=re.M)))


@pytest.fixture(scope="module")
def lp():
    import paper_2512_16229_amd as lp
    return lp


def test_header_declares_the_four_hot_path_calls():
    names = declared()
    for n in ("lopa_build_branches", "lopa_verify_forward", "lopa_branch_confidence_select",
              "lopa_commit_kv"):
        assert n in names


def test_library_exports_every_declared_symbol(lp):
    raw = C.CDLL(lp.LIB_PATH)
    missing = [n for n in declared() if not hasattr(raw, n)]
    assert not missing, missing
    assert set(declared()) == set(lp.EXPORTS)


def test_strerror(lp):
    for code in (0, -1, -2, -3, -4, -5):
        assert lp.lib.lopa_strerror(code)
    assert lp.lib.lopa_strerror(-99) == b"unknown status"


FAKE = C.c_void_p(0x1000)  # never dereferenced: every case fails validation first


@pytest.mark.parametrize("L,mask,tau,k,code", [
    (0, 5, 0.9, 3, -2), (257, 5, 0.9, 3, -2), (16, 5, 1.5, 3, -1), (16, 5, -0.1, 3, -1),
    (16, 5, float("nan"), 3, -1), (16, 5, 0.9, -1, -1), (16, -1, 0.9, 3, -1)])
def test_build_branches_validation(lp, L, mask, tau, k, code):
    rc = lp.lib.lopa_build_branches(FAKE, FAKE, FAKE, L, mask, tau, k, FAKE, FAKE, FAKE, FAKE, None)
    assert rc == code, lp.lib.lopa_last_error()


def test_null_pointers(lp):
    assert lp.lib.lopa_build_branches(None, FAKE, FAKE, 16, 5, 0.9, 3, FAKE, FAKE, FAKE, FAKE, None) == -1
    assert lp.lib.lopa_verify_forward(None, None, 0, FAKE, 1, 16, FAKE, FAKE, None) == -1
    assert lp.lib.lopa_verify_forward_noalloc(None, None, 0, FAKE, 1, 16, FAKE, FAKE, None) == -1
    assert lp.lib.lopa_verify_forward_noalloc(FAKE, FAKE, 0, FAKE, 1, 16, None, FAKE, None) == -1
    assert lp.lib.lopa_branch_confidence_select(FAKE, FAKE, FAKE, FAKE, 4, 16, 5, FAKE, None,
                                                FAKE, FAKE, FAKE, FAKE, None) == -1
    assert lp.lib.lopa_commit_kv(None, FAKE, 0, 16, FAKE, None) == -1
    assert lp.lib.lopa_kv_read(None, 0, 0, 1, FAKE, FAKE, None) == -1


def test_select_validation(lp):
    f = lp.lib.lopa_branch_confidence_select
    assert f(FAKE, FAKE, FAKE, FAKE, 0, 16, 5, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == -2
    assert f(FAKE, FAKE, FAKE, FAKE, 4, 257, 5, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == -2
    assert f(FAKE, FAKE, FAKE, FAKE, 4, 16, -3, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == -1


def test_select_metric_validation(lp):
    f = lp.lib.lopa_branch_confidence_select_metric
    o = (FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None)
    assert f(FAKE, FAKE, FAKE, FAKE, 4, 16, 5, 3, 1, 1.0, *o) == -1        # unknown metric
    assert f(FAKE, FAKE, FAKE, FAKE, 4, 16, 5, -1, 1, 1.0, *o) == -1
    assert f(FAKE, FAKE, FAKE, FAKE, 4, 16, 5, 1, 0, 1.0, *o) == -1        # window < 1
    assert f(FAKE, FAKE, FAKE, FAKE, 4, 16, 5, 2, 1, 0.0, *o) == -1        # eta outside (0, 1]
    assert f(FAKE, FAKE, FAKE, FAKE, 4, 16, 5, 2, 1, 1.5, *o) == -1
    assert f(FAKE, FAKE, FAKE, FAKE, 4, 16, 5, 2, 1, float("nan"), *o) == -1
    assert f(FAKE, FAKE, FAKE, FAKE, 4, 257, 5, 1, 2, 1.0, *o) == -2       # L too large
    assert f(None, FAKE, FAKE, FAKE, 4, 16, 5, 0, 1, 1.0, *o) == -1


@pytest.mark.parametrize("field,value,code", [
    ("hidden", 200, -2), ("head_dim", 96, -2), ("kv_heads", 3, -2), ("ffn", 700, -2),
    ("mask_id", 1024, -1), ("mask_id", -1, -1), ("layers", 0, -1), ("rms_eps", 0.0, -1),
    ("heads", 5, -2)])
def test_model_cfg_validation(lp, field, value, code):
    cfg = lp.lopa_model_cfg(2, 256, 4, 2, 64, 704, 1024, 1023, 1e-6, 1e4, 1)
    setattr(cfg, field, value)
    w = lp.lopa_weight_ptrs()
    h = C.c_void_p()
    rc = lp.lib.lopa_model_create(C.byref(cfg), C.byref(w), None, C.byref(h))
    assert rc == code, lp.lib.lopa_last_error()
    assert not h.value


def test_model_create_null_weights(lp):
    cfg = lp.lopa_model_cfg(2, 256, 4, 2, 64, 704, 1024, 1023, 1e-6, 1e4, 1)
    h = C.c_void_p()
    assert lp.lib.lopa_model_create(C.byref(cfg), None, None, C.byref(h)) == -1
    w = lp.lopa_weight_ptrs(FAKE, None, FAKE, FAKE)
    assert lp.lib.lopa_model_create(C.byref(cfg), C.byref(w), None, C.byref(h)) == -1


@pytest.mark.parametrize("precision", [-1, 3, 7])
def test_model_create_unknown_precision(lp, precision):
    """lopa_model_create_ex rejects a precision outside {BF16, FP8_MLP, FP8}
    before any HIP call; the known ones pass that check and stop at the null
    weight pointers."""
    cfg = lp.lopa_model_cfg(2, 256, 4, 2, 64, 704, 1024, 1023, 1e-6, 1e4, 1)
    h = C.c_void_p()
    w = lp.lopa_weight_ptrs()
    rc = lp.lib.lopa_model_create_ex(C.byref(cfg), C.byref(w), precision, None, C.byref(h))
    assert rc == -1 and "precision" in lp.lib.lopa_last_error().decode()
    assert not h.value
    for known in lp.PRECISIONS.values():
        rc = lp.lib.lopa_model_create_ex(C.byref(cfg), C.byref(w), known, None, C.byref(h))
        assert rc == -1 and "weight pointer" in lp.lib.lopa_last_error().decode()


def test_kv_create_validation(lp):
    h = C.c_void_p()
    assert lp.lib.lopa_kv_create(None, 128, 8, 32, C.byref(h)) == -1
    assert lp.lib.lopa_kv_create(FAKE, 0, 8, 32, C.byref(h)) == -1
    assert lp.lib.lopa_kv_create(FAKE, 128, 8, 257, C.byref(h)) == -2
    assert lp.lib.lopa_kv_create(FAKE, 128, 16, 256, C.byref(h)) == -2  # 4096 rows > 2048


def test_window_entry_points_validation(lp):
    f = lp.lib.lopa_build_branches_window
    o = (FAKE, FAKE, FAKE, FAKE, None)
    assert f(FAKE, FAKE, FAKE, 32, 0, 5, 0.9, 3, *o) == -1        # n_eligible < 1
    assert f(FAKE, FAKE, FAKE, 32, 33, 5, 0.9, 3, *o) == -1       # n_eligible > L
    assert f(FAKE, FAKE, FAKE, 257, 32, 5, 0.9, 3, *o) == -2      # L too large
    assert f(None, FAKE, FAKE, 32, 16, 5, 0.9, 3, *o) == -1
    assert lp.lib.lopa_commit_kv_rows(None, FAKE, 0, 32, 16, FAKE, None) == -1


def test_window_state_validation(lp):
    """lopa_window_init / _update / _commit reject bad arguments on the host,
    before any launch (the window's sizes and gates; null pointers)."""
    init = lp.lib.lopa_window_init
    t = (FAKE, FAKE, FAKE)
    assert init(None, *t, 32, 2, 4, 0, 5, 0.1, 0.9, None) == -1
    assert init(FAKE, None, FAKE, FAKE, 32, 2, 4, 0, 5, 0.1, 0.9, None) == -1
    assert init(FAKE, *t, 32, 0, 4, 0, 5, 0.1, 0.9, None) == -2                 # w_max < 1
    assert init(FAKE, *t, 16, lp.WINDOW_MAX_BLOCKS + 1, 4, 0, 5, 0.1, 0.9, None) == -2
    assert init(FAKE, *t, 32, 9, 4, 0, 5, 0.1, 0.9, None) == -2                 # 288 positions
    assert init(FAKE, *t, 0, 2, 4, 0, 5, 0.1, 0.9, None) == -2                  # L < 1
    assert init(FAKE, *t, 32, 2, 0, 0, 5, 0.1, 0.9, None) == -1                 # no blocks
    assert init(FAKE, *t, 32, 2, 4, -1, 5, 0.1, 0.9, None) == -1                # prefix < 0
    assert init(FAKE, *t, 32, 2, 4, 0, 5, 1.5, 0.9, None) == -1                 # tau_add > 1
    assert init(FAKE, *t, 32, 2, 4, 0, 5, 0.1, float("nan"), None) == -1
    assert lp.lib.lopa_window_update(None, *t, FAKE, None) == -1
    assert lp.lib.lopa_window_update(FAKE, *t, None, None) == -1
    assert lp.lib.lopa_window_commit(None, FAKE, FAKE, None) == -1
    assert lp.lib.lopa_window_commit(FAKE, None, FAKE, None) == -1


def test_window_struct_layout(lp):
    """The ctypes mirror of lopa_window has the header's field order and size
    (16 header words, then the activation flags)."""
    assert C.sizeof(lp.lopa_window) == 4 * (16 + lp.WINDOW_MAX_BLOCKS)
    assert [f[0] for f in lp.lopa_window._fields_][:5] == ["blocks", "eligible", "prefix_len",
                                                            "need_initial", "done"]
