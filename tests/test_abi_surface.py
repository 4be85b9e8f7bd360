"""The C-ABI library loads and exports every function include/batchsim.h declares; the
Python binding mirrors the ABI structs. No device work (runs without a GPU)."""
import ctypes as C
import os
import re

from paper_2607_05272_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "batchsim.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*([a-z][a-z_0-9]*)\s*\(",
                                 src, flags=re.M)))


def test_header_declares_the_mdp_calls():
    names = declared_functions()
    for n in ("sim_create", "sim_reset", "sim_step", "sim_rollout", "returns_gae"):
        assert n in names
    assert set(names) == set(_lib.SYMBOLS)


def test_library_exports_every_declared_symbol():
    L = _lib.load()
    for n in declared_functions():
        assert hasattr(L, n), n
    assert L.sim_abi_version() == _lib.ABI_VERSION


def test_struct_sizes_match_header_layout():
    # sizes implied by the header's field list on x86-64 (natural alignment)
    # 472 by the header's field list; sim_create also rejects a struct_size mismatch
    assert C.sizeof(_lib.SimCfg) == 472
    assert C.sizeof(_lib.SimTraj) == 7 * 8
    assert C.sizeof(_lib.SimWLayout) == 7 * 8 + 8
    assert C.sizeof(_lib.SimUpdateCfg) == 4 * 4 + 8 + 7 * 4 + 4  # padded to 8


def test_invalid_config_is_rejected_without_device_work():
    from workloads import preset
    L = _lib.load()
    lay = _lib.SimWLayout()
    bad = _lib.make_cfg(preset("C1"))
    bad.mlp_h1 = 0
    assert L.sim_weights_layout(C.byref(bad), C.byref(lay)) == -1
    assert b"MLP" in L.sim_last_error()
    ok = _lib.make_cfg(preset("C5"))
    assert L.sim_weights_layout(C.byref(ok), C.byref(lay)) == 0
    assert lay.n_out == 97 and lay.elem_bytes == 2
    ctx = C.c_void_p()
    bad = _lib.make_cfg(preset("C2"))
    bad.obs_dim = 4
    assert L.sim_create(C.byref(bad), None, C.byref(ctx)) == -1
    assert b"obs_dim" in L.sim_last_error()
    for sigma in (float("nan"), -0.5, 100.0):
        bad = _lib.make_cfg(preset("C4"))
        bad.svc_sigma = sigma
        assert L.sim_create(C.byref(bad), None, C.byref(ctx)) == -1
        assert b"svc_sigma" in L.sim_last_error()
        assert not ctx.value
    bad = _lib.make_cfg(preset("C2"))
    bad.abi_version = 99
    assert L.sim_create(C.byref(bad), None, C.byref(ctx)) == -1
    assert not ctx.value
