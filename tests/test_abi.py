"""The C ABI: the library loads and exports every function include/hetpipe.h
declares (no device work, runs without a GPU)."""
import ctypes
import os
import re

from paper_2005_14038_amd import hetpipe

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "hetpipe.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(hp_\w+)\s*\(", src, flags=re.M)))


def test_header_declares_the_hot_path_calls():
    names = declared_functions()
    for f in ["hp_stage_forward", "hp_stage_backward", "hp_wsp_local_update",
              "hp_wsp_push_wave", "hp_wsp_pull"]:
        assert f in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(hetpipe.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing
    assert sorted(hetpipe.EXPORTS) == declared_functions()


def test_library_resolves_every_symbol_at_load():
    # immediate binding: a reference the library makes but does not define
    # fails here instead of at its first call on a GPU
    ctypes.CDLL(hetpipe.LIB_PATH, mode=os.RTLD_NOW | os.RTLD_LOCAL)


def test_layer_struct_matches_header():
    # 10 int32 fields and one float: 44 bytes, no padding
    assert ctypes.sizeof(hetpipe.hp_layer) == 44
    # one int64 and eight int32: 40 bytes, no padding
    assert ctypes.sizeof(hetpipe.hp_wsp_state_t) == 8 + 8 * 4


def test_error_text_without_device_work():
    lib = hetpipe.lib()
    out = ctypes.c_void_p()
    rc = lib.hp_stage_create(None, 0, 1, 1, 1, 1, 0, None, ctypes.byref(out))
    assert rc == hetpipe.HP_ERR_ARG
    assert b"bad arguments" in lib.hp_last_error()
    rc = lib.hp_ps_create(0, None, 1, 0, None, ctypes.byref(out))
    assert rc == hetpipe.HP_ERR_ARG
