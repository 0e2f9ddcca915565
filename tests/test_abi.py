"""The C ABI: libtgm.so loads and exports every function include/tgm.h
declares, and the binding covers exactly that list.  No compute calls (no GPU
here)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tgm.h")


def declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tgm_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def libtgm():
    from paper_2402_15113_amd import _build, tgm
    if not os.path.exists(tgm.LIB_PATH):
        _build.build(force=False)
    return ctypes.CDLL(tgm.LIB_PATH)


def test_header_declares_the_stage_calls():
    names = declared()
    for f in ("tgm_sample", "tgm_node_set", "tgm_fetch_memory", "tgm_update_memory",
              "tgm_embed", "tgm_batch_roots", "tgm_graph_create", "tgm_state_create",
              "tgm_model_create"):
        assert f in names


def test_every_declared_symbol_is_exported(libtgm):
    for name in declared():
        assert hasattr(libtgm, name), name


def test_binding_covers_the_header():
    from paper_2402_15113_amd import tgm
    assert sorted(tgm.SYMBOLS) == declared()


def test_status_strings_and_version(libtgm):
    from paper_2402_15113_amd import tgm
    assert tgm.version() == 100
    assert tgm.status_str(tgm.TGM_OK) == "ok"
    assert tgm.status_str(tgm.TGM_EORDER) == "iteration protocol violated"
    assert tgm.status_str(12345) == "unknown status"


def test_null_handles_rejected_without_device(libtgm):
    """Argument checks run on the host before anything touches the device."""
    from paper_2402_15113_amd import tgm
    L = tgm.lib()
    assert L.tgm_graph_destroy(None) == tgm.TGM_EINVAL
    assert L.tgm_state_destroy(None) == tgm.TGM_EINVAL
    assert L.tgm_model_destroy(None) == tgm.TGM_EINVAL
    assert L.tgm_sample(None, None, None, 0, 10, None, None, None, None, None) == tgm.TGM_EINVAL
    assert L.tgm_state_flush(None, None) == tgm.TGM_EINVAL
    assert L.tgm_graph_create(0, 0, None, None, None, None, None, 0, None, None) == tgm.TGM_EINVAL
    out = ctypes.c_void_p()
    assert L.tgm_state_create(10, 0, 4, 0, 5, None, ctypes.byref(out)) == tgm.TGM_EINVAL


def test_binding_constants_match_the_header():
    from paper_2402_15113_amd import tgm
    text = open(HEADER).read()
    defs = dict(re.findall(r"#define\s+(TGM_\w+)\s+\(?(-?\d+)", text))
    assert int(defs["TGM_MAX_SAMPLE_SETS"]) == tgm.MAX_SAMPLE_SETS
    assert int(defs["TGM_MITIGATE_NOALLOC_MAX_NODES"]) == tgm.MITIGATE_NOALLOC_MAX_NODES
    for name in ("TGM_OK", "TGM_EINVAL", "TGM_ERANGE", "TGM_EORDER", "TGM_ESIZE", "TGM_EDEVICE",
                 "TGM_ENOMEM"):
        assert int(defs[name]) == getattr(tgm, name), name


def test_alloc_count_without_device(libtgm):
    from paper_2402_15113_amd import tgm
    assert tgm.lib().tgm_alloc_count(None) == tgm.TGM_EINVAL
    assert tgm.alloc_count() >= 0
