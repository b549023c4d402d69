"""The C ABI library loads and exports every entry point include/chimera.h
declares; host-side argument checks return the documented codes (no GPU)."""
import ctypes
import os
import re

import pytest

from paper_2608_23553_amd import chimera

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "chimera.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(chimera_[a-z_0-9]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    names = _declared()
    assert "chimera_search" in names and "chimera_index_load" in names and len(names) >= 19
    L = ctypes.CDLL(chimera.LIB_PATH)
    for n in names:
        assert hasattr(L, n), n


def test_null_arguments_are_rejected_without_gpu():
    L = chimera.lib()
    assert L.chimera_last_error() is not None
    rc = L.chimera_search(None, None, 0, 1, 32, 128, 2, 256, 10, None, None, None)
    assert rc == chimera.E_INVAL and b"null index" in L.chimera_last_error()
    assert L.chimera_probe(None, None, 0, 1, 32, 128, 2, None, None, None) == chimera.E_INVAL
    assert L.chimera_prune(None, None, 0, 1, 32, 128, 2, 10, None, None, None, None) == chimera.E_INVAL
    assert L.chimera_candidates(None, None, 0, 1, 32, 128, 2, None, None, 0, None) == chimera.E_INVAL
    assert L.chimera_search_refine(None, None, 0, 1, 32, 128, 2, 256, 10, chimera.REFINE_TOKEN, None, None,
                                   None) == chimera.E_INVAL
    assert L.chimera_prune_refine(None, None, 0, 1, 32, 128, 2, 10, chimera.REFINE_TOKEN, None, None, None,
                                  None) == chimera.E_INVAL
    assert L.chimera_search_collab(None, None, 0, 1, 32, 128, 2, 256, 40, 4, 10, None, None, None, 0,
                                   None) == chimera.E_INVAL
    assert L.chimera_fullbit_attach(None, None, 0) == chimera.E_INVAL
    assert L.chimera_index_info_get(None, None) == chimera.E_INVAL
    assert L.chimera_index_load(None, 0, None) == chimera.E_INVAL
    assert L.chimera_stage_times(None, None) == chimera.E_INVAL
    L.chimera_index_free(None)
    L.chimera_builder_free(None)
