"""Host-side checks of the graph-cache ABI (no GPU): exports and argument
validation that happens before any HIP call."""
import ctypes
import os
import re

import pytest

from paper_2404_11068_amd import evo_attn as ea
from paper_2404_11068_amd import graph as gr

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _lib():
    if not os.path.exists(ea.LIB_PATH):
        pytest.skip("libevoattn.so not built")
    return gr._lib()


def test_exports():
    lib = _lib()
    decls = re.findall(r"^\s*(?:int|int32_t)\s*(evo_graph_\w+)\s*\(",
                       open(os.path.join(ROOT, "include", "evo_graph.h")).read(), flags=re.M)
    assert set(decls) == {"evo_graph_cache_create", "evo_graph_cache_destroy", "evo_graph_cache_run",
                          "evo_graph_cache_size", "evo_graph_cache_clear"}
    for n in decls:
        assert hasattr(lib, n)


def test_validation_without_hip():
    lib = _lib()
    h = ctypes.c_void_p()
    assert lib.evo_graph_cache_create(0, ctypes.byref(h)) == 1
    assert lib.evo_graph_cache_create(2, None) == 1
    assert lib.evo_graph_cache_create(2, ctypes.byref(h)) == 0 and h.value
    assert lib.evo_graph_cache_size(h) == 0
    assert lib.evo_graph_cache_size(None) == -1
    noop = gr.RECORD_FN(lambda u, s: None)
    assert lib.evo_graph_cache_run(h, 1, noop, None, None, None) == 1          # null stream
    assert lib.evo_graph_cache_run(None, 1, noop, None, ctypes.c_void_p(8), None) == 1
    assert lib.evo_graph_cache_run(h, 1, gr.RECORD_FN(), None, ctypes.c_void_p(8), None) == 1  # null record
    assert lib.evo_graph_cache_clear(h) == 0 and lib.evo_graph_cache_clear(None) == 1
    assert lib.evo_graph_cache_destroy(h) == 0 and lib.evo_graph_cache_destroy(None) == 1
