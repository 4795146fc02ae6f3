"""The C ABI library loads without a GPU, exports every declared symbol, and
rejects bad arguments on the host before any HIP call."""
import ctypes
import os
import re

import pytest

import paper_2502_01637_amd as S

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                      "include", "scone.h")


def declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(scone_\w+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared()
    assert len(names) >= 9, names
    L = S.scone.lib()
    for n in names:
        assert hasattr(L, n), n
    assert {"scone_build_fgram_table", "scone_lookup", "scone_gather"} <= set(names)


def test_status_strings():
    L = S.scone.lib()
    for code in range(10):
        assert L.scone_strerror(code)
    assert L.scone_strerror(S.scone.EROW) == b"row id outside [0, n_rows)"
    assert L.scone_strerror(1234) == b"unknown status"


def test_host_side_argument_errors():
    L = S.scone.lib()
    h = ctypes.c_void_p()
    E = S.scone.EINVAL
    # build: no output pointer, bad K, bad load factor, negative n, missing inputs
    assert L.scone_build_fgram_table(None, None, None, 0, 3, 0.5, None, None) == E
    assert L.scone_build_fgram_table(None, None, None, 0, 8, 0.5, None, ctypes.byref(h)) == E
    assert L.scone_build_fgram_table(None, None, None, 0, 1, 0.5, None, ctypes.byref(h)) == E
    assert L.scone_build_fgram_table(None, None, None, 0, 3, 0.0, None, ctypes.byref(h)) == E
    assert L.scone_build_fgram_table(None, None, None, 0, 3, 0.95, None, ctypes.byref(h)) == E
    assert L.scone_build_fgram_table(None, None, None, -1, 3, 0.5, None, ctypes.byref(h)) == E
    assert L.scone_build_fgram_table(None, None, None, 5, 3, 0.5, None, ctypes.byref(h)) == E
    assert h.value is None
    # lookup: no table, bad window, negative sizes
    assert L.scone_lookup(None, None, 1, 1, 3, None, None, None) == E
    # gather: negative sizes, zero row width, bad placement, missing pointers
    assert L.scone_gather(None, -1, None, 0, 16, None, 0, None) == E
    assert L.scone_gather(None, 1, None, 0, 0, None, 0, None) == E
    assert L.scone_gather(None, 1, None, 1, 16, None, 7, None) == E
    assert L.scone_gather(None, 1, None, 1, 16, None, 0, None) == E
    assert L.scone_gather(None, 0, None, 0, 16, None, 0, None) == S.scone.OK  # nothing to do
    # host memory and table bookkeeping
    assert L.scone_host_alloc(0, ctypes.byref(h), ctypes.byref(h)) == E
    assert L.scone_host_free(None) == S.scone.OK
    assert L.scone_table_info(None, None, None, None, None) == E
    L.scone_table_destroy(None)


def test_binding_rejects_non_device_tensors():
    import torch
    with pytest.raises(TypeError):
        S.gather(torch.zeros(3, dtype=torch.int32), torch.zeros(4, 2))
    with pytest.raises(TypeError):
        S.build_fgram_table(torch.zeros((1, 2), dtype=torch.int32),
                            torch.zeros(1, dtype=torch.int32), torch.zeros(1, dtype=torch.int32))
