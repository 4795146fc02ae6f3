"""The C ABI library loads without a GPU, exports every declared symbol, and
rejects bad arguments on the host before any HIP call."""
import ctypes
import os
import re

import pytest
import torch

import paper_2502_01637_amd as S

# These tests pass fake device addresses and count on the first HIP call
# failing: a call that got past its host checks in a process with a GPU would
# launch kernels on them.  They run only where no GPU is visible
# (torch.cuda.device_count does not initialise one).
pytestmark = pytest.mark.skipif(torch.cuda.device_count() > 0,
                                reason="fake device addresses: for a process without a GPU")

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
    for code in range(11):
        assert L.scone_strerror(code) and L.scone_strerror(code) != b"unknown status"
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
    # pipelined step: no table, bad window, negative sizes, bad placement
    assert L.scone_embed_pipelined(None, None, 0, 0, 3, None, None, None, 0, None, 0, 16, 0,
                                   None, None) == E
    # discovery: corpora whose candidates a 32-bit counter cannot count
    n = ctypes.c_int64(-1)
    assert L.scone_discover_fgrams(None, 1, 1 << 31, 3, 5, 10, None, None, None,
                                   ctypes.byref(n), None, 0, None) == E          # B * T >= 2^31
    assert L.scone_discover_fgrams(None, 1, (1 << 31) - 1, 7, 5, 10, None, None, None,
                                   ctypes.byref(n), None, 0, None) == E          # 6 * B * T >= 2^32
    assert L.scone_discover_fgrams(None, 1, 1 << 30, 5, 5, 10, None, None, None,
                                   ctypes.byref(n), None, 0, None) == E          # 4 * B * T = 2^32
    assert n.value == 0
    assert L.scone_discover_workspace(1, 1 << 30, 5) == -1
    assert L.scone_discover_workspace(1, 1 << 20, 5) > 2 * (1 << 20) * 16
    # host memory and table bookkeeping
    assert L.scone_host_alloc(0, ctypes.byref(h), ctypes.byref(h)) == E
    assert L.scone_host_free(None) == S.scone.OK
    assert L.scone_table_info(None, None, None, None, None, None) == E
    L.scone_table_destroy(None)


def test_binding_rejects_non_device_tensors():
    import torch
    with pytest.raises(TypeError):
        S.gather(torch.zeros(3, dtype=torch.int32), torch.zeros(4, 2))
    with pytest.raises(TypeError):
        S.build_fgram_table(torch.zeros((1, 2), dtype=torch.int32),
                            torch.zeros(1, dtype=torch.int32), torch.zeros(1, dtype=torch.int32))


def test_fgram_model_layout_and_argument_errors():
    L = S.scone.lib()
    E = S.scone.EINVAL
    n_par, total = ctypes.c_int64(), ctypes.c_int64()
    for d, h, f, nl, K in [(512, 8, 1024, 2, 7), (1024, 16, 4096, 6, 3), (2048, 16, 8192, 0, 5)]:
        assert L.scone_fgram_model_layout(d, h, f, nl, K, None, ctypes.byref(n_par),
                                          ctypes.byref(total)) == S.scone.OK
        assert n_par.value == 3 + 12 * nl
        offs = (ctypes.c_int64 * n_par.value)()
        assert L.scone_fgram_model_layout(d, h, f, nl, K, offs, None, None) == S.scone.OK
        sizes = [K * d] + [s for _ in range(nl) for s in
                           (d, d, 3 * d * d, 3 * d, d * d, d, d, d, f * d, f, d * f, d)] + [d, d]
        o = list(offs)
        assert o[0] == 0 and all(x % 128 == 0 for x in o)
        for k in range(len(o) - 1):   # each tensor fits before the next one starts
            assert o[k] + sizes[k] <= o[k + 1] < o[k] + sizes[k] + 128
        assert o[-1] + sizes[-1] <= total.value < o[-1] + sizes[-1] + 128
    # unsupported sizes: d not a multiple of 512, head width not 64/128, d_ff, K
    for d, h, f, nl, K in [(768, 12, 3072, 1, 3), (512, 16, 1024, 1, 3), (512, 8, 1000, 1, 3),
                           (512, 8, 1024, 1, 8), (512, 8, 1024, 1, 1), (512, 8, 1024, -1, 3),
                           (8192, 64, 1024, 1, 3)]:
        assert L.scone_fgram_model_layout(d, h, f, nl, K, None, None, None) == E
        assert L.scone_fgram_model_forward(None, None, None, 1, K, None, 10, None, d, h, f, nl,
                                           None, 10, None) == E
    # good sizes, bad pointers or counts: rejected before any device work
    assert L.scone_fgram_model_forward(None, None, None, 1, 3, None, 10, None, 512, 8, 1024, 1,
                                       None, 10, None) == E
    assert L.scone_fgram_model_forward(None, None, None, -1, 3, None, 10, None, 512, 8, 1024, 1,
                                       None, 10, None) == E
    assert L.scone_fgram_model_forward(None, None, None, 0, 3, None, 10, None, 512, 8, 1024, 1,
                                       None, 10, None) == S.scone.OK


def _fake(base: int):
    """A fake device address: the calls below reject aliasing before any
    device access, so no memory is behind it."""
    return ctypes.c_void_p(base)


def test_aliasing_outputs_are_rejected_before_any_device_work():
    """Outputs that share memory with an input (or another output) that other
    workgroups of the same launch still read are argument errors.  A call
    whose buffers do not alias gets past these checks and only then fails
    here, at its first HIP call (SCONE_EHIP: no GPU in this process)."""
    L = S.scone.lib()
    E, H = S.scone.EINVAL, S.scone.EHIP
    tbl = ctypes.create_string_buffer(64)          # stands in for a table handle
    B, T, R = 4, 256, 4096
    n = B * T
    tok, ids, ln = _fake(1 << 32), _fake(2 << 32), _fake(3 << 32)
    out, rows, cur = _fake(4 << 32), _fake(5 << 32), _fake(6 << 32)
    # scone_lookup: ids or lengths over the tokens, lengths over the ids
    assert L.scone_lookup(tbl, tok, B, T, 3, _fake((1 << 32) + 4 * n - 4), None, None) == E
    assert L.scone_lookup(tbl, tok, B, T, 3, ids, _fake((1 << 32) + 8), None) == E
    assert L.scone_lookup(tbl, tok, B, T, 3, ids, _fake((2 << 32) + 4 * n - 1), None) == E
    assert L.scone_lookup(tbl, tok, B, T, 3, ids, ln, None) == H
    # scone_tag: lengths over the tokens
    assert L.scone_tag(tbl, tok, B, T, 3, _fake(1 << 32), None, None) == E
    # scone_gather: output over the ids or over the row table
    assert L.scone_gather(ids, n, rows, 100, R, _fake((2 << 32) - n * R + 1), 0, None) == E
    assert L.scone_gather(ids, n, rows, 100, R, _fake((5 << 32) + 99 * R), 0, None) == E
    assert L.scone_gather(ids, n, rows, 100, R, out, 0, None) == H
    # scone_embed: output over tokens, ids over output, lengths over ids
    assert L.scone_embed(tbl, tok, B, T, 3, rows, 100, R, 0, _fake(1 << 32), ids, ln,
                         None) == E
    assert L.scone_embed(tbl, tok, B, T, 3, rows, 100, R, 0, out, _fake((4 << 32) + 64), ln,
                         None) == E
    assert L.scone_embed(tbl, tok, B, T, 3, rows, 100, R, 0, out, ids, _fake(2 << 32),
                         None) == E
    assert L.scone_embed(tbl, tok, B, T, 3, rows, 100, R, 0, out, ids, ln, None) == H
    # scone_embed_pipelined: every output against next_tokens, cur_ids and the
    # other outputs
    P = L.scone_embed_pipelined
    assert P(tbl, tok, B, T, 3, ids, ln, cur, n, rows, 100, R, 0, out, None) == H
    assert P(tbl, tok, B, T, 3, _fake(6 << 32), ln, cur, n, rows, 100, R, 0, out, None) == E
    assert P(tbl, tok, B, T, 3, ids, _fake(6 << 32), cur, n, rows, 100, R, 0, out, None) == E
    assert P(tbl, tok, B, T, 3, ids, ln, cur, n, rows, 100, R, 0, _fake(6 << 32), None) == E
    assert P(tbl, tok, B, T, 3, ids, ln, cur, n, rows, 100, R, 0,
             _fake((1 << 32) + 4 * n - 16), None) == E                      # out over tokens
    assert P(tbl, tok, B, T, 3, _fake((1 << 32) + 4), ln, cur, n, rows, 100, R, 0, out,
             None) == E                                                     # ids over tokens
    assert P(tbl, tok, B, T, 3, ids, ln, cur, n, rows, 100, R, 0, _fake((2 << 32) + 4),
             None) == E                                                     # out over next ids
    assert P(tbl, tok, B, T, 3, ids, _fake((4 << 32) + 7), cur, n, rows, 100, R, 0, out,
             None) == E                                                     # lengths over out
    # scone_decode_step: outputs against the context, lengths, new tokens, rows
    D = L.scone_decode_step
    ctx, clen, newt = _fake(7 << 32), _fake(8 << 32), _fake(9 << 32)
    assert D(tbl, ctx, clen, 4, newt, B, 3, rows, 100, R, 0, out, ids, ln, None) == H
    assert D(tbl, ctx, clen, 4, newt, B, 3, rows, 100, R, 0, _fake(7 << 32), ids, ln,
             None) == E
    assert D(tbl, ctx, clen, 4, newt, B, 3, rows, 100, R, 0, out, _fake(9 << 32), ln,
             None) == E
    assert D(tbl, ctx, clen, 4, newt, B, 3, rows, 100, R, 0, out, ids, _fake(8 << 32),
             None) == E
    assert D(tbl, ctx, _fake(9 << 32), 4, newt, B, 3, rows, 100, R, 0, out, ids, ln,
             None) == E


def test_decode_host_argument_errors():
    L = S.scone.lib()
    E = S.scone.EINVAL
    tbl = ctypes.create_string_buffer(64)
    D = L.scone_decode_step
    p = _fake(1 << 40)
    assert D(None, p, p, 4, p, 1, 3, p, 10, 16, 0, p, None, None, None) == E     # no table
    assert D(tbl, p, p, 4, p, -1, 3, p, 10, 16, 0, p, None, None, None) == E     # S < 0
    assert D(tbl, p, p, 4, p, 1, 0, p, 10, 16, 0, p, None, None, None) == E      # max_n < 1
    assert D(tbl, p, p, 4, p, 1, 3, p, 10, 0, 0, p, None, None, None) == E       # row_bytes
    assert D(tbl, p, p, 4, p, 1, 3, p, 10, 16, 2, p, None, None, None) == E      # placement
    assert D(tbl, p, p, 64, p, 1, 3, p, 10, 16, 0, p, None, None, None) == E     # ctx_cap > 63
    assert D(tbl, p, None, 4, p, 1, 3, p, 10, 16, 0, p, None, None, None) == E   # no ctx_len
    assert D(tbl, p, p, 4, p, 0, 3, p, 10, 16, 0, p, None, None, None) == S.scone.OK


def test_static_split_gather_checks_its_scratch_limit_on_the_host():
    """scone_gather_split_static refuses work beyond its fixed scratch before
    any device work (SCONE_ESCRATCH) and checks arguments like
    scone_gather_split; a call that fits gets past the checks and only then
    fails here, at its first HIP call."""
    L = S.scone.lib()
    F = L.scone_gather_split_static
    ids, near, far, out = _fake(1 << 32), _fake(2 << 32), _fake(3 << 32), _fake(4 << 32)
    R = 4096
    limit = S.scone.SPLIT_STATIC_BYTES
    fits = max(n for n in range(1, 20000) if L.scone_gather_split_workspace(n, R) <= limit)
    assert 7000 < fits < 8192
    assert F(ids, fits + 1, near, 10, far, 10, R, out, None, None) == S.scone.ESCRATCH
    assert F(ids, fits, near, 10, far, 10, R, out, None, None) == S.scone.EHIP
    assert F(ids, 0, near, 10, far, 10, R, out, None, None) == S.scone.OK
    assert F(ids, 5, near, 10, far, 10, 24, out, None, None) == S.scone.EINVAL   # width % 16
    assert F(None, 5, near, 10, far, 10, R, out, None, None) == S.scone.EINVAL
    assert F(ids, 5, near, 10, far, 10, R, _fake((1 << 32) + 8), None, None) == S.scone.EINVAL


def test_split_gather_rejects_workspace_and_count_aliasing():
    """scone_gather_split's workspace (the part the call uses) may not share
    memory with any input or output, and n_unique may not share memory with
    out or the ids; the static variant checks n_unique the same way.  A call
    whose buffers do not alias gets past the checks and only then fails here,
    at its first HIP call."""
    L = S.scone.lib()
    E, H = S.scone.EINVAL, S.scone.EHIP
    G, F = L.scone_gather_split, L.scone_gather_split_static
    n, R, nn, nf = 100, 4096, 10, 10
    ids, near, far, out = _fake(1 << 32), _fake(2 << 32), _fake(3 << 32), _fake(4 << 32)
    cnt, ws = _fake(5 << 32), _fake(6 << 32)
    need = L.scone_gather_split_workspace(n, R)
    assert need > n * R
    assert G(ids, n, near, nn, far, nf, R, out, ws, need, cnt, None) == H
    assert G(ids, n, near, nn, far, nf, R, out, ws, need - 16, cnt, None) == E  # too small
    for bad in ((1 << 32) - need + 16,            # workspace ends inside the ids
                (2 << 32) + 16 * (nn * R // 16 - 1),   # starts inside near_rows
                (3 << 32) - 16,                   # runs into far_rows
                (4 << 32) + 1024 * 16,            # starts inside out
                (5 << 32) - need + 16):           # ends inside n_unique
        assert G(ids, n, near, nn, far, nf, R, out, _fake(bad), need, cnt, None) == E, bad
    # n_unique inside out or inside the ids, for both entry points
    for c in (_fake((4 << 32) + 4096), _fake((1 << 32) + 8)):
        assert G(ids, n, near, nn, far, nf, R, out, ws, need, c, None) == E
        assert F(ids, n, near, nn, far, nf, R, out, c, None) == E
    assert F(ids, n, near, nn, far, nf, R, out, cnt, None) == H


def test_discovery_rejects_shared_buffers():
    """No two of the corpus, the three outputs and the workspace may share
    memory; a call whose buffers are apart gets past the checks and only
    then fails here, at its first HIP call."""
    L = S.scone.lib()
    E, H = S.scone.EINVAL, S.scone.EHIP
    D = L.scone_discover_fgrams
    B, T, K, Sn = 4, 1000, 3, 500
    tok, fg, ln, cnt, ws = (_fake(k << 32) for k in (1, 2, 3, 4, 5))
    need = L.scone_discover_workspace(B, T, K)
    assert need > 0
    nf = ctypes.c_int64(-1)
    assert D(tok, B, T, K, 5, Sn, fg, ln, cnt, ctypes.byref(nf), ws, need, None) == H
    assert nf.value == 0
    assert D(tok, B, T, K, 5, Sn, fg, _fake((1 << 32) + 4 * B * T - 4), cnt, ctypes.byref(nf),
             ws, need, None) == E                                      # lengths ends in corpus
    assert D(tok, B, T, K, 5, Sn, _fake((3 << 32) - 4 * Sn * K + 4), ln, cnt, ctypes.byref(nf),
             ws, need, None) == E                                      # fgrams runs into lengths
    assert D(tok, B, T, K, 5, Sn, fg, ln, _fake((3 << 32) + 4 * Sn - 4), ctypes.byref(nf),
             ws, need, None) == E                                      # counts over lengths
    assert D(tok, B, T, K, 5, Sn, fg, ln, cnt, ctypes.byref(nf), _fake((2 << 32) + 256), need,
             None) == E                                                # workspace in fgrams
    assert D(tok, B, T, K, 5, Sn, fg, ln, cnt, ctypes.byref(nf),
             _fake(((1 << 32) - need + 512) // 256 * 256), need, None) == E  # into corpus


def test_fgram_model_rejects_rows_over_its_inputs():
    """The output table may not share memory with the f-grams, lengths, row
    ids or parameters (the token rows may lie inside it); a call whose
    buffers are apart gets past the checks and only then fails here, at its
    first allocation."""
    L = S.scone.lib()
    E = S.scone.EINVAL
    Fw = L.scone_fgram_model_forward
    n, K, V, d, heads, dff, layers, n_rows = 100, 3, 50, 512, 8, 1024, 1, 200
    total = ctypes.c_int64()
    assert L.scone_fgram_model_layout(d, heads, dff, layers, K, None, None,
                                      ctypes.byref(total)) == S.scone.OK
    fg, ln, ids, prm, rows = (_fake(k << 32) for k in (1, 2, 3, 4, 5))
    tok = _fake((5 << 32))                       # the unified table: T inside rows
    rb = n_rows * d * 2

    def call(fg=fg, ln=ln, ids=ids, prm=prm, rows=rows):
        return Fw(fg, ln, ids, n, K, tok, V, prm, d, heads, dff, layers, rows, n_rows, None)
    assert call() not in (E, S.scone.OK)         # past the checks: fails allocating
    assert call(rows=_fake((1 << 32) - rb + 16)) == E           # rows end in the f-grams
    assert call(ln=_fake((5 << 32) + rb - 4)) == E              # lengths at the table's end
    assert call(ids=_fake((5 << 32) + 1024)) == E               # row ids inside the table
    assert call(prm=_fake((5 << 32) - 2 * total.value + 16)) == E  # params run into it


def test_counted_lookup_host_checks():
    """scone_lookup_counted needs its counter, and the counter may not share
    memory with the tokens or the outputs; otherwise it checks like
    scone_lookup and gets as far as its first HIP call."""
    L = S.scone.lib()
    E, H = S.scone.EINVAL, S.scone.EHIP
    C = L.scone_lookup_counted
    tbl = ctypes.create_string_buffer(64)
    B, T = 4, 256
    n = B * T
    tok, ids, ln, cnt = _fake(1 << 32), _fake(2 << 32), _fake(3 << 32), _fake(4 << 32)
    assert C(tbl, tok, B, T, 3, ids, ln, None, None) == E                 # no counter
    assert C(None, tok, B, T, 3, ids, ln, cnt, None) == E                 # no table
    assert C(tbl, tok, B, T, 0, ids, ln, cnt, None) == E                  # max_n < 1
    assert C(tbl, tok, B, T, 3, ids, ln, _fake((1 << 32) + 4 * n - 8), None) == E  # in tokens
    assert C(tbl, tok, B, T, 3, ids, ln, _fake((2 << 32) + 64), None) == E         # in ids
    assert C(tbl, tok, B, T, 3, ids, ln, _fake((3 << 32) + n - 1), None) == E      # in lengths
    assert C(tbl, tok, B, T, 3, _fake((1 << 32) + 4), ln, cnt, None) == E          # ids over tokens
    assert C(tbl, tok, B, T, 3, ids, ln, cnt, None) == H
    assert C(tbl, tok, 0, T, 3, ids, ln, cnt, None) == S.scone.OK
