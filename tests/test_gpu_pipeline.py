"""The pipelined step (scone_embed_pipelined: the lookup of the next batch and
the gather of the current batch in one launch) against the oracle.

A stream of batches of different shapes, an empty one among them, runs
through the documented schedule (a lookup-only first step, steady steps, a
gather-only last step) with the ids alternating between two buffers; every
step's ids and match lengths and every batch's rows are compared with the
oracle's lookup and memcpy gather.  Cases cover both slot widths, every lane
group (windows 1 to 7), every one-wavefront row width (1, 2, 4, 8 KiB) and
the two-launch fallback (odd and misaligned rows, a table without rows)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2502_01637_amd as S
from gpu_util import as_bytes, build_gpu, dev, device_rows
from workloads import CONFIGS, make_workload, query_batches, scaled

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _clean_error_word():
    S.check()
    yield
    assert S.check() == S.scone.OK, "a test left a device error behind"


def case_config(case):
    c2, c3, tiny = CONFIGS["c2_1m"], CONFIGS["c3_10m_k5"], CONFIGS["tiny"]
    return {
        "c2_2k": scaled(c2, n_fgrams=20_000, B=3, T=1500),                 # slots 16, G 2, 2 KiB
        "c3_4k": scaled(c3, n_fgrams=40_000, B=2, T=2100),                 # slots 16, G 4, 4 KiB
        "c3_win2": scaled(c3, n_fgrams=40_000, B=2, T=900, max_n=2, d=512),  # G 1, 1 KiB
        "k7_8k": scaled(tiny, V=40, n_fgrams=3000, max_len=7, max_n=7, B=3, T=700,
                        d=2048),                                           # slots 32, G 8, 8 KiB
        "k6_win4": scaled(tiny, V=60, n_fgrams=4000, max_len=6, max_n=4, B=2, T=800,
                          d=1024, dtype="bf16"),                           # slots 32, G 4, 2 KiB
        "win1": scaled(tiny, max_n=1, d=256),                              # no probes, 1 KiB
        "odd_rows": scaled(tiny, d=7, B=5, T=333),                         # 28-byte rows
    }[case]


def stream_batches(w, n_rows_cap=None):
    """Batches of several shapes: the workload's own, a ragged one, an empty
    one and a fresh full one."""
    b = query_batches(w, 3)
    return [b[0], np.ascontiguousarray(b[1][:1, :517]), b[1][:, :0].copy(), b[2]]


def run_stream(tb, batches, max_n, rows, check_step=None):
    """The pipelined schedule with two alternating id buffers.  Returns the
    per-batch outputs; check_step(k, ids, lens) sees batch k's ids right after
    the step that looked them up."""
    cap = max(X.size for X in batches)
    ids_buf = [torch.empty(cap, dtype=torch.int32, device="cuda") for _ in range(2)]
    len_buf = [torch.empty(cap, dtype=torch.int8, device="cuda") for _ in range(2)]
    Xd = [dev(X) for X in batches]
    outs = [None] * len(batches)

    def views(k):
        n = batches[k].size
        return ids_buf[k % 2][:n].view(batches[k].shape), len_buf[k % 2][:n].view(batches[k].shape)

    ids0, len0 = views(0)
    assert S.embed_pipelined(tb, Xd[0], max_n, ids0, None, rows, next_len=len0) is None
    if check_step:
        check_step(0, ids0, len0)
    for k in range(1, len(batches) + 1):
        cur, _ = views(k - 1)
        if k < len(batches):
            nid, nlen = views(k)
            outs[k - 1] = S.embed_pipelined(tb, Xd[k], max_n, nid, cur, rows, next_len=nlen)
            if check_step:
                check_step(k, nid, nlen)
        else:
            outs[k - 1] = S.embed_pipelined(tb, None, max_n, None, cur, rows)
    return outs


@pytest.mark.parametrize("case", ["c2_2k", "c3_4k", "c3_win2", "k7_8k", "k6_win4", "win1",
                                  "odd_rows"])
def test_pipelined_stream_matches_oracle(case):
    cfg = case_config(case)
    w = make_workload(cfg)
    o = oracle.OracleTable(w.fgrams, w.lengths, w.ids)
    tb = build_gpu(w.fgrams, w.lengths, w.ids)
    E = device_rows(cfg)
    table = E.cpu().view(torch.uint8).numpy().reshape(cfg.n_rows, -1)
    batches = stream_batches(w)
    exp = [o.lookup(X, cfg.max_n) for X in batches]

    def check_step(k, ids, lens):
        np.testing.assert_array_equal(ids.cpu().numpy(), exp[k][0], err_msg=f"{case} batch {k}")
        np.testing.assert_array_equal(lens.cpu().numpy(), exp[k][1], err_msg=f"{case} batch {k}")

    outs = run_stream(tb, batches, cfg.max_n, E, check_step)
    S.check_ok()
    for k, (out, (exp_ids, _)) in enumerate(zip(outs, exp)):
        assert tuple(out.shape) == batches[k].shape + (cfg.d,)
        assert as_bytes(out).tobytes() == oracle.gather(exp_ids, table).tobytes(), (case, k)


def test_pipelined_misaligned_rows_take_the_fallback():
    cfg = scaled(CONFIGS["tiny"], d=256, B=3, T=600)          # 1 KiB rows, 4-byte aligned
    w = make_workload(cfg)
    o = oracle.OracleTable(w.fgrams, w.lengths, w.ids)
    tb = build_gpu(w.fgrams, w.lengths, w.ids)
    base = torch.empty(cfg.n_rows * cfg.d + 1, dtype=torch.float32, device="cuda")
    E = base[1:].view(cfg.n_rows, cfg.d)
    E.copy_(device_rows(cfg))
    table = E.cpu().view(torch.uint8).numpy()
    batches = stream_batches(w)
    outs = run_stream(tb, batches, cfg.max_n, E)
    S.check_ok()
    for k, X in enumerate(batches):
        exp_ids, _ = o.lookup(X, cfg.max_n)
        assert as_bytes(outs[k]).tobytes() == oracle.gather(exp_ids, table).tobytes(), k


def raises_code(code, fn, *a, **kw):
    with pytest.raises(S.SconeError) as e:
        fn(*a, **kw)
    assert e.value.code == code, (e.value.code, code)


def test_pipelined_errors_and_overlap():
    fg = np.array([[1, 2, -1], [2, 3, 4]], dtype=np.int32)
    tb = build_gpu(fg, [2, 3], [10, 11])
    E = torch.arange(12 * 512, dtype=torch.int32, device="cuda").view(12, 512)  # 2 KiB rows
    Xn = np.array([[1, 2, 3, 4, 9]], dtype=np.int32)
    X = dev(Xn)
    exp_ids = oracle.OracleTable(fg, [2, 3], [10, 11]).lookup(Xn, 3)[0].ravel().tolist()
    assert exp_ids == [1, 10, 3, 11, 9]
    buf = torch.zeros(64, dtype=torch.int32, device="cuda")
    cur = dev(np.array([10, 11, 0], dtype=np.int32))
    # the same buffer, or overlapping ranges, for the next and current ids
    raises_code(S.scone.EINVAL, S.embed_pipelined, tb, X, 3, buf[:5], buf[:5], E)
    raises_code(S.scone.EINVAL, S.embed_pipelined, tb, X, 3, buf[:5], buf[4:9], E)
    raises_code(S.scone.EINVAL, S.embed_pipelined, tb, X, 3, buf[10:15], buf[4:11], E)
    raises_code(S.scone.EINVAL, S.embed_pipelined, tb, X, 3, buf[:5], buf[20:23], E,
                next_len=buf[21:23].view(torch.int8)[:5])
    raises_code(S.scone.EINVAL, S.embed_pipelined, tb, X, 0, buf[:5], None, E)
    # adjacent ranges are fine
    buf[5:8].copy_(cur)
    out = S.embed_pipelined(tb, X, 3, buf[:5], buf[5:8], E)
    S.check_ok()
    assert buf[:5].cpu().tolist() == exp_ids
    assert torch.equal(out, E[[10, 11, 0]])
    # bad ids in the current batch: zero rows and SCONE_EROW, while the lookup
    # half of the same launch stays right
    ids = torch.empty(5, dtype=torch.int32, device="cuda")
    out = S.embed_pipelined(tb, X, 3, ids, dev(np.array([3, 12, -1, 11], dtype=np.int32)), E)
    assert S.check() == S.scone.EROW
    assert ids.cpu().tolist() == exp_ids
    got = out.cpu()
    assert torch.equal(got[0], E[3].cpu()) and torch.equal(got[3], E[11].cpu())
    assert (got[1] == 0).all() and (got[2] == 0).all()
    # a bad token in the next batch: SCONE_ETOKEN, the gather half stays right
    Xbad = dev(np.array([[1, 2, 70000, -3]], dtype=np.int32))
    ids4 = torch.empty(4, dtype=torch.int32, device="cuda")
    out = S.embed_pipelined(tb, Xbad, 3, ids4, cur, E)
    assert S.check() == S.scone.ETOKEN
    assert ids4.cpu().tolist()[:2] == [1, 10]
    assert torch.equal(out, E[[10, 11, 0]])
    # a table without rows: every id is out of range
    out = S.embed_pipelined(tb, X, 3, ids, cur, E[:0])
    assert S.check() == S.scone.EROW
    assert (out == 0).all() and ids.cpu().tolist() == exp_ids
    # nothing to do
    assert S.embed_pipelined(tb, None, 3, None, None, E) is None
    S.check_ok()


@pytest.mark.parametrize("d", [1024, 2048, 4096])   # 2, 4 and 8 KiB rows (whole, 2- and 4-way split)
def test_split_row_copies_zero_bad_rows(d):
    """Rows of 4 and 8 KiB are copied in parts by several wavefronts: every
    part of a row with a bad id is zeroed, the error is raised, and the other
    rows are exact, in the standalone gather and in the pipelined step."""
    rng = np.random.default_rng(d)
    n_rows, n_tok = 97, 777
    E = torch.from_numpy(rng.integers(-2**31, 2**31, size=(n_rows, d // 2), dtype=np.int64)
                         .astype(np.int32)).cuda()
    ids_np = rng.integers(0, n_rows, size=n_tok).astype(np.int32)
    bad = rng.choice(n_tok, 40, replace=False)
    ids_np[bad[:20]] = n_rows + rng.integers(0, 1000, 20)
    ids_np[bad[20:]] = -1 - rng.integers(0, 1000, 20)
    exp = E.cpu().numpy()[np.clip(ids_np, 0, n_rows - 1)]
    exp[bad] = 0
    ids = dev(ids_np)
    out = S.gather(ids, E)
    assert S.check() == S.scone.EROW
    assert np.array_equal(out.cpu().numpy(), exp)
    fg = np.array([[1, 2, -1]], dtype=np.int32)
    tb = build_gpu(fg, [2], [5])
    X = dev(np.arange(40, dtype=np.int32).reshape(2, 20) % 7)
    nxt = torch.empty((2, 20), dtype=torch.int32, device="cuda")
    outp = S.embed_pipelined(tb, X, 3, nxt, ids, E)
    assert S.check() == S.scone.EROW
    assert np.array_equal(outp.cpu().numpy(), exp)
    exp_n = oracle.OracleTable(fg, [2], [5]).lookup(X.cpu().numpy(), 3)[0]
    assert np.array_equal(nxt.cpu().numpy(), exp_n)
