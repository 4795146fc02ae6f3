"""The allocation-free split gather (scone_gather_split_static), called through
the C ABI, against scone_gather_split with a caller workspace and against the
oracle's gather over the concatenated table: two calls in a row on the same
GPU scratch, the second one smaller, then a request beyond the scratch."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2502_01637_amd as S

pytestmark = pytest.mark.gpu

D = 2048                      # bf16 elements per row: 4 KiB rows
N_NEAR, N_FAR = 3000, 60000


def static_split(ids, near, far, out, n_unique):
    """scone_gather_split_static through ctypes, on torch's current stream."""
    L = S.scone.lib()
    return L.scone_gather_split_static(
        ctypes.c_void_p(ids.data_ptr()), ids.numel(), ctypes.c_void_p(near.data_ptr()),
        near.shape[0], ctypes.c_void_p(far.device_ptr), far.n_rows, far.row_bytes,
        ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(n_unique.data_ptr()),
        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))


@pytest.fixture(scope="module")
def tables():
    g = torch.Generator(device="cuda")
    g.manual_seed(11)
    near = torch.randn((N_NEAR, D), generator=g, device="cuda").to(torch.bfloat16)
    far = S.HostRows(N_FAR, (D,), torch.bfloat16)
    stage = torch.randn((N_FAR, D), generator=g, device="cuda").to(torch.bfloat16)
    far.tensor().copy_(stage.cpu())
    concat = torch.cat([near.cpu(), far.tensor()]).view(torch.uint8).numpy()
    yield near, far, concat
    far.close()


def batch(rng, n_tok, far_lo, far_hi):
    """Near ids, far ids in [far_lo, far_hi) with repeats (so the dedupe set
    has work), shuffled."""
    n_far_ids = n_tok * 2 // 3
    pool = rng.integers(N_NEAR + far_lo, N_NEAR + far_hi, size=max(1, n_far_ids // 3))
    ids = np.concatenate([rng.choice(pool, n_far_ids),
                          rng.integers(0, N_NEAR, n_tok - n_far_ids)]).astype(np.int32)
    rng.shuffle(ids)
    return ids


def test_static_split_matches_workspace_split_two_calls(tables):
    near, far, concat = tables
    rng = np.random.default_rng(5)
    # the first call nearly fills the scratch; the second, smaller one uses
    # far rows the first never staged
    for n_tok, lo, hi in ((7800, 0, 30000), (1500, 30000, 60000)):
        assert S.split_workspace_bytes(n_tok, 2 * D) <= S.scone.SPLIT_STATIC_BYTES
        ids_np = batch(rng, n_tok, lo, hi)
        ids = torch.from_numpy(ids_np).cuda()
        ws = torch.empty(S.split_workspace_bytes(n_tok, 2 * D), dtype=torch.uint8,
                         device="cuda")
        nu_ref = torch.zeros(1, dtype=torch.int32, device="cuda")
        ref = S.gather_split(ids, near, far, ws, n_unique=nu_ref)
        out = torch.full((n_tok, D), float("nan"), dtype=torch.bfloat16, device="cuda")
        nu = torch.full((1,), -1, dtype=torch.int32, device="cuda")
        assert static_split(ids, near, far, out, nu) == S.scone.OK
        S.check_ok()
        assert torch.equal(out.view(torch.int16), ref.view(torch.int16)), n_tok
        assert int(nu.item()) == int(nu_ref.item()) == len(np.unique(ids_np[ids_np >= N_NEAR]))
        exp = oracle.gather(ids_np, concat)
        assert out.cpu().view(torch.uint8).numpy().tobytes() == exp.tobytes(), n_tok


def test_static_split_beyond_scratch_launches_nothing(tables):
    near, far, _ = tables
    n_tok = 8200                                     # 4 KiB rows: just over 32 MiB
    assert S.split_workspace_bytes(n_tok, 2 * D) > S.scone.SPLIT_STATIC_BYTES
    ids = torch.zeros(n_tok, dtype=torch.int32, device="cuda")
    out = torch.full((n_tok, D), 3.0, dtype=torch.bfloat16, device="cuda")
    nu = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    assert static_split(ids, near, far, out, nu) == S.scone.ESCRATCH
    torch.cuda.synchronize()
    assert bool((out == 3.0).all()) and int(nu.item()) == -1


def test_static_split_in_a_captured_graph(tables):
    """The allocation-free call captured in a HIP graph (its use case: it
    allocates nothing and launches kernels only) and replayed three times,
    with other work on the same scratch between the replays; every replay
    equals the eager result."""
    near, far, concat = tables
    rng = np.random.default_rng(9)
    n_tok = 2048
    ids_np = batch(rng, n_tok, 0, N_FAR)
    ids = torch.from_numpy(ids_np).cuda()
    other = torch.from_numpy(batch(rng, 3000, 0, N_FAR)).cuda()
    eager = torch.empty((n_tok, D), dtype=torch.bfloat16, device="cuda")
    nu = torch.zeros(1, dtype=torch.int32, device="cuda")
    assert static_split(ids, near, far, eager, nu) == S.scone.OK
    S.check_ok()
    exp = oracle.gather(ids_np, concat)
    assert eager.cpu().view(torch.uint8).numpy().tobytes() == exp.tobytes()
    out = torch.zeros_like(eager)
    nu_g = torch.zeros(1, dtype=torch.int32, device="cuda")
    scratch_out = torch.empty((3000, D), dtype=torch.bfloat16, device="cuda")
    nu_o = torch.zeros(1, dtype=torch.int32, device="cuda")
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            assert static_split(ids, near, far, out, nu_g) == S.scone.OK
    torch.cuda.current_stream().wait_stream(s)
    for r in range(3):
        out.zero_()
        # eager work that reuses the same scratch between replays
        assert static_split(other, near, far, scratch_out, nu_o) == S.scone.OK
        g.replay()
        torch.cuda.synchronize()
        S.check_ok()
        assert torch.equal(out.view(torch.int16), eager.view(torch.int16)), r
        assert int(nu_g.item()) == int(nu.item()), r
