"""The scoring entry point that allocates nothing (eogp_score_topk_noalloc)
against the workspace entry point (eogp_score_topk) and the oracle, through
the C ABI: two calls in a row on the same GPU (the second with a smaller
input, so it reuses the scratch the first one filled), and a call whose
workspace would exceed the scratch array, rejected before anything runs."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_37842_amd import eogp as E

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def store(seed, N, ks, Q):
    g = np.random.default_rng(seed)
    codes = g.integers(0, 256, size=(N, sum(k // 8 for k in ks)), dtype=np.uint8)
    scales = np.exp(g.standard_normal((N, len(ks)))).astype(np.float16).view(np.uint16)
    Y = g.standard_normal((Q, sum(ks))).astype(np.float32)
    return codes, scales, Y


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


@pytest.mark.parametrize("first,second", [
    ((3000, [128, 512, 64], 20, 37), (700, [256], 5, 10)),       # several modules, then one
    ((70_000, [1024], 33, 100), (1000, [64, 64], 3, 7)),          # one module, then several
])
def test_noalloc_matches_workspace_entry_point_and_oracle(first, second):
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    E.load()
    for i, (N, ks, Q, topk) in enumerate((first, second)):
        print(f"[no-alloc] call {i}: N={N} ks={ks} Q={Q} topk={topk}", flush=True)
        codes, scales, Y = store(N + 13 * i, N, ks, Q)
        c, s, y = dev(codes), dev(scales.view(np.int16)), dev(Y)
        idx_w, sc_w, full_w = E.eogp_score_topk(c, s, ks, y, topk, full_scores=True)
        idx_n = torch.empty((Q, topk), dtype=torch.int64, device=DEV)
        sc_n = torch.empty((Q, topk), dtype=torch.float32, device=DEV)
        full_n = torch.empty((Q, N), dtype=torch.float32, device=DEV)
        E.eogp_score_topk_noalloc(c, s, ks, y, topk, idx_n, sc_n, full_scores=full_n)
        torch.cuda.synchronize()
        assert torch.equal(idx_n, idx_w) and torch.equal(sc_n, sc_w)
        assert torch.equal(full_n, full_w)
        rows = np.sort(np.random.default_rng(i).choice(N, min(N, 512), replace=False))
        ref = O.score(codes[rows], scales[rows], ks, Y)
        assert np.array_equal(full_n.cpu().numpy()[:, rows], ref.astype(np.float32))
        if N <= 5000:
            oi, ov = O.topk(O.score(codes, scales, ks, Y), topk)
            assert np.array_equal(idx_n.cpu().numpy(), oi)
            assert np.array_equal(sc_n.cpu().numpy(), ov)


def test_noalloc_rejects_calls_beyond_its_scratch():
    """48 modules x 8,192 bits need 64 bytes per stored row and module for
    each 16 queries; 50,000 rows exceed the 128 MiB array: invalid argument,
    and the outputs stay untouched."""
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    N, ks, Q, topk = 50_000, [8192] * 48, 16, 10
    assert E.eogp_score_topk_workspace_size(N, Q, ks, topk) > (128 << 20)
    codes = torch.zeros((N, 48 * 1024), dtype=torch.uint8, device=DEV)
    scales = torch.zeros((N, 48), dtype=torch.int16, device=DEV)
    Y = torch.zeros((Q, 48 * 8192), dtype=torch.float32, device=DEV)
    idx = torch.full((Q, topk), 7, dtype=torch.int64, device=DEV)
    sc = torch.full((Q, topk), 3.0, dtype=torch.float32, device=DEV)
    with pytest.raises(E.EogpError) as ei:
        E.eogp_score_topk_noalloc(codes, scales, ks, Y, topk, idx, sc)
    assert ei.value.status == -1 and "scratch" in str(ei.value)
    torch.cuda.synchronize()
    assert torch.all(idx == 7) and torch.all(sc == 3.0)
