"""GPU parity: every C-ABI entry point against the fp64 oracle on the same
seeded inputs.

Bars (stated per test): bit-exact for integer/byte/index work (selection,
codes from given coordinates, scores and top-k from given codes); relative
error per example-module row, ||gpu - oracle|| / ||oracle||, at most 1e-3 for
fp32 inputs in accurate mode and 2e-2 for bf16 inputs; sign bits of the full
pipeline identical except where |x| < 1e-3 * rms(x) of the oracle row.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_37842_amd import eogp as E
from paper_2609_37842_amd import synth as S
from tiled_helpers import rows_from_tiled, tiled_from_rows

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    E.load()
    yield


def d(x, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(x)).to(DEV)
    return t if dtype is None else t.to(dtype)


def rel_rows(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    num = np.linalg.norm(a - b, axis=-1)
    den = np.linalg.norm(b, axis=-1)
    return num / np.maximum(den, 1e-300)


def random_problem(seed, N, T, d_in, d_out, m, lens_lo=None, nan_masked=True):
    g = np.random.default_rng(seed)
    a = (g.standard_normal((N, T, d_in)) * np.sqrt(g.lognormal(0, 1, d_in))).astype(np.float32)
    ds = (0.01 * g.standard_normal((N, T, d_out))).astype(np.float32)
    lo = T if lens_lo is None else lens_lo
    lens = g.integers(lo, T + 1, size=N)
    mask = S.prefix_mask(lens, T)
    QA = S.haar_orthogonal(g, d_in).astype(np.float32)
    QS = S.haar_orthogonal(g, d_out).astype(np.float32)
    lam = (g.lognormal(0, 1, d_out)[:, None] * g.lognormal(0, 1, d_in)[None, :]
           * np.exp(0.25 * g.standard_normal((d_out, d_in))) * 1e-3).astype(np.float32)
    if nan_masked:
        a = S.fill_masked(a, mask)
        ds = S.fill_masked(ds, mask)
    return a, ds, mask, QA, QS, lam


def oracle_Z(a, ds, mask, QA, QS, lam, damping, m):
    ret = O.select_retained(lam, damping, m)
    return O.first_stage_batch(a, ds, mask, QA, QS, ret), ret


# ---------------------------------------------------------------------------
# One-bit encoding
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("k", [64, 128, 100, 8192, 13, 16384, 32768])
def test_sign_pack_bit_exact(k):
    say(f"[sign_pack] k={k}")
    g = np.random.default_rng(k)
    X = g.standard_normal((37, k)).astype(np.float32)
    X[0, :5] = [0.0, -0.0, 1e-30, -1e-30, 0.0]
    X[1, :] = 0.0
    codes, scales = E.eogp_sign_pack(d(X))
    torch.cuda.synchronize()
    oc, os_ = O.encode(X)
    assert np.array_equal(codes.cpu().numpy(), oc)
    assert np.array_equal(scales.cpu().numpy().view(np.uint16)[:, 0], os_)


def test_sign_pack_into_multi_module_rows():
    say("[sign_pack] strided rows")
    g = np.random.default_rng(5)
    ks = [128, 64, 256]
    N = 19
    row = sum(k // 8 for k in ks)
    codes = torch.zeros((N, row + 8), dtype=torch.uint8, device=DEV)
    scales = torch.zeros((N, len(ks)), dtype=torch.int16, device=DEV)
    Xs = [g.standard_normal((N, k)).astype(np.float32) * (u + 1) for u, k in enumerate(ks)]
    off = 0
    for u, (k, X) in enumerate(zip(ks, Xs)):
        E.eogp_sign_pack(d(X), codes[:, off:off + k // 8], scales[:, u:u + 1])
        off += k // 8
    torch.cuda.synchronize()
    c = codes.cpu().numpy()
    s = scales.cpu().numpy().view(np.uint16)
    off = 0
    for u, (k, X) in enumerate(zip(ks, Xs)):
        oc, os_ = O.encode(X)
        assert np.array_equal(c[:, off:off + k // 8], oc)
        assert np.array_equal(s[:, u], os_)
        off += k // 8
    assert np.all(c[:, row:] == 0)


def test_sign_pack_tiled_layout():
    """Three modules (512, 1024 and 2,048 bits) packed into a tiled store of
    77 rows written in two row ranges; converted back to row-major by the
    layout's definition, codes and scales equal the oracle's bit for bit."""
    say("[sign_pack] tiled")
    g = np.random.default_rng(512)
    ks, N = [512, 1024, 2048], 77
    S_row = sum(ks) // 512
    store = torch.zeros(E.tiled_store_bytes(N, ks), dtype=torch.uint8, device=DEV)
    scales = torch.zeros((N, len(ks)), dtype=torch.int16, device=DEV)
    Xs = [g.standard_normal((N, k)).astype(np.float32) for k in ks]
    Xs[0][3, :7] = [0.0, -0.0, 1e-30, -1e-30, 0.0, -1.0, 2.0]
    step0 = 0
    for u, (k, X) in enumerate(zip(ks, Xs)):
        for r0, r1 in ((0, 40), (40, N)):
            E.eogp_sign_pack_tiled(d(X[r0:r1]), store, r0, S_row, step0, scales[r0:r1, u:u + 1])
        step0 += k // 512
    torch.cuda.synchronize()
    rows = rows_from_tiled(store.cpu().numpy(), S_row)[:N]
    off = 0
    sc = scales.cpu().numpy().view(np.uint16)
    for u, (k, X) in enumerate(zip(ks, Xs)):
        oc, os_ = O.encode(X)
        assert np.array_equal(rows[:, off:off + k // 8], oc)
        assert np.array_equal(sc[:, u], os_)
        off += k // 8


@pytest.mark.parametrize("N,ks,Q,topk", [
    (5000, [16384], 16, 100),          # one module
    (3000, [512, 1024, 512], 20, 37),  # several modules (ranges split across workgroups)
    (19, [1024], 5, 10),               # less than one tile, fewer rows than topk
    (600_000, [512], 16, 100),         # many blocks per workgroup
])
def test_score_topk_tiled_layout(N, ks, Q, topk):
    """Scores and top-k of a tiled store equal the oracle's (and the
    row-major entry point's) for the same bits."""
    say(f"[score] tiled N={N} ks={ks} Q={Q}")
    codes, scales, Y = random_store(N + 99, N, ks, Q)
    tiled = d(tiled_from_rows(codes))
    idx, sc, full = E.eogp_score_topk_tiled(tiled, d(scales.view(np.int16)), N, ks, d(Y), topk,
                                            full_scores=True)
    idx_r, sc_r, full_r = E.eogp_score_topk(d(codes), d(scales.view(np.int16)), ks, d(Y), topk,
                                            full_scores=True)
    torch.cuda.synchronize()
    assert torch.equal(full, full_r) and torch.equal(idx, idx_r) and torch.equal(sc, sc_r)
    rows = np.sort(np.random.default_rng(N).choice(N, min(N, 2000), replace=False))
    ref = O.score(codes[rows], scales[rows], ks, Y)
    assert np.array_equal(full.cpu().numpy()[:, rows], ref.astype(np.float32))
    if N <= 5000:
        oi, ov = O.topk(O.score(codes, scales, ks, Y), topk)
        assert np.array_equal(idx.cpu().numpy(), oi)
        assert np.array_equal(sc.cpu().numpy(), ov)


# ---------------------------------------------------------------------------
# Second stage
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("p_dtype,prec,tol", [
    (torch.float32, E.PREC_ACCURATE, 1e-5),
    (torch.float16, E.PREC_ACCURATE, 1e-5),
    (torch.float16, E.PREC_FAST, 1e-3),
    (torch.bfloat16, E.PREC_ACCURATE, 1e-5),
    (torch.bfloat16, E.PREC_FAST, 2e-2),
    (torch.float32, E.PREC_FAST, 2e-2),
])
def test_pca_project(p_dtype, prec, tol):
    say(f"[pca] {p_dtype} prec={prec}")
    g = np.random.default_rng(7)
    N, m, k = 300, 1000, 200          # several tiles plus ragged tails in every dim
    Z = g.standard_normal((N, m)).astype(np.float32)
    P = S.haar_orthogonal(g, m)[:, :k]
    Pt = torch.from_numpy(np.ascontiguousarray(P.T).astype(np.float32)).to(DEV).to(p_dtype)
    X = E.eogp_pca_project(d(Z), Pt, prec=prec)
    torch.cuda.synchronize()
    P_used = Pt.float().cpu().numpy().astype(np.float64).T      # P exactly as stored
    ref = O.pca_project(Z, P_used)
    err = rel_rows(X.cpu().numpy(), ref)
    say(f"   max rel {err.max():.2e}")
    assert err.max() <= tol


def test_pca_project_leading_dims_and_empty():
    g = np.random.default_rng(8)
    Zbig = torch.from_numpy(g.standard_normal((40, 300)).astype(np.float32)).to(DEV)
    Z = Zbig[:, :256]                                   # ldz = 300
    P = S.haar_orthogonal(g, 256)[:, :64]
    Pt = torch.from_numpy(np.ascontiguousarray(P.T).astype(np.float32)).to(DEV).half()
    Xbig = torch.full((40, 70), 7.0, device=DEV)
    E.eogp_pca_project(Z, Pt, X=Xbig[:, :64], prec=E.PREC_ACCURATE)
    torch.cuda.synchronize()
    ref = O.pca_project(Z.cpu().numpy(), Pt.float().cpu().numpy().T)
    assert rel_rows(Xbig[:, :64].cpu().numpy(), ref).max() < 1e-5
    assert torch.all(Xbig[:, 64:] == 7.0)
    empty = E.eogp_pca_project(torch.empty((0, 256), device=DEV), Pt)
    assert empty.shape == (0, 64)


# ---------------------------------------------------------------------------
# Selection (plan)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("d_out,d_in,m", [(64, 64, 512), (130, 97, 1000), (3, 5, 15), (300, 200, 1)])
def test_plan_selection_bit_exact(d_out, d_in, m):
    say(f"[plan] {d_out}x{d_in} m={m}")
    g = np.random.default_rng(d_out * 1000 + d_in)
    lam = g.lognormal(0, 1, (d_out, d_in)).astype(np.float32)
    QA = S.haar_orthogonal(g, d_in).astype(np.float32)
    QS = S.haar_orthogonal(g, d_out).astype(np.float32)
    damping = 0.05
    plan = E.eogp_plan_create(d(lam), damping, m, d(QA), d(QS))
    flat, w = plan.retained()
    torch.cuda.synchronize()
    ret = O.select_retained(lam, damping, m)
    assert np.array_equal(flat.cpu().numpy().astype(np.int64), ret.flat)
    assert np.array_equal(w.cpu().numpy(), ret.w.astype(np.float32))
    assert plan.n_rows == np.unique(ret.j).size
    assert plan.n_cols == np.unique(ret.k).size
    plan.close()


def test_plan_ties_and_negative_values():
    say("[plan] ties")
    lam = np.array([[1.0, 3.0, 3.0, -1.0], [3.0, 2.0, 3.0, 3.0], [0.5, 3.0, -0.0, 0.0]],
                   dtype=np.float32)
    QA = np.eye(4, dtype=np.float32)
    QS = np.eye(3, dtype=np.float32)
    for m in range(1, 11):
        plan = E.eogp_plan_create(d(lam), 2.0, m, d(QA), d(QS))
        flat, _ = plan.retained()
        torch.cuda.synchronize()
        assert flat.cpu().numpy().tolist() == O.select_retained(lam, 2.0, m).flat.tolist()
        plan.close()


def test_plan_rejects_nan_and_nonpositive_weights():
    lam = np.ones((8, 8), dtype=np.float32)
    I8 = d(np.eye(8, dtype=np.float32))
    lam_nan = lam.copy()
    lam_nan[3, 3] = np.nan
    with pytest.raises(E.EogpError):
        E.eogp_plan_create(d(lam_nan), 0.1, 4, I8, I8)
    with pytest.raises(E.EogpError):
        E.eogp_plan_create(d(-2.0 * lam), 0.5, 4, I8, I8)   # Lambda + lambda <= 0


# ---------------------------------------------------------------------------
# First stage
# ---------------------------------------------------------------------------
def test_rotate_retain_tiny_workload(tiny_fit):
    say("[first stage] tiny workload")
    raw, art = tiny_fit["raw"], tiny_fit["art"]
    w = S.TINY
    Z = E.eogp_rotate_retain(d(raw["a"]), d(raw["ds"]), d(raw["mask"]), d(art["Q_A"]),
                             d(art["Q_S"]), d(art["eigvals"]), art["damping"], w.m,
                             prec=E.PREC_ACCURATE)
    torch.cuda.synchronize()
    ref, _ = oracle_Z(raw["a"], raw["ds"], raw["mask"], art["Q_A"], art["Q_S"], art["eigvals"],
                      art["damping"], w.m)
    err = rel_rows(Z.cpu().numpy(), ref)
    say(f"   max rel {err.max():.2e} median {np.median(err):.2e}")
    assert err.max() <= 1e-3


@pytest.mark.parametrize("shape", [
    # N, T, d_in, d_out, m, lens_lo
    (5, 37, 97, 130, 1000, 0),       # ragged masks incl. empty examples, odd widths
    (3, 200, 769, 64, 700, 64),      # GPT-2-like input width (bias column)
    (2, 16, 5, 3, 15, 16),           # full basis retained
    (4, 70, 64, 257, 333, 1),
])
def test_rotate_retain_planned_fp32(shape):
    N, T, d_in, d_out, m, lo = shape
    say(f"[first stage] fp32 planned {shape}")
    a, ds, mask, QA, QS, lam = random_problem(sum(shape), N, T, d_in, d_out, m, lens_lo=lo)
    if lo == 0:
        mask[0, :] = 0                # an example with no valid token
    damping = 1e-4
    plan = E.eogp_plan_create(d(lam), damping, m, d(QA), d(QS))
    Z = E.eogp_rotate_retain_planned(plan, d(a), d(ds), d(mask), prec=E.PREC_ACCURATE)
    torch.cuda.synchronize()
    ref, _ = oracle_Z(a, ds, mask, QA, QS, lam, damping, m)
    Zg = Z.cpu().numpy()
    assert np.all(np.isfinite(Zg))
    nz = np.linalg.norm(ref, axis=1) > 0
    err = rel_rows(Zg[nz], ref[nz])
    say(f"   max rel {err.max():.2e}")
    assert err.max() <= 1e-3
    assert np.all(Zg[~nz] == 0)
    plan.close()


def test_rotate_retain_bf16_inputs_fast_and_accurate():
    say("[first stage] bf16")
    N, T, d_in, d_out, m = 6, 96, 256, 384, 2048
    a, ds, mask, QA, QS, lam = random_problem(11, N, T, d_in, d_out, m, lens_lo=8)
    at = d(a, torch.bfloat16)
    dt = d(ds, torch.bfloat16)
    a_used = at.float().cpu().numpy()
    d_used = dt.float().cpu().numpy()
    plan = E.eogp_plan_create(d(lam), 1e-4, m, d(QA), d(QS))
    ref, _ = oracle_Z(a_used, d_used, mask, QA, QS, lam, 1e-4, m)
    # the fp16 mode takes bf16 inputs exactly (inside fp16's normal range) and
    # rounds only the bases and the rotated tokens: the 1e-3 bound of fp32
    # accumulation holds, with and without power-of-two input scaling
    for prec, tol, ex in ((E.PREC_FAST, 2e-2, None), (E.PREC_ACCURATE, 1e-3, None),
                          (E.PREC_F16, 1e-3, None), (E.PREC_F16, 1e-3, (-2, 9))):
        if ex is not None:
            E.eogp_plan_set_input_exponents(plan, *ex)
        Z = E.eogp_rotate_retain_planned(plan, at, dt, d(mask), prec=prec)
        torch.cuda.synchronize()
        err = rel_rows(Z.cpu().numpy(), ref)
        say(f"   prec={prec} exponents={ex} max rel {err.max():.2e}")
        assert err.max() <= tol
    plan.close()


def test_fp16_coordinates_feed_the_pca_unchanged():
    """fp16 first-stage coordinates are the fp32 ones rounded once (nearest
    even); the PCA projection of a 16-bit Z with a P of the same type equals,
    bit for bit, the projection of the fp32 Z (which is rounded to P's type as
    it is staged); mismatched 16-bit types are refused."""
    say("[first stage] fp16 Z")
    N, T, d_in, d_out, m, k = 40, 48, 96, 80, 1000, 200
    a, ds, mask, QA, QS, lam = random_problem(31, N, T, d_in, d_out, m, lens_lo=5)
    plan = E.eogp_plan_create(d(lam), 1e-3, m, d(QA), d(QS))
    for prec in (E.PREC_F16, E.PREC_ACCURATE, E.PREC_FAST):
        Z32 = E.eogp_rotate_retain_planned(plan, d(a), d(ds), d(mask), prec=prec)
        Z16 = E.eogp_rotate_retain_planned(plan, d(a), d(ds), d(mask), prec=prec,
                                           Z=torch.empty((N, m), dtype=torch.float16, device=DEV))
        torch.cuda.synchronize()
        assert torch.equal(Z16, Z32.half())
    plan.close()
    g = np.random.default_rng(32)
    Pt = torch.from_numpy(np.ascontiguousarray(S.haar_orthogonal(g, m)[:, :k].T)).to(DEV)
    for pt in (Pt.half(), Pt.bfloat16()):
        X32 = E.eogp_pca_project(Z32, pt, prec=E.PREC_FAST)
        X16 = E.eogp_pca_project(Z32.to(pt.dtype), pt, prec=E.PREC_FAST)
        torch.cuda.synchronize()
        assert torch.equal(X16, X32)
    with pytest.raises(Exception):
        E.eogp_pca_project(Z16, Pt.bfloat16(), prec=E.PREC_FAST)


def test_rotate_retain_no_mask_and_ldz():
    N, T, d_in, d_out, m = 3, 20, 40, 50, 100
    a, ds, mask, QA, QS, lam = random_problem(12, N, T, d_in, d_out, m, nan_masked=False)
    plan = E.eogp_plan_create(d(lam), 1e-3, m, d(QA), d(QS))
    Zbig = torch.full((N, m + 9), -5.0, device=DEV)
    E.eogp_rotate_retain_planned(plan, d(a), d(ds), None, Z=Zbig[:, :m], prec=E.PREC_ACCURATE)
    torch.cuda.synchronize()
    ref, _ = oracle_Z(a, ds, np.ones((N, T), np.uint8), QA, QS, lam, 1e-3, m)
    assert rel_rows(Zbig[:, :m].cpu().numpy(), ref).max() <= 1e-3
    assert torch.all(Zbig[:, m:] == -5.0)
    plan.close()


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_rotate_retain_strided_token_rows(dtype):
    """Tokens passed as column slices of wider, 16-byte aligned buffers
    (769 -> 776 and 65 -> 72 columns), the way a caller hands over GPT-2's
    bias-augmented activations."""
    N, T, d_in, d_out, m = 3, 50, 769, 65, 900
    say(f"[first stage] strided rows {dtype}")
    a, ds, mask, QA, QS, lam = random_problem(14, N, T, d_in, d_out, m, lens_lo=5)
    abuf = torch.full((N, T, 776), float("nan"), device=DEV, dtype=dtype)
    gbuf = torch.full((N, T, 72), float("nan"), device=DEV, dtype=dtype)
    abuf[:, :, :d_in] = d(a, dtype)
    gbuf[:, :, :d_out] = d(ds, dtype)
    a_used = abuf[:, :, :d_in].float().cpu().numpy()
    d_used = gbuf[:, :, :d_out].float().cpu().numpy()
    plan = E.eogp_plan_create(d(lam), 1e-4, m, d(QA), d(QS))
    Z = E.eogp_rotate_retain_planned(plan, abuf[:, :, :d_in], gbuf[:, :, :d_out], d(mask),
                                     prec=E.PREC_ACCURATE)
    Z1 = E.eogp_rotate_retain(abuf[:, :, :d_in], gbuf[:, :, :d_out], d(mask), d(QA), d(QS),
                              d(lam), 1e-4, m, prec=E.PREC_ACCURATE)
    torch.cuda.synchronize()
    ref, _ = oracle_Z(S.fill_masked(a_used, mask), S.fill_masked(d_used, mask), mask, QA, QS,
                      lam, 1e-4, m)
    for got in (Z, Z1):
        err = rel_rows(got.cpu().numpy(), ref)
        say(f"   max rel {err.max():.2e}")
        assert err.max() <= 1e-3
    plan.close()


@pytest.mark.parametrize("shape", [
    # N, T, d_in, d_out, m, lens_lo
    (4, 288, 769, 768, 16384, 64),     # GPT-2 attn.c_proj-like widths and m
    (3, 100, 97, 130, 1000, 0),        # ragged, odd widths, an empty example
])
def test_rotate_retain_fp16_mode(shape):
    """fp32 inputs and bases rounded once to fp16, one MFMA pass: rows of Z
    within 1e-3 relative of the fp64 oracle."""
    N, T, d_in, d_out, m, lo = shape
    say(f"[first stage] fp16 mode {shape}")
    a, ds, mask, QA, QS, lam = random_problem(sum(shape) + 1, N, T, d_in, d_out, m, lens_lo=lo)
    if lo == 0:
        mask[0, :] = 0
    plan = E.eogp_plan_create(d(lam), 1e-4, m, d(QA), d(QS))
    Z = E.eogp_rotate_retain_planned(plan, d(a), d(ds), d(mask), prec=E.PREC_F16)
    torch.cuda.synchronize()
    ref, _ = oracle_Z(a, ds, mask, QA, QS, lam, 1e-4, m)
    Zg = Z.cpu().numpy()
    nz = np.linalg.norm(ref, axis=1) > 0
    err = rel_rows(Zg[nz], ref[nz])
    say(f"   max rel {err.max():.2e}")
    assert err.max() <= 1e-3
    assert np.all(Zg[~nz] == 0)
    plan.close()


@pytest.mark.parametrize("axis", ["rows", "cols"])
def test_rotate_retain_block_groups(axis):
    """Retained set inside one row block of S~ (or one column block of A~):
    the retained products then load that block once for a group of active
    blocks; both 16-bit modes match the oracle."""
    N, T, d_in, d_out, m = 5, 120, 300, 260, 4000
    say(f"[first stage] block groups sharing {axis}")
    a, ds, mask, QA, QS, lam = random_problem(71 if axis == "rows" else 72, N, T, d_in, d_out, m,
                                              lens_lo=3)
    if axis == "rows":
        lam[:32, :] += 100.0          # 32 x 300 > m entries: J = rows 0..31, one row block
    else:
        lam[:, :32] += 100.0          # K = columns 0..31, one column block
    plan = E.eogp_plan_create(d(lam), 1e-4, m, d(QA), d(QS))
    assert (plan.n_rows if axis == "rows" else plan.n_cols) == 32
    ref, _ = oracle_Z(a, ds, mask, QA, QS, lam, 1e-4, m)
    for prec, tol in ((E.PREC_F16, 1e-3), (E.PREC_FAST, 2e-2)):
        Z = E.eogp_rotate_retain_planned(plan, d(a), d(ds), d(mask), prec=prec)
        torch.cuda.synchronize()
        err = rel_rows(Z.cpu().numpy(), ref)
        say(f"   prec={prec} max rel {err.max():.2e}")
        assert err.max() <= tol
    plan.close()


def test_rotate_retain_compacted_matches_planned():
    """One token list (eogp_compact_tokens) serves several modules of a batch:
    eogp_rotate_retain_compacted gives the planned call's Z bit for bit, in
    every precision, for two plans of different widths, with empty and
    ragged examples."""
    say("[first stage] shared token list")
    N, T = 6, 90
    probs = []
    for seed, (d_in, d_out, m) in ((81, (97, 130, 900)), (82, (64, 257, 1200))):
        a, ds, _, QA, QS, lam = random_problem(seed, N, T, d_in, d_out, m, nan_masked=False)
        probs.append((a, ds, QA, QS, lam, m))
    g = np.random.default_rng(83)
    lens = g.integers(0, T + 1, size=N)
    lens[1] = 0                                          # an example with no valid token
    mask = S.prefix_mask(lens, T)
    plans = [E.eogp_plan_create(d(lam), 1e-4, m, d(QA), d(QS)) for (_, _, QA, QS, lam, m) in probs]
    need = max(E.eogp_rotate_retain_workspace_size(p, N, T) for p in plans)
    ws = torch.empty(need, dtype=torch.uint8, device=DEV)
    for prec in (E.PREC_F16, E.PREC_FAST, E.PREC_ACCURATE):
        E.eogp_compact_tokens(d(mask), N, T, prec, ws)
        for p, (a, ds, QA, QS, lam, m) in zip(plans, probs):
            af, df = d(S.fill_masked(a, mask)), d(S.fill_masked(ds, mask))
            Zc = E.eogp_rotate_retain_compacted(p, af, df, ws, prec=prec)
            Zp = E.eogp_rotate_retain_planned(p, af, df, d(mask), prec=prec)
            torch.cuda.synchronize()
            assert torch.equal(Zc, Zp), f"prec {prec}"
            assert torch.all(Zc[1] == 0)
    for p in plans:
        p.close()


def test_rotate_retain_fp16_mode_input_exponents():
    """Gradients of order 1e-7 (below fp16's normal range) are brought into
    range by the plan's exponent; the result is then as accurate as for
    ordinary magnitudes, and scaled back exactly."""
    N, T, d_in, d_out, m = 3, 64, 128, 96, 2000
    say("[first stage] fp16 mode exponents")
    a, ds, mask, QA, QS, lam = random_problem(21, N, T, d_in, d_out, m, lens_lo=16)
    ds = (ds * 1e-5).astype(np.float32)
    lam = (lam * 1e-10).astype(np.float32)
    ref, _ = oracle_Z(a, ds, mask, QA, QS, lam, 1e-14, m)
    plan = E.eogp_plan_create(d(lam), 1e-14, m, d(QA), d(QS))
    Z0 = E.eogp_rotate_retain_planned(plan, d(a), d(ds), d(mask), prec=E.PREC_F16)
    E.eogp_plan_set_input_exponents(plan, -2, 20)
    Z1 = E.eogp_rotate_retain_planned(plan, d(a), d(ds), d(mask), prec=E.PREC_F16)
    torch.cuda.synchronize()
    e0 = rel_rows(Z0.cpu().numpy(), ref).max()
    e1 = rel_rows(Z1.cpu().numpy(), ref).max()
    say(f"   without exponents {e0:.2e}, with {e1:.2e}")
    assert e1 <= 1e-3
    assert e0 > 3 * e1
    with pytest.raises(E.EogpError):
        E.eogp_plan_set_input_exponents(plan, 61, 0)
    # bf16 inputs of the same magnitudes: taken exactly into fp16 once the
    # exponents bring them into range
    ab, db = d(a, torch.bfloat16), d(ds, torch.bfloat16)
    refb, _ = oracle_Z(ab.float().cpu().numpy(), db.float().cpu().numpy(), mask, QA, QS, lam,
                       1e-14, m)
    Zb = E.eogp_rotate_retain_planned(plan, ab, db, d(mask), prec=E.PREC_F16)
    torch.cuda.synchronize()
    eb = rel_rows(Zb.cpu().numpy(), refb).max()
    say(f"   bf16 inputs with exponents {eb:.2e}")
    assert eb <= 1e-3
    plan.close()


def test_rotate_retain_deterministic():
    N, T, d_in, d_out, m = 4, 64, 128, 96, 500
    a, ds, mask, QA, QS, lam = random_problem(13, N, T, d_in, d_out, m, lens_lo=10)
    plan = E.eogp_plan_create(d(lam), 1e-3, m, d(QA), d(QS))
    Z1 = E.eogp_rotate_retain_planned(plan, d(a), d(ds), d(mask))
    Z2 = E.eogp_rotate_retain_planned(plan, d(a), d(ds), d(mask))
    torch.cuda.synchronize()
    assert torch.equal(Z1, Z2)
    plan.close()


# ---------------------------------------------------------------------------
# EK-FAC corrected eigenvalues (the fitting pass before selection)
# ---------------------------------------------------------------------------
def rel_fro(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return np.linalg.norm(a - b) / np.linalg.norm(b)


def test_ekfac_eigenvalues_tiny_workload(tiny_fit):
    """Mean over the 256 tiny examples of the squared rotated gradients, in
    the oracle-fitted eigenbases, against the oracle's fitting pass."""
    raw, f = tiny_fit["raw"], tiny_fit["fit"]
    QA = f["Q_A"].astype(np.float32)
    QS = f["Q_S"].astype(np.float32)
    sq = E.eogp_ekfac_eigenvalues(d(raw["a"]), d(raw["ds"]), d(raw["mask"]), d(QA), d(QS))
    torch.cuda.synchronize()
    lam = sq.cpu().numpy() / raw["a"].shape[0]
    ref = O.ekfac_eigenvalues(raw["a"], raw["ds"], raw["mask"], QA, QS)
    rel = np.abs(lam - ref) / np.maximum(np.abs(ref), 1e-30)
    say(f"[ekfac] tiny: fro {rel_fro(lam, ref):.2e}, max entry rel {rel.max():.2e}")
    assert rel_fro(lam, ref) <= 1e-4
    assert np.all(rel <= 1e-3)


def test_ekfac_ragged_batches_accumulate():
    """Odd widths, ragged masks with an empty example, NaN in masked tokens;
    two accumulated batches equal one batch of all examples."""
    N, T, d_in, d_out, m = 9, 37, 97, 130, 10
    a, ds, mask, QA, QS, _ = random_problem(71, N, T, d_in, d_out, m, lens_lo=0)
    mask[3, :] = 0
    a = S.fill_masked(a, mask)
    ds = S.fill_masked(ds, mask)
    ref = O.ekfac_eigenvalues(a, ds, mask, QA, QS) * N
    one = E.eogp_ekfac_eigenvalues(d(a), d(ds), d(mask), d(QA), d(QS))
    two = E.eogp_ekfac_eigenvalues(d(a[:4]), d(ds[:4]), d(mask[:4]), d(QA), d(QS))
    E.eogp_ekfac_eigenvalues(d(a[4:]), d(ds[4:]), d(mask[4:]), d(QA), d(QS), sq_sum=two,
                             accumulate=True)
    again = E.eogp_ekfac_eigenvalues(d(a), d(ds), d(mask), d(QA), d(QS))
    torch.cuda.synchronize()
    say(f"[ekfac] ragged: fro {rel_fro(one.cpu().numpy(), ref):.2e}")
    assert rel_fro(one.cpu().numpy(), ref) <= 1e-4
    assert rel_fro(two.cpu().numpy(), ref) <= 1e-4
    assert torch.equal(one, again)                       # fixed summation order


def test_ekfac_bf16_inputs():
    N, T, d_in, d_out = 4, 64, 256, 192
    a, ds, mask, QA, QS, _ = random_problem(72, N, T, d_in, d_out, 10, lens_lo=8)
    at, dt = d(a, torch.bfloat16), d(ds, torch.bfloat16)
    ref = O.ekfac_eigenvalues(at.float().cpu().numpy(), dt.float().cpu().numpy(), mask, QA, QS) * N
    for prec, tol, ex in ((E.PREC_FAST, 2e-2, (0, 0)), (E.PREC_ACCURATE, 1e-4, (0, 0)),
                          (E.PREC_F16, 3e-3, (0, 0)), (E.PREC_F16, 3e-3, (-1, 8))):
        sq = E.eogp_ekfac_eigenvalues(at, dt, d(mask), d(QA), d(QS), prec=prec, exponents=ex)
        torch.cuda.synchronize()
        err = rel_fro(sq.cpu().numpy(), ref)
        say(f"[ekfac] bf16 prec={prec} exponents={ex}: fro {err:.2e}")
        assert err <= tol


# fp16 mode: inputs, bases and the rotated tokens are each rounded once to
# fp16 (unit roundoff u = 2^-11 ~ 4.9e-4), products and sums in fp32. A block
# sum C = sum_t S~ A~ then carries a relative error of a few u (the rounding
# of both input factors, of both bases and of both rotated factors), and C^2
# twice that; over the whole matrix the errors are independent, so the
# Frobenius-relative error of sq_sum stays near 2u ~ 1e-3: the tolerance
# below is 3e-3.
F16_EKFAC_TOL = 3e-3


@pytest.mark.parametrize("N,T,d_in,d_out,lens_lo", [
    (9, 37, 97, 130, 0),          # odd widths, ragged runs, an empty example
    (40, 64, 384, 320, 1),        # several column groups, example ranges split
    (3, 200, 256, 128, 150),      # few examples: one range
])
def test_ekfac_fp16_mode_matches_oracle(N, T, d_in, d_out, lens_lo):
    say(f"[ekfac fp16] N={N} T={T} d_in={d_in} d_out={d_out}")
    a, ds, mask, QA, QS, _ = random_problem(73 + N, N, T, d_in, d_out, 10, lens_lo=lens_lo)
    if N == 9:
        mask[3, :] = 0
        a = S.fill_masked(a, mask)
        ds = S.fill_masked(ds, mask)
    ref = O.ekfac_eigenvalues(a, ds, mask, QA, QS) * N
    ex = (0, 7)                                         # gradients are of order 1e-2
    sq = E.eogp_ekfac_eigenvalues(d(a), d(ds), d(mask), d(QA), d(QS), prec=E.PREC_F16, exponents=ex)
    again = E.eogp_ekfac_eigenvalues(d(a), d(ds), d(mask), d(QA), d(QS), prec=E.PREC_F16, exponents=ex)
    torch.cuda.synchronize()
    err = rel_fro(sq.cpu().numpy(), ref)
    say(f"   fro {err:.2e}")
    assert err <= F16_EKFAC_TOL
    assert torch.equal(sq, again)                       # fixed summation order
    # two accumulated batches give the one-batch result
    h = N // 2
    two = E.eogp_ekfac_eigenvalues(d(a[:h]), d(ds[:h]), d(mask[:h]), d(QA), d(QS), prec=E.PREC_F16,
                                   exponents=ex)
    E.eogp_ekfac_eigenvalues(d(a[h:]), d(ds[h:]), d(mask[h:]), d(QA), d(QS), sq_sum=two,
                             accumulate=True, prec=E.PREC_F16, exponents=ex)
    torch.cuda.synchronize()
    assert rel_fro(two.cpu().numpy(), ref) <= F16_EKFAC_TOL


@pytest.mark.parametrize("prec", [0, 1, 2])
def test_ekfac_empty_batches(prec):
    """No examples, or every token masked: the sums are zero (accumulate=False)
    or left unchanged (accumulate=True), in every precision mode."""
    d_in, d_out = 96, 64
    a, ds, mask, QA, QS, _ = random_problem(75, 3, 16, d_in, d_out, 10)
    for n, msk in ((0, mask[:0]), (3, np.zeros_like(mask))):
        sq = E.eogp_ekfac_eigenvalues(d(a[:n]), d(ds[:n]), d(msk), d(QA), d(QS), prec=prec)
        prev = torch.full((d_out, d_in), 2.5, dtype=torch.float32, device=DEV)
        E.eogp_ekfac_eigenvalues(d(a[:n]), d(ds[:n]), d(msk), d(QA), d(QS), sq_sum=prev,
                                 accumulate=True, prec=prec)
        torch.cuda.synchronize()
        assert torch.all(sq == 0)
        assert torch.all(prev == 2.5)


def test_ekfac_fp16_mode_tiny_workload(tiny_fit):
    raw, f = tiny_fit["raw"], tiny_fit["fit"]
    QA = f["Q_A"].astype(np.float32)
    QS = f["Q_S"].astype(np.float32)
    sq = E.eogp_ekfac_eigenvalues(d(raw["a"]), d(raw["ds"]), d(raw["mask"]), d(QA), d(QS),
                                  prec=E.PREC_F16)
    torch.cuda.synchronize()
    lam = sq.cpu().numpy() / raw["a"].shape[0]
    ref = O.ekfac_eigenvalues(raw["a"], raw["ds"], raw["mask"], QA, QS)
    say(f"[ekfac fp16] tiny: fro {rel_fro(lam, ref):.2e}")
    assert rel_fro(lam, ref) <= F16_EKFAC_TOL


def test_ekfac_fp16_mode_input_exponents():
    """Gradients of order 1e-7 leave fp16's normal range; the exponents bring
    them back, and the result is scaled back exactly."""
    N, T, d_in, d_out = 6, 48, 160, 96
    a, ds, mask, QA, QS, _ = random_problem(74, N, T, d_in, d_out, 10, lens_lo=20)
    ds = (ds * 1e-5).astype(np.float32)
    ref = O.ekfac_eigenvalues(a, ds, mask, QA, QS) * N
    plain = E.eogp_ekfac_eigenvalues(d(a), d(ds), d(mask), d(QA), d(QS), prec=E.PREC_F16)
    scaled = E.eogp_ekfac_eigenvalues(d(a), d(ds), d(mask), d(QA), d(QS), prec=E.PREC_F16,
                                      exponents=(-1, 24))
    torch.cuda.synchronize()
    e0, e1 = rel_fro(plain.cpu().numpy(), ref), rel_fro(scaled.cpu().numpy(), ref)
    say(f"[ekfac fp16] without exponents {e0:.2e}, with {e1:.2e}")
    assert e1 <= F16_EKFAC_TOL
    assert e0 > 10 * e1
    with pytest.raises(E.EogpError):
        E.eogp_ekfac_eigenvalues(d(a), d(ds), d(mask), d(QA), d(QS), prec=E.PREC_F16,
                                 exponents=(0, 61))


# ---------------------------------------------------------------------------
# Random second stage (EOGP-R)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("N,m,k", [
    (5, 1, 1), (7, 3, 4), (9, 512, 128), (4, 700, 300), (3, 16384, 8192), (2, 32768, 16384),
    (0, 64, 8),
    # every width of the register form (p = 2^10 .. 2^15), k up to p
    (4, 1500, 700), (3, 3000, 3000), (2, 5000, 8192), (3, 9000, 16384),
    # two-stage form (p > 32768): padded 40000 -> 65536, the OLMo-2-32B-shaped
    # module (m = 65,536, k = 32,768), the paper's timing configuration
    # (m = 262,144, k = 2,048), and the largest supported width
    (3, 40000, 8192), (2, 65536, 32768), (2, 262144, 2048), (1, 1 << 20, 4096), (0, 70000, 8),
])
def test_srht_project(N, m, k):
    """Against the fp64 oracle; fp32 butterflies keep about 1e-6 relative."""
    say(f"[srht] N={N} m={m} k={k}")
    p = O.srht_width(m)
    signs, rows = S.srht_draws(9, m + k, m, p, k)
    Z = np.random.default_rng(m).standard_normal((N, m)).astype(np.float32)
    X = E.eogp_srht_project(d(Z), d(signs), d(rows))
    torch.cuda.synchronize()
    if N == 0:
        assert X.shape == (0, k)
        return
    ref = O.srht_project(Z, signs, rows)
    err = rel_rows(X.cpu().numpy(), ref)
    say(f"   max rel {err.max():.2e}")
    assert err.max() <= 1e-5


@pytest.mark.parametrize("m", [1000, 40000])
def test_srht_project_strides_and_bad_rows(m):
    k = 64
    p = O.srht_width(m)
    signs, rows = S.srht_draws(9, 1, m, p, k)
    rows[5] = p                                  # outside the transform
    Z = np.random.default_rng(2).standard_normal((3, m + 24)).astype(np.float32)
    Xb = torch.full((3, k + 7), 7.0, device=DEV)
    E.eogp_srht_project(d(Z)[:, :m], d(signs), d(rows), X=Xb[:, :k])
    torch.cuda.synchronize()
    Xg = Xb.cpu().numpy()
    assert np.all(np.isnan(Xg[:, 5]))
    good = np.r_[0:5, 6:k]
    ref = O.srht_project(Z[:, :m], signs, np.where(rows < p, rows, 0))
    assert rel_rows(Xg[:, good], ref[:, good]).max() <= 1e-5
    assert np.all(Xg[:, k:] == 7.0)


# ---------------------------------------------------------------------------
# Scoring
# ---------------------------------------------------------------------------
def random_store(seed, N, ks, Q):
    g = np.random.default_rng(seed)
    nbytes = sum(k // 8 for k in ks)
    codes = g.integers(0, 256, size=(N, nbytes), dtype=np.uint8)
    scales = np.exp(g.standard_normal((N, len(ks)))).astype(np.float16).view(np.uint16)
    Y = g.standard_normal((Q, sum(ks))).astype(np.float32)
    return codes, scales, Y


@pytest.mark.parametrize("N,ks,Q,topk", [
    (300, [128], 8, 10),
    (1000, [64, 512, 192], 20, 37),
    (5, [256], 3, 10),               # fewer examples than topk
    (4097, [1024], 17, 100),
    (256, [64] * 5, 16, 256),
])
def test_score_topk_bit_exact(N, ks, Q, topk):
    say(f"[score] N={N} ks={ks} Q={Q} topk={topk}")
    codes, scales, Y = random_store(N + Q, N, ks, Q)
    Y[0, :] = 0.0                      # an all-zero query
    idx, sc, full = E.eogp_score_topk(d(codes), d(scales.view(np.int16)), ks, d(Y), topk,
                                      full_scores=True)
    torch.cuda.synchronize()
    ref = O.score(codes, scales, ks, Y)
    assert np.array_equal(full.cpu().numpy(), ref.astype(np.float32))
    oi, ov = O.topk(ref, topk)
    assert np.array_equal(idx.cpu().numpy(), oi)
    assert np.array_equal(sc.cpu().numpy(), ov)


@pytest.mark.parametrize("N,ks,Q,topk", [
    (600_000, [64], 16, 100),        # one module: several 1024-row blocks per workgroup
    (300_000, [64, 64], 9, 128),     # two modules: several 512-row blocks per workgroup
    (70_000, [128], 5, 200),         # the 512-slot candidate lists
])
def test_score_topk_bit_exact_large_stores(N, ks, Q, topk):
    """More rows than one pass of workgroups covers, so every workgroup keeps
    its candidate lists over several blocks (pruning and re-offering)."""
    say(f"[score] large N={N} ks={ks} Q={Q} topk={topk}")
    codes, scales, Y = random_store(N + 7, N, ks, Q)
    idx, sc, _ = E.eogp_score_topk(d(codes), d(scales.view(np.int16)), ks, d(Y), topk)
    torch.cuda.synchronize()
    ref = O.score(codes, scales, ks, Y)
    oi, ov = O.topk(ref, topk)
    assert np.array_equal(idx.cpu().numpy(), oi)
    assert np.array_equal(sc.cpu().numpy(), ov)


@pytest.mark.parametrize("N,ks,stride", [
    (1, [64], 8),            # an 8-byte store: the pass reads a zero-padded copy
    (1, [64, 64], 16),       # exactly 16 readable bytes
    (2, [64], 8),
    (3, [192], 32),          # rows wider than their codes (stride > sum k_u / 8)
])
def test_score_tiny_stores(N, ks, stride):
    """Stores of a few bytes: every lane's 16-byte reads stay inside the
    store (or its padded copy) and the scores are exact."""
    say(f"[score] tiny N={N} ks={ks} stride={stride}")
    codes, scales, Y = random_store(N + 40, N, ks, 5)
    wide = np.zeros((N, stride), np.uint8)
    wide[:, :codes.shape[1]] = codes
    ct = d(wide)[:, :codes.shape[1]] if stride > codes.shape[1] else d(wide)
    idx, sc, full = E.eogp_score_topk(ct, d(scales.view(np.int16)), ks, d(Y), 3,
                                      full_scores=True)
    torch.cuda.synchronize()
    ref = O.score(codes, scales, ks, Y)
    assert np.array_equal(full.cpu().numpy(), ref.astype(np.float32))
    oi, ov = O.topk(ref, 3)
    assert np.array_equal(idx.cpu().numpy(), oi)
    assert np.array_equal(sc.cpu().numpy(), ov)


def test_score_empty_store_and_no_queries():
    """An empty store pads every query's list (index -1, score -inf); no
    queries is a no-op."""
    ks = [128, 64]
    codes, scales, Y = random_store(23, 0, ks, 4)
    idx, sc, _ = E.eogp_score_topk(d(codes), d(scales.view(np.int16)), ks, d(Y), 10)
    torch.cuda.synchronize()
    assert torch.all(idx == -1)
    assert torch.all(sc == float("-inf"))
    codes, scales, _ = random_store(24, 50, ks, 1)
    idx, sc, _ = E.eogp_score_topk(d(codes), d(scales.view(np.int16)), ks,
                                   torch.empty((0, 192), device=DEV), 10)
    torch.cuda.synchronize()
    assert idx.shape == (0, 10) and sc.shape == (0, 10)


def test_score_integral_queries_give_exact_real_scores():
    g = np.random.default_rng(21)
    ks = [256, 128]
    codes, scales, _ = random_store(22, 200, ks, 5)
    Y = g.integers(-3000, 3000, size=(5, 384)).astype(np.float32)
    idx, sc, full = E.eogp_score_topk(d(codes), d(scales.view(np.int16)), ks, d(Y), 10,
                                      full_scores=True)
    torch.cuda.synchronize()
    real = O.score_real(codes, scales, ks, Y)
    assert np.array_equal(full.cpu().numpy(), real.astype(np.float32))


@pytest.mark.parametrize("ks", [[1 << 18], [1 << 18, 64]])
def test_score_long_modules_with_same_signed_queries(ks):
    """k_u = 2^18 with every query coordinate positive: sum_c y_int reaches
    about 3.2e9 > 2^31, so it must be carried in 64 bits (the one-module
    kernel) and the per-module dots stored in 64 bits (several modules).
    Scores of sampled rows are exact against the oracle (eq. onebit_influence)."""
    N, Q = 1100, 3
    say(f"[score] long modules ks={ks} N={N}")
    g = np.random.default_rng(1 << 18)
    nbytes = sum(k // 8 for k in ks)
    codes = g.integers(0, 256, size=(N, nbytes), dtype=np.uint8)
    scales = np.exp(g.standard_normal((N, len(ks)))).astype(np.float16).view(np.uint16)
    Y = g.uniform(0.5, 1.0, size=(Q, sum(ks))).astype(np.float32)
    fx = O.query_fixed_point(Y[0, :ks[0]])[0]
    assert int(fx.sum()) > 2 ** 31                       # the case the 64-bit sums exist for
    idx, sc, full = E.eogp_score_topk(d(codes), d(scales.view(np.int16)), ks, d(Y), 10,
                                      full_scores=True)
    torch.cuda.synchronize()
    rows = np.sort(g.choice(N, 48, replace=False))
    ref = O.score(codes[rows], scales[rows], ks, Y)
    assert np.array_equal(full.cpu().numpy()[:, rows], ref.astype(np.float32))
    f = full.double()
    for q in range(Q):
        assert torch.equal(sc[q], full[q, idx[q]])
        rest = torch.ones(N, dtype=torch.bool, device=DEV)
        rest[idx[q]] = False
        assert float(f[q][rest].max()) <= float(sc[q, -1])


def test_score_gpt2_store_layout_sampled_rows():
    """The GPT-2-small-shaped store as the bench scores it: 20,000 rows of 48
    modules x 8,192 bits (983 MB of codes), 16 queries, top-100. 256 sampled
    rows are scored exactly against the oracle; the top-100 is checked by the
    properties that define it on the full score vector."""
    N, U, k, Q, topk = 20000, 48, 8192, 16, 100
    say(f"[score] gpt2 store N={N} U={U} k={k}")
    gen = torch.Generator(device=DEV)
    gen.manual_seed(48)
    codes = torch.randint(0, 256, (N, U * k // 8), dtype=torch.uint8, device=DEV, generator=gen)
    scales = torch.exp(torch.randn((N, U), device=DEV, generator=gen)).half().view(torch.int16)
    Y = torch.randn((Q, U * k), device=DEV, generator=gen)
    idx, sc, full = E.eogp_score_topk(codes, scales, [k] * U, Y, topk, full_scores=True)
    torch.cuda.synchronize()
    rows = np.sort(np.random.default_rng(48).choice(N, 256, replace=False))
    rows[-1] = N - 1
    ri = torch.from_numpy(rows).to(DEV)
    ref = O.score(codes[ri].cpu().numpy(), scales[ri].cpu().numpy().view(np.uint16), [k] * U,
                  Y.cpu().numpy())
    assert np.array_equal(full[:, ri].cpu().numpy(), ref.astype(np.float32))
    f = full.double()
    for q in range(Q):
        iq = idx[q]
        assert torch.equal(sc[q], full[q, iq])
        assert bool(torch.all(sc[q, :-1] >= sc[q, 1:]))
        rest = torch.ones(N, dtype=torch.bool, device=DEV)
        rest[iq] = False
        assert float(f[q][rest].max()) <= float(sc[q, -1])
        ties = iq[sc[q] == sc[q, -1]]
        # among equal scores the smaller index ranks first, and nothing left
        # out ties the last entry with a smaller index
        assert bool(torch.all(ties[:-1] < ties[1:]))
        left = torch.nonzero(rest & (full[q] == sc[q, -1])).flatten()
        assert left.numel() == 0 or int(left.min()) > int(ties.max())


def test_score_ties_resolved_by_index():
    # identical codes and scales: every score ties; ranking must be by index
    N, ks = 600, [128]
    codes = np.tile(np.random.default_rng(3).integers(0, 256, (1, 16), dtype=np.uint8), (N, 1))
    scales = np.full((N, 1), np.float16(1.5)).view(np.uint16)
    Y = np.random.default_rng(4).standard_normal((3, 128)).astype(np.float32)
    idx, sc, _ = E.eogp_score_topk(d(codes), d(scales.view(np.int16)), ks, d(Y), 50)
    torch.cuda.synchronize()
    assert np.array_equal(idx.cpu().numpy(), np.tile(np.arange(50), (3, 1)))


# ---------------------------------------------------------------------------
# Whole path on the tiny workload
# ---------------------------------------------------------------------------
def test_end_to_end_tiny(tiny_fit):
    say("[end to end] tiny")
    raw, art = tiny_fit["raw"], tiny_fit["art"]
    w = S.TINY
    plan = E.eogp_plan_create(d(art["eigvals"]), art["damping"], w.m, d(art["Q_A"]), d(art["Q_S"]))
    Pt = d(np.ascontiguousarray(art["P"].T))
    Z = E.eogp_rotate_retain_planned(plan, d(raw["a"]), d(raw["ds"]), d(raw["mask"]),
                                     prec=E.PREC_ACCURATE)
    X = E.eogp_pca_project(Z, Pt, prec=E.PREC_ACCURATE)
    codes, scales = E.eogp_sign_pack(X)
    Zq = E.eogp_rotate_retain_planned(plan, d(raw["qa"]), d(raw["qds"]), d(raw["qmask"]),
                                      prec=E.PREC_ACCURATE)
    Y = E.eogp_pca_project(Zq, Pt, prec=E.PREC_ACCURATE)
    idx, sc, full = E.eogp_score_topk(codes, scales, [w.k], Y, w.topk, full_scores=True)
    torch.cuda.synchronize()

    Zo, Xo, co, so = O.store(raw["a"], raw["ds"], raw["mask"], art["Q_A"], art["Q_S"],
                             art["eigvals"], art["damping"], w.m, art["P"])
    Yo = O.query(raw["qa"], raw["qds"], raw["qmask"], art["Q_A"], art["Q_S"], art["eigvals"],
                 art["damping"], w.m, art["P"])
    ex = rel_rows(X.cpu().numpy(), Xo)
    ey = rel_rows(Y.cpu().numpy(), Yo)
    say(f"   x max rel {ex.max():.2e}, y max rel {ey.max():.2e}")
    assert ex.max() <= 1e-3 and ey.max() <= 1e-3
    # sign bits: identical except where |x| < 1e-3 rms(x)
    bits_g = O.unpack_bits(codes.cpu().numpy(), w.k)
    bits_o = O.unpack_bits(co, w.k)
    rms = np.sqrt(np.mean(Xo ** 2, axis=1, keepdims=True))
    diff = bits_g != bits_o
    assert not np.any(diff & (np.abs(Xo) >= 1e-3 * rms))
    say(f"   sign mismatch fraction {diff.mean():.2e}")
    # scales: within one fp16 ulp of the oracle
    sg = scales.cpu().numpy().view(np.float16)[:, 0].astype(np.float64)
    so16 = so.view(np.float16).astype(np.float64)
    assert np.all(np.abs(sg - so16) <= np.spacing(so.view(np.float16)).astype(np.float64))
    # scores and top-k: bit-exact for the codes, scales and queries the GPU produced
    cg = codes.cpu().numpy()
    sgb = scales.cpu().numpy().view(np.uint16)
    Yg = Y.cpu().numpy()
    ref = O.score(cg, sgb, [w.k], Yg)
    assert np.array_equal(full.cpu().numpy(), ref.astype(np.float32))
    oi, ov = O.topk(ref, w.topk)
    assert np.array_equal(idx.cpu().numpy(), oi)
    assert np.array_equal(sc.cpu().numpy(), ov)
    plan.close()
