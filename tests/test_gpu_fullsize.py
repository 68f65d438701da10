"""GPU parity at the workloads' full sizes, on sampled outputs.

The oracle cannot evaluate whole full-size problems in seconds, so each test
runs the HIP path at the real shape (for the GPT-2-small-shaped workload in
the launch configuration bench.py times: 1,266 examples x 512 tokens per call)
and checks

* sampled examples, or sampled retained coordinates, of the first stage
  against the fp64 oracle on the same inputs (relative error per row);
* the retained-axis selection bit-exactly against an independent O(n)
  selection (a partition for the m-th key, then a sort of the candidates);
* the PCA projection on sampled output columns, sign bits and scales;
* 8M-code scoring on sampled rows (exact) and its top-k by the properties
  that define it (sorted, tie rule, nothing better left out).

Tolerances are the ones stated in test_gpu_parity.py: 1e-3 relative for fp32
accumulation of fp32 inputs (accurate and fp16 modes), 2e-2 for bf16 inputs.
"""
import sys

import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_37842_amd import eogp as E
from paper_2609_37842_amd import synth as S
from select_helpers import restrict, select_large
from tiled_helpers import rows_from_tiled

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

DEV = "cuda:0"


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    E.load()
    yield
    torch.cuda.empty_cache()


def rel_rows(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return np.linalg.norm(a - b, axis=-1) / np.maximum(np.linalg.norm(b, axis=-1), 1e-300)


def padded_inputs(w, si, N, T, d_in, d_out, dtype):
    """Token rows in buffers padded to 32-element (128-byte) strides, as the
    bench lays them out; returns views [N, T, d] and the mask."""
    a, ds, mask = S.torch_inputs(w, si, N, T, d_in, d_out, DEV, dtype)
    bufs = []
    for x, width in ((a, d_in), (ds, d_out)):
        ld = -(-width // 32) * 32
        b = torch.zeros((N, T, ld), dtype=dtype, device=DEV)
        b[:, :, :width] = x
        bufs.append(b[:, :, :width])
    return bufs[0], bufs[1], mask


def check_selection(plan, ret: O.Retained):
    flat, wgt = plan.retained()
    torch.cuda.synchronize()
    assert np.array_equal(flat.cpu().numpy().astype(np.int64), ret.flat)
    assert np.allclose(wgt.cpu().numpy(), ret.w, rtol=1e-6, atol=0)


def first_stage_sampled(w, si, name, d_in, d_out, N, T, dtype, precs, examples, coords=None):
    """Run the first stage at full width; compare sampled examples (and, if
    given, sampled retained coordinates) with the oracle."""
    a, ds, mask = padded_inputs(w, si, N, T, d_in, d_out, dtype)
    art = S.torch_module_artifacts(w, si, d_in, d_out, DEV, torch.float16, {})
    lam = art["eigvals"].cpu().numpy()
    ret = select_large(lam, art["damping"], w.m)
    plan = E.eogp_plan_create(art["eigvals"], art["damping"], w.m, art["Q_A"], art["Q_S"])
    check_selection(plan, ret)
    say(f"   {name}: |J|={plan.n_rows} |K|={plan.n_cols} tiles={plan.n_tiles}")
    if coords is None:
        coords = np.arange(w.m)
    sub, J, K = restrict(ret, coords)
    QS = art["Q_S"][:, torch.from_numpy(J).to(DEV)].cpu().numpy()
    QA = art["Q_A"][:, torch.from_numpy(K).to(DEV)].cpu().numpy()
    ex = torch.tensor(examples, device=DEV)
    a_s = a[ex].float().cpu().numpy()
    d_s = ds[ex].float().cpu().numpy()
    m_s = mask[ex].cpu().numpy()
    ref = np.stack([O.first_stage_tokens(a_s[i], d_s[i], m_s[i], QA, QS, sub)
                    for i in range(len(examples))])
    out = {}
    for prec, tol in precs:
        Z = E.eogp_rotate_retain_planned(plan, a, ds, mask, prec=prec)
        torch.cuda.synchronize()
        got = Z[ex][:, torch.from_numpy(coords).to(DEV)].cpu().numpy()
        err = rel_rows(got, ref)
        say(f"   prec={prec}: max rel {err.max():.2e}")
        assert err.max() <= tol
        out[prec] = Z
    plan.close()
    return out, ref, art


SIGN_RECORD = {}


def record_sign_mismatch(key, value):
    """Keeps the measured sign-mismatch fractions and writes them to
    gpurun_out/sign_mismatch_gpt2.json (a run record, not an input)."""
    import json
    import os
    SIGN_RECORD[key] = value
    out = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "gpurun_out")
    os.makedirs(out, exist_ok=True)
    with open(os.path.join(out, "sign_mismatch_gpt2.json"), "w") as f:
        json.dump(SIGN_RECORD, f, indent=1, sort_keys=True)


@pytest.mark.parametrize("si", [0, 1, 2, 3])   # c_attn, attn.c_proj, c_fc, mlp.c_proj
def test_gpt2_small_full_step_shape(si):
    """Each GPT-2-small-shaped linear at the bench's launch shape (1,266
    examples x 512 tokens, fp32 inputs): the first stage in the bench's fp16
    mode and in the accurate mode against the oracle on eight sampled
    examples (all retained coordinates), then the PCA projection with the
    module's fp16 P, sign bits and scales. The accurate path must keep every
    sign outside the band |x| < 1e-3 rms (eq. onebit); the bench's fp16 path
    (fp16 first stage, fp16 coordinates into the PCA) is held to a bound on
    the fraction outside the band, and both fractions are recorded."""
    w = S.GPT2_SMALL
    name, d_in, d_out = w.block[si]
    N, T = 1266, w.T
    examples = [0, 181, 362, 633, 790, 1000, 1200, 1265]
    say(f"[full size] gpt2 {name}")
    Zs, zref, art = first_stage_sampled(w, si, name, d_in, d_out, N, T, torch.float32,
                                        [(E.PREC_F16, 1e-3), (E.PREC_ACCURATE, 1e-3)], examples)
    P = art["Pt"].double().cpu().numpy().T                 # [m, k], the fp16 values
    xref = O.pca_project(zref, P)
    rms = np.sqrt(np.mean(xref ** 2, axis=1, keepdims=True))
    so = O.onebit_scale(xref).view(np.float16)
    ei = torch.tensor(examples, device=DEV)
    band = np.abs(xref) < 1e-3 * rms
    for prec, pca_prec, label in ((E.PREC_ACCURATE, E.PREC_ACCURATE, "accurate"),
                                  (E.PREC_F16, E.PREC_FAST, "bench_f16")):
        Zin = Zs[prec]
        if label == "bench_f16":
            Zin = Zin.half()                               # the bench keeps Z in fp16
        X = E.eogp_pca_project(Zin, art["Pt"], prec=pca_prec)
        codes, scales = E.eogp_sign_pack(X)
        torch.cuda.synchronize()
        err = rel_rows(X[ei].cpu().numpy(), xref)
        bits_g = O.unpack_bits(codes[ei].cpu().numpy(), w.k)
        diff = bits_g != O.sign_bits(xref)
        outside = diff & ~band
        say(f"   {label}: pca max rel {err.max():.2e}, sign mismatch fraction "
            f"{diff.mean():.2e} ({outside.mean():.2e} outside the band)")
        record_sign_mismatch(f"{name}/{label}", {
            "bits": int(diff.size), "mismatch": int(diff.sum()),
            "mismatch_outside_band": int(outside.sum()),
            "fraction": float(diff.mean()), "fraction_outside_band": float(outside.mean()),
            "in_band_fraction_of_bits": float(band.mean()),
            "x_max_rel_err": float(err.max())})
        assert err.max() <= 1e-3
        if label == "accurate":
            assert not np.any(outside)                   # strict in accurate mode
        else:
            assert outside.mean() <= 1e-3                # bounded and recorded
        sg = scales[ei].cpu().numpy().view(np.float16)[:, 0]
        assert np.all(np.abs(sg.astype(np.float64) - so.astype(np.float64))
                      <= 2 * np.spacing(so).astype(np.float64))


@pytest.mark.parametrize("si", [0, 4, 6])     # q_proj 2048 -> 2048 (the shape of k, v, o too),
def test_olmo2_1b_bf16_modules(si):            # gate_proj 2048 -> 8192, down_proj 8192 -> 2048
    """OLMo-2-1B-shaped modules (every distinct shape of the block), bf16
    inputs, T = 1024 with lengths U{64..1024}, m = 32768: two sampled
    examples, all retained coordinates,
    in the bf16 mode, the accurate mode and the fp16 mode (bf16 inputs taken
    exactly, bases and rotated tokens rounded to fp16)."""
    w = S.OLMO2_1B
    name, d_in, d_out = w.block[si]
    say(f"[full size] olmo2-1b {name}")
    first_stage_sampled(w, si, name, d_in, d_out, 12, w.T, torch.bfloat16,
                        [(E.PREC_FAST, 2e-2), (E.PREC_ACCURATE, 2e-3), (E.PREC_F16, 1e-3)],
                        [0, 11])


@pytest.mark.parametrize("si", [0, 1, 5, 6])  # q_proj 5120 -> 5120, k_proj 5120 -> 1024, up
def test_olmo2_32b_bf16_modules(si):            # 5120 -> 27648, down 27648 -> 5120
    """OLMo-2-32B-shaped modules (every distinct shape of the block: q_proj
    as o_proj, grouped-query k_proj as v_proj, MLP up as gate, down), bf16
    inputs, T = 2048, m = 65536: 512 sampled retained coordinates of two
    examples; the whole retained set is checked bit-exactly."""
    w = S.OLMO2_32B
    name, d_in, d_out = w.block[si]
    say(f"[full size] olmo2-32b {name}")
    g = np.random.default_rng(si)
    coords = np.sort(g.choice(w.m, 512, replace=False))
    first_stage_sampled(w, si, name, d_in, d_out, 3, w.T, torch.bfloat16,
                        [(E.PREC_FAST, 2e-2), (E.PREC_F16, 1e-3)], [0, 2], coords=coords)


@pytest.mark.parametrize("wl", ["olmo2-1b", "olmo2-32b"])
def test_pca_full_size_sampled_columns(wl):
    """PCA projection with the workload's fp16 P at full size (m x k =
    32768 x 16384 and 65536 x 32768) on synthetic first-stage rows; 384
    sampled output columns against the oracle."""
    w = S.OLMO2_1B if wl == "olmo2-1b" else S.OLMO2_32B
    say(f"[full size] pca {wl}")
    Pt = S.torch_pca_directions_t(S.rng(w.config_id, 600000 + w.m), w.m, w.k, DEV).half()
    g = torch.Generator(device=DEV)
    g.manual_seed(w.config_id)
    Z = torch.randn((40, w.m), device=DEV, generator=g)
    X = E.eogp_pca_project(Z, Pt, prec=E.PREC_FAST)
    torch.cuda.synchronize()
    cols = np.sort(np.random.default_rng(5).choice(w.k, 384, replace=False))
    ci = torch.from_numpy(cols).to(DEV)
    P = Pt[ci].double().cpu().numpy().T                   # [m, 384]
    zr = Z.double().cpu().numpy()
    xref = zr @ P
    err = rel_rows(X[:, ci].cpu().numpy(), xref)
    say(f"   max rel {err.max():.2e}")
    # fast mode rounds z to fp16 once: 2^-11 relative per coordinate
    assert err.max() <= 1e-3


def test_scoring_8m_codes_one_pass():
    """8,388,608 stored codes x 16,384 bits, 16 queries, top-100: 4096
    sampled rows scored exactly; the top-100 equals the best 100 of the full
    score vector under the (score desc, index asc) rule."""
    w = S.SCORING
    N, k, Q, topk = w.N, w.k, 16, w.topk
    say(f"[full size] scoring N={N} k={k}")
    g = torch.Generator(device=DEV)
    g.manual_seed(77)
    codes = torch.empty((N, k // 8), dtype=torch.uint8, device=DEV)
    for i0 in range(0, N, 1 << 20):
        codes[i0:i0 + (1 << 20)] = torch.randint(0, 256, (1 << 20, k // 8), dtype=torch.uint8,
                                                 device=DEV, generator=g)
    scales = torch.exp(torch.randn((N, 1), device=DEV, generator=g)).half().view(torch.int16)
    Y = torch.randn((Q, k), device=DEV, generator=g)
    idx, sc, full = E.eogp_score_topk(codes, scales, [k], Y, topk, full_scores=True)
    torch.cuda.synchronize()
    rows = np.sort(np.random.default_rng(9).choice(N, 4096, replace=False))
    ri = torch.from_numpy(rows).to(DEV)
    ref = O.score(codes[ri].cpu().numpy(), scales[ri].cpu().numpy().view(np.uint16), [k],
                  Y.cpu().numpy())
    assert np.array_equal(full[:, ri].cpu().numpy(), ref.astype(np.float32))
    # top-k properties on the full score vector (fp32 values of exact fp64 scores)
    f = full.double()
    for q in range(Q):
        iq = idx[q]
        assert torch.equal(sc[q], full[q, iq])
        kth = float(sc[q, -1])
        assert int((f[q] > kth).sum()) <= topk
        assert bool(torch.all(sc[q, :-1] >= sc[q, 1:]))
        # nothing outside the list scores strictly higher than its last entry
        mask = torch.ones(N, dtype=torch.bool, device=DEV)
        mask[iq] = False
        assert float(f[q][mask].max()) <= kth


def test_scoring_8m_codes_tiled_store():
    """The same 8,388,608 x 16,384-bit workload in the tiled store layout
    (random bytes are a valid tiled store): 128 sampled tiles (4,096 rows),
    converted to row-major by the layout's definition, scored exactly against
    the oracle; the top-100 by its defining properties."""
    w = S.SCORING
    N, k, Q, topk = w.N, w.k, 16, w.topk
    S_row = k // 512
    say(f"[full size] tiled scoring N={N} k={k}")
    g = torch.Generator(device=DEV)
    g.manual_seed(78)
    nbytes = E.tiled_store_bytes(N, [k])
    codes = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    for i0 in range(0, nbytes, 1 << 30):
        i1 = min(nbytes, i0 + (1 << 30))
        codes[i0:i1] = torch.randint(0, 256, (i1 - i0,), dtype=torch.uint8, device=DEV, generator=g)
    scales = torch.exp(torch.randn((N, 1), device=DEV, generator=g)).half().view(torch.int16)
    Y = torch.randn((Q, k), device=DEV, generator=g)
    idx, sc, full = E.eogp_score_topk_tiled(codes, scales, N, [k], Y, topk, full_scores=True)
    torch.cuda.synchronize()
    tiles = np.sort(np.random.default_rng(10).choice(N // 32, 128, replace=False))
    blk = S_row * 2048
    sub = np.concatenate([codes[t * blk:(t + 1) * blk].cpu().numpy() for t in tiles])
    rows_codes = rows_from_tiled(sub, S_row)
    rows = (tiles[:, None] * 32 + np.arange(32)[None, :]).reshape(-1)
    ri = torch.from_numpy(rows).to(DEV)
    ref = O.score(rows_codes, scales[ri].cpu().numpy().view(np.uint16), [k], Y.cpu().numpy())
    assert np.array_equal(full[:, ri].cpu().numpy(), ref.astype(np.float32))
    f = full.double()
    for q in range(Q):
        iq = idx[q]
        assert torch.equal(sc[q], full[q, iq])
        assert bool(torch.all(sc[q, :-1] >= sc[q, 1:]))
        rest = torch.ones(N, dtype=torch.bool, device=DEV)
        rest[iq] = False
        assert float(f[q][rest].max()) <= float(sc[q, -1])


def test_scoring_olmo2_1b_store_tiled():
    """The OLMo-2-1B-shaped store the bench scores: 100,000 rows x 112 modules
    x 16,384 bits in the tiled layout (23 GB; random bytes are a valid tiled
    store), per-module fp16 scales, 16 queries, top-100 (the several-module
    pass: module ranges split across workgroups, exact per-module dots summed
    in module order). 8 sampled tiles (256 rows), converted to row-major by
    the layout's definition, are scored exactly against the oracle; the
    top-100 is checked by the properties that define it."""
    w = S.OLMO2_1B
    U = len(w.modules)
    N, k, Q, topk = w.N, w.k, 16, w.topk
    ks = [k] * U
    S_row = U * k // 512
    say(f"[full size] olmo2-1b store N={N} U={U} k={k}")
    g = torch.Generator(device=DEV)
    g.manual_seed(112)
    nbytes = E.tiled_store_bytes(N, ks)
    codes = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    for i0 in range(0, nbytes, 1 << 30):
        i1 = min(nbytes, i0 + (1 << 30))
        codes[i0:i1] = torch.randint(0, 256, (i1 - i0,), dtype=torch.uint8, device=DEV, generator=g)
    scales = torch.exp(torch.randn((N, U), device=DEV, generator=g)).half().view(torch.int16)
    Y = torch.randn((Q, U * k), device=DEV, generator=g)
    idx, sc, full = E.eogp_score_topk_tiled(codes, scales, N, ks, Y, topk, full_scores=True)
    torch.cuda.synchronize()
    n_tiles = -(-N // 32)
    tiles = np.sort(np.random.default_rng(11).choice(n_tiles - 1, 7, replace=False))
    tiles = np.append(tiles, n_tiles - 1)            # the last tile (rows past N unused)
    blk = S_row * 2048
    sub = np.concatenate([codes[t * blk:(t + 1) * blk].cpu().numpy() for t in tiles])
    rows_codes = rows_from_tiled(sub, S_row)
    rows = (tiles[:, None] * 32 + np.arange(32)[None, :]).reshape(-1)
    keep = rows < N
    rows, rows_codes = rows[keep], rows_codes[keep]
    ri = torch.from_numpy(rows).to(DEV)
    ref = O.score(rows_codes, scales[ri].cpu().numpy().view(np.uint16), ks, Y.cpu().numpy())
    assert np.array_equal(full[:, ri].cpu().numpy(), ref.astype(np.float32))
    f = full.double()
    for q in range(Q):
        iq = idx[q]
        assert torch.equal(sc[q], full[q, iq])
        assert bool(torch.all(sc[q, :-1] >= sc[q, 1:]))
        rest = torch.ones(N, dtype=torch.bool, device=DEV)
        rest[iq] = False
        assert float(f[q][rest].max()) <= float(sc[q, -1])
    del codes
    torch.cuda.empty_cache()
