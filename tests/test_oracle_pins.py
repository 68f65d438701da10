"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: a brute-force
loop, a closed form, an identity from the paper, a textbook special case, or a
number the paper prints. None of these tests needs a GPU.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle as O
from paper_2609_37842_amd import synth as S

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def small_problem(seed, N=3, T=5, d_in=4, d_out=3, mask=None):
    g = np.random.default_rng(seed)
    a = g.standard_normal((N, T, d_in))
    ds = g.standard_normal((N, T, d_out))
    if mask is None:
        mask = np.ones((N, T), dtype=np.uint8)
    QA = S.haar_orthogonal(g, d_in)
    QS = S.haar_orthogonal(g, d_out)
    lam = g.lognormal(0, 1, size=(d_out, d_in))
    return a, ds, mask, QA, QS, lam


# --------------------------------------------------------------------------
# Selection (first stage, Section 3.2; eq. sigma_ekfac)
# --------------------------------------------------------------------------
def test_selection_matches_brute_force_sort():
    g = np.random.default_rng(1)
    lam = g.lognormal(0, 1, size=(7, 9))
    for m in (1, 5, 30, 63):
        ret = O.select_retained(lam, 0.1, m)
        items = [(lam[j, k], j * 9 + k) for j in range(7) for k in range(9)]
        brute = sorted(items, key=lambda t: (-t[0], t[1]))[:m]
        assert [f for _, f in brute] == ret.flat.tolist()
        assert np.array_equal(ret.j * 9 + ret.k, ret.flat)


def test_selection_ties_break_by_flat_index():
    lam = np.array([[1.0, 3.0, 3.0], [3.0, 2.0, 3.0]])
    ret = O.select_retained(lam, 1.0, 4)
    assert ret.flat.tolist() == [1, 2, 3, 5]
    ret = O.select_retained(lam, 1.0, 2)
    assert ret.flat.tolist() == [1, 2]


def test_selection_is_top_m_of_sigma_proxy_diagonal():
    # eq. sigma_ekfac: lambda_j/(lambda_j + lambda) is increasing in lambda_j,
    # so the m largest corrected eigenvalues are the m largest proxy variances.
    g = np.random.default_rng(2)
    lam = g.lognormal(0, 2, size=(11, 13))
    damping = 0.37
    m = 40
    ret = O.select_retained(lam, damping, m)
    proxy = (lam / (lam + damping)).ravel()
    kth = np.sort(proxy)[::-1][m - 1]
    assert np.all(proxy[ret.flat] >= kth)
    assert np.allclose(ret.w, 1.0 / np.sqrt(lam.ravel()[ret.flat] + damping), rtol=0, atol=0)


def test_selection_validation():
    lam = np.ones((2, 2))
    with pytest.raises(ValueError):
        O.select_retained(lam, 0.1, 0)
    with pytest.raises(ValueError):
        O.select_retained(lam, 0.1, 5)
    with pytest.raises(ValueError):
        O.select_retained(lam, 0.0, 2)
    with pytest.raises(ValueError):
        O.select_retained(-np.ones((2, 2)), 0.5, 2)


# --------------------------------------------------------------------------
# First stage (eq. first_stage, eq. app_projection_maps; K-FAC paragraph)
# --------------------------------------------------------------------------
def test_kronecker_identity_with_explicit_kron():
    # Coordinates of vec(G) in Q_A (x) Q_S equal the entries of Q_S^T G Q_A,
    # with (j, k) at position k*d_out + j of the column-major vec.
    a, ds, mask, QA, QS, lam = small_problem(3, d_in=4, d_out=3)
    G = O.per_example_gradient(a[0], ds[0], mask[0])
    coords = np.kron(QA, QS).T @ G.flatten(order="F")
    Gt = O.rotate(G, QA, QS)
    for j, k in itertools.product(range(3), range(4)):
        assert abs(coords[k * 3 + j] - Gt[j, k]) < 1e-12


def test_token_form_equals_explicit_gradient_form():
    a, ds, mask, QA, QS, lam = small_problem(4, N=4, T=7, d_in=6, d_out=5)
    mask = np.array([[1, 1, 0, 1, 1, 0, 1], [1] * 7, [0, 0, 1, 0, 0, 0, 0], [1, 0, 1, 0, 1, 0, 1]],
                    dtype=np.uint8)
    ret = O.select_retained(lam, 0.05, 17)
    for i in range(4):
        ze = O.first_stage_explicit(a[i], ds[i], mask[i], QA, QS, ret)
        zt = O.first_stage_tokens(a[i], ds[i], mask[i], QA, QS, ret)
        assert np.max(np.abs(ze - zt)) <= 1e-12 * max(1.0, np.max(np.abs(ze)))


def test_token_form_brute_force_loops():
    # Pure-Python loops over tokens and channels on a tiny case.
    a, ds, mask, QA, QS, lam = small_problem(5, N=1, T=3, d_in=3, d_out=2)
    mask = np.array([[1, 0, 1]], dtype=np.uint8)
    damping = 0.2
    ret = O.select_retained(lam, damping, 4)
    z = O.first_stage_tokens(a[0], ds[0], mask[0], QA, QS, ret)
    for r in range(4):
        j, k = int(ret.j[r]), int(ret.k[r])
        acc = 0.0
        for t in range(3):
            if mask[0, t] == 0:
                continue
            sj = sum(QS[c, j] * ds[0, t, c] for c in range(2))
            ak = sum(QA[c, k] * a[0, t, c] for c in range(3))
            acc += sj * ak
        expect = acc / math.sqrt(lam[j, k] + damping)
        assert abs(z[r] - expect) < 1e-12


def test_frobenius_norm_preserved_under_full_basis():
    # m = d_in*d_out and Lambda + lambda == 1 (unit weights): the first stage is
    # an orthogonal change of basis, so ||z||_2 = ||G||_F.
    a, ds, mask, QA, QS, _ = small_problem(6, N=2, T=9, d_in=5, d_out=4)
    damping = 1e-3
    lam = np.full((4, 5), 1.0 - damping)
    ret = O.select_retained(lam, damping, 20)
    assert np.allclose(ret.w, 1.0)
    for i in range(2):
        G = O.per_example_gradient(a[i], ds[i], mask[i])
        z = O.first_stage_tokens(a[i], ds[i], mask[i], QA, QS, ret)
        assert abs(np.linalg.norm(z) - np.linalg.norm(G)) < 1e-12 * np.linalg.norm(G)


def test_identity_bases_reduce_to_masked_gemm():
    # Q_A = Q_S = I: z_r = w_r * (DS^T diag(mask) A)[j_r, k_r].
    a, ds, mask, _, _, lam = small_problem(7, N=1, T=6, d_in=4, d_out=3)
    mask = np.array([[1, 1, 0, 0, 1, 1]], dtype=np.uint8)
    ret = O.select_retained(lam, 0.3, 7)
    z = O.first_stage_tokens(a[0], ds[0], mask[0], np.eye(4), np.eye(3), ret)
    G = ds[0].T @ np.diag(mask[0].astype(float)) @ a[0]
    assert np.allclose(z, ret.w * G[ret.j, ret.k], rtol=1e-13, atol=1e-14)


def test_masked_tokens_are_ignored_even_if_nan():
    a, ds, mask, QA, QS, lam = small_problem(8, N=2, T=6, d_in=4, d_out=3)
    mask = np.array([[1, 1, 1, 0, 0, 0], [0, 1, 0, 1, 0, 1]], dtype=np.uint8)
    ret = O.select_retained(lam, 0.1, 6)
    an = S.fill_masked(a, mask)
    dn = S.fill_masked(ds, mask)
    for i in range(2):
        keep = mask[i] != 0
        z_nan = O.first_stage_tokens(an[i], dn[i], mask[i], QA, QS, ret)
        z_cut = O.first_stage_tokens(a[i][keep], ds[i][keep], np.ones(keep.sum()), QA, QS, ret)
        assert np.all(np.isfinite(z_nan))
        assert np.allclose(z_nan, z_cut, rtol=0, atol=1e-14)


def test_all_tokens_masked_gives_zero():
    a, ds, mask, QA, QS, lam = small_problem(9, N=1, T=4)
    ret = O.select_retained(lam, 0.1, 5)
    z = O.first_stage_tokens(a[0], ds[0], np.zeros(4, np.uint8), QA, QS, ret)
    assert np.array_equal(z, np.zeros(5))


# --------------------------------------------------------------------------
# Half-whitening (eq. sigma_ekfac diagonal) on the tiny workload
# --------------------------------------------------------------------------
def test_half_whitened_second_moment_matches_proxy_diagonal(tiny_fit):
    # With Lambda fitted as the mean square of each coordinate over the same
    # examples, E_i[z_{i,r}^2] = Lambda_r / (Lambda_r + lambda) exactly.
    f = tiny_fit["fit"]
    ret = f["retained"]
    lhs = np.mean(f["Z"] ** 2, axis=0)
    rhs = ret.lam / (ret.lam + S.TINY.damping)
    assert np.max(np.abs(lhs - rhs)) < 1e-12


def test_ekfac_eigenvalues_parseval_identity_basis_and_symmetries():
    """Corrected eigenvalues (Section 2.2, eq. ekfac_eigendecompose) against
    gradients summed by explicit loops: with identity bases Lambda is the mean of
    the squared gradient entries; for any orthogonal bases the entries sum to the
    mean squared Frobenius norm (the rotation preserves it); permuting or
    negating basis columns permutes Lambda and leaves it unchanged otherwise."""
    a, ds, mask, QA, QS, _ = small_problem(81, N=4, T=6, d_in=5, d_out=3)
    mask[1, 4:] = 0
    mask[2, :] = 0
    N, T = mask.shape
    G = np.zeros((N, 3, 5))
    for i in range(N):
        for t in range(T):
            if mask[i, t]:
                for j in range(3):
                    for k in range(5):
                        G[i, j, k] += ds[i, t, j] * a[i, t, k]
    lam_id = O.ekfac_eigenvalues(a, ds, mask, np.eye(5), np.eye(3))
    assert np.allclose(lam_id, (G * G).mean(axis=0), rtol=1e-13, atol=0)
    lam = O.ekfac_eigenvalues(a, ds, mask, QA, QS)
    assert np.isclose(lam.sum(), (G * G).sum(axis=(1, 2)).mean(), rtol=1e-12)
    assert np.all(lam >= 0)
    pa, ps = np.array([3, 0, 4, 1, 2]), np.array([2, 0, 1])
    sa, ss = np.array([1, -1, 1, -1, -1]), np.array([-1, 1, 1])
    lam_p = O.ekfac_eigenvalues(a, ds, mask, QA[:, pa] * sa, QS[:, ps] * ss)
    assert np.allclose(lam_p, lam[np.ix_(ps, pa)], rtol=1e-12, atol=0)


def test_kfac_factors_loop_sum_over_valid_tokens():
    """K-FAC factors (Section 2.2, eq. kfac_factorization; Appendix C.2: factor
    statistics averaged over non-padding tokens) against outer products summed
    token by token in pure Python and divided by the number of valid tokens.
    Masked tokens hold NaN, so reading one poisons the result; the valid count
    (11) differs from N*T (15) and from the per-example mean, so a wrong
    normaliser fails too."""
    g = np.random.default_rng(91)
    N, T, d_in, d_out = 3, 5, 4, 3
    a = g.standard_normal((N, T, d_in))
    ds = g.standard_normal((N, T, d_out))
    mask = np.array([[1, 1, 1, 0, 0], [1, 1, 1, 1, 1], [0, 1, 1, 1, 0]], dtype=np.uint8)
    a[mask == 0] = np.nan
    ds[mask == 0] = np.nan
    n_valid = int(mask.sum())
    assert n_valid == 11
    A_ref = [[0.0] * d_in for _ in range(d_in)]
    S_ref = [[0.0] * d_out for _ in range(d_out)]
    for i in range(N):
        for t in range(T):
            if not mask[i, t]:
                continue
            for p in range(d_in):
                for q in range(d_in):
                    A_ref[p][q] += float(a[i, t, p]) * float(a[i, t, q])
            for p in range(d_out):
                for q in range(d_out):
                    S_ref[p][q] += float(ds[i, t, p]) * float(ds[i, t, q])
    A, Sf = O.kfac_factors(a, ds, mask)
    assert np.all(np.isfinite(A)) and np.all(np.isfinite(Sf))
    assert np.allclose(A, np.array(A_ref) / n_valid, rtol=1e-13, atol=0)
    assert np.allclose(Sf, np.array(S_ref) / n_valid, rtol=1e-13, atol=0)


def test_kfac_factors_closed_form_with_basis_vector_tokens():
    """Closed form: when every valid activation token is a standard basis
    vector e_c and every output-gradient token is 2 e_c', the factors are
    diagonal with entries count_c / n_valid and 4 count_c' / n_valid."""
    N, T, d = 2, 6, 3
    a = np.full((N, T, d), np.nan)
    ds = np.full((N, T, d), np.nan)
    mask = np.zeros((N, T), dtype=np.uint8)
    cols = {(0, 0): 0, (0, 1): 0, (0, 3): 2, (1, 0): 1, (1, 2): 0, (1, 5): 2}
    for (i, t), c in cols.items():
        mask[i, t] = 1
        a[i, t] = np.eye(d)[c]
        ds[i, t] = 2.0 * np.eye(d)[(c + 1) % d]
    A, Sf = O.kfac_factors(a, ds, mask)
    counts = np.bincount(list(cols.values()), minlength=d).astype(np.float64)
    assert np.array_equal(A, np.diag(counts / 6.0))
    assert np.array_equal(Sf, np.diag(4.0 * np.roll(counts, 1) / 6.0))


def test_relative_damping_hand_computed():
    """Appendix C.2 (eq. app_module_damping): lambda_u = 0.1 tr(Lambda_u) / d_u
    over the module's full set of corrected eigenvalues. Hand-computed:
    Lambda = [[1, 2, 3], [4, 5, 9]] has trace of the diagonal matrix 24 over
    d_u = 6 parameters, so lambda_u = 0.4. The rule is linear in Lambda and
    depends only on the multiset of eigenvalues (not their layout)."""
    lam = np.array([[1.0, 2.0, 3.0], [4.0, 5.0, 9.0]])
    assert O.relative_damping(lam) == pytest.approx(0.4, rel=1e-15)
    assert O.relative_damping(7.0 * lam) == pytest.approx(2.8, rel=1e-15)
    assert O.relative_damping(lam.T) == pytest.approx(0.4, rel=1e-15)
    assert O.relative_damping(np.full((5, 7), 3.0)) == pytest.approx(0.3, rel=1e-15)


def test_kfac_eigenbasis_diagonalises_factors(tiny_fit):
    f = tiny_fit["fit"]
    for F, Q in ((f["A"], f["Q_A"]), (f["S"], f["Q_S"])):
        D = Q.T @ F @ Q
        assert np.max(np.abs(D - np.diag(np.diag(D)))) < 1e-10 * np.max(np.abs(F))
        assert np.allclose(Q.T @ Q, np.eye(Q.shape[0]), atol=1e-12)


# --------------------------------------------------------------------------
# Second stage (eq. second_stage; Propositions 1 and 2)
# --------------------------------------------------------------------------
def test_pca_directions_orthonormal_and_eigen(tiny_fit):
    f = tiny_fit["fit"]
    P, mu, Z = f["P"], f["mu"], f["Z"]
    k = P.shape[1]
    assert np.allclose(P.T @ P, np.eye(k), atol=1e-12)
    C = Z.T @ Z / Z.shape[0]
    assert np.max(np.abs(C @ P - P * mu[:k][None, :])) < 1e-10 * mu[0]
    assert np.all(np.diff(mu) <= 1e-15)


def test_pca_fit_equals_svd_and_gram_routes():
    # PCA fitting (appendix on PCA fitting): the columns of P are the top-k
    # right singular vectors of Z, equivalently eigenvectors of Z^T Z / n, and
    # they follow from the n x n Gram matrix Z Z^T as Z^T v / sqrt(lambda).
    # Both routes (an SVD, and the Gram eigendecomposition) must give the
    # oracle's P up to the sign rule, for n < m and n > m.
    g = np.random.default_rng(31)
    for n, m, k in ((40, 64, 12), (90, 30, 10)):
        U, _ = np.linalg.qr(g.standard_normal((n, min(n, m))))
        W, _ = np.linalg.qr(g.standard_normal((m, min(n, m))))
        s = 2.0 ** -np.arange(min(n, m)) * 10.0          # well separated
        Z = (U * s) @ W.T
        P, mu = O.pca_fit(Z, k)
        _, sv, Vt = np.linalg.svd(Z, full_matrices=False)
        V = Vt[:k].T
        assert np.allclose(np.abs(np.sum(P * V, axis=0)), 1.0, atol=1e-10)
        assert np.allclose(mu[:k], sv[:k] ** 2 / n, rtol=1e-10)
        lam, Vg = np.linalg.eigh(Z @ Z.T)
        lam, Vg = lam[::-1][:k], Vg[:, ::-1][:, :k]
        Pg = Z.T @ Vg / np.sqrt(lam)[None, :]
        assert np.allclose(np.abs(np.sum(P * Pg, axis=0)), 1.0, atol=1e-10)
        # sign rule: the largest-magnitude entry of every column is positive
        piv = np.argmax(np.abs(P), axis=0)
        assert np.all(P[piv, np.arange(k)] > 0)


def test_proposition1_optimal_value(tiny_fit):
    # Within the first-stage span, the PCA reconstruction error equals the sum
    # of the trailing eigenvalues (eq. app_optimal_value) and beats random
    # k-dimensional orthonormal bases.
    f = tiny_fit["fit"]
    P, mu, Z = f["P"], f["mu"], f["Z"]
    k = P.shape[1]
    err = np.mean(np.sum((Z - (Z @ P) @ P.T) ** 2, axis=1))
    assert abs(err - mu[k:].sum()) < 1e-10 * mu.sum()
    g = np.random.default_rng(10)
    for _ in range(3):
        W, _ = np.linalg.qr(g.standard_normal((Z.shape[1], k)))
        err_w = np.mean(np.sum((Z - (Z @ W) @ W.T) ** 2, axis=1))
        assert err_w >= err


def test_proposition2_correction_beats_leading_axes(tiny_fit):
    # Full-space EK-FAC half-whitened gradients t = Q (Lambda+lambda)^-1/2 Q^T g;
    # the corrected basis Q_m P reconstructs them at least as well as the
    # leading k retained axes, and the error splits as in
    # eq. app_restricted_reconstruction.
    raw, f = tiny_fit["raw"], tiny_fit["fit"]
    QA, QS, lam, ret, P = f["Q_A"], f["Q_S"], f["eigvals"], f["retained"], f["P"]
    d_out, d_in = lam.shape
    damping = S.TINY.damping
    Q = np.kron(QA, QS)                          # column k*d_out + j
    lam_col = lam.flatten(order="F")
    cols = ret.k * d_out + ret.j                 # retained axes as columns of Q
    Qm = Q[:, cols]
    k = P.shape[1]
    err_star = err_lead = err_out = 0.0
    for i in range(raw["a"].shape[0]):
        g = O.per_example_gradient(raw["a"][i], raw["ds"][i], raw["mask"][i]).flatten(order="F")
        t = Q @ ((Q.T @ g) / np.sqrt(lam_col + damping))
        U = Qm @ P
        Qk = Qm[:, :k]
        err_star += np.sum((t - U @ (U.T @ t)) ** 2)
        err_lead += np.sum((t - Qk @ (Qk.T @ t)) ** 2)
        err_out += np.sum((t - Qm @ (Qm.T @ t)) ** 2)
    n = raw["a"].shape[0]
    assert err_star <= err_lead
    within = np.mean(np.sum((f["Z"] - (f["Z"] @ P) @ P.T) ** 2, axis=1))
    assert abs(err_star / n - (err_out / n + within)) < 1e-9 * err_star / n


# --------------------------------------------------------------------------
# One-bit encoding (eq. onebit, eq. app_onebit_scale, eq. app_payload)
# --------------------------------------------------------------------------
def test_onebit_scale_is_least_squares_optimum():
    g = np.random.default_rng(11)
    x = g.standard_normal(97)
    b = 2.0 * O.sign_bits(x) - 1.0
    k = x.size
    assert abs(b @ x - np.abs(x).sum()) < 1e-12
    s_star = np.abs(x).sum() / k
    resid = np.sum((x - s_star * b) ** 2)
    assert abs(resid - (x @ x - np.abs(x).sum() ** 2 / k)) < 1e-10
    for s in (0.0, 0.5 * s_star, 1.5 * s_star, s_star + 1e-3):
        lhs = np.sum((x - s * b) ** 2)
        rhs = k * (s - s_star) ** 2 + x @ x - np.abs(x).sum() ** 2 / k
        assert abs(lhs - rhs) < 1e-9
        assert lhs >= resid - 1e-12


def test_sign_of_zero_and_negative_zero():
    x = np.array([0.0, -0.0, -1e-300, 1e-300, -2.0, np.inf, -np.inf])
    assert O.sign_bits(x).tolist() == [1, 1, 0, 1, 0, 1, 0]


def test_pack_bits_brute_force_layout():
    g = np.random.default_rng(12)
    for k in (8, 13, 64, 100):
        bits = g.integers(0, 2, size=(3, k)).astype(np.uint8)
        packed = O.pack_bits(bits)
        assert packed.shape == (3, -(-k // 8))
        for i in range(3):
            manual = [0] * (-(-k // 8))
            for c in range(k):
                if bits[i, c]:
                    manual[c >> 3] |= 1 << (c & 7)
            assert packed[i].tolist() == manual
        assert np.array_equal(O.unpack_bits(packed, k), bits)


def test_scale_rounds_once_to_nearest_even():
    # 1 + 2^-11 lies halfway between fp16 1.0 and 1 + 2^-10: ties to even -> 1.0;
    # 1 + 3*2^-11 is halfway between 1+2^-10 and 1+2^-9: ties to even -> 1+2^-9.
    for target, expect in ((1 + 2.0 ** -11, 1.0), (1 + 3 * 2.0 ** -11, 1 + 2.0 ** -9),
                           (1 + 2.0 ** -11 + 2.0 ** -30, 1 + 2.0 ** -10)):
        x = np.array([target, -target, target, -target])
        s = O.onebit_scale(x).view(np.float16)
        assert float(s) == expect
    # overflow of the fp16 range gives +inf
    assert np.isinf(O.onebit_scale(np.array([1e6, -1e6])).view(np.float16))


def test_payload_and_storage_figures_reproduce_paper_numbers():
    gold = json.load(open(os.path.join(GOLDEN, "storage_costs.json")))
    assert O.payload_bytes([2048]) == gold["bytes_per_module_k2048"]
    # Linear modules per transformer block (q, k, v, o, gate, up, down).
    def olmo(hidden, mlp, blocks, kv=None):
        kv = hidden if kv is None else kv
        per = [(hidden, hidden), (hidden, kv), (hidden, kv), (hidden, hidden),
               (hidden, mlp), (hidden, mlp), (mlp, hidden)]
        return per * blocks
    models = {"olmo2-1b": olmo(2048, 8192, 16), "olmo2-7b": olmo(4096, 11008, 32),
              "olmo2-13b": olmo(5120, 13824, 40), "olmo2-32b": olmo(5120, 27648, 64, kv=1024)}
    for name, mods in models.items():
        row = gold["payload_table"][name]
        kb = O.payload_bytes([2048] * len(mods)) / 1000.0
        gb = 2 * sum(di * do for di, do in mods) / 1e9
        assert round(kb, 3) == row["onebit_KB"]
        assert round(gb, 3) == row["uncompressed_fp16_GB"]
    n32 = len(models["olmo2-32b"])
    assert n32 == gold["olmo2-32b_modules"]
    m = gold["olmo2-32b_m"]
    p_mod = 2 * m * 2048                        # eq. app_correction_storage
    assert round(p_mod / 1e9, 2) == gold["olmo2-32b_P_GB_per_module"]
    assert round(n32 * p_mod / 1e9) == gold["olmo2-32b_P_GB_total"]
    assert round(n32 * 2 * m * 256 / 1e9, 1) == gold["olmo2-32b_P_GB_total_k256"]
    payload = O.payload_bytes([2048] * n32)
    assert round(n32 * p_mod / (1e8 * payload), 3) == gold["P_share_of_payload_1e8"]
    assert round(n32 * p_mod / (1e9 * payload), 4) == gold["P_share_of_payload_1e9"]
    # GPT-2 small: attention and MLP linears with biases, 12 blocks, FP16.
    gpt2 = 12 * sum(di * do for _, di, do in S.GPT2_BLOCK)
    assert round(2 * gpt2 / 2 ** 20) == gold["gpt2_uncompressed_fp16_MB"]


# --------------------------------------------------------------------------
# Scoring (eq. onebit_influence, eq. app_stored_influence) and top-k
# --------------------------------------------------------------------------
def random_store(seed, N, ks, Q):
    g = np.random.default_rng(seed)
    nbytes = sum(-(-k // 8) for k in ks)
    codes = g.integers(0, 256, size=(N, nbytes), dtype=np.uint8)
    scales = np.exp(g.standard_normal((N, len(ks)))).astype(np.float16).view(np.uint16)
    Y = g.standard_normal((Q, sum(ks))).astype(np.float32)
    return codes, scales, Y


def test_score_brute_force_loops():
    ks = [16, 8]
    codes, scales, Y = random_store(13, 5, ks, 3)
    sc = O.score(codes, scales, ks, Y)
    s16 = scales.view(np.float16).astype(np.float64)
    for q in range(3):
        for i in range(5):
            total = 0.0
            off_c, off_b = 0, 0
            for u, k in enumerate(ks):
                y_int, f = O.query_fixed_point(Y[q, off_c:off_c + k])
                n = 0
                for c in range(k):
                    bit = (int(codes[i, off_b + (c >> 3)]) >> (c & 7)) & 1
                    n += int(y_int[c]) * (1 if bit else -1)
                total = total + float(s16[i, u]) * n * 2.0 ** (-f)
                off_c += k
                off_b += k // 8
            assert sc[q, i] == total


def test_score_signed_identity_and_fixed_point_bounds():
    ks = [64]
    codes, scales, Y = random_store(14, 7, ks, 4)
    b = O.unpack_bits(codes, 64).astype(np.int64)
    for q in range(4):
        y_int, f = O.query_fixed_point(Y[q])
        assert np.max(np.abs(y_int)) <= 2 ** 14
        assert 2 ** 13 <= np.max(np.abs(y_int))
        lhs = (2 * b - 1) @ y_int
        rhs = 2 * (b @ y_int) - y_int.sum()
        assert np.array_equal(lhs, rhs)
        # fixed point keeps each coordinate within half a unit of the last place
        assert np.max(np.abs(np.ldexp(y_int.astype(float), -f) - Y[q])) <= 2.0 ** (-f - 1)


def test_integral_queries_score_exactly_the_real_formula():
    ks = [32, 64]
    codes, scales, _ = random_store(15, 9, ks, 3)
    g = np.random.default_rng(16)
    Y = g.integers(-9000, 9000, size=(3, 96)).astype(np.float32)
    assert np.array_equal(O.score(codes, scales, ks, Y), O.score_real(codes, scales, ks, Y))


def test_zero_query_scores_zero():
    ks = [64]
    codes, scales, _ = random_store(17, 4, ks, 1)
    assert np.array_equal(O.score(codes, scales, ks, np.zeros((1, 64), np.float32)),
                          np.zeros((1, 4)))


def test_fixed_point_score_close_to_real_score():
    ks = [256, 128]
    codes, scales, Y = random_store(18, 50, ks, 6)
    exact = O.score_real(codes, scales, ks, Y)
    fixed = O.score(codes, scales, ks, Y)
    s16 = scales.view(np.float16).astype(np.float64)
    # each coordinate moves by at most half an ulp of the fixed point
    bound = np.zeros_like(exact)
    off = 0
    for u, k in enumerate(ks):
        for q in range(6):
            _, f = O.query_fixed_point(Y[q, off:off + k])
            bound[q] += s16[:, u] * k * 2.0 ** (-f - 1)
        off += k
    assert np.all(np.abs(exact - fixed) <= bound * (1 + 1e-12))


def test_topk_brute_force_with_ties_and_padding():
    S_ = np.array([[3.0, 1.0, 3.0, -2.0, 1.0], [0.0, 0.0, 0.0, 0.0, 0.0]])
    idx, val = O.topk(S_, 3)
    assert idx.tolist() == [[0, 2, 1], [0, 1, 2]]
    assert val.dtype == np.float32
    idx, val = O.topk(S_, 7)
    assert idx[0].tolist() == [0, 2, 1, 4, 3, -1, -1]
    assert np.isneginf(val[0, 5]) and np.isneginf(val[0, 6])
    g = np.random.default_rng(19)
    R = np.round(g.standard_normal((4, 40)), 1)
    idx, val = O.topk(R, 10)
    for q in range(4):
        brute = sorted(range(40), key=lambda i: (-R[q, i], i))[:10]
        assert idx[q].tolist() == brute


# --------------------------------------------------------------------------
# Whole passes on the tiny workload
# --------------------------------------------------------------------------
def test_tiny_store_and_query_roundtrip(tiny_fit):
    raw, art = tiny_fit["raw"], tiny_fit["art"]
    w = S.TINY
    Z, X, codes, scales = O.store(raw["a"], raw["ds"], raw["mask"], art["Q_A"], art["Q_S"],
                                  art["eigvals"], art["damping"], w.m, art["P"])
    assert codes.shape == (w.N, w.k // 8) and scales.shape == (w.N,)
    Y = O.query(raw["qa"], raw["qds"], raw["qmask"], art["Q_A"], art["Q_S"],
                art["eigvals"], art["damping"], w.m, art["P"])
    sc = O.score(codes, scales, [w.k], Y.astype(np.float32))
    # One-bit scores track the unquantized influence <y, x> (Section 3.3). For
    # roughly Gaussian coordinates the correlation of s*sign(x) with x is
    # sqrt(2/pi) ~ 0.798, and the score correlation sits near it.
    full = Y @ X.T
    rho = [np.corrcoef(sc[q], full[q])[0, 1] for q in range(w.Q)]
    assert min(rho) > 0.6
    assert abs(np.median(rho) - math.sqrt(2 / math.pi)) < 0.08


def test_partition_selection_helper_matches_full_sort():
    """The tests' O(n) selection for very large Lambda agrees with the
    oracle's full sort, ties included."""
    from select_helpers import restrict, select_large
    g = np.random.default_rng(31)
    lam = np.round(g.lognormal(0, 1, (97, 53)), 1)        # many exact ties
    for m in (1, 100, 2000, 97 * 53):
        a = O.select_retained(lam, 0.01, m)
        b = select_large(lam, 0.01, m)
        assert np.array_equal(a.flat, b.flat)
        assert np.allclose(a.w, b.w, rtol=0, atol=0)
    sub, J, K = restrict(a, np.arange(0, 97 * 53, 7))
    assert np.array_equal(J[sub.j], a.j[::7]) and np.array_equal(K[sub.k], a.k[::7])


# ---------------------------------------------------------------------------
# SRHT second stage (Appendix B.2)
# ---------------------------------------------------------------------------
def test_walsh_hadamard_matches_sylvester_matrix():
    import scipy.linalg
    g = np.random.default_rng(41)
    for p in (1, 2, 8, 64, 1024):
        x = g.standard_normal((3, p))
        H = scipy.linalg.hadamard(p).astype(np.float64)
        assert np.allclose(O.walsh_hadamard(x), x @ H.T, rtol=0, atol=1e-10)


def test_srht_width_and_padding():
    assert [O.srht_width(m) for m in (1, 2, 3, 512, 513, 16384, 32767)] == \
        [1, 2, 4, 512, 1024, 16384, 32768]
    # padding: the transform of a width-m vector equals that of its zero-padded copy
    g = np.random.default_rng(42)
    z = g.standard_normal((2, 300))
    signs = g.choice([-1, 1], 300)
    rows = g.choice(512, 40, replace=False)
    zp = np.concatenate([z, np.zeros((2, 212))], axis=1)
    sp = np.concatenate([signs, np.ones(212, int)])
    assert np.allclose(O.srht_project(z, signs, rows), O.srht_project(zp, sp, rows), atol=1e-12)


def test_srht_full_rows_is_orthonormal():
    """With all p rows kept the map is sqrt(p/p) H D J: orthonormal, so the
    norm and inner products of the (padded) inputs are preserved."""
    g = np.random.default_rng(43)
    m = 200
    z = g.standard_normal((4, m))
    signs = g.choice([-1, 1], m)
    p = O.srht_width(m)
    x = O.srht_project(z, signs, np.arange(p))
    assert np.allclose(x @ x.T, z @ z.T, rtol=0, atol=1e-9)


def test_srht_explicit_matrix_small_case():
    """Against the printed definition with explicit matrices: R (k x p row
    selector), H_p / sqrt(p), D = diag(signs), J (p x m zero padding)."""
    import scipy.linalg
    g = np.random.default_rng(44)
    m, k = 13, 5
    p = 16
    z = g.standard_normal((3, m))
    signs = g.choice([-1, 1], m)
    rows = g.choice(p, k, replace=False)
    R = np.eye(p)[rows]
    H = scipy.linalg.hadamard(p) / np.sqrt(p)
    D = np.diag(np.concatenate([signs, np.ones(p - m)]))
    J = np.eye(p)[:, :m]
    S_ = np.sqrt(p / k) * R @ H @ D @ J
    assert np.allclose(O.srht_project(z, signs, rows), z @ S_.T, rtol=0, atol=1e-12)


def test_srht_preserves_squared_norm_in_expectation():
    """E over row subsets of ||S z||^2 = ||z||^2 (each row of H D J z has
    mean square ||z||^2 / p); averaged over many draws."""
    g = np.random.default_rng(45)
    m, k = 100, 16
    z = g.standard_normal((1, m))
    signs = g.choice([-1, 1], m)
    p = O.srht_width(m)
    tot = np.mean([np.sum(O.srht_project(z, signs, g.choice(p, k, replace=False)) ** 2)
                   for _ in range(4000)])
    assert abs(tot / np.sum(z ** 2) - 1.0) < 0.03

