"""EOGP oracle: a plain, slow, fp64 CPU statement of the hot path.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package. The product path
(the HIP library and its Python binding) never calls into it, and this package
imports nothing from the product path.

Every function follows the paper's definitions in their order and notation
(Section 3, Algorithm 1 and the appendix on projection implementation), in
numpy float64. Library primitives (matmul, sort, eigh, float16 rounding) serve
as steps; there is no blocking, fusion or reordering beyond what the
definitions state. Inputs are float64 copies of exactly the arrays handed to the
GPU.

Readings of points the paper leaves open (each is also listed in the design doc):
  * index convention: corrected eigenvalues are given as Lambda[j, k] with row
    j <-> output-side eigenvector Q_S[:, j] and column k <-> input-side
    eigenvector Q_A[:, k]; coordinate (j, k) of the rotated gradient is
    (Q_S^T G Q_A)[j, k], the entry of (Q_A (x) Q_S)^T vec(G) at k*d_out + j
    (Section 2, K-FAC paragraph);
  * retained order and ties: all coordinates sorted by (Lambda descending,
    flat index j*d_in + k ascending); the first m are kept in that order;
  * mask: the per-example gradient sums only valid tokens (token-summed loss);
  * sign of zero: bit = 1 (+1) iff x >= 0, so -0.0 encodes as +1;
  * bit layout: coordinate c of a module lands in byte c >> 3, bit c & 7
    (least significant bit first); codes of several modules are concatenated,
    and scales are stored apart from the bits, one fp16 per (example, module);
  * scale: fp16 of ||x||_1 / k, rounded once, to nearest even;
  * random second stage (EOGP-R): the Walsh-Hadamard matrix is in Sylvester
    (natural) order, entry (r, i) = (-1)^popcount(r & i); the random signs
    and the k kept rows are inputs (drawn by the caller), and coordinate c of
    the output is transform row rows[c];
  * scoring: the query coordinates are kept to 15 significant bits by a
    per-(query, module) power of two (fixed point), so <y, b> is an exact
    integer; module terms are summed in float64 in ascending module order;
    ranking is by (score descending, example index ascending).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


# ---------------------------------------------------------------------------
# Fitting shared projections (Algorithm 1, first block)
# ---------------------------------------------------------------------------
@dataclass
class Retained:
    """The retained EK-FAC axes of one module, in canonical order."""
    flat: np.ndarray   # int64 [m], flat index j*d_in + k
    j: np.ndarray      # int64 [m], output-side eigenvector index
    k: np.ndarray      # int64 [m], input-side eigenvector index
    lam: np.ndarray    # float64 [m], corrected eigenvalues Lambda_m
    w: np.ndarray      # float64 [m], half-whitening weights (Lambda_m + lambda)^-1/2


def select_retained(eigvals: np.ndarray, damping: float, m: int) -> Retained:
    """Keep the m axes with the largest corrected eigenvalues (first stage of
    Section 3.2; eq. sigma_ekfac: lambda_j/(lambda_j+lambda) grows with lambda_j,
    so these axes span the top-m PCA subspace of Sigma_proxy)."""
    lam = np.asarray(eigvals, dtype=np.float64)
    d_out, d_in = lam.shape
    if not (1 <= m <= d_out * d_in):
        raise ValueError("need 1 <= m <= d_in*d_out")
    if not damping > 0:
        raise ValueError("damping must be positive")
    flat_lam = lam.reshape(-1)
    flat_idx = np.arange(flat_lam.size, dtype=np.int64)
    # Primary key: Lambda descending; secondary key: flat index ascending.
    order = np.lexsort((flat_idx, -flat_lam))
    keep = order[:m]
    lam_m = flat_lam[keep]
    if np.any(~np.isfinite(lam_m)) or np.any(lam_m + damping <= 0):
        raise ValueError("retained Lambda + lambda must be positive and finite")
    # eq. first_stage: scaling by (Lambda_m + lambda I)^-1/2
    w = 1.0 / np.sqrt(lam_m + float(damping))
    return Retained(flat=keep, j=keep // d_in, k=keep % d_in, lam=lam_m, w=w)


def kfac_factors(a: np.ndarray, ds: np.ndarray, mask: np.ndarray):
    """K-FAC factors A = E[a a^T], S = E[ds ds^T] (eq. kfac_factorization),
    averaged over non-padding tokens of all examples."""
    valid = np.asarray(mask) != 0
    av = np.asarray(a, dtype=np.float64)[valid]
    dv = np.asarray(ds, dtype=np.float64)[valid]
    n = av.shape[0]
    return av.T @ av / n, dv.T @ dv / n


def eigenbasis(F: np.ndarray) -> np.ndarray:
    """Orthonormal eigenbasis of a symmetric factor (columns = eigenvectors),
    each column's largest-magnitude entry made positive."""
    _, V = np.linalg.eigh(F)
    piv = np.argmax(np.abs(V), axis=0)
    sgn = np.sign(V[piv, np.arange(V.shape[1])])
    sgn[sgn == 0] = 1.0
    return V * sgn[None, :]


def ekfac_eigenvalues(a, ds, mask, Q_A, Q_S) -> np.ndarray:
    """Corrected eigenvalues (eq. ekfac_eigendecompose): the mean over examples
    of the squared coordinates of each sequence-level gradient in Q_A (x) Q_S,
    returned as Lambda[j, k]."""
    N = a.shape[0]
    acc = 0.0
    for i in range(N):
        Gt = rotate(per_example_gradient(a[i], ds[i], mask[i]), Q_A, Q_S)
        acc = acc + Gt * Gt
    return acc / N


def relative_damping(eigvals: np.ndarray) -> float:
    """lambda_u = 0.1 tr(Lambda_u) / d_u (eq. app_module_damping)."""
    lam = np.asarray(eigvals, dtype=np.float64)
    return 0.1 * float(lam.sum()) / lam.size


def pca_fit(Z: np.ndarray, k: int):
    """Uncentered PCA of first-stage coordinates (appendix on PCA fitting):
    P = top-k eigenvectors of Z^T Z / n, sorted by eigenvalue descending, each
    column's largest-magnitude entry made positive. Returns (P [m,k], mu [m])."""
    Z = np.asarray(Z, dtype=np.float64)
    C = Z.T @ Z / Z.shape[0]
    mu, V = np.linalg.eigh(C)
    order = np.argsort(-mu, kind="stable")
    mu = mu[order]
    V = V[:, order]
    P = V[:, :k]
    piv = np.argmax(np.abs(P), axis=0)
    sgn = np.sign(P[piv, np.arange(k)])
    sgn[sgn == 0] = 1.0
    return P * sgn[None, :], mu


# ---------------------------------------------------------------------------
# First stage: z = L_u g = (Lambda_m + lambda I)^-1/2 Q_m^T g  (eq. first_stage,
# eq. app_projection_maps)
# ---------------------------------------------------------------------------
def valid_tokens(mask_row: np.ndarray) -> np.ndarray:
    """Token positions that enter the token-summed loss."""
    return np.flatnonzero(np.asarray(mask_row) != 0)


def per_example_gradient(a_i, ds_i, mask_i) -> np.ndarray:
    """g_i of one linear module as a matrix: G = sum_{valid t} ds_t a_t^T
    ([d_out, d_in])."""
    V = valid_tokens(mask_i)
    A = np.asarray(a_i, dtype=np.float64)[V]
    D = np.asarray(ds_i, dtype=np.float64)[V]
    return D.T @ A


def rotate(G, Q_A, Q_S) -> np.ndarray:
    """Coordinates of G in the Kronecker eigenbasis: Q_S^T G Q_A."""
    return np.asarray(Q_S, np.float64).T @ G @ np.asarray(Q_A, np.float64)


def first_stage_explicit(a_i, ds_i, mask_i, Q_A, Q_S, ret: Retained) -> np.ndarray:
    """z_i formed from the explicit gradient matrix (small sizes only)."""
    Gt = rotate(per_example_gradient(a_i, ds_i, mask_i), Q_A, Q_S)
    return ret.w * Gt[ret.j, ret.k]


def first_stage_tokens(a_i, ds_i, mask_i, Q_A, Q_S, ret: Retained,
                       coords: np.ndarray | None = None) -> np.ndarray:
    """The same z_i through the two Kronecker factors, without forming G:
    z_r = w_r * sum_{valid t} (Q_S[:, j_r] . ds_t) (Q_A[:, k_r] . a_t).
    ``coords`` restricts the output to those retained positions r."""
    r = np.arange(ret.flat.size) if coords is None else np.asarray(coords)
    jr, kr, wr = ret.j[r], ret.k[r], ret.w[r]
    V = valid_tokens(mask_i)
    A = np.asarray(a_i, dtype=np.float64)[V]
    D = np.asarray(ds_i, dtype=np.float64)[V]
    J, jinv = np.unique(jr, return_inverse=True)
    K, kinv = np.unique(kr, return_inverse=True)
    At = A @ np.asarray(Q_A, np.float64)[:, K]        # [T_eff, |K|]
    St = D @ np.asarray(Q_S, np.float64)[:, J]        # [T_eff, |J|]
    return wr * np.einsum("tr,tr->r", St[:, jinv], At[:, kinv])


def first_stage_batch(a, ds, mask, Q_A, Q_S, ret: Retained) -> np.ndarray:
    """Z [N, m]: first-stage coordinates of every example (token form)."""
    return np.stack([first_stage_tokens(a[i], ds[i], mask[i], Q_A, Q_S, ret)
                     for i in range(a.shape[0])])


# ---------------------------------------------------------------------------
# Second stage: x = P^T z  (eq. second_stage)
# ---------------------------------------------------------------------------
def pca_project(Z: np.ndarray, P: np.ndarray) -> np.ndarray:
    """Rows of X are P^T z_i for the rows z_i of Z. P is [m, k]."""
    return np.asarray(Z, np.float64) @ np.asarray(P, np.float64)


# ---------------------------------------------------------------------------
# Random second stage, EOGP-R (Appendix B.2, eq. app_srht_definition)
# ---------------------------------------------------------------------------
def srht_width(m: int) -> int:
    """p = 2^ceil(log2 m), the zero-padded width of the transform."""
    return 1 << max(0, int(m - 1).bit_length())


def walsh_hadamard(x: np.ndarray) -> np.ndarray:
    """Unnormalised Walsh-Hadamard transform in Sylvester (natural) order
    along the last axis: y[r] = sum_i (-1)^popcount(r & i) x[i], computed by
    the butterfly recursion H_2n = [[H_n, H_n], [H_n, -H_n]]."""
    y = np.array(x, dtype=np.float64, copy=True)
    p = y.shape[-1]
    h = 1
    while h < p:
        v = y.reshape(y.shape[:-1] + (p // (2 * h), 2, h))
        a = v[..., 0, :].copy()
        b = v[..., 1, :].copy()
        v[..., 0, :] = a + b
        v[..., 1, :] = a - b
        h *= 2
    return y


def srht_project(Z: np.ndarray, signs: np.ndarray, rows: np.ndarray) -> np.ndarray:
    """x = sqrt(p/k) R H_p D J z for each row z of Z [N, m]: J zero-pads to
    p, D multiplies by the random signs [m] (+1 / -1), H_p is the orthonormal
    Walsh-Hadamard matrix (the unnormalised one over sqrt(p)), and R keeps
    the rows `rows` [k] in that order; so x = (H (D J z))[rows] / sqrt(k)."""
    Z = np.asarray(Z, np.float64)
    N, m = Z.shape
    p = srht_width(m)
    k = len(rows)
    zp = np.zeros((N, p))
    zp[:, :m] = Z * np.where(np.asarray(signs) < 0, -1.0, 1.0)[None, :]
    y = walsh_hadamard(zp) / np.sqrt(p)
    return np.sqrt(p / k) * y[:, np.asarray(rows, np.int64)]


# ---------------------------------------------------------------------------
# One-bit encoding (eq. onebit; Algorithm 1, storing one example)
# ---------------------------------------------------------------------------
def sign_bits(x: np.ndarray) -> np.ndarray:
    """b = sign(x) as bits: 1 for +1 (x >= 0, including -0.0), 0 for -1."""
    return (np.asarray(x, dtype=np.float64) >= 0).astype(np.uint8)


def pack_bits(bits: np.ndarray) -> np.ndarray:
    """Byte-pack the last axis, coordinate c -> byte c >> 3, bit c & 7."""
    return np.packbits(np.asarray(bits, dtype=np.uint8), axis=-1, bitorder="little")


def onebit_scale(x: np.ndarray) -> np.ndarray:
    """s = FP16(||x||_1 / k) over the last axis (eq. onebit), one rounding
    from float64 to fp16 (nearest even). Returned as fp16 bit patterns."""
    x = np.asarray(x, dtype=np.float64)
    k = x.shape[-1]
    with np.errstate(over="ignore"):          # IEEE overflow to +inf is the rule
        return (np.sum(np.abs(x), axis=-1) / k).astype(np.float16).view(np.uint16)


def encode(X: np.ndarray):
    """Codes [N, ceil(k/8)] and fp16 scales [N] of projected coordinates X."""
    return pack_bits(sign_bits(X)), onebit_scale(X)


def unpack_bits(codes: np.ndarray, k: int) -> np.ndarray:
    """Inverse of :func:`pack_bits`: bits [..., k] in {0, 1}."""
    return np.unpackbits(np.asarray(codes, dtype=np.uint8), axis=-1,
                         bitorder="little", count=k)


def payload_bytes(k_per_module) -> int:
    """Per-example payload sum_u (ceil(k_u/8) + 2) bytes (eq. app_payload)."""
    return int(sum(-(-int(k) // 8) + 2 for k in k_per_module))


# ---------------------------------------------------------------------------
# Scoring (eq. onebit_influence, eq. app_stored_influence)
# ---------------------------------------------------------------------------
Y_FRAC_BITS = 14


def query_fixed_point(y_u: np.ndarray):
    """Fixed-point form of one query's module coordinates: y_int = rint(y 2^f)
    with f = 14 - e for max|y| = mu 2^e, mu in [0.5, 1) (so |y_int| <= 2^14).
    An all-zero y gives y_int = 0, f = 0."""
    y = np.asarray(y_u, dtype=np.float64)
    M = float(np.max(np.abs(y))) if y.size else 0.0
    if M == 0.0:
        return np.zeros(y.shape, dtype=np.int64), 0
    _, e = np.frexp(M)
    f = Y_FRAC_BITS - int(e)
    return np.rint(np.ldexp(y, f)).astype(np.int64), f


def module_offsets(k_per_module):
    """Coordinate offsets and code byte offsets of each module in a row."""
    ks = [int(k) for k in k_per_module]
    coord = np.concatenate([[0], np.cumsum(ks)]).astype(np.int64)
    byte = np.concatenate([[0], np.cumsum([-(-k // 8) for k in ks])]).astype(np.int64)
    return coord, byte


def score(codes, scales, k_per_module, Y) -> np.ndarray:
    """float64 [Q, N]: I(i) = sum_u s_{i,u} <y_u, b_{i,u}> with b in {-1,+1},
    y in fixed point (exact integer inner products), modules summed in
    ascending order.

    The integer inner products go through a float64 matmul: every operand is
    an integer with |y_int| <= 2^14 and every partial sum is bounded by
    k * 2^14 <= 2^29 < 2^53, so the float64 result is the exact integer. Each
    module term s * n * 2^-f is exact too (11-bit s times a <= 30-bit n)."""
    codes = np.asarray(codes, dtype=np.uint8)
    scales16 = np.asarray(scales, dtype=np.uint16).view(np.float16).astype(np.float64)
    Y = np.asarray(Y, dtype=np.float64)
    N = codes.shape[0]
    Qn = Y.shape[0]
    if scales16.ndim == 1:
        scales16 = scales16[:, None]
    coord, byte = module_offsets(k_per_module)
    out = np.zeros((Qn, N), dtype=np.float64)
    for u, k in enumerate(k_per_module):
        pm = 2.0 * unpack_bits(codes[:, byte[u]:byte[u + 1]], int(k)) - 1.0
        Yint = np.empty((Qn, int(k)))
        pow2 = np.empty(Qn)
        for q in range(Qn):
            y_int, f = query_fixed_point(Y[q, coord[u]:coord[u + 1]])
            Yint[q] = y_int
            pow2[q] = np.ldexp(1.0, -f)
        n = Yint @ pm.T                                    # exact integers
        term = (scales16[:, u][None, :] * n) * pow2[:, None]
        out = out + term
    return out


def score_real(codes, scales, k_per_module, Y) -> np.ndarray:
    """The paper's score with y used as given (no fixed point), in float64."""
    codes = np.asarray(codes, dtype=np.uint8)
    scales16 = np.asarray(scales, dtype=np.uint16).view(np.float16).astype(np.float64)
    if scales16.ndim == 1:
        scales16 = scales16[:, None]
    Y = np.asarray(Y, dtype=np.float64)
    coord, byte = module_offsets(k_per_module)
    out = np.zeros((Y.shape[0], codes.shape[0]))
    for u, k in enumerate(k_per_module):
        pm = 2.0 * unpack_bits(codes[:, byte[u]:byte[u + 1]], int(k)) - 1.0
        out = out + (Y[:, coord[u]:coord[u + 1]] @ pm.T) * scales16[:, u][None, :]
    return out


def topk(scores: np.ndarray, k: int):
    """Per query: the k largest scores, ordered by (score desc, index asc).
    Fewer than k examples pad with index -1 and score -inf. Scores are returned
    as float32 (one rounding of the float64 score)."""
    S = np.asarray(scores, dtype=np.float64)
    Qn, N = S.shape
    idx = np.full((Qn, k), -1, dtype=np.int64)
    val = np.full((Qn, k), -np.inf, dtype=np.float32)
    ar = np.arange(N, dtype=np.int64)
    for q in range(Qn):
        order = np.lexsort((ar, -S[q]))[:k]
        idx[q, :order.size] = order
        val[q, :order.size] = S[q, order].astype(np.float32)
    return idx, val


# ---------------------------------------------------------------------------
# Whole passes (Algorithm 1: storing examples, scoring a query)
# ---------------------------------------------------------------------------
def store(a, ds, mask, Q_A, Q_S, eigvals, damping, m, P):
    """Codes and scales of a batch of examples for one module: x = P^T L g,
    then packed signs and FP16 scale. Returns (Z, X, codes, scales)."""
    ret = select_retained(eigvals, damping, m)
    Z = first_stage_batch(a, ds, mask, Q_A, Q_S, ret)
    X = pca_project(Z, P)
    codes, scales = encode(X)
    return Z, X, codes, scales


def query(qa, qds, qmask, Q_A, Q_S, eigvals, damping, m, P):
    """Unquantized query coordinates y = P^T L q for one module."""
    ret = select_retained(eigvals, damping, m)
    return pca_project(first_stage_batch(qa, qds, qmask, Q_A, Q_S, ret), P)


def fit(a, ds, mask, damping, m, k):
    """Fitting shared projections for one module from its own examples
    (Algorithm 1, first block): K-FAC factors and their eigenbases, EK-FAC
    corrected eigenvalues, the m retained axes, cached first-stage
    coordinates, and P by uncentered PCA. Returns a dict of float64 arrays."""
    A, S = kfac_factors(a, ds, mask)
    Q_A, Q_S = eigenbasis(A), eigenbasis(S)
    lam = ekfac_eigenvalues(a, ds, mask, Q_A, Q_S)
    ret = select_retained(lam, damping, m)
    Z = first_stage_batch(a, ds, mask, Q_A, Q_S, ret)
    P, mu = pca_fit(Z, k)
    return dict(A=A, S=S, Q_A=Q_A, Q_S=Q_S, eigvals=lam, retained=ret, Z=Z,
                P=P, mu=mu)
