"""Seeded synthetic inputs for the EOGP hot path.

This module only draws random numbers and lays them out in the shapes of the
paper's workloads (GPT-2 and OLMo-2 linear layers, Section 4 and the appendix on
models and data). It holds none of the method's arithmetic: no selection, no
rotation, no projection, no encoding and no scoring. Both the GPU path and the
oracle receive exactly the arrays made here.

Two back ends draw the same distributions:
  * numpy (``default_rng([config_id, stream_id])``), one stream per array, for
    the small cases the oracle finishes in seconds;
  * torch on a device (``torch.Generator`` seeded from the same pair), for the
    full-size workloads that only fit in device memory. Parity tests copy the
    device arrays they check back to the host.

Distributions (stand-ins for WikiText-2 / Tulu-3 activations and gradients,
which are not available here):
  * activations a_t ~ N(0, diag(s)), s_c ~ LogNormal(0, 1) per input channel;
    an optional trailing constant-1 column models an attributed bias;
  * output-gradients ds_t = sigma * eps_t + U_i c_t, with a per-example
    low-rank factor U_i (entries N(0, sigma_u^2)) and c_t ~ N(0, c_var * I);
  * padding masks: example i keeps its first L_i tokens, L_i ~ U{lo..T};
  * eigenbases: Haar-random orthogonal matrices (QR of a Gaussian, sign fixed),
    or a Kronecker product of two such factors for large widths;
  * corrected eigenvalues: Lambda[j, k] = c * sigma_j * alpha_k * exp(0.25 xi_jk)
    with sigma, alpha ~ LogNormal(0, 1), xi ~ N(0, 1);
  * PCA directions: the first k columns of a Kronecker product of two
    Haar-random orthogonal factors (dense, orthonormal columns);
  * stored codes: uniform random bits; scales fp16(exp(N(0, 1)));
    query projections N(0, 1).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

# ---------------------------------------------------------------------------
# Workload shapes (per linear module: (name, d_in, d_out)).
# GPT-2 small: hidden 768, MLP 3072, 12 blocks; biases attributed, so every
# input width carries one extra constant column (769 / 3073).
# OLMo-2 1B: hidden 2048, MLP 8192, 16 blocks.
# OLMo-2 32B: hidden 5120, MLP 27648, 64 blocks, grouped-query k/v (1024 wide).
# ---------------------------------------------------------------------------
GPT2_BLOCK = (("c_attn", 769, 2304), ("attn.c_proj", 769, 768),
              ("c_fc", 769, 3072), ("mlp.c_proj", 3073, 768))
OLMO1B_BLOCK = (("q_proj", 2048, 2048), ("k_proj", 2048, 2048),
                ("v_proj", 2048, 2048), ("o_proj", 2048, 2048),
                ("gate_proj", 2048, 8192), ("up_proj", 2048, 8192),
                ("down_proj", 8192, 2048))
OLMO32B_BLOCK = (("q_proj", 5120, 5120), ("k_proj", 5120, 1024),
                 ("v_proj", 5120, 1024), ("o_proj", 5120, 5120),
                 ("gate_proj", 5120, 27648), ("up_proj", 5120, 27648),
                 ("down_proj", 27648, 5120))


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: shapes, sizes and generator parameters."""
    config_id: int
    name: str
    block: tuple            # per-block module list
    n_blocks: int           # blocks whose modules are processed
    N: int                  # stored (training) examples
    T: int                  # padded tokens per example
    len_lo: int             # lengths ~ U{len_lo..T}; len_lo == T means no padding
    m: int                  # retained first-stage coordinates per module
    k: int                  # code bits (PCA outputs) per module
    Q: int                  # queries
    topk: int
    act_dtype: str          # "f32" or "bf16"
    grad_rank: int          # rank of the per-example component of ds
    grad_c_var: float       # variance of c_t
    damping: float | None = None   # absolute damping; None = recipe value
    bias_column: bool = False
    extra: dict = field(default_factory=dict)

    @property
    def modules(self):
        return [(f"blocks.{b}.{n}", di, do)
                for b in range(self.n_blocks) for (n, di, do) in self.block]


TINY = Workload(1, "tiny-64x64", (("linear", 64, 64),), 1, N=256, T=16, len_lo=16,
                m=512, k=128, Q=8, topk=10, act_dtype="f32", grad_rank=2,
                grad_c_var=1.0, damping=1e-3)
GPT2_SMALL = Workload(2, "gpt2-small-shaped", GPT2_BLOCK, 12, N=20000, T=512,
                      len_lo=64, m=16384, k=8192, Q=256, topk=100, act_dtype="f32",
                      grad_rank=8, grad_c_var=1.0 / 8, bias_column=True)
OLMO2_1B = Workload(3, "olmo2-1b-shaped", OLMO1B_BLOCK, 16, N=100000, T=1024,
                    len_lo=64, m=32768, k=16384, Q=1024, topk=100, act_dtype="bf16",
                    grad_rank=8, grad_c_var=1.0 / 8)
OLMO2_32B = Workload(4, "olmo2-32b-shaped-4-blocks", OLMO32B_BLOCK, 4, N=10000,
                     T=2048, len_lo=2048, m=65536, k=32768, Q=0, topk=100,
                     act_dtype="bf16", grad_rank=8, grad_c_var=1.0 / 8)
SCORING = Workload(5, "scoring-8M-codes-16384-bits", (("module", 0, 0),), 1,
                   N=8 * 1024 * 1024, T=0, len_lo=0, m=0, k=16384, Q=512, topk=100,
                   act_dtype="f32", grad_rank=0, grad_c_var=0.0)

WORKLOADS = {w.config_id: w for w in (TINY, GPT2_SMALL, OLMO2_1B, OLMO2_32B, SCORING)}

# Scalar recipe constants shared by every generator.
GRAD_SIGMA = 0.01      # isotropic part of ds
GRAD_SIGMA_U = 0.01    # entries of the per-example factor U_i
LAMBDA_XI = 0.25       # log-jitter of the synthetic corrected eigenvalues
RELATIVE_DAMPING = 0.1


def rng(config_id: int, stream: int) -> np.random.Generator:
    """The numpy stream ``stream`` of workload ``config_id``."""
    return np.random.default_rng([int(config_id), int(stream)])


# ---------------------------------------------------------------------------
# numpy back end (small cases)
# ---------------------------------------------------------------------------
def channel_variances(g: np.random.Generator, d: int) -> np.ndarray:
    return g.lognormal(0.0, 1.0, size=d)


def lengths(g: np.random.Generator, N: int, T: int, lo: int) -> np.ndarray:
    if lo >= T:
        return np.full(N, T, dtype=np.int64)
    return g.integers(lo, T + 1, size=N)


def prefix_mask(lens: np.ndarray, T: int) -> np.ndarray:
    """uint8 [N, T]: 1 on the first lens[i] tokens of example i."""
    return (np.arange(T)[None, :] < np.asarray(lens)[:, None]).astype(np.uint8)


def activations(g: np.random.Generator, N: int, T: int, d_in: int,
                s: np.ndarray, bias_column: bool = False) -> np.ndarray:
    """float64 [N, T, d_in]; with ``bias_column`` the last channel is 1."""
    d = d_in - 1 if bias_column else d_in
    a = g.standard_normal((N, T, d)) * np.sqrt(s[:d])
    if bias_column:
        a = np.concatenate([a, np.ones((N, T, 1))], axis=2)
    return a


def output_grads(g: np.random.Generator, N: int, T: int, d_out: int, rank: int,
                 c_var: float) -> np.ndarray:
    """float64 [N, T, d_out]: sigma*eps + U_i c_t (per-example rank ``rank``)."""
    ds = GRAD_SIGMA * g.standard_normal((N, T, d_out))
    if rank > 0:
        U = GRAD_SIGMA_U * g.standard_normal((N, d_out, rank))
        c = math.sqrt(c_var) * g.standard_normal((N, T, rank))
        ds = ds + np.matmul(c, np.transpose(U, (0, 2, 1)))
    return ds


def fill_masked(x: np.ndarray, mask: np.ndarray, value=np.nan) -> np.ndarray:
    """Copy of ``x`` [N, T, d] with masked tokens overwritten by ``value``."""
    y = np.array(x, copy=True)
    y[np.asarray(mask) == 0] = value
    return y


def haar_orthogonal(g: np.random.Generator, d: int) -> np.ndarray:
    """Haar-random orthogonal d x d (QR of a Gaussian, R's diagonal made positive)."""
    q, r = np.linalg.qr(g.standard_normal((d, d)))
    return q * np.sign(np.diag(r))[None, :]


def kron_factors(d: int) -> tuple[int, int]:
    """A factorisation d = p * q with p <= q as close to sqrt(d) as possible."""
    p = int(math.isqrt(d))
    while d % p:
        p -= 1
    return p, d // p


def eigenbasis(g: np.random.Generator, d: int, kron_above: int = 4096) -> np.ndarray:
    """Dense orthogonal d x d: Haar for d <= kron_above, else a Kronecker
    product of two Haar factors (kept dense, as a K-FAC eigenbasis would be)."""
    if d <= kron_above:
        return haar_orthogonal(g, d)
    p, q = kron_factors(d)
    if p == 1:
        return haar_orthogonal(g, d)
    return np.kron(haar_orthogonal(g, p), haar_orthogonal(g, q))


def synthetic_eigvals(g: np.random.Generator, d_out: int, d_in: int,
                      scale: float) -> np.ndarray:
    """float64 [d_out, d_in]: scale * sigma_j * alpha_k * exp(0.25 xi_jk)."""
    sig = g.lognormal(0.0, 1.0, size=d_out)
    alp = g.lognormal(0.0, 1.0, size=d_in)
    xi = g.standard_normal((d_out, d_in))
    return scale * sig[:, None] * alp[None, :] * np.exp(LAMBDA_XI * xi)


def expected_coord_energy(mean_len: float, d_in_var: float, rank: int,
                          c_var: float) -> float:
    """Recipe constant: the expected square of one rotated gradient entry,
    mean_len * E[(q.a)^2] * E[(q'.ds)^2] for unit q, q' under this recipe."""
    ds_var = GRAD_SIGMA ** 2 + rank * c_var * GRAD_SIGMA_U ** 2
    return mean_len * d_in_var * ds_var


def eigval_scale(w: Workload) -> float:
    """Scale c of the synthetic Lambda so that its mean matches the expected
    rotated-gradient energy (so half-whitened coordinates are O(1))."""
    mean_len = 0.5 * (w.len_lo + w.T)
    e_s = math.exp(0.5)                      # E[LogNormal(0,1)]
    target = expected_coord_energy(mean_len, e_s, w.grad_rank, w.grad_c_var)
    mean_lam = math.exp(0.5) * math.exp(0.5) * math.exp(0.5 * LAMBDA_XI ** 2)
    return target / mean_lam


def recipe_damping(w: Workload) -> float:
    """Damping of a synthetic workload: the given absolute value, else the
    relative rule 0.1 * (mean corrected eigenvalue) applied to the recipe's
    expected eigenvalue (a constant of the recipe, not computed from data)."""
    if w.damping is not None:
        return float(w.damping)
    return RELATIVE_DAMPING * eigval_scale(w) * math.exp(1.0 + 0.5 * LAMBDA_XI ** 2)


def pca_directions(g: np.random.Generator, m: int, k: int) -> np.ndarray:
    """float64 [m, k] with orthonormal columns: first k columns of
    kron(H1, H2) for Haar H1, H2 (or of one Haar factor if m is prime)."""
    p, q = kron_factors(m)
    if p == 1:
        return haar_orthogonal(g, m)[:, :k]
    a = haar_orthogonal(g, p)
    b = haar_orthogonal(g, q)
    ncols_a = -(-k // q)
    full = np.kron(a[:, :ncols_a], b)
    return full[:, :k]


def random_codes(g: np.random.Generator, N: int, row_bytes: int) -> np.ndarray:
    return g.integers(0, 256, size=(N, row_bytes), dtype=np.uint8)


def random_scales(g: np.random.Generator, N: int, U: int) -> np.ndarray:
    """fp16 bit patterns (uint16) of exp(N(0, 1))."""
    return np.exp(g.standard_normal((N, U))).astype(np.float16).view(np.uint16)


def query_projections(g: np.random.Generator, Q: int, width: int) -> np.ndarray:
    return g.standard_normal((Q, width)).astype(np.float32)


def srht_draws(config_id: int, stream: int, m: int, p: int, k: int):
    """The random draws of one module's SRHT (the same realised transform for
    the store and the queries): signs [m] (int8, +1 / -1) and k distinct rows
    of the width-p transform (int32), uniformly without replacement."""
    g = rng(config_id, 700000 + stream)
    signs = np.where(g.random(m) < 0.5, -1, 1).astype(np.int8)
    rows = g.choice(p, size=k, replace=False).astype(np.int32)
    return signs, rows


# ---------------------------------------------------------------------------
# Tiny workload (numpy): raw per-token inputs for stored examples and queries.
# ---------------------------------------------------------------------------
def tiny_raw(w: Workload = TINY, N: int | None = None, T: int | None = None,
             len_lo: int | None = None):
    """Stored-example and query inputs of the tiny workload, as float32 arrays
    (the dtype handed to the GPU) plus uint8 masks."""
    N = w.N if N is None else N
    T = w.T if T is None else T
    len_lo = T if len_lo is None else len_lo
    _, d_in, d_out = w.block[0]
    s = channel_variances(rng(w.config_id, 0), d_in)
    a = activations(rng(w.config_id, 1), N, T, d_in, s).astype(np.float32)
    ds = output_grads(rng(w.config_id, 2), N, T, d_out, w.grad_rank,
                      w.grad_c_var).astype(np.float32)
    mask = prefix_mask(lengths(rng(w.config_id, 3), N, T, len_lo), T)
    qa = activations(rng(w.config_id, 11), w.Q, T, d_in, s).astype(np.float32)
    qds = output_grads(rng(w.config_id, 12), w.Q, T, d_out, w.grad_rank,
                       w.grad_c_var).astype(np.float32)
    qmask = prefix_mask(lengths(rng(w.config_id, 13), w.Q, T, len_lo), T)
    return dict(a=a, ds=ds, mask=mask, qa=qa, qds=qds, qmask=qmask,
                d_in=d_in, d_out=d_out)


def module_artifacts(w: Workload, module_index: int, d_in: int, d_out: int,
                     m: int | None = None, k: int | None = None):
    """Shared artifacts of one synthetic module (numpy): eigenbases Q_A, Q_S
    (float32), corrected eigenvalues (float32), damping, PCA directions P
    (float32, [m, k])."""
    m = w.m if m is None else m
    k = w.k if k is None else k
    base = 1000 + 16 * module_index
    QA = eigenbasis(rng(w.config_id, base + 0), d_in).astype(np.float32)
    QS = eigenbasis(rng(w.config_id, base + 1), d_out).astype(np.float32)
    lam = synthetic_eigvals(rng(w.config_id, base + 2), d_out, d_in,
                            eigval_scale(w)).astype(np.float32)
    P = pca_directions(rng(w.config_id, base + 3), m, k).astype(np.float32)
    return dict(Q_A=QA, Q_S=QS, eigvals=lam, damping=recipe_damping(w), P=P)


def module_inputs(w: Workload, module_index: int, N: int, T: int, d_in: int,
                  d_out: int, len_lo: int | None = None, stream_base: int = 0):
    """Per-token inputs of one module for N examples (numpy, float32 + mask)."""
    len_lo = w.len_lo if len_lo is None else len_lo
    base = 100000 + 64 * module_index + stream_base
    s = channel_variances(rng(w.config_id, base + 0), d_in)
    a = activations(rng(w.config_id, base + 1), N, T, d_in, s,
                    bias_column=w.bias_column).astype(np.float32)
    ds = output_grads(rng(w.config_id, base + 2), N, T, d_out, w.grad_rank,
                      w.grad_c_var).astype(np.float32)
    mask = prefix_mask(lengths(rng(w.config_id, base + 3), N, T, len_lo), T)
    return a, ds, mask


# ---------------------------------------------------------------------------
# torch back end (full-size workloads, generated directly in device memory)
# ---------------------------------------------------------------------------
def torch_generator(config_id: int, stream: int, device):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed((int(config_id) << 32) ^ (int(stream) * 0x9E3779B1 & 0xFFFFFFFF))
    return g


def torch_inputs(w: Workload, module_index: int, N: int, T: int, d_in: int,
                 d_out: int, device, dtype, stream_base: int = 0):
    """Per-token inputs (device tensors) for one module shape: a [N,T,d_in],
    ds [N,T,d_out] in ``dtype`` and a uint8 prefix mask [N,T]."""
    import torch
    base = 100000 + 64 * module_index + stream_base
    g0 = torch_generator(w.config_id, base + 0, device)
    d = d_in - 1 if w.bias_column else d_in
    s = torch.empty(d, device=device).log_normal_(0.0, 1.0, generator=g0)
    g1 = torch_generator(w.config_id, base + 1, device)
    a = torch.empty((N, T, d_in), device=device, dtype=dtype)
    chunk = max(1, (1 << 27) // max(1, T * d_in))
    for i0 in range(0, N, chunk):
        i1 = min(N, i0 + chunk)
        blk = torch.randn((i1 - i0, T, d), device=device, generator=g1) * s.sqrt()
        a[i0:i1, :, :d] = blk.to(dtype)
        if w.bias_column:
            a[i0:i1, :, d] = 1.0
    g2 = torch_generator(w.config_id, base + 2, device)
    ds = torch.empty((N, T, d_out), device=device, dtype=dtype)
    chunk = max(1, (1 << 27) // max(1, T * d_out))
    for i0 in range(0, N, chunk):
        i1 = min(N, i0 + chunk)
        n = i1 - i0
        blk = GRAD_SIGMA * torch.randn((n, T, d_out), device=device, generator=g2)
        if w.grad_rank > 0:
            U = GRAD_SIGMA_U * torch.randn((n, d_out, w.grad_rank), device=device,
                                           generator=g2)
            c = math.sqrt(w.grad_c_var) * torch.randn((n, T, w.grad_rank),
                                                      device=device, generator=g2)
            blk = blk + torch.matmul(c, U.transpose(1, 2).contiguous())
        ds[i0:i1] = blk.to(dtype)
    g3 = torch_generator(w.config_id, base + 3, device)
    if w.len_lo >= T:
        lens = torch.full((N,), T, device=device, dtype=torch.int64)
    else:
        lens = torch.randint(w.len_lo, T + 1, (N,), device=device, generator=g3)
    mask = (torch.arange(T, device=device)[None, :] < lens[:, None]).to(torch.uint8)
    return a, ds, mask


def torch_eigenbasis(g: np.random.Generator, d: int, device, kron_above: int = 4096):
    """Device float32 d x d orthogonal matrix with the same recipe as
    :func:`eigenbasis`; Kronecker products are formed on the device."""
    import torch
    if d <= kron_above:
        return torch.from_numpy(haar_orthogonal(g, d).astype(np.float32)).to(device)
    p, q = kron_factors(d)
    if p == 1:
        return torch.from_numpy(haar_orthogonal(g, d).astype(np.float32)).to(device)
    a = torch.from_numpy(haar_orthogonal(g, p)).to(device)
    b = torch.from_numpy(haar_orthogonal(g, q)).to(device)
    return torch.kron(a, b).float().contiguous()


def torch_pca_directions_t(g: np.random.Generator, m: int, k: int, device):
    """Device float32 [k, m]: the transpose of :func:`pca_directions` (each
    direction stored contiguously), formed on the device."""
    import torch
    p, q = kron_factors(m)
    if p == 1:
        return torch.from_numpy(
            np.ascontiguousarray(haar_orthogonal(g, m)[:, :k].T).astype(np.float32)
        ).to(device)
    a = haar_orthogonal(g, p)
    b = haar_orthogonal(g, q)
    ncols_a = -(-k // q)
    at = torch.from_numpy(np.ascontiguousarray(a[:, :ncols_a].T)).to(device)
    bt = torch.from_numpy(np.ascontiguousarray(b.T)).to(device)
    return torch.kron(at, bt)[:k].float().contiguous()


def torch_module_artifacts(w: Workload, module_index: int, d_in: int, d_out: int,
                           device, p_dtype, base_cache: dict | None = None):
    """Shared artifacts of one module as device tensors. Eigenbases are a
    Haar (or Kronecker-Haar) matrix per distinct width, drawn once and made
    distinct per module by a random signed column permutation; P is stored
    column-major ([k, m] row-major, i.e. each direction contiguous)."""
    import torch
    cache = {} if base_cache is None else base_cache
    base = 1000 + 16 * module_index

    def basis(d, stream):
        key = ("basis", d)
        if key not in cache:
            cache[key] = torch_eigenbasis(rng(w.config_id, 500000 + d), d, device)
        g = torch_generator(w.config_id, base + stream, device)
        perm = torch.randperm(d, device=device, generator=g)
        sign = torch.randint(0, 2, (d,), device=device, generator=g).float() * 2 - 1
        return (cache[key][:, perm] * sign[None, :]).contiguous()

    QA = basis(d_in, 0)
    QS = basis(d_out, 1)
    g2 = torch_generator(w.config_id, base + 2, device)
    sig = torch.empty(d_out, device=device).log_normal_(0.0, 1.0, generator=g2)
    alp = torch.empty(d_in, device=device).log_normal_(0.0, 1.0, generator=g2)
    xi = torch.randn((d_out, d_in), device=device, generator=g2)
    lam = (eigval_scale(w) * sig[:, None] * alp[None, :]
           * torch.exp(LAMBDA_XI * xi)).float().contiguous()
    key = ("P", w.m, w.k)
    if key not in cache:
        cache[key] = torch_pca_directions_t(rng(w.config_id, 600000 + w.m), w.m,
                                            w.k, device)
    Pt = cache[key].to(p_dtype).clone()    # distinct memory per module
    return dict(Q_A=QA, Q_S=QS, eigvals=lam, damping=recipe_damping(w), Pt=Pt)
