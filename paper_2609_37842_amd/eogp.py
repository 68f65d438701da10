"""Python binding of the EOGP C ABI (include/eogp.h).

Argument marshalling only: every step of the hot path runs in the HIP kernels of
libeogp.so. torch supplies device memory (tensors) and the current HIP stream.
The functions carry the same names as the C entry points. If the library is
missing the import of any entry point raises; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libeogp.so")

F32, BF16, F16 = 0, 1, 2
PREC_FAST, PREC_ACCURATE, PREC_F16 = 0, 1, 2

_DTYPE_CODE = {torch.float32: F32, torch.bfloat16: BF16, torch.float16: F16}

c_i64 = ctypes.c_int64
c_i32 = ctypes.c_int32
c_vp = ctypes.c_void_p
c_sz = ctypes.c_size_t


class EogpError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"eogp status {status}: {msg}")
        self.status = status


class PlanInfo(ctypes.Structure):
    _fields_ = [("d_out", c_i64), ("d_in", c_i64), ("m", c_i64), ("damping", ctypes.c_double),
                ("n_rows", c_i64), ("n_cols", c_i64), ("n_tiles", c_i64),
                ("retained_flat", c_vp), ("retained_weight", c_vp)]


_lib = None

EXPORTED = (
    "eogp_plan_create", "eogp_plan_destroy", "eogp_plan_get_info", "eogp_plan_copy_retained",
    "eogp_plan_set_input_exponents",
    "eogp_rotate_retain_workspace_size", "eogp_rotate_retain_planned",
    "eogp_compact_tokens_workspace_size", "eogp_compact_tokens", "eogp_rotate_retain_compacted",
    "eogp_rotate_retain_oneshot_workspace_size", "eogp_rotate_retain",
    "eogp_pca_project_workspace_size", "eogp_pca_project",
    "eogp_sign_pack", "eogp_sign_pack_tiled", "eogp_srht_project_workspace_size",
    "eogp_srht_project",
    "eogp_pca_fit_workspace_size", "eogp_pca_fit",
    "eogp_ekfac_workspace_size", "eogp_ekfac_eigenvalues",
    "eogp_score_topk_workspace_size", "eogp_score_topk", "eogp_score_topk_tiled",
    "eogp_score_topk_noalloc",
    "eogp_timing_enable", "eogp_timing_read",
    "eogp_status_string", "eogp_last_error", "eogp_version",
)


def load(path: str | None = None):
    """Load libeogp.so once and declare the C signatures."""
    global _lib
    if _lib is not None:
        return _lib
    path = path or LIB_PATH
    if not os.path.exists(path):
        raise RuntimeError(f"{path} not found; build it with "
                           "`python -m paper_2609_37842_amd.build`")
    L = ctypes.CDLL(path)
    sig = {
        "eogp_plan_create": (c_i32, [c_vp, c_i64, c_i64, ctypes.c_double, c_i64, c_vp, c_vp, c_vp,
                                     ctypes.POINTER(c_vp)]),
        "eogp_plan_destroy": (None, [c_vp]),
        "eogp_plan_get_info": (c_i32, [c_vp, ctypes.POINTER(PlanInfo)]),
        "eogp_plan_copy_retained": (c_i32, [c_vp, c_vp, c_vp, c_vp]),
        "eogp_plan_set_input_exponents": (c_i32, [c_vp, c_i32, c_i32]),
        "eogp_rotate_retain_workspace_size": (c_sz, [c_vp, c_i64, c_i64]),
        "eogp_rotate_retain_planned": (c_i32, [c_vp, c_vp, c_i64, c_vp, c_i64, c_i32, c_vp, c_i64,
                                               c_i64, c_vp, c_i32, c_i64, c_i32, c_vp, c_sz, c_vp]),
        "eogp_compact_tokens_workspace_size": (c_sz, [c_i64, c_i64]),
        "eogp_compact_tokens": (c_i32, [c_vp, c_i64, c_i64, c_i32, c_vp, c_sz, c_vp]),
        "eogp_rotate_retain_compacted": (c_i32, [c_vp, c_vp, c_i64, c_vp, c_i64, c_i32, c_i64, c_i64,
                                                 c_vp, c_i32, c_i64, c_i32, c_vp, c_sz, c_vp]),
        "eogp_rotate_retain_oneshot_workspace_size": (c_sz, [c_i64, c_i64, c_i64, c_i64, c_i64]),
        "eogp_rotate_retain": (c_i32, [c_vp, c_i64, c_vp, c_i64, c_i32, c_vp, c_i64, c_i64, c_i64,
                                       c_i64, c_vp, c_vp, c_vp, ctypes.c_double, c_i64, c_vp, c_i64,
                                       c_i32, c_vp, c_sz, c_vp]),
        "eogp_pca_project_workspace_size": (c_sz, [c_i64, c_i64, c_i64, c_i32, c_i32]),
        "eogp_pca_project": (c_i32, [c_vp, c_i32, c_i64, c_i64, c_i64, c_vp, c_i32, c_i64, c_i64,
                                     c_vp, c_i64, c_i32, c_vp, c_sz, c_vp]),
        "eogp_sign_pack": (c_i32, [c_vp, c_i64, c_i64, c_i64, c_vp, c_i64, c_vp, c_i64, c_vp]),
        "eogp_sign_pack_tiled": (c_i32, [c_vp, c_i64, c_i64, c_i64, c_i64, c_vp, c_i64, c_i64, c_vp,
                                         c_i64, c_vp]),
        "eogp_ekfac_workspace_size": (c_sz, [c_i64, c_i64, c_i64, c_i64]),
        "eogp_ekfac_eigenvalues": (c_i32, [c_vp, c_i64, c_vp, c_i64, c_i32, c_vp, c_i64, c_i64,
                                           c_i64, c_i64, c_vp, c_vp, c_i32, c_i32, c_i32, c_vp,
                                           c_i32, c_vp, c_sz, c_vp]),
        "eogp_srht_project_workspace_size": (c_sz, [c_i64, c_i64]),
        "eogp_srht_project": (c_i32, [c_vp, c_i64, c_i64, c_i64, c_vp, c_vp, c_i64, c_vp, c_i64,
                                      c_vp, c_sz, c_vp]),
        "eogp_pca_fit_workspace_size": (c_sz, [c_i64, c_i64, c_i64]),
        "eogp_pca_fit": (c_i32, [c_vp, c_i64, c_i64, c_i64, c_i64, c_vp, c_i64, c_vp, c_vp, c_sz,
                                 c_vp]),
        "eogp_score_topk_workspace_size": (c_sz, [c_i64, c_i64, c_i32, ctypes.POINTER(c_i64),
                                                  c_i32]),
        "eogp_score_topk": (c_i32, [c_vp, c_i64, c_vp, c_i64, c_i32, ctypes.POINTER(c_i64), c_vp,
                                    c_i64, c_i64, c_i32, c_vp, c_vp, c_vp, c_vp, c_sz, c_vp]),
        "eogp_score_topk_tiled": (c_i32, [c_vp, c_vp, c_i64, c_i32, ctypes.POINTER(c_i64), c_vp,
                                          c_i64, c_i64, c_i32, c_vp, c_vp, c_vp, c_vp, c_sz, c_vp]),
        "eogp_score_topk_noalloc": (c_i32, [c_vp, c_i64, c_vp, c_i64, c_i32, ctypes.POINTER(c_i64),
                                            c_vp, c_i64, c_i64, c_i32, c_vp, c_vp, c_vp, c_vp]),
        "eogp_timing_enable": (c_i32, [c_i32]),
        "eogp_timing_read": (c_i32, [c_i32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(c_i64)]),
        "eogp_status_string": (ctypes.c_char_p, [c_i32]),
        "eogp_last_error": (ctypes.c_char_p, []),
        "eogp_version": (c_i32, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


def _check(status: int):
    if status != 0:
        L = load()
        raise EogpError(status, L.eogp_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _need_cuda(*ts):
    for t in ts:
        if t is not None and (not t.is_cuda):
            raise ValueError("EOGP arguments must be device tensors")


def _workspace(nbytes: int, device, ws=None):
    if nbytes == 0:
        return None, 0
    if ws is not None:
        if ws.numel() * ws.element_size() < nbytes:
            raise ValueError(f"workspace needs {nbytes} bytes")
        return ws, ws.numel() * ws.element_size()
    return torch.empty(nbytes, dtype=torch.uint8, device=device), nbytes


# ---------------------------------------------------------------------------
# Plans (fitting shared projections)
# ---------------------------------------------------------------------------
class eogp_plan:
    """Retained-axis plan of one module; see eogp_plan_create in eogp.h."""

    def __init__(self, eigvals, damping: float, m: int, Q_A, Q_S, stream=None):
        L = load()
        _need_cuda(eigvals, Q_A, Q_S)
        for t in (eigvals, Q_A, Q_S):
            if t.dtype != torch.float32 or not t.is_contiguous():
                raise ValueError("eigvals, Q_A, Q_S must be contiguous float32")
        d_out, d_in = eigvals.shape
        if tuple(Q_A.shape) != (d_in, d_in) or tuple(Q_S.shape) != (d_out, d_out):
            raise ValueError("Q_A must be [d_in, d_in] and Q_S [d_out, d_out]")
        h = c_vp()
        _check(L.eogp_plan_create(_ptr(eigvals), d_out, d_in, float(damping), int(m), _ptr(Q_A),
                                  _ptr(Q_S), _stream(stream), ctypes.byref(h)))
        self._h = h
        self.device = eigvals.device
        info = PlanInfo()
        _check(L.eogp_plan_get_info(h, ctypes.byref(info)))
        self.d_out, self.d_in, self.m = int(info.d_out), int(info.d_in), int(info.m)
        self.damping = float(info.damping)
        self.n_rows, self.n_cols, self.n_tiles = int(info.n_rows), int(info.n_cols), int(info.n_tiles)
        self._flat_ptr, self._w_ptr = info.retained_flat, info.retained_weight

    def retained(self):
        """(flat index int32 [m], weight float32 [m]) copied to new device tensors."""
        flat = torch.empty(self.m, dtype=torch.int32, device=self.device)
        w = torch.empty(self.m, dtype=torch.float32, device=self.device)
        _check(load().eogp_plan_copy_retained(self._h, _ptr(flat), _ptr(w), _stream()))
        return flat, w

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            load().eogp_plan_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def eogp_plan_create(eigvals, damping, m, Q_A, Q_S, stream=None) -> eogp_plan:
    return eogp_plan(eigvals, damping, m, Q_A, Q_S, stream)


def eogp_plan_set_input_exponents(plan: eogp_plan, e_acts: int, e_grads: int) -> None:
    """Power-of-two input scaling of the plan's fp16 first stage (see eogp.h)."""
    _check(load().eogp_plan_set_input_exponents(plan._h, int(e_acts), int(e_grads)))


# ---------------------------------------------------------------------------
# First stage
# ---------------------------------------------------------------------------
def _token_stride(x, name):
    """Row stride (elements) of a [N, T, d] token tensor whose tokens are laid
    out at a constant stride, e.g. a column slice of a wider padded buffer."""
    if x.dim() != 3 or x.stride(2) != 1 or x.stride(0) != x.shape[1] * x.stride(1):
        raise ValueError(f"{name} must be [N, T, d] with unit column stride and tokens at a "
                         "constant row stride")
    return x.stride(1)


def _acts_dtype(acts, out_grads):
    if acts.dtype != out_grads.dtype or acts.dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("acts and out_grads must both be float32 or both bfloat16")
    return _DTYPE_CODE[acts.dtype]


def eogp_rotate_retain_workspace_size(plan: eogp_plan, N: int, T: int) -> int:
    return int(load().eogp_rotate_retain_workspace_size(plan._h, N, T))


def _first_stage_args(plan, acts, out_grads, Z):
    """Checks shared by the planned first-stage calls; returns (N, T, ld_a, ld_g, Z)."""
    _need_cuda(acts, out_grads, Z)
    N, T, d_in = acts.shape
    if tuple(out_grads.shape) != (N, T, plan.d_out) or d_in != plan.d_in:
        raise ValueError("acts [N,T,d_in] / out_grads [N,T,d_out] do not match the plan")
    ld_a, ld_g = _token_stride(acts, "acts"), _token_stride(out_grads, "out_grads")
    if Z is None:
        Z = torch.empty((N, plan.m), dtype=torch.float32, device=acts.device)
    if (Z.dtype not in (torch.float32, torch.float16) or Z.dim() != 2 or Z.stride(1) != 1
            or Z.shape[0] != N):
        raise ValueError("Z must be float32 or float16 [N, >= m] with unit column stride")
    return N, T, ld_a, ld_g, Z


def eogp_rotate_retain_planned(plan: eogp_plan, acts, out_grads, token_mask=None, Z=None,
                               prec=PREC_ACCURATE, ws=None, stream=None):
    """Z [N, m] (float32) of the batch; see eogp_rotate_retain_planned in eogp.h."""
    L = load()
    _need_cuda(token_mask)
    N, T, ld_a, ld_g, Z = _first_stage_args(plan, acts, out_grads, Z)
    if token_mask is not None and (token_mask.dtype != torch.uint8 or tuple(token_mask.shape) != (N, T)
                                   or not token_mask.is_contiguous()):
        raise ValueError("token_mask must be contiguous uint8 [N, T]")
    need = eogp_rotate_retain_workspace_size(plan, N, T)
    ws, wsb = _workspace(need, acts.device, ws)
    _check(L.eogp_rotate_retain_planned(plan._h, _ptr(acts), ld_a, _ptr(out_grads), ld_g,
                                        _acts_dtype(acts, out_grads), _ptr(token_mask), N, T,
                                        _ptr(Z), _DTYPE_CODE[Z.dtype], Z.stride(0), prec, _ptr(ws),
                                        wsb, _stream(stream)))
    return Z


def eogp_compact_tokens_workspace_size(N: int, T: int) -> int:
    return int(load().eogp_compact_tokens_workspace_size(N, T))


def eogp_compact_tokens(token_mask, N: int, T: int, prec, ws, stream=None):
    """Valid-token list of (token_mask, N, T) into the head of the first-stage
    workspace `ws` (a uint8 device tensor); see eogp_compact_tokens in eogp.h."""
    L = load()
    if ws is None:
        raise ValueError("eogp_compact_tokens writes into a caller's first-stage workspace")
    _need_cuda(token_mask, ws)
    if token_mask is not None and (token_mask.dtype != torch.uint8 or tuple(token_mask.shape) != (N, T)
                                   or not token_mask.is_contiguous()):
        raise ValueError("token_mask must be contiguous uint8 [N, T]")
    ws, wsb = _workspace(eogp_compact_tokens_workspace_size(N, T), ws.device, ws)
    _check(L.eogp_compact_tokens(_ptr(token_mask), N, T, prec, _ptr(ws), wsb, _stream(stream)))


def eogp_rotate_retain_compacted(plan: eogp_plan, acts, out_grads, ws, Z=None, prec=PREC_ACCURATE,
                                 stream=None):
    """The planned first stage with the token list already in `ws` (written by
    eogp_compact_tokens for the same N, T and precision layout)."""
    L = load()
    if ws is None:
        raise ValueError("the compacted first stage reads the token list from ws")
    _need_cuda(ws)
    N, T, ld_a, ld_g, Z = _first_stage_args(plan, acts, out_grads, Z)
    ws, wsb = _workspace(eogp_rotate_retain_workspace_size(plan, N, T), acts.device, ws)
    _check(L.eogp_rotate_retain_compacted(plan._h, _ptr(acts), ld_a, _ptr(out_grads), ld_g,
                                          _acts_dtype(acts, out_grads), N, T, _ptr(Z),
                                          _DTYPE_CODE[Z.dtype], Z.stride(0), prec, _ptr(ws), wsb,
                                          _stream(stream)))
    return Z


def eogp_rotate_retain(acts, out_grads, token_mask, Q_A, Q_S, eigvals, damping, m, Z=None,
                       prec=PREC_ACCURATE, ws=None, stream=None):
    """One-shot first stage with the paper's arguments (builds and frees a plan)."""
    L = load()
    _need_cuda(acts, out_grads, token_mask, Q_A, Q_S, eigvals, Z)
    N, T, d_in = acts.shape
    d_out = out_grads.shape[2]
    ld_a, ld_g = _token_stride(acts, "acts"), _token_stride(out_grads, "out_grads")
    if Z is None:
        Z = torch.empty((N, m), dtype=torch.float32, device=acts.device)
    need = int(L.eogp_rotate_retain_oneshot_workspace_size(N, T, d_in, d_out, int(m)))
    ws, wsb = _workspace(need, acts.device, ws)
    _check(L.eogp_rotate_retain(_ptr(acts), ld_a, _ptr(out_grads), ld_g, _acts_dtype(acts, out_grads),
                                _ptr(token_mask), N, T, d_in, d_out, _ptr(Q_A), _ptr(Q_S),
                                _ptr(eigvals), float(damping), int(m), _ptr(Z), Z.stride(0), prec,
                                _ptr(ws), wsb, _stream(stream)))
    return Z


# ---------------------------------------------------------------------------
# Second stage, encoding, scoring
# ---------------------------------------------------------------------------
def eogp_pca_project_workspace_size(N: int, m: int, k: int, p_dtype: int, prec: int) -> int:
    """Bytes of workspace eogp_pca_project needs for these sizes."""
    return int(load().eogp_pca_project_workspace_size(N, m, k, p_dtype, prec))


def eogp_pca_project(Z, Pt, X=None, prec=PREC_FAST, ws=None, stream=None):
    """X [N, k] = Z [N, m] @ P, with P given as Pt [k, m] (each direction
    contiguous, i.e. P column-major) in float16, bfloat16 or float32; Z in
    float32, or in P's own 16-bit type."""
    L = load()
    _need_cuda(Z, Pt, X)
    N, m = Z.shape
    k, m2 = Pt.shape
    if m2 != m or Pt.stride(1) != 1 or Z.stride(1) != 1:
        raise ValueError("Pt must be [k, m] with unit column stride; Z [N, m]")
    if Z.dtype not in (torch.float32, torch.float16, torch.bfloat16):
        raise ValueError("Z must be float32, float16 or bfloat16")
    if X is None:
        X = torch.empty((N, k), dtype=torch.float32, device=Z.device)
    pd = _DTYPE_CODE[Pt.dtype]
    need = int(L.eogp_pca_project_workspace_size(N, m, k, pd, prec))
    ws, wsb = _workspace(need, Z.device, ws)
    _check(L.eogp_pca_project(_ptr(Z), _DTYPE_CODE[Z.dtype], Z.stride(0), N, m, _ptr(Pt), pd,
                              Pt.stride(0), k, _ptr(X), X.stride(0), prec, _ptr(ws), wsb,
                              _stream(stream)))
    return X


def eogp_ekfac_workspace_size(N: int, T: int, d_in: int, d_out: int) -> int:
    """Bytes of workspace eogp_ekfac_eigenvalues needs for these sizes."""
    return int(load().eogp_ekfac_workspace_size(N, T, d_in, d_out))


def eogp_ekfac_eigenvalues(acts, out_grads, token_mask, Q_A, Q_S, sq_sum=None, accumulate=False,
                           prec=PREC_ACCURATE, exponents=(0, 0), ws=None, stream=None):
    """Sum over the batch of the squared rotated gradients (Q_S^T G_i Q_A)^2,
    [d_out, d_in] float32 (divide by the total number of examples for the
    corrected eigenvalues). exponents = (e_acts, e_grads), the power-of-two
    input scaling of the fp16 mode; see eogp_ekfac_eigenvalues in eogp.h."""
    L = load()
    _need_cuda(acts, out_grads, token_mask, Q_A, Q_S, sq_sum)
    N, T, d_in = acts.shape
    d_out = out_grads.shape[2]
    ld_a, ld_g = _token_stride(acts, "acts"), _token_stride(out_grads, "out_grads")
    if sq_sum is None:
        sq_sum = torch.empty((d_out, d_in), dtype=torch.float32, device=acts.device)
        accumulate = False
    if sq_sum.dtype != torch.float32 or tuple(sq_sum.shape) != (d_out, d_in) or not sq_sum.is_contiguous():
        raise ValueError("sq_sum must be contiguous float32 [d_out, d_in]")
    need = int(L.eogp_ekfac_workspace_size(N, T, d_in, d_out))
    ws, wsb = _workspace(need, acts.device, ws)
    _check(L.eogp_ekfac_eigenvalues(_ptr(acts), ld_a, _ptr(out_grads), ld_g,
                                    _acts_dtype(acts, out_grads), _ptr(token_mask), N, T, d_in,
                                    d_out, _ptr(Q_A), _ptr(Q_S), prec, int(exponents[0]),
                                    int(exponents[1]), _ptr(sq_sum), 1 if accumulate else 0,
                                    _ptr(ws), wsb, _stream(stream)))
    return sq_sum


def eogp_srht_project_workspace_size(N: int, m: int) -> int:
    return int(load().eogp_srht_project_workspace_size(N, m))


def eogp_srht_project(Z, signs, rows, X=None, ws=None, stream=None):
    """X [N, k] = the SRHT of each row of Z [N, m] (float32) with random signs
    [m] (int8) and kept rows [k] (int32); see eogp_srht_project in eogp.h."""
    L = load()
    _need_cuda(Z, signs, rows, X)
    N, m = Z.shape
    k = rows.shape[0]
    if Z.dtype != torch.float32 or (Z.numel() > 0 and Z.stride(1) != 1):
        raise ValueError("Z must be float32 [N, m] with unit column stride")
    if signs.dtype != torch.int8 or signs.shape[0] != m or not signs.is_contiguous():
        raise ValueError("signs must be contiguous int8 [m]")
    if rows.dtype != torch.int32 or not rows.is_contiguous():
        raise ValueError("rows must be contiguous int32 [k]")
    if X is None:
        X = torch.empty((N, k), dtype=torch.float32, device=Z.device)
    ws, wsb = _workspace(int(L.eogp_srht_project_workspace_size(N, m)), Z.device, ws)
    _check(L.eogp_srht_project(_ptr(Z), max(Z.stride(0), m), N, m, _ptr(signs), _ptr(rows), k,
                               _ptr(X), max(X.stride(0), k), _ptr(ws), wsb, _stream(stream)))
    return X


def eogp_pca_fit_workspace_size(n: int, m: int, k: int) -> int:
    return int(load().eogp_pca_fit_workspace_size(n, m, k))


def eogp_pca_fit(Z, k, Pt=None, mu=None, ws=None, stream=None):
    """Fit the PCA projection from first-stage coordinates Z [n, m] (float32):
    returns (Pt [k, m] float32, mu [k] float32); see eogp_pca_fit in eogp.h.
    Synchronises the stream."""
    L = load()
    _need_cuda(Z, Pt, mu)
    n, m = Z.shape
    if Z.dtype != torch.float32 or Z.stride(1) != 1:
        raise ValueError("Z must be float32 [n, m] with unit column stride")
    if Pt is None:
        Pt = torch.empty((k, m), dtype=torch.float32, device=Z.device)
    if mu is None:
        mu = torch.empty((k,), dtype=torch.float32, device=Z.device)
    need = int(L.eogp_pca_fit_workspace_size(n, m, k))
    if need == 0:
        bad_sizes = not (1 <= k <= min(n, m))
        raise EogpError(-1 if bad_sizes else -3, L.eogp_last_error().decode())
    ws, wsb = _workspace(need, Z.device, ws)
    _check(L.eogp_pca_fit(_ptr(Z), max(Z.stride(0), m), n, m, k, _ptr(Pt), Pt.stride(0), _ptr(mu),
                          _ptr(ws), wsb, _stream(stream)))
    return Pt, mu


def eogp_sign_pack(X, codes=None, scales=None, stream=None):
    """Packed sign bits [N, ceil(k/8)] (uint8) and fp16 scales [N] (uint16 bits)."""
    L = load()
    _need_cuda(X, codes, scales)
    N, k = X.shape
    if codes is None:
        codes = torch.empty((N, (k + 7) // 8), dtype=torch.uint8, device=X.device)
    if scales is None:
        scales = torch.empty((N, 1), dtype=torch.int16, device=X.device)
    sstride = scales.stride(0) if scales.dim() == 2 else 1
    _check(L.eogp_sign_pack(_ptr(X), X.stride(0), N, k, _ptr(codes), codes.stride(0),
                            _ptr(scales), sstride, _stream(stream)))
    return codes, scales


def tiled_store_bytes(N: int, k_per_module) -> int:
    """Bytes of a tiled store of N rows (see eogp_sign_pack_tiled in eogp.h)."""
    steps = sum(int(k) for k in k_per_module) // 512
    return -(-int(N) // 32) * steps * 2048


def eogp_sign_pack_tiled(X, codes, row0, steps_per_row, step0, scales, stream=None):
    """Sign bits of X [N, k] into rows row0 .. row0+N-1 of a tiled store
    (uint8, tiled_store_bytes long) at the module's first step step0, and
    the fp16 scales into scales (int16 [N] or a column of an [N, U] array)."""
    L = load()
    _need_cuda(X, codes, scales)
    N, k = X.shape
    if codes.dtype != torch.uint8 or not codes.is_contiguous():
        raise ValueError("codes must be a contiguous uint8 tiled store")
    need = -(-(int(row0) + N) // 32) * int(steps_per_row) * 2048
    if N > 0 and codes.numel() < need:
        raise ValueError(f"the tiled store needs at least {need} bytes for these rows")
    sstride = scales.stride(0) if scales.dim() == 2 else 1
    _check(L.eogp_sign_pack_tiled(_ptr(X), X.stride(0), N, k, int(row0), _ptr(codes),
                                  int(steps_per_row), int(step0), _ptr(scales), sstride,
                                  _stream(stream)))
    return codes, scales


def eogp_score_topk_tiled(codes, scales, N, k_per_module, Y, topk, full_scores=False,
                          out_idx=None, out_score=None, ws=None, stream=None):
    """eogp_score_topk over a tiled store of N rows (codes: the uint8 store)."""
    L = load()
    U = len(k_per_module)
    if codes.dtype != torch.uint8 or not codes.is_contiguous():
        raise ValueError("codes must be a contiguous uint8 tiled store")
    if N > 0 and codes.numel() < tiled_store_bytes(N, k_per_module):
        raise ValueError("the tiled store is too small for N rows")
    if scales.dtype not in (torch.int16, torch.float16) or not scales.is_contiguous() or \
            scales.numel() != N * U:
        raise ValueError("scales must be contiguous fp16 bits [N, U]")
    if Y.dtype != torch.float32 or Y.dim() != 2 or (Y.shape[0] > 0 and Y.stride(1) != 1):
        raise ValueError("Y must be float32 [Q, sum k_u] with unit column stride")
    _need_cuda(codes, scales, Y)
    Q = Y.shape[0]
    ks = (c_i64 * U)(*[int(k) for k in k_per_module])
    if out_idx is None:
        out_idx = torch.empty((Q, topk), dtype=torch.int64, device=Y.device)
    if out_score is None:
        out_score = torch.empty((Q, topk), dtype=torch.float32, device=Y.device)
    full = torch.empty((Q, N), dtype=torch.float32, device=Y.device) if full_scores else None
    need = int(L.eogp_score_topk_workspace_size(N, Q, U, ks, topk))
    ws, wsb = _workspace(need, Y.device, ws)
    ldy = Y.stride(0) if Q > 0 else sum(int(k) for k in k_per_module)
    _check(L.eogp_score_topk_tiled(_ptr(codes), _ptr(scales), N, U, ks, _ptr(Y), ldy, Q, topk,
                                   _ptr(out_idx), _ptr(out_score), _ptr(full), _ptr(ws), wsb,
                                   _stream(stream)))
    return out_idx, out_score, full


def eogp_score_topk_workspace_size(N, Q, k_per_module, topk) -> int:
    ks = (c_i64 * len(k_per_module))(*[int(k) for k in k_per_module])
    return int(load().eogp_score_topk_workspace_size(N, Q, len(k_per_module), ks, topk))


def _score_layout(codes, scales, k_per_module, Y):
    U = len(k_per_module)
    if codes.dtype != torch.uint8 or codes.dim() != 2 or (codes.shape[0] > 0 and codes.stride(1) != 1):
        raise ValueError("codes must be uint8 [N, row bytes] with unit column stride")
    N = codes.shape[0]
    if scales.dtype not in (torch.int16, torch.float16):
        raise ValueError("scales must hold fp16 bit patterns (int16 or float16)")
    if not ((scales.dim() == 2 and tuple(scales.shape) == (N, U)) or
            (scales.dim() == 1 and U == 1 and scales.shape[0] == N)) or not scales.is_contiguous():
        raise ValueError("scales must be contiguous [N, U] (or [N] for one module)")
    if Y.dtype != torch.float32 or Y.dim() != 2 or (Y.shape[0] > 0 and Y.stride(1) != 1):
        raise ValueError("Y must be float32 [Q, sum k_u] with unit column stride")
    _need_cuda(codes, scales, Y)
    ksum = sum(int(k) for k in k_per_module)
    # an empty tensor may report stride 0; with no rows any valid stride will do
    cstride = codes.stride(0) if N > 0 else ksum // 8
    ldy = Y.stride(0) if Y.shape[0] > 0 else ksum
    return N, Y.shape[0], U, cstride, ldy


def eogp_score_topk_noalloc(codes, scales, k_per_module, Y, topk, out_idx, out_score,
                            full_scores=None, stream=None):
    """eogp_score_topk without a workspace (see eogp_score_topk_noalloc in
    eogp.h): the library's per-GPU scratch array serves as workspace, so the
    call allocates nothing; outputs are the caller's (index int64 [Q, topk],
    score float32 [Q, topk], optionally every score float32 [Q, N])."""
    L = load()
    N, Q, U, cstride, ldy = _score_layout(codes, scales, k_per_module, Y)
    _need_cuda(out_idx, out_score, full_scores)
    if (out_idx.dtype != torch.int64 or tuple(out_idx.shape) != (Q, topk) or not out_idx.is_contiguous()
            or out_score.dtype != torch.float32 or tuple(out_score.shape) != (Q, topk)
            or not out_score.is_contiguous()):
        raise ValueError("out_idx / out_score must be contiguous int64 / float32 [Q, topk]")
    if full_scores is not None and (full_scores.dtype != torch.float32 or
                                    tuple(full_scores.shape) != (Q, N) or
                                    not full_scores.is_contiguous()):
        raise ValueError("full_scores must be contiguous float32 [Q, N]")
    ks = (c_i64 * U)(*[int(k) for k in k_per_module])
    _check(L.eogp_score_topk_noalloc(_ptr(codes), cstride, _ptr(scales), N, U, ks, _ptr(Y), ldy, Q,
                                     topk, _ptr(out_idx), _ptr(out_score), _ptr(full_scores),
                                     _stream(stream)))
    return out_idx, out_score, full_scores


def eogp_score_topk(codes, scales, k_per_module, Y, topk, full_scores=False, out_idx=None,
                    out_score=None, ws=None, stream=None):
    """Per-query top-k (index int64 [Q, topk], score float32 [Q, topk]) and
    optionally every score (float32 [Q, N])."""
    L = load()
    N, Q, U, cstride, ldy = _score_layout(codes, scales, k_per_module, Y)
    ks = (c_i64 * U)(*[int(k) for k in k_per_module])
    if out_idx is None:
        out_idx = torch.empty((Q, topk), dtype=torch.int64, device=Y.device)
    if out_score is None:
        out_score = torch.empty((Q, topk), dtype=torch.float32, device=Y.device)
    full = torch.empty((Q, N), dtype=torch.float32, device=Y.device) if full_scores else None
    need = int(L.eogp_score_topk_workspace_size(N, Q, U, ks, topk))
    ws, wsb = _workspace(need, Y.device, ws)
    _check(L.eogp_score_topk(_ptr(codes), cstride, _ptr(scales), N, U, ks, _ptr(Y), ldy, Q,
                             topk, _ptr(out_idx), _ptr(out_score), _ptr(full), _ptr(ws), wsb,
                             _stream(stream)))
    return out_idx, out_score, full


def eogp_version() -> int:
    return int(load().eogp_version())


# ---------------------------------------------------------------------------
# Kernel timing (measurement harnesses)
# ---------------------------------------------------------------------------
KT_ROTATION_GEMM, KT_RETAINED, KT_PCA_GEMM, KT_SIGN_PACK = 0, 1, 2, 3
KT_SCORE_PASS, KT_SCORE_MERGE, KT_SCORE_PREP, KT_COMPACTION = 4, 5, 6, 7
KT_SRHT, KT_EKFAC, KT_PCA_FIT = 8, 9, 10
KERNEL_CLASSES = {"rotation_gemm": 0, "retained": 1, "pca_gemm": 2, "sign_pack": 3,
                  "score_pass": 4, "score_merge": 5, "score_prep": 6, "compaction": 7,
                  "srht": 8, "ekfac": 9, "pca_fit": 10}


def eogp_timing_enable(on: bool = True):
    _check(load().eogp_timing_enable(1 if on else 0))


def eogp_timing_read(kernel_class: int):
    """(total milliseconds, launches) of one kernel class since the last read."""
    ms = ctypes.c_double()
    n = c_i64()
    _check(load().eogp_timing_read(int(kernel_class), ctypes.byref(ms), ctypes.byref(n)))
    return float(ms.value), int(n.value)
