"""PAIR hot path on AMD Instinct MI355X: thin Python binding over libpair.so.

Each ``pair_*`` function mirrors the C entry point of the same name declared
in ``include/pair.h``: it checks device, dtype and contiguity of the torch
tensors it is given, passes their device pointers and the current HIP stream,
and turns a negative return code into :class:`PairError`.  Every step of the
computation runs in the library's HIP kernels; torch only provides device
memory and the stream.  There is no fallback: if ``libpair.so`` is missing the
import of the library fails loudly (build it with
``python -m paper_2608_11368_amd.build``).

The lower-case helpers (``design_inclusion``, ``edge_coeffs``,
``weighted_grad``, ``audit``) allocate the outputs with torch and call the
``pair_*`` functions.  Given an explicit ``stream``, a helper makes it torch's
current stream while it allocates, clears and launches, so the zero-fills are
ordered before the kernels and the caching allocator hands a temporary
workspace to later work only behind them.
"""
from __future__ import annotations

import ctypes
import functools
import inspect
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# PAIR_LIB names another build of the same library to load instead (the test
# suite's host-sanitizer build); it must exist like the default one.
LIB_PATH = os.environ.get("PAIR_LIB") or os.path.join(_HERE, "libpair.so")

PAIR_F32 = 0
PAIR_BF16 = 1
ST_BAD_GROUP = 1
ST_RHO_RANGE = 2
ST_P_RANGE = 4
ST_NONFINITE = 8
ST_BUDGET = 16
ST_SOLVER = 32
DESIGN_PAIR = 0
DESIGN_POINTWISE = 1
DESIGN_UNIFORM = 2
GMAX_LIMIT = 64
# Bytes of the static device scratch that pair_audit_noalloc uses as its workspace.
AUDIT_SCRATCH_BYTES = 64 << 20

RULE_HT = 0
RULE_UNWEIGHTED = 1
RULE_RATIO_KE = 2
RULE_CLIPPED = 3
RULE_SELFNORM = 4
RULE_MARGINAL = 5

EXPORTED = ("pair_design_coeffs", "pair_design_alloc", "pair_design_alloc_ex", "pair_cps_fit", "pair_cps_draw", "pair_design_inclusion", "pair_edge_coeffs", "pair_edge_coeffs_rule",
            "pair_weighted_grad", "pair_audit_workspace_bytes", "pair_audit", "pair_audit_rule",
            "pair_audit_exact_workspace_bytes", "pair_audit_exact",
            "pair_audit_direction_workspace_bytes", "pair_audit_direction", "pair_audit_noalloc",
            "pair_strerror", "pair_version")


class PairError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {strerror(code)} (code {code})")


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded libpair.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_2608_11368_amd.build` (hipcc, gfx950)")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        i64, i32, u64 = ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64
        L.pair_design_inclusion.argtypes = [i64, i64, i32, P, P, u64, i64, i64, P, P, P, P, P, P]
        L.pair_design_inclusion.restype = ctypes.c_int
        L.pair_edge_coeffs.argtypes = [i64, i64, i32, P, P, P, P, P, P, P, P]
        L.pair_edge_coeffs.restype = ctypes.c_int
        f32 = ctypes.c_float
        L.pair_edge_coeffs_rule.argtypes = [i64, i64, i32, P, P, P, P, i32, f32, P, P, P, P, P, P]
        L.pair_edge_coeffs_rule.restype = ctypes.c_int
        L.pair_audit_rule.argtypes = [i64, i64, i32, P, i64, P, i32, i64, P, P, P, i32, f32, u64,
                                      i64, i64, P, P, P, P, P, ctypes.c_size_t, P, P]
        L.pair_audit_rule.restype = ctypes.c_int
        L.pair_audit_exact_workspace_bytes.argtypes = [i64, i32, i64]
        L.pair_audit_exact_workspace_bytes.restype = ctypes.c_size_t
        L.pair_audit_exact.argtypes = [i64, i64, i32, P, i64, P, i32, i64, P, P, P, i32, f32, P, P,
                                       P, P, ctypes.c_size_t, P, P]
        L.pair_audit_exact.restype = ctypes.c_int
        L.pair_design_alloc.argtypes = [i64, i64, i32, P, P, P, P, P, f32, i32, P, P, P, P, P]
        L.pair_design_alloc.restype = ctypes.c_int
        L.pair_design_alloc_ex.argtypes = [i64, i64, i32, P, P, P, P, P, f32, i32, P, i32, P, P, P,
                                           P, P, P]
        L.pair_design_alloc_ex.restype = ctypes.c_int
        L.pair_audit_direction_workspace_bytes.argtypes = [i64, i32, i64, i64]
        L.pair_audit_direction_workspace_bytes.restype = ctypes.c_size_t
        L.pair_audit_direction.argtypes = [i64, i64, i32, P, i64, P, i32, i64, P, P, P, i32, f32,
                                           u64, i64, i64, P, P, P, ctypes.c_size_t, P, P]
        L.pair_audit_direction.restype = ctypes.c_int
        L.pair_design_coeffs.argtypes = [i64, i64, i32, P, P, P, u64, i64, P, P, P, P, P, P, P]
        L.pair_design_coeffs.restype = ctypes.c_int
        L.pair_cps_fit.argtypes = [i64, i64, i32, P, P, P, P, P, P, P, P]
        L.pair_cps_fit.restype = ctypes.c_int
        L.pair_cps_draw.argtypes = [i64, i64, i32, P, P, P, u64, i64, i64, P, P, P, P]
        L.pair_cps_draw.restype = ctypes.c_int
        L.pair_weighted_grad.argtypes = [i64, i64, P, i64, P, i32, i64, P, P, i32, P, P]
        L.pair_weighted_grad.restype = ctypes.c_int
        L.pair_audit_workspace_bytes.argtypes = [i64, i32, i64, i64]
        L.pair_audit_workspace_bytes.restype = ctypes.c_size_t
        L.pair_audit.argtypes = [i64, i64, i32, P, i64, P, i32, i64, P, P, P, u64, i64, i64,
                                 P, P, P, P, P, ctypes.c_size_t, P, P]
        L.pair_audit.restype = ctypes.c_int
        L.pair_audit_noalloc.argtypes = [i64, i64, i32, P, i64, P, i32, i64, P, P, P, u64, i64,
                                         i64, P, P, P, P, P, P]
        L.pair_audit_noalloc.restype = ctypes.c_int
        L.pair_strerror.argtypes = [ctypes.c_int]
        L.pair_strerror.restype = ctypes.c_char_p
        L.pair_version.argtypes = []
        L.pair_version.restype = ctypes.c_int
        _lib = L
    return _lib


def strerror(code: int) -> str:
    return lib().pair_strerror(int(code)).decode()


def version() -> int:
    return lib().pair_version()


# ----------------------------------------------------------- marshalling ---
def _dev(t, name, dtype, numel=None, allow_none=False):
    if t is None:
        if allow_none:
            return None
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise ValueError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} holds {t.numel()} elements, needs {numel}")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _scores_arg(scores):
    if not isinstance(scores, torch.Tensor) or scores.device.type != "cuda" or scores.dim() != 2:
        raise ValueError("scores must be a 2-D CUDA tensor [nv][ld-strided rows]")
    if scores.stride(1) != 1:
        raise ValueError("scores rows must be contiguous")
    if scores.dtype == torch.float32:
        code = PAIR_F32
    elif scores.dtype == torch.bfloat16:
        code = PAIR_BF16
    else:
        raise TypeError("scores must be float32 or bfloat16")
    return ctypes.c_void_p(scores.data_ptr()), code, scores.stride(0), scores.shape[1]


def _rc(code, where):
    if code != 0:
        raise PairError(code, where)


# ------------------------------------------------------- C-ABI mirrors -----
def pair_design_inclusion(B, nv, gmax, offsets, p, seed, rep0, R, mask=None, pi=None,
                          edge_count=None, completed=None, d_status=None, stream=None):
    _rc(lib().pair_design_inclusion(
        B, nv, gmax, _dev(offsets, "offsets", torch.int64, B + 1), _dev(p, "p", torch.float32, nv),
        ctypes.c_uint64(seed & ((1 << 64) - 1)), rep0, R,
        _dev(mask, "mask", torch.uint8, R * nv, True),
        _dev(pi, "pi", torch.float32, B * gmax * gmax, True),
        _dev(edge_count, "edge_count", torch.int32, R * B, True),
        _dev(completed, "completed", torch.int32, R * B, True),
        _dev(d_status, "d_status", torch.int32, 1, True), _stream(stream)), "pair_design_inclusion")


def pair_design_coeffs(B, nv, gmax, offsets, p, rewards, seed, rep, coeff, mask=None, pi=None,
                       edge_count=None, completed=None, d_status=None, stream=None):
    _rc(lib().pair_design_coeffs(
        B, nv, gmax, _dev(offsets, "offsets", torch.int64, B + 1), _dev(p, "p", torch.float32, nv),
        _dev(rewards, "rewards", torch.float32, nv), ctypes.c_uint64(seed & ((1 << 64) - 1)), rep,
        _dev(mask, "mask", torch.uint8, nv, True),
        _dev(pi, "pi", torch.float32, B * gmax * gmax, True),
        _dev(coeff, "coeff", torch.float32, nv),
        _dev(edge_count, "edge_count", torch.int32, B, True),
        _dev(completed, "completed", torch.int32, B, True),
        _dev(d_status, "d_status", torch.int32, 1, True), _stream(stream)), "pair_design_coeffs")


def pair_design_alloc(B, nv, gmax, offsets, p_hat, c_hat, m_hat, budget, pi_min, design, pi,
                      objective=None, iters=None, d_status=None, stream=None):
    _rc(lib().pair_design_alloc(
        B, nv, gmax, _dev(offsets, "offsets", torch.int64, B + 1),
        _dev(p_hat, "p_hat", torch.float32, nv), _dev(c_hat, "c_hat", torch.float32, nv),
        _dev(m_hat, "m_hat", torch.float32, nv, True), _dev(budget, "budget", torch.float32, B),
        float(pi_min), int(design), _dev(pi, "pi", torch.float32, nv),
        _dev(objective, "objective", torch.float64, B, True),
        _dev(iters, "iters", torch.int32, B, True),
        _dev(d_status, "d_status", torch.int32, 1, True), _stream(stream)), "pair_design_alloc")


def pair_design_alloc_ex(B, nv, gmax, offsets, p_hat, c_hat, m_hat, budget, pi_min, design,
                         pi_prev, max_sweeps, pi, objective=None, iters=None, residual=None,
                         d_status=None, stream=None):
    _rc(lib().pair_design_alloc_ex(
        B, nv, gmax, _dev(offsets, "offsets", torch.int64, B + 1),
        _dev(p_hat, "p_hat", torch.float32, nv), _dev(c_hat, "c_hat", torch.float32, nv),
        _dev(m_hat, "m_hat", torch.float32, nv, True), _dev(budget, "budget", torch.float32, B),
        float(pi_min), int(design), _dev(pi_prev, "pi_prev", torch.float32, nv, True),
        int(max_sweeps), _dev(pi, "pi", torch.float32, nv),
        _dev(objective, "objective", torch.float64, B, True),
        _dev(iters, "iters", torch.int32, B, True),
        _dev(residual, "residual", torch.float64, B, True),
        _dev(d_status, "d_status", torch.int32, 1, True), _stream(stream)), "pair_design_alloc_ex")


def pair_cps_fit(B, nv, gmax, offsets, pi_target, w, n_out=None, pi_joint=None, iters=None,
                 d_status=None, stream=None):
    _rc(lib().pair_cps_fit(
        B, nv, gmax, _dev(offsets, "offsets", torch.int64, B + 1),
        _dev(pi_target, "pi_target", torch.float32, nv), _dev(w, "w", torch.float64, nv),
        _dev(n_out, "n_out", torch.int32, B, True),
        _dev(pi_joint, "pi_joint", torch.float32, B * gmax * gmax, True),
        _dev(iters, "iters", torch.int32, B, True),
        _dev(d_status, "d_status", torch.int32, 1, True), _stream(stream)), "pair_cps_fit")


def pair_cps_draw(B, nv, gmax, offsets, w, n, seed, rep0, R, mask, edge_count=None,
                  d_status=None, stream=None):
    _rc(lib().pair_cps_draw(
        B, nv, gmax, _dev(offsets, "offsets", torch.int64, B + 1), _dev(w, "w", torch.float64, nv),
        _dev(n, "n", torch.int32, B), ctypes.c_uint64(seed & ((1 << 64) - 1)), rep0, R,
        _dev(mask, "mask", torch.uint8, R * nv),
        _dev(edge_count, "edge_count", torch.int32, R * B, True),
        _dev(d_status, "d_status", torch.int32, 1, True), _stream(stream)), "pair_cps_draw")


def pair_edge_coeffs(B, nv, gmax, offsets, rewards, mask, pi, coeff, edge_count=None,
                     d_status=None, stream=None):
    _rc(lib().pair_edge_coeffs(
        B, nv, gmax, _dev(offsets, "offsets", torch.int64, B + 1),
        _dev(rewards, "rewards", torch.float32, nv), _dev(mask, "mask", torch.uint8, nv, True),
        _dev(pi, "pi", torch.float32, B * gmax * gmax, True),
        _dev(coeff, "coeff", torch.float32, nv),
        _dev(edge_count, "edge_count", torch.int32, B, True),
        _dev(d_status, "d_status", torch.int32, 1, True), _stream(stream)), "pair_edge_coeffs")


def pair_edge_coeffs_rule(B, nv, gmax, offsets, rewards, mask, pi, rule, wmax, coeff,
                          edge_count=None, ess=None, max_weight=None, d_status=None, stream=None):
    _rc(lib().pair_edge_coeffs_rule(
        B, nv, gmax, _dev(offsets, "offsets", torch.int64, B + 1),
        _dev(rewards, "rewards", torch.float32, nv), _dev(mask, "mask", torch.uint8, nv, True),
        _dev(pi, "pi", torch.float32, B * gmax * gmax, True), int(rule), float(wmax),
        _dev(coeff, "coeff", torch.float32, nv),
        _dev(edge_count, "edge_count", torch.int32, B, True),
        _dev(ess, "ess", torch.float32, B, True), _dev(max_weight, "max_weight", torch.float32, B, True),
        _dev(d_status, "d_status", torch.int32, 1, True), _stream(stream)), "pair_edge_coeffs_rule")


def pair_weighted_grad(B, nv, offsets, scores, coeff, out, reduce=0, d_status=None, stream=None):
    sp, code, ld, D = _scores_arg(scores)
    _rc(lib().pair_weighted_grad(
        B, nv, _dev(offsets, "offsets", torch.int64, B + 1), D, sp, code, ld,
        _dev(coeff, "coeff", torch.float32, nv),
        _dev(out, "out", torch.float32, D if reduce else B * D), int(reduce),
        _dev(d_status, "d_status", torch.int32, 1, True), _stream(stream)), "pair_weighted_grad")


def pair_audit_workspace_bytes(B, gmax, D, R) -> int:
    return int(lib().pair_audit_workspace_bytes(B, gmax, D, R))


def pair_audit(B, nv, gmax, offsets, scores, rewards, p, pi_w, seed, rep0, R, mse, bias_norm,
               rep_sqerr, edge_count, workspace, d_status=None, stream=None):
    pair_audit_rule(B, nv, gmax, offsets, scores, rewards, p, pi_w, RULE_HT, 0.0, seed, rep0, R,
                    mse, bias_norm, rep_sqerr, edge_count, workspace, d_status, stream,
                    _name="pair_audit")


def pair_audit_rule(B, nv, gmax, offsets, scores, rewards, p, pi_w, rule, wmax, seed, rep0, R,
                    mse, bias_norm, rep_sqerr, edge_count, workspace, d_status=None, stream=None,
                    _name="pair_audit_rule"):
    sp, code, ld, D = _scores_arg(scores)
    ws = _dev(workspace, "workspace", torch.uint8)
    fn = lib().pair_audit if _name == "pair_audit" else lib().pair_audit_rule
    extra = () if _name == "pair_audit" else (int(rule), float(wmax))
    _rc(fn(
        B, nv, gmax, _dev(offsets, "offsets", torch.int64, B + 1), D, sp, code, ld,
        _dev(rewards, "rewards", torch.float32, nv), _dev(p, "p", torch.float32, nv),
        _dev(pi_w, "pi_w", torch.float32, B * gmax * gmax, True), *extra,
        ctypes.c_uint64(seed & ((1 << 64) - 1)), rep0, R,
        _dev(mse, "mse", torch.float64, B), _dev(bias_norm, "bias_norm", torch.float64, B),
        _dev(rep_sqerr, "rep_sqerr", torch.float32, B * R, True),
        _dev(edge_count, "edge_count", torch.int32, B * R, True),
        ws, workspace.numel(), _dev(d_status, "d_status", torch.int32, 1, True),
        _stream(stream)), _name)


def pair_audit_noalloc(B, nv, gmax, offsets, scores, rewards, p, pi_w, seed, rep0, R, mse,
                       bias_norm, rep_sqerr=None, edge_count=None, d_status=None, stream=None):
    """pair_audit with the library's static device scratch as its workspace."""
    sp, code, ld, D = _scores_arg(scores)
    _rc(lib().pair_audit_noalloc(
        B, nv, gmax, _dev(offsets, "offsets", torch.int64, B + 1), D, sp, code, ld,
        _dev(rewards, "rewards", torch.float32, nv), _dev(p, "p", torch.float32, nv),
        _dev(pi_w, "pi_w", torch.float32, B * gmax * gmax, True),
        ctypes.c_uint64(seed & ((1 << 64) - 1)), rep0, R,
        _dev(mse, "mse", torch.float64, B), _dev(bias_norm, "bias_norm", torch.float64, B),
        _dev(rep_sqerr, "rep_sqerr", torch.float32, B * R, True),
        _dev(edge_count, "edge_count", torch.int32, B * R, True),
        _dev(d_status, "d_status", torch.int32, 1, True), _stream(stream)), "pair_audit_noalloc")


def pair_audit_direction_workspace_bytes(B, gmax, D, R) -> int:
    return int(lib().pair_audit_direction_workspace_bytes(B, gmax, D, R))


def pair_audit_direction(B, nv, gmax, offsets, scores, rewards, p, pi_w, rule, wmax, seed, rep0,
                         R, cosine, target_norm, workspace, d_status=None, stream=None):
    sp, code, ld, D = _scores_arg(scores)
    ws = _dev(workspace, "workspace", torch.uint8)
    _rc(lib().pair_audit_direction(
        B, nv, gmax, _dev(offsets, "offsets", torch.int64, B + 1), D, sp, code, ld,
        _dev(rewards, "rewards", torch.float32, nv), _dev(p, "p", torch.float32, nv),
        _dev(pi_w, "pi_w", torch.float32, B * gmax * gmax, True), int(rule), float(wmax),
        ctypes.c_uint64(seed & ((1 << 64) - 1)), rep0, R,
        _dev(cosine, "cosine", torch.float64, B), _dev(target_norm, "target_norm", torch.float64, B),
        ws, workspace.numel(), _dev(d_status, "d_status", torch.int32, 1, True),
        _stream(stream)), "pair_audit_direction")


def pair_audit_exact_workspace_bytes(B, gmax, D) -> int:
    return int(lib().pair_audit_exact_workspace_bytes(B, gmax, D))


def pair_audit_exact(B, nv, gmax, offsets, scores, rewards, p, pi_w, rule, wmax, mse, bias_norm,
                     gram, workspace, d_status=None, stream=None):
    sp, code, ld, D = _scores_arg(scores)
    _rc(lib().pair_audit_exact(
        B, nv, gmax, _dev(offsets, "offsets", torch.int64, B + 1), D, sp, code, ld,
        _dev(rewards, "rewards", torch.float32, nv), _dev(p, "p", torch.float32, nv),
        _dev(pi_w, "pi_w", torch.float32, B * gmax * gmax, True), int(rule), float(wmax),
        _dev(mse, "mse", torch.float64, B), _dev(bias_norm, "bias_norm", torch.float64, B),
        _dev(gram, "gram", torch.float64, B * gmax * gmax, True),
        _dev(workspace, "workspace", torch.uint8), workspace.numel(),
        _dev(d_status, "d_status", torch.int32, 1, True), _stream(stream)), "pair_audit_exact")


# ------------------------------------------------ allocating helpers -------
def _nv(offsets):
    return int(offsets[-1].item())


def _allocating(fn):
    """Run an allocating helper with its `stream` argument (when given) as
    torch's current stream: outputs, status words and temporary workspaces
    are then allocated and zero-filled on the stream the kernels run on."""
    sig = inspect.signature(fn)

    @functools.wraps(fn)
    def wrapper(*args, **kwargs):
        stream = sig.bind(*args, **kwargs).arguments.get("stream")
        if stream is None:
            return fn(*args, **kwargs)
        with torch.cuda.stream(stream):
            return fn(*args, **kwargs)

    return wrapper


@_allocating
def design_inclusion(offsets, p, seed, rep0, R, gmax, want_mask=True, want_pi=True, nv=None,
                     stream=None):
    B = offsets.numel() - 1
    nv = _nv(offsets) if nv is None else nv
    dev = p.device
    out = {
        "mask": torch.empty((R, nv), dtype=torch.uint8, device=dev) if want_mask else None,
        "pi": torch.empty((B, gmax, gmax), dtype=torch.float32, device=dev) if want_pi else None,
        "edge_count": torch.empty((R, B), dtype=torch.int32, device=dev),
        "completed": torch.empty((R, B), dtype=torch.int32, device=dev),
        "status": torch.zeros(1, dtype=torch.int32, device=dev),
    }
    pair_design_inclusion(B, nv, gmax, offsets, p, seed, rep0, R, out["mask"], out["pi"],
                          out["edge_count"], out["completed"], out["status"], stream)
    return out


@_allocating
def design_coeffs(offsets, p, rewards, seed, rep, gmax, want_mask=True, want_pi=True, nv=None,
                  stream=None):
    """One replicate's design draw and its sequence advantages A~ in one
    launch (the per-rollout weights a trainer applies to the log-probability
    gradients), with the mask and the logged rho block."""
    B = offsets.numel() - 1
    nv = _nv(offsets) if nv is None else nv
    dev = p.device
    out = {
        "coeff": torch.empty(nv, dtype=torch.float32, device=dev),
        "mask": torch.empty(nv, dtype=torch.uint8, device=dev) if want_mask else None,
        "pi": torch.empty((B, gmax, gmax), dtype=torch.float32, device=dev) if want_pi else None,
        "edge_count": torch.empty(B, dtype=torch.int32, device=dev),
        "completed": torch.empty(B, dtype=torch.int32, device=dev),
        "status": torch.zeros(1, dtype=torch.int32, device=dev),
    }
    pair_design_coeffs(B, nv, gmax, offsets, p, rewards, seed, rep, out["coeff"], out["mask"],
                       out["pi"], out["edge_count"], out["completed"], out["status"], stream)
    return out


@_allocating
def edge_coeffs(offsets, rewards, mask, pi, gmax, nv=None, rule=None, wmax=0.0, stream=None):
    """Coefficients; with `rule` (RULE_*) also returns the ESS and the maximum weight."""
    B = offsets.numel() - 1
    nv = _nv(offsets) if nv is None else nv
    dev = rewards.device
    coeff = torch.empty(nv, dtype=torch.float32, device=dev)
    ec = torch.empty(B, dtype=torch.int32, device=dev)
    st = torch.zeros(1, dtype=torch.int32, device=dev)
    if rule is None:
        pair_edge_coeffs(B, nv, gmax, offsets, rewards, mask, pi, coeff, ec, st, stream)
        return {"coeff": coeff, "edge_count": ec, "status": st}
    ess = torch.empty(B, dtype=torch.float32, device=dev)
    mw = torch.empty(B, dtype=torch.float32, device=dev)
    pair_edge_coeffs_rule(B, nv, gmax, offsets, rewards, mask, pi, rule, wmax, coeff, ec, ess, mw,
                          st, stream)
    return {"coeff": coeff, "edge_count": ec, "ess": ess, "max_weight": mw, "status": st}


@_allocating
def weighted_grad(offsets, scores, coeff, nv=None, reduce=False, stream=None):
    B = offsets.numel() - 1
    nv = _nv(offsets) if nv is None else nv
    D = scores.shape[1]
    shape = (D,) if reduce else (B, D)
    out = torch.empty(shape, dtype=torch.float32, device=scores.device)
    st = torch.zeros(1, dtype=torch.int32, device=scores.device)
    pair_weighted_grad(B, nv, offsets, scores, coeff, out, int(bool(reduce)), st, stream)
    return {"out": out, "status": st}


@_allocating
def audit(offsets, scores, rewards, p, seed, rep0, R, gmax, pi_w=None, want_reps=True, nv=None,
          workspace=None, rule=None, wmax=0.0, stream=None):
    B = offsets.numel() - 1
    nv = _nv(offsets) if nv is None else nv
    dev = scores.device
    need = pair_audit_workspace_bytes(B, gmax, scores.shape[1], R)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    out = {
        "mse": torch.empty(B, dtype=torch.float64, device=dev),
        "bias_norm": torch.empty(B, dtype=torch.float64, device=dev),
        "rep_sqerr": torch.empty((B, R), dtype=torch.float32, device=dev) if want_reps else None,
        "edge_count": torch.empty((B, R), dtype=torch.int32, device=dev) if want_reps else None,
        "status": torch.zeros(1, dtype=torch.int32, device=dev),
    }
    if rule is None:
        pair_audit(B, nv, gmax, offsets, scores, rewards, p, pi_w, seed, rep0, R, out["mse"],
                   out["bias_norm"], out["rep_sqerr"], out["edge_count"], workspace, out["status"],
                   stream)
    else:
        pair_audit_rule(B, nv, gmax, offsets, scores, rewards, p, pi_w, rule, wmax, seed, rep0, R,
                        out["mse"], out["bias_norm"], out["rep_sqerr"], out["edge_count"],
                        workspace, out["status"], stream)
    return out


@_allocating
def audit_direction(offsets, scores, rewards, p, seed, rep0, R, gmax, pi_w=None, rule=RULE_HT,
                    wmax=0.0, nv=None, workspace=None, stream=None):
    """Mean per-replicate cosine between estimate and target, and |t|."""
    B = offsets.numel() - 1
    nv = _nv(offsets) if nv is None else nv
    dev = scores.device
    need = pair_audit_direction_workspace_bytes(B, gmax, scores.shape[1], R)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    out = {
        "cosine": torch.empty(B, dtype=torch.float64, device=dev),
        "target_norm": torch.empty(B, dtype=torch.float64, device=dev),
        "status": torch.zeros(1, dtype=torch.int32, device=dev),
    }
    pair_audit_direction(B, nv, gmax, offsets, scores, rewards, p, pi_w, rule, wmax, seed, rep0, R,
                         out["cosine"], out["target_norm"], workspace, out["status"], stream)
    return out


@_allocating
def audit_exact(offsets, scores, rewards, p, gmax, pi_w=None, rule=RULE_HT, wmax=0.0,
                want_gram=False, nv=None, workspace=None, stream=None):
    """Exact design MSE and bias norm per prompt (no draws); optional Gram."""
    B = offsets.numel() - 1
    nv = _nv(offsets) if nv is None else nv
    dev = scores.device
    need = pair_audit_exact_workspace_bytes(B, gmax, scores.shape[1])
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    out = {
        "mse": torch.empty(B, dtype=torch.float64, device=dev),
        "bias_norm": torch.empty(B, dtype=torch.float64, device=dev),
        "gram": torch.zeros((B, gmax, gmax), dtype=torch.float64, device=dev) if want_gram else None,
        "status": torch.zeros(1, dtype=torch.int32, device=dev),
    }
    pair_audit_exact(B, nv, gmax, offsets, scores, rewards, p, pi_w, rule, wmax, out["mse"],
                     out["bias_norm"], out["gram"], workspace, out["status"], stream)
    return out


@_allocating
def design_alloc(offsets, p_hat, c_hat, budget, gmax, pi_min=0.08, design=DESIGN_PAIR, m_hat=None,
                 nv=None, pi_prev=None, max_sweeps=0, stream=None):
    """Continuation probabilities of every prompt (fp32 [nv]) with the
    objective, sweep counts (negative: solver fallback), KKT residual and
    status; `pi_prev` warm-starts the solver, `max_sweeps` caps it."""
    B = offsets.numel() - 1
    nv = _nv(offsets) if nv is None else nv
    dev = p_hat.device
    out = {
        "pi": torch.empty(nv, dtype=torch.float32, device=dev),
        "objective": torch.empty(B, dtype=torch.float64, device=dev),
        "iters": torch.empty(B, dtype=torch.int32, device=dev),
        "residual": torch.empty(B, dtype=torch.float64, device=dev),
        "status": torch.zeros(1, dtype=torch.int32, device=dev),
    }
    pair_design_alloc_ex(B, nv, gmax, offsets, p_hat, c_hat, m_hat, budget, pi_min, design,
                         pi_prev, max_sweeps, out["pi"], out["objective"], out["iters"],
                         out["residual"], out["status"], stream)
    return out


@_allocating
def cps_fit(offsets, pi_target, gmax, nv=None, stream=None):
    """Fixed-size design from target probabilities: dict(w, n, pi_joint, iters, status)."""
    B = offsets.numel() - 1
    nv = _nv(offsets) if nv is None else nv
    dev = pi_target.device
    out = {
        "w": torch.empty(nv, dtype=torch.float64, device=dev),
        "n": torch.empty(B, dtype=torch.int32, device=dev),
        "pi_joint": torch.empty((B, gmax, gmax), dtype=torch.float32, device=dev),
        "iters": torch.empty(B, dtype=torch.int32, device=dev),
        "status": torch.zeros(1, dtype=torch.int32, device=dev),
    }
    pair_cps_fit(B, nv, gmax, offsets, pi_target, out["w"], out["n"], out["pi_joint"],
                 out["iters"], out["status"], stream)
    return out


@_allocating
def cps_draw(offsets, w, n, seed, rep0, R, gmax, nv=None, stream=None):
    """Fixed-size draws: dict(mask[R][nv], edge_count[R][B], status)."""
    B = offsets.numel() - 1
    nv = _nv(offsets) if nv is None else nv
    dev = w.device
    out = {
        "mask": torch.empty((R, nv), dtype=torch.uint8, device=dev),
        "edge_count": torch.empty((R, B), dtype=torch.int32, device=dev),
        "status": torch.zeros(1, dtype=torch.int32, device=dev),
    }
    pair_cps_draw(B, nv, gmax, offsets, w, n, seed, rep0, R, out["mask"], out["edge_count"],
                  out["status"], stream)
    return out
