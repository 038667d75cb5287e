"""ctypes binding of libgmc.so: the C-ABI entry points under the same names,
plus a thin tensor-level wrapper (argument marshalling only).

Every step of the operator runs inside the HIP library.  If the library has
not been built, ``lib()`` raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libgmc.so")

GMC_OK, GMC_ERR_ARG, GMC_ERR_CAPACITY, GMC_ERR_STATE, GMC_ERR_HIP = 0, -1, -2, -3, -4
GMC_ERR_DEVICE, GMC_ERR_NONFINITE = -5, -6
GMC_STATUS_SELECT_TIMEOUT, GMC_STATUS_BANK_TIMEOUT, GMC_STATUS_NONFINITE = 1, 2, 4
GMC_DIAG_CERT, GMC_DIAG_FINITE = 1, 2
GMC_CERT_MAX_ROUNDS = 64
GMC_STATIC_SCRATCH_BYTES = 64 << 20
GMC_F32, GMC_BF16 = 0, 1
GMC_STATS = 15
GMC_MAX_HIST_VIEWS = 3
GMC_MAX_IMAGES = 64
GMC_AUDIT_ROW, GMC_AUDIT_OUT = 8, 8
GMC_STATUS_INPUT = 8
GMC_MAX_GATHER_TENSORS = 64

_i32, _f32, _i64, _vp = ctypes.c_int32, ctypes.c_float, ctypes.c_int64, ctypes.c_void_p


class GmcConfig(ctypes.Structure):
    """Mirror of ``gmc_config`` in include/gmc.h (same field order)."""
    _fields_ = [
        ("d", _i32), ("n_q_heads", _i32), ("n_kv_heads", _i32), ("head_dim", _i32),
        ("probe_rank", _i32), ("dtype", _i32), ("max_batch", _i32), ("max_n", _i32),
        ("max_t", _i32), ("max_k", _i32),
        ("value_probe", _vp), ("app_projection", _vp),
        ("lambda_mass", _f32), ("eps_mass", _f32),
        ("beta_msg", _f32), ("beta_app", _f32), ("beta_spa", _f32),
        ("tau_v", _f32), ("tau_s", _f32),
        ("landmarks", _i32),
        ("batch_b", _i32), ("pool_mult", _i32),
        ("tau_r", _f32), ("resp_eps", _f32),
        ("spatial_w", _f32), ("gate_t", _f32), ("gate_p", _f32),
        ("amb_margin", _f32), ("amb_p", _f32),
        ("g_form", _i32),
        ("pop_strength", _f32), ("tau_j", _f32),
        ("max_head_clusters", _i32),
        ("disp_eps", _f32), ("terminal_q_weight", _f32),
        ("rms_eps", _f32), ("norm_eps", _f32), ("restore_eps", _f32),
        ("bounded_threshold_n", _i32),
        ("app_rank", _i32), ("app_max_clients", _i32),
        ("batch_b_bounded", _i32),
        ("value_probe_bias", _vp),
        ("max_hist_views", _i32), ("hist_mass", _f32),
        ("value_probe_hist", _vp), ("value_probe_bias_hist", _vp),
        ("max_images", _i32),
    ]


class GmcTrace(ctypes.Structure):
    """Mirror of ``gmc_trace``: optional device output pointers."""
    _fields_ = [("round_pool", _vp), ("round_batch", _vp), ("assign", _vp), ("omega", _vp),
                ("ebar", _vp), ("client", _vp), ("stats", _vp), ("round_gains", _vp),
                ("round_scores", _vp)]


class GmcView(ctypes.Structure):
    """Mirror of ``gmc_view``: one historical message view's device tensors."""
    _fields_ = [("hidden", _vp), ("text_q", _vp), ("vis_k", _vp), ("nonvis_lse", _vp)]


class GmcDiag(ctypes.Structure):
    """Mirror of ``gmc_diag``: host-side diagnostics of the last call."""
    _fields_ = [("status", ctypes.c_uint32), ("identity", _i32), ("has_certificate", _i32),
                ("k", _i32), ("rounds", _i32), ("m_rows", _i32), ("n_discarded", _i32),
                ("s_x", _f32), ("dbar", _f32), ("f_s", _f32), ("f_v", _f32),
                ("f_bank_s", _f32 * 3), ("f_bank_v", _f32 * 3), ("c_b", _f32),
                ("max_rounds", _i32),
                ("u_top", ctypes.POINTER(_f32)), ("gain", ctypes.POINTER(_f32)),
                ("q", ctypes.POINTER(_f32)), ("pool_margin", ctypes.POINTER(_f32)),
                ("batch_margin", ctypes.POINTER(_f32))]


# name -> (restype, argtypes) of every symbol include/gmc.h declares
SIGNATURES = {
    "gmc_config_default": (None, [ctypes.POINTER(GmcConfig)]),
    "gmc_init": (ctypes.c_int, [ctypes.POINTER(GmcConfig)]),
    "gmc_set_stream": (ctypes.c_int, [_vp]),
    "gmc_prune": (ctypes.c_int, [_vp, _vp, _vp, _vp, _i64, _i64, _i64, _vp, _vp, _vp]),
    "gmc_prune_ex": (ctypes.c_int, [_i64, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _vp, _vp, _vp, _vp,
                                    ctypes.POINTER(GmcTrace)]),
    "gmc_prune_views": (ctypes.c_int, [_i64, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _vp, _vp, _vp, _vp, _i64,
                                       ctypes.POINTER(GmcView), ctypes.POINTER(GmcTrace)]),
    "gmc_prune_full": (ctypes.c_int, [_i64, _vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64, _vp, _vp, _vp, _vp,
                                      _i64, ctypes.POINTER(GmcView), ctypes.POINTER(GmcTrace)]),
    "gmc_realized_budget": (_i64, [_i64, _i64, _i64]),
    "gmc_audit_message": (ctypes.c_int, [_i64, _i64, _i64, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                         _vp]),
    "gmc_trace_dims_full": (ctypes.c_int, [_i64, _i64, _i64, _i64, _i64, ctypes.POINTER(_i64), ctypes.POINTER(_i64),
                                           ctypes.POINTER(_i64), ctypes.POINTER(_i64)]),
    "gmc_realized_k": (_i64, [_i64, _i64]),
    "gmc_trace_dims": (ctypes.c_int, [_i64, _i64, _i64, ctypes.POINTER(_i64), ctypes.POINTER(_i64),
                                      ctypes.POINTER(_i64), ctypes.POINTER(_i64)]),
    "gmc_compact_sequence": (ctypes.c_int, [_i64, _i64, _i64, _i64, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _i64,
                                            _vp, _vp]),
    "gmc_gather_rows": (ctypes.c_int, [_i64, ctypes.POINTER(_vp), ctypes.POINTER(_vp), _i64, _i64, _i64, _i64,
                                       _i64, _vp]),
    "gmc_set_diag": (ctypes.c_int, [_i32]),
    "gmc_get_diag": (ctypes.c_int, [_i64, ctypes.POINTER(GmcDiag)]),
    "gmc_prune_static": (ctypes.c_int, [ctypes.POINTER(GmcConfig), _i64, _vp, _vp, _vp, _vp, _i64, _i64, _i64,
                                        _vp, _vp, _vp, _vp, _vp]),
    "gmc_workspace_bytes": (_i64, []),
    "gmc_last_error": (ctypes.c_char_p, []),
    "gmc_free": (None, []),
}

_LIB = None


def lib():
    """Load libgmc.so (raises if it has not been built)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -c 'import __graft_entry__ as g; g.build()'`")
        so = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(so, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = so
    return _LIB


class GmcError(RuntimeError):
    def __init__(self, code: int, where: str):
        msg = lib().gmc_last_error().decode(errors="replace")
        super().__init__(f"{where} failed ({code}): {msg}")
        self.code = code


def _check(code: int, where: str):
    if code != GMC_OK:
        raise GmcError(code, where)


# --- C-ABI entry points under their own names ------------------------------
def gmc_config_default() -> GmcConfig:
    cfg = GmcConfig()
    lib().gmc_config_default(ctypes.byref(cfg))
    return cfg


def gmc_init(cfg: GmcConfig) -> int:
    return lib().gmc_init(ctypes.byref(cfg))


def gmc_set_stream(stream: int) -> int:
    return lib().gmc_set_stream(_vp(stream))


def gmc_prune(hidden, text_q, vis_k, pos3d, n, t, k, out_hidden, out_pos, out_idx) -> int:
    return lib().gmc_prune(hidden, text_q, vis_k, pos3d, n, t, k, out_hidden, out_pos, out_idx)


def gmc_prune_ex(b, hidden, text_q, vis_k, pos3d, n, t, k, out_hidden, out_pos, out_idx,
                 nonvis_lse=None, trace: Optional[GmcTrace] = None) -> int:
    tr = ctypes.byref(trace) if trace is not None else None
    return lib().gmc_prune_ex(b, hidden, text_q, vis_k, pos3d, n, t, k, out_hidden, out_pos,
                              out_idx, nonvis_lse, tr)


def gmc_prune_views(b, hidden, text_q, vis_k, pos3d, n, t, k, out_hidden, out_pos, out_idx, nonvis_lse,
                    hist_views, trace: Optional[GmcTrace] = None) -> int:
    """hist_views: a sequence of GmcView."""
    nh = len(hist_views)
    arr = (GmcView * max(nh, 1))(*hist_views)
    tr = ctypes.byref(trace) if trace is not None else None
    return lib().gmc_prune_views(b, hidden, text_q, vis_k, pos3d, n, t, k, out_hidden, out_pos, out_idx,
                                 nonvis_lse, nh, arr, tr)


def gmc_prune_full(b, hidden, text_q, vis_k, pos3d, image_id, n_images, n, t, k, out_hidden, out_pos, out_idx,
                   nonvis_lse=None, hist_views=(), trace: Optional[GmcTrace] = None) -> int:
    nh = len(hist_views)
    arr = (GmcView * max(nh, 1))(*hist_views)
    tr = ctypes.byref(trace) if trace is not None else None
    return lib().gmc_prune_full(b, hidden, text_q, vis_k, pos3d, image_id, n_images, n, t, k, out_hidden,
                                out_pos, out_idx, nonvis_lse, nh, arr, tr)


def gmc_audit_message(b, n, t, k, text_q, vis_k, vis_v, comp_k, comp_v, carrier, weights, nonvis_lse, rows_out,
                      vec_out, out) -> int:
    return lib().gmc_audit_message(b, n, t, k, text_q, vis_k, vis_v, comp_k, comp_v, carrier, weights, nonvis_lse,
                                   rows_out, vec_out, out)


def gmc_realized_budget(n: int, k_req: int, n_images: int) -> int:
    return int(lib().gmc_realized_budget(n, k_req, n_images))


def gmc_trace_dims_full(n: int, t: int, k: int, n_hist: int, n_images: int):
    vals = [_i64() for _ in range(4)]
    code = lib().gmc_trace_dims_full(n, t, k, n_hist, n_images, *[ctypes.byref(v) for v in vals])
    _check(code, "gmc_trace_dims_full")
    return tuple(int(v.value) for v in vals)


def gmc_realized_k(n: int, k_req: int) -> int:
    return int(lib().gmc_realized_k(n, k_req))


def gmc_trace_dims(n: int, t: int, k: int):
    vals = [_i64() for _ in range(4)]
    code = lib().gmc_trace_dims(n, t, k, *[ctypes.byref(v) for v in vals])
    _check(code, "gmc_trace_dims")
    return tuple(int(v.value) for v in vals)


def gmc_compact_sequence(b, seq_len, vis_start, n, k, out_idx, iota, keep, seq_rows, vis_rows, out_rows,
                         row_bytes, seq_pos, out_pos) -> int:
    return lib().gmc_compact_sequence(b, seq_len, vis_start, n, k, out_idx, iota, keep, seq_rows, vis_rows,
                                      out_rows, row_bytes, seq_pos, out_pos)


def gmc_gather_rows(src_ptrs, dst_ptrs, n_seq, seqs_per_keep, seq_len, seq_len2, row_bytes, keep) -> int:
    n = len(src_ptrs)
    src = (_vp * max(n, 1))(*src_ptrs)
    dst = (_vp * max(len(dst_ptrs), 1))(*dst_ptrs)
    return lib().gmc_gather_rows(n, src, dst, n_seq, seqs_per_keep, seq_len, seq_len2, row_bytes, keep)


def check_prune_inputs(cfg: GmcConfig, dtype, hidden, text_q, vis_k, pos3d, nonvis_lse=None):
    """Shapes, dtypes and devices of a pruning call's tensors against the
    context's configuration (the library itself sees raw pointers only).
    Returns (B, N, T); raises ValueError."""
    import torch
    if hidden.dim() != 3 or hidden.shape[2] != cfg.d:
        raise ValueError(f"hidden must be [B][N][{cfg.d}], got {tuple(hidden.shape)}")
    b, n, _ = hidden.shape
    hd = cfg.n_q_heads * cfg.head_dim
    if text_q.dim() < 3 or text_q.shape[0] != b or int(np.prod(text_q.shape[2:])) != hd:
        raise ValueError(f"text_q must be [B][T][{cfg.n_q_heads}][{cfg.head_dim}] (or [B][T][Hq*dh]), "
                         f"got {tuple(text_q.shape)}")
    t = text_q.shape[1]
    if vis_k.dim() < 3 or vis_k.shape[0] != b or vis_k.shape[1] != n or \
            int(np.prod(vis_k.shape[2:])) != cfg.n_kv_heads * cfg.head_dim:
        raise ValueError(f"vis_k must be [B][N][{cfg.n_kv_heads}][{cfg.head_dim}] (or [B][N][Hkv*dh]), "
                         f"got {tuple(vis_k.shape)}")
    if tuple(pos3d.shape) != (b, n, 3) or pos3d.dtype != torch.int32:
        raise ValueError(f"pos3d must be int32 [B][N][3] = ({b}, {n}, 3), got {pos3d.dtype} {tuple(pos3d.shape)}")
    for name, x in (("hidden", hidden), ("text_q", text_q), ("vis_k", vis_k)):
        if x.dtype != dtype:
            raise ValueError(f"{name} has dtype {x.dtype}, the context computes in {dtype}")
    tensors = [("hidden", hidden), ("text_q", text_q), ("vis_k", vis_k), ("pos3d", pos3d)]
    if nonvis_lse is not None:
        if nonvis_lse.dtype != torch.float32 or tuple(nonvis_lse.shape) != (b, cfg.n_q_heads, t):
            raise ValueError(f"nonvis_lse must be float32 [B][Hq][T] = ({b}, {cfg.n_q_heads}, {t}), "
                             f"got {nonvis_lse.dtype} {tuple(nonvis_lse.shape)}")
        tensors.append(("nonvis_lse", nonvis_lse))
    for name, x in tensors:
        if not x.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    dev = hidden.device
    for name, x in tensors:
        if x.device.type != "cuda" or x.device != dev:
            raise ValueError(f"{name} must be on the GPU, on hidden's device; got {x.device}")
    return b, n, t


def check_gather_inputs(caches, keep, seqs_per_keep):
    """Every cache contiguous with the same [n_seq][L] leading shape and row
    bytes, on keep's device; keep int32 [n_seq / seqs_per_keep][L2].  Raises
    ValueError."""
    import torch
    if not caches:
        raise ValueError("gather_rows needs at least one cache")
    c0 = caches[0]
    if c0.dim() < 2:
        raise ValueError("caches must be [n_seq][L][...]")
    n_seq, seq_len = c0.shape[:2]
    row_bytes = (c0.numel() // max(n_seq * seq_len, 1)) * c0.element_size()
    for i, c in enumerate(caches):
        if c.dim() < 2 or tuple(c.shape[:2]) != (n_seq, seq_len):
            raise ValueError(f"cache {i} has leading shape {tuple(c.shape[:2])}, expected {(n_seq, seq_len)}")
        if (c.numel() // max(n_seq * seq_len, 1)) * c.element_size() != row_bytes:
            raise ValueError(f"cache {i} rows are not {row_bytes} bytes")
        if not c.is_contiguous():
            raise ValueError(f"cache {i} must be contiguous")
    if keep.dtype != torch.int32 or keep.dim() != 2 or not keep.is_contiguous():
        raise ValueError("keep must be a contiguous int32 [n_seq / seqs_per_keep][L2] tensor")
    if seqs_per_keep < 1 or keep.shape[0] * seqs_per_keep != n_seq:
        raise ValueError(f"keep has {keep.shape[0]} lists; {n_seq} sequences need {n_seq} / seqs_per_keep")
    for i, c in enumerate(caches):
        if c.device.type != "cuda" or c.device != keep.device:
            raise ValueError(f"cache {i} must be on the GPU, on keep's device; got {c.device}")
    return n_seq, seq_len, row_bytes


def check_compact_inputs(out_idx, n, seq_rows, vis_rows, seq_pos, seq_len):
    """out_idx int32 [B][K]; seq_rows [B][L][...] and vis_rows [B][K][...] of one
    dtype and row size; seq_pos int32 [B][L][3]; all on out_idx's device.
    Raises ValueError."""
    import torch
    if out_idx.dtype != torch.int32 or out_idx.dim() != 2 or not out_idx.is_contiguous():
        raise ValueError("out_idx must be a contiguous int32 [B][K] tensor")
    b, k = out_idx.shape
    if not 1 <= k <= n:
        raise ValueError(f"need 1 <= K <= N, got K={k}, N={n}")
    tensors = [("out_idx", out_idx)]
    if (seq_rows is None) != (vis_rows is None):
        raise ValueError("seq_rows and vis_rows must be given together")
    if seq_rows is not None:
        if seq_rows.shape[0] != b or seq_rows.shape[1] != seq_len or vis_rows.shape[0] != b or vis_rows.shape[1] != k:
            raise ValueError(f"seq_rows must be [B][L][...] and vis_rows [B][K][...] with B={b}, L={seq_len}, K={k}")
        if seq_rows.dtype != vis_rows.dtype or seq_rows[0, 0].numel() != vis_rows[0, 0].numel():
            raise ValueError("seq_rows and vis_rows must share dtype and row size")
        tensors += [("seq_rows", seq_rows), ("vis_rows", vis_rows)]
    if seq_pos is not None:
        if seq_pos.dtype != torch.int32 or tuple(seq_pos.shape) != (b, seq_len, 3):
            raise ValueError(f"seq_pos must be int32 [B][L][3] = ({b}, {seq_len}, 3)")
        tensors.append(("seq_pos", seq_pos))
    for name, x in tensors:
        if not x.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    for name, x in tensors:
        if x.device.type != "cuda" or x.device != out_idx.device:
            raise ValueError(f"{name} must be on the GPU, on out_idx's device; got {x.device}")


def compact_sequence(out_idx, vis_start, n, seq_rows=None, vis_rows=None, seq_pos=None, seq_len=None):
    """Tensor-level sequence compaction on torch's current stream (argument
    marshalling only): out_idx [B][K] int32 device; seq_rows [B][L][...] and
    vis_rows [B][K][...] of one dtype; seq_pos [B][L][3] int32.  Returns
    (iota [B][L], keep [B][L2], out_rows or None, out_pos or None)."""
    import torch
    b, k = out_idx.shape
    if seq_len is None:
        seq_len = seq_rows.shape[1] if seq_rows is not None else seq_pos.shape[1]
    check_compact_inputs(out_idx, n, seq_rows, vis_rows, seq_pos, seq_len)
    l2 = seq_len - n + k
    dev = out_idx.device
    iota = torch.empty((b, seq_len), dtype=torch.int32, device=dev)
    keep = torch.empty((b, l2), dtype=torch.int32, device=dev)
    out_rows = out_pos = None
    row_bytes = 0
    if seq_rows is not None:
        out_rows = torch.empty((b, l2) + tuple(seq_rows.shape[2:]), dtype=seq_rows.dtype, device=dev)
        row_bytes = seq_rows[0, 0].numel() * seq_rows.element_size()
    if seq_pos is not None:
        out_pos = torch.empty((b, l2, 3), dtype=torch.int32, device=dev)
    _check(gmc_set_stream(torch.cuda.current_stream(dev).cuda_stream), "gmc_set_stream")
    ptr = (lambda t: None if t is None else t.data_ptr())
    _check(gmc_compact_sequence(b, seq_len, vis_start, n, k, out_idx.data_ptr(), iota.data_ptr(), keep.data_ptr(),
                                ptr(seq_rows), ptr(vis_rows), ptr(out_rows), row_bytes, ptr(seq_pos), ptr(out_pos)),
           "gmc_compact_sequence")
    return iota, keep, out_rows, out_pos


def gather_rows(caches, keep, seqs_per_keep=1):
    """Tensor-level row gather on torch's current stream: each cache is
    [n_seq][L][...] (contiguous), keep [n_seq / seqs_per_keep][L2] int32;
    returns the gathered [n_seq][L2][...] caches."""
    import torch
    n_seq, seq_len, row_bytes = check_gather_inputs(caches, keep, seqs_per_keep)
    l2 = keep.shape[1]
    outs = [torch.empty((n_seq, l2) + tuple(c.shape[2:]), dtype=c.dtype, device=c.device) for c in caches]
    _check(gmc_set_stream(torch.cuda.current_stream(caches[0].device).cuda_stream), "gmc_set_stream")
    for i in range(0, len(caches), GMC_MAX_GATHER_TENSORS):
        part = slice(i, i + GMC_MAX_GATHER_TENSORS)
        _check(gmc_gather_rows([c.data_ptr() for c in caches[part]], [o.data_ptr() for o in outs[part]], n_seq,
                               seqs_per_keep, seq_len, l2, row_bytes, keep.data_ptr()), "gmc_gather_rows")
    return outs


def gmc_set_diag(flags: int) -> int:
    return lib().gmc_set_diag(flags)


def gmc_get_diag(problem: int = 0, max_rounds: int = GMC_CERT_MAX_ROUNDS):
    """Diagnostics of the last pruning call for one problem (synchronises).
    Returns (code, dict); the per-round arrays hold `rounds` entries."""
    arrs = {k: (_f32 * max(max_rounds, 1))() for k in ("u_top", "gain", "q", "pool_margin", "batch_margin")}
    d = GmcDiag()
    d.max_rounds = max_rounds
    for k, a in arrs.items():
        setattr(d, k, ctypes.cast(a, ctypes.POINTER(_f32)))
    code = lib().gmc_get_diag(problem, ctypes.byref(d))
    out = {k: getattr(d, k) for k in ("status", "identity", "has_certificate", "k", "rounds", "m_rows",
                                       "n_discarded", "s_x", "dbar", "f_s", "f_v", "c_b")}
    out["f_bank_s"] = list(d.f_bank_s)
    out["f_bank_v"] = list(d.f_bank_v)
    nr = min(d.rounds, max_rounds) if d.has_certificate else 0
    for k, a in arrs.items():
        out[k] = [a[i] for i in range(nr)]
    return code, out


def gmc_prune_static(cfg: GmcConfig, b, hidden, text_q, vis_k, pos3d, n, t, k, out_hidden, out_pos, out_idx,
                     nonvis_lse=None, stream=None) -> int:
    return lib().gmc_prune_static(ctypes.byref(cfg), b, hidden, text_q, vis_k, pos3d, n, t, k, out_hidden,
                                  out_pos, out_idx, nonvis_lse, stream)


def gmc_workspace_bytes() -> int:
    return int(lib().gmc_workspace_bytes())


def gmc_last_error() -> str:
    return lib().gmc_last_error().decode(errors="replace")


def gmc_free() -> None:
    lib().gmc_free()


# --- tensor-level wrapper ----------------------------------------------------
class Pruner:
    """Owns one library context for a model shape and capacity.

    ``probe`` [Hq][r][d] and ``app_projection`` [app_rank][d] are device
    tensors in the operator dtype, ``probe_bias`` [Hq][r] an optional fp32
    device tensor; the wrapper keeps them alive.  ``prune``
    allocates outputs with torch and calls gmc_prune_ex on torch's current
    stream.
    """

    def __init__(self, *, d, n_q_heads, n_kv_heads, head_dim, probe, dtype, max_batch, max_n,
                 max_t, max_k=0, app_projection=None, probe_bias=None, probe_hist=None, **overrides):
        import torch
        self.torch = torch
        cfg = gmc_config_default()
        cfg.d, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim = d, n_q_heads, n_kv_heads, head_dim
        cfg.probe_rank = probe.shape[1]
        cfg.dtype = GMC_BF16 if dtype == torch.bfloat16 else GMC_F32
        cfg.max_batch, cfg.max_n, cfg.max_t, cfg.max_k = max_batch, max_n, max_t, max_k
        for key, val in overrides.items():
            setattr(cfg, key, val)
        self.probe = probe.contiguous()
        self.app_projection = None if app_projection is None else app_projection.contiguous()
        cfg.value_probe = self.probe.data_ptr()
        cfg.app_projection = 0 if self.app_projection is None else self.app_projection.data_ptr()
        self.probe_bias = None if probe_bias is None else probe_bias.contiguous()
        if self.probe_bias is not None and (self.probe_bias.dtype != torch.float32 or
                                            tuple(self.probe_bias.shape) != (n_q_heads, cfg.probe_rank)):
            raise ValueError("probe_bias must be a float32 [n_q_heads][probe_rank] tensor")
        cfg.value_probe_bias = 0 if self.probe_bias is None else self.probe_bias.data_ptr()
        # probes of the historical message views [n_hist][Hq][r][d]
        self.probe_hist = None if probe_hist is None else probe_hist.contiguous()
        if self.probe_hist is not None:
            if self.probe_hist.dim() != 4 or tuple(self.probe_hist.shape[1:]) != tuple(self.probe.shape) or \
                    self.probe_hist.dtype != self.probe.dtype:
                raise ValueError("probe_hist must be [n_hist] x the probe's shape and dtype")
            cfg.max_hist_views = self.probe_hist.shape[0]
            cfg.value_probe_hist = self.probe_hist.data_ptr()
        self.cfg = cfg
        self.dtype = dtype
        _check(gmc_init(cfg), "gmc_init")

    def trace_dims(self, n, t, k):
        return gmc_trace_dims(n, t, k)

    def prune(self, hidden, text_q, vis_k, pos3d, k, nonvis_lse=None, trace: bool = False, hist=None,
              image_id=None, n_images: int = 1):
        """hist: optional list of historical views, each (hidden, text_q,
        vis_k[, nonvis_lse]) shaped like the current view's tensors;
        image_id: optional int32 [B][N] device tensor of image ids in
        [0, n_images) for a multi-image prompt."""
        torch = self.torch
        b, n, t = check_prune_inputs(self.cfg, self.dtype, hidden, text_q, vis_k, pos3d, nonvis_lse)
        hist = list(hist or [])
        views = []
        for i, hv in enumerate(hist):
            hv = tuple(hv) + (None,) * (4 - len(hv))
            try:
                check_prune_inputs(self.cfg, self.dtype, hv[0], hv[1], hv[2], pos3d, hv[3])
                if hv[0].shape != hidden.shape or hv[1].shape != text_q.shape:
                    raise ValueError("shapes differ from the current view's")
                if hv[0].device != hidden.device:
                    raise ValueError("not on hidden's device")
            except ValueError as e:
                raise ValueError(f"historical view {i}: {e}") from None
            views.append(GmcView(hv[0].data_ptr(), hv[1].data_ptr(), hv[2].data_ptr(),
                                 None if hv[3] is None else hv[3].data_ptr()))
        if image_id is not None:
            if image_id.dtype != torch.int32 or tuple(image_id.shape) != (b, n) or not image_id.is_contiguous() \
                    or image_id.device != hidden.device:
                raise ValueError(f"image_id must be a contiguous int32 [B][N] = ({b}, {n}) tensor on hidden's device")
        multi = image_id is not None and n_images > 1
        d = hidden.shape[2]
        kk = gmc_realized_budget(n, k, n_images if image_id is not None else 1)
        dev = hidden.device
        out_h = torch.empty((b, kk, d), dtype=hidden.dtype, device=dev)
        out_p = torch.empty((b, kk, 3), dtype=torch.int32, device=dev)
        out_i = torch.empty((b, kk), dtype=torch.int32, device=dev)
        tr, bufs = None, {}
        if trace:
            rounds, pool_cap, bcap, m_rows = gmc_trace_dims_full(n, t, k, len(views),
                                                                 n_images if multi else 1)
            hq = self.cfg.n_q_heads
            r1 = max(rounds, 1)
            bufs = dict(
                round_pool=torch.full((b, r1, pool_cap), -1, dtype=torch.int32, device=dev),
                round_batch=torch.full((b, r1, bcap), -1, dtype=torch.int32, device=dev),
                assign=torch.full((b, n), -1, dtype=torch.int32, device=dev),
                omega=torch.zeros((b, hq), dtype=torch.float32, device=dev),
                ebar=torch.zeros((b, n), dtype=torch.float32, device=dev),
                client=torch.zeros((b, m_rows, n), dtype=torch.float32, device=dev),
                stats=torch.zeros((b, GMC_STATS), dtype=torch.float32, device=dev),
                round_gains=torch.full((b, r1, n), -1.0, dtype=torch.float32, device=dev),
                round_scores=torch.full((b, r1, pool_cap), -1.0, dtype=torch.float32, device=dev))
            tr = GmcTrace(**{key: v.data_ptr() for key, v in bufs.items()})
        _check(gmc_set_stream(torch.cuda.current_stream(dev).cuda_stream), "gmc_set_stream")
        nv = None if nonvis_lse is None else nonvis_lse.data_ptr()
        if multi:
            code = gmc_prune_full(b, hidden.data_ptr(), text_q.data_ptr() if t > 0 else None,
                                  vis_k.data_ptr(), pos3d.data_ptr(), image_id.data_ptr(), n_images, n, t, k,
                                  out_h.data_ptr(), out_p.data_ptr(), out_i.data_ptr(), nv, views, tr)
            _check(code, "gmc_prune_full")
        elif views:
            code = gmc_prune_views(b, hidden.data_ptr(), text_q.data_ptr() if t > 0 else None,
                                   vis_k.data_ptr(), pos3d.data_ptr(), n, t, k, out_h.data_ptr(),
                                   out_p.data_ptr(), out_i.data_ptr(), nv, views, tr)
            _check(code, "gmc_prune_views")
        else:
            code = gmc_prune_ex(b, hidden.data_ptr(), text_q.data_ptr() if t > 0 else None,
                                vis_k.data_ptr(), pos3d.data_ptr(), n, t, k, out_h.data_ptr(),
                                out_p.data_ptr(), out_i.data_ptr(), nv, tr)
            _check(code, "gmc_prune_ex")
        if trace:
            return out_h, out_p, out_i, bufs
        return out_h, out_p, out_i

    def audit(self, text_q, vis_k, vis_v, comp_k, comp_v, carrier, weights=None, nonvis_lse=None,
              rows: bool = False, vectors: bool = False):
        """gmc_audit_message on torch's current stream: text_q [B][T][Hq][dh],
        vis_k / vis_v [B][N][Hkv][dh], comp_k / comp_v [B][K][Hkv][dh] in the
        context dtype, carrier [B][N] int32 slots, weights / nonvis_lse
        [B][Hq][T] fp32 or None.  Returns (out [B][8], rows [B][Hq][T][8] or
        None, vectors [B][Hq][T][4][dh] or None)."""
        torch = self.torch
        cfg = self.cfg
        b, t = text_q.shape[:2]
        n, k = vis_k.shape[1], comp_k.shape[1]
        hd = (cfg.n_kv_heads, cfg.head_dim)
        for name, x, lead in (("vis_k", vis_k, (b, n)), ("vis_v", vis_v, (b, n)), ("comp_k", comp_k, (b, k)),
                              ("comp_v", comp_v, (b, k))):
            if tuple(x.shape) != lead + hd or x.dtype != self.dtype or not x.is_contiguous():
                raise ValueError(f"{name} must be a contiguous {self.dtype} {lead + hd} tensor")
        if tuple(text_q.shape) != (b, t, cfg.n_q_heads, cfg.head_dim) or text_q.dtype != self.dtype:
            raise ValueError("text_q must be [B][T][Hq][dh] in the context dtype")
        if tuple(carrier.shape) != (b, n) or carrier.dtype != torch.int32 or not carrier.is_contiguous():
            raise ValueError("carrier must be a contiguous int32 [B][N] tensor")
        for name, x in (("weights", weights), ("nonvis_lse", nonvis_lse)):
            if x is not None and (tuple(x.shape) != (b, cfg.n_q_heads, t) or x.dtype != torch.float32):
                raise ValueError(f"{name} must be float32 [B][Hq][T]")
        dev = text_q.device
        out = torch.zeros((b, GMC_AUDIT_OUT), dtype=torch.float32, device=dev)
        ro = torch.zeros((b, cfg.n_q_heads, t, GMC_AUDIT_ROW), dtype=torch.float32, device=dev) if rows else None
        vo = torch.zeros((b, cfg.n_q_heads, t, 4, cfg.head_dim), dtype=torch.float32, device=dev) if vectors else None
        _check(gmc_set_stream(torch.cuda.current_stream(dev).cuda_stream), "gmc_set_stream")
        ptr = (lambda x: None if x is None else x.contiguous().data_ptr())
        _check(gmc_audit_message(b, n, t, k, text_q.data_ptr(), vis_k.data_ptr(), vis_v.data_ptr(), comp_k.data_ptr(),
                                 comp_v.data_ptr(), carrier.data_ptr(), ptr(weights), ptr(nonvis_lse), ptr(ro),
                                 ptr(vo), out.data_ptr()), "gmc_audit_message")
        return out, ro, vo

    def set_diag(self, flags: int):
        _check(gmc_set_diag(flags), "gmc_set_diag")

    def diag(self, problem: int = 0):
        """(code, dict) of gmc_get_diag for the last call (synchronises)."""
        return gmc_get_diag(problem)

    def close(self):
        gmc_free()


def gmc_timing_enable(enable: bool) -> int:
    return lib().gmc_timing_enable(1 if enable else 0)


def gmc_timing_read():
    """Per-stage (total ms, span count) since the last read (syncs the stream)."""
    n = GMC_TIMERS
    ms = (ctypes.c_double * n)()
    cnt = (_i64 * n)()
    _check(lib().gmc_timing_read(ms, cnt, n), "gmc_timing_read")
    return list(ms), list(cnt)


GMC_TIMERS = 13
STAGE_NAMES = ["probe", "logits", "heads", "appearance", "spatial", "cov", "gains", "resp",
               "objective", "assign", "transport", "init", "select"]
SIGNATURES["gmc_timing_enable"] = (ctypes.c_int, [ctypes.c_int])
SIGNATURES["gmc_timing_read"] = (ctypes.c_int, [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_i64),
                                                ctypes.c_int32])


# --- host <-> device marshalling of seeded workloads --------------------------
def to_device(a, dtype: str, torch):
    """A float32 numpy array holding exact values of `dtype` ("f32" or
    "bf16") as a contiguous device tensor of that dtype."""
    from . import synth
    if dtype == "bf16":
        bits = synth.bf16_bits(a).view(np.int16)
        return torch.from_numpy(np.ascontiguousarray(bits)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def from_device(t, torch) -> np.ndarray:
    return t.float().cpu().numpy() if t.dtype == torch.bfloat16 else t.cpu().numpy()


def make_pruner(prob, torch, max_k=0, probe_bias=None, hist=None, **overrides) -> Pruner:
    """A Pruner sized for a seeded workload (synth.Problem): its shape, dtype,
    batch and token capacity, probe and bounded-bank projection, and the
    probes of its historical views (synth.HistView list) when given."""
    w = prob.workload
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    probe = to_device(prob.probe, w.dtype, torch)
    proj = None if prob.app_proj is None else to_device(prob.app_proj, w.dtype, torch)
    bias = None if probe_bias is None else torch.from_numpy(np.ascontiguousarray(probe_bias, np.float32)).cuda()
    ph = None if not hist else to_device(np.stack([v.probe for v in hist]), w.dtype, torch)
    return Pruner(d=w.d, n_q_heads=w.hq, n_kv_heads=w.hkv, head_dim=w.dh, probe=probe, dtype=tdt,
                  max_batch=w.batch, max_n=w.n, max_t=max(w.t, 1), max_k=max_k, app_projection=proj,
                  probe_bias=bias, probe_hist=ph, **overrides)
