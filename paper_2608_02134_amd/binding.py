"""ctypes binding of libgmc.so: the C-ABI entry points under the same names,
plus a thin tensor-level wrapper (argument marshalling only).

Every step of the operator runs inside the HIP library.  If the library has
not been built, ``lib()`` raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libgmc.so")

GMC_OK, GMC_ERR_ARG, GMC_ERR_CAPACITY, GMC_ERR_STATE, GMC_ERR_HIP = 0, -1, -2, -3, -4
GMC_F32, GMC_BF16 = 0, 1
GMC_STATS = 15
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
    ]


class GmcTrace(ctypes.Structure):
    """Mirror of ``gmc_trace``: optional device output pointers."""
    _fields_ = [("round_pool", _vp), ("round_batch", _vp), ("assign", _vp), ("omega", _vp),
                ("ebar", _vp), ("client", _vp), ("stats", _vp)]


# name -> (restype, argtypes) of every symbol include/gmc.h declares
SIGNATURES = {
    "gmc_config_default": (None, [ctypes.POINTER(GmcConfig)]),
    "gmc_init": (ctypes.c_int, [ctypes.POINTER(GmcConfig)]),
    "gmc_set_stream": (ctypes.c_int, [_vp]),
    "gmc_prune": (ctypes.c_int, [_vp, _vp, _vp, _vp, _i64, _i64, _i64, _vp, _vp, _vp]),
    "gmc_prune_ex": (ctypes.c_int, [_i64, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _vp, _vp, _vp, _vp,
                                    ctypes.POINTER(GmcTrace)]),
    "gmc_realized_k": (_i64, [_i64, _i64]),
    "gmc_trace_dims": (ctypes.c_int, [_i64, _i64, _i64, ctypes.POINTER(_i64), ctypes.POINTER(_i64),
                                      ctypes.POINTER(_i64), ctypes.POINTER(_i64)]),
    "gmc_compact_sequence": (ctypes.c_int, [_i64, _i64, _i64, _i64, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _i64,
                                            _vp, _vp]),
    "gmc_gather_rows": (ctypes.c_int, [_i64, ctypes.POINTER(_vp), ctypes.POINTER(_vp), _i64, _i64, _i64, _i64,
                                       _i64, _vp]),
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


def compact_sequence(out_idx, vis_start, n, seq_rows=None, vis_rows=None, seq_pos=None, seq_len=None):
    """Tensor-level sequence compaction on torch's current stream (argument
    marshalling only): out_idx [B][K] int32 device; seq_rows [B][L][...] and
    vis_rows [B][K][...] of one dtype; seq_pos [B][L][3] int32.  Returns
    (iota [B][L], keep [B][L2], out_rows or None, out_pos or None)."""
    import torch
    b, k = out_idx.shape
    if seq_len is None:
        seq_len = seq_rows.shape[1] if seq_rows is not None else seq_pos.shape[1]
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
    n_seq, seq_len = caches[0].shape[:2]
    l2 = keep.shape[1]
    outs = [torch.empty((n_seq, l2) + tuple(c.shape[2:]), dtype=c.dtype, device=c.device) for c in caches]
    row_bytes = caches[0][0, 0].numel() * caches[0].element_size()
    _check(gmc_set_stream(torch.cuda.current_stream(caches[0].device).cuda_stream), "gmc_set_stream")
    for i in range(0, len(caches), GMC_MAX_GATHER_TENSORS):
        part = slice(i, i + GMC_MAX_GATHER_TENSORS)
        _check(gmc_gather_rows([c.data_ptr() for c in caches[part]], [o.data_ptr() for o in outs[part]], n_seq,
                               seqs_per_keep, seq_len, l2, row_bytes, keep.data_ptr()), "gmc_gather_rows")
    return outs


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
                 max_t, max_k=0, app_projection=None, probe_bias=None, **overrides):
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
        self.cfg = cfg
        self.dtype = dtype
        _check(gmc_init(cfg), "gmc_init")

    def trace_dims(self, n, t, k):
        return gmc_trace_dims(n, t, k)

    def prune(self, hidden, text_q, vis_k, pos3d, k, nonvis_lse=None, trace: bool = False):
        torch = self.torch
        b, n, d = hidden.shape
        t = text_q.shape[1]
        for x in (hidden, text_q, vis_k, pos3d):
            if not x.is_contiguous():
                raise ValueError("inputs must be contiguous")
        kk = gmc_realized_k(n, k)
        dev = hidden.device
        out_h = torch.empty((b, kk, d), dtype=hidden.dtype, device=dev)
        out_p = torch.empty((b, kk, 3), dtype=torch.int32, device=dev)
        out_i = torch.empty((b, kk), dtype=torch.int32, device=dev)
        tr, bufs = None, {}
        if trace:
            rounds, pool_cap, bcap, m_rows = gmc_trace_dims(n, t, k)
            hq = self.cfg.n_q_heads
            bufs = dict(
                round_pool=torch.full((b, max(rounds, 1), pool_cap), -1, dtype=torch.int32, device=dev),
                round_batch=torch.full((b, max(rounds, 1), bcap), -1, dtype=torch.int32, device=dev),
                assign=torch.full((b, n), -1, dtype=torch.int32, device=dev),
                omega=torch.zeros((b, hq), dtype=torch.float32, device=dev),
                ebar=torch.zeros((b, n), dtype=torch.float32, device=dev),
                client=torch.zeros((b, m_rows, n), dtype=torch.float32, device=dev),
                stats=torch.zeros((b, GMC_STATS), dtype=torch.float32, device=dev))
            tr = GmcTrace(**{key: v.data_ptr() for key, v in bufs.items()})
        _check(gmc_set_stream(torch.cuda.current_stream(dev).cuda_stream), "gmc_set_stream")
        nv = None if nonvis_lse is None else nonvis_lse.contiguous().data_ptr()
        code = gmc_prune_ex(b, hidden.data_ptr(), text_q.data_ptr() if t > 0 else None,
                            vis_k.data_ptr(), pos3d.data_ptr(), n, t, k, out_h.data_ptr(),
                            out_p.data_ptr(), out_i.data_ptr(), nv, tr)
        _check(code, "gmc_prune_ex")
        if trace:
            return out_h, out_p, out_i, bufs
        return out_h, out_p, out_i

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
