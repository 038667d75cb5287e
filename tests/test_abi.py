"""C-ABI contract on the CPU: the built library loads, exports every entry
point include/gmc.h declares, the ctypes config mirrors the C layout, and
host-side validation rejects bad arguments before touching a device."""
import ctypes
import os
import re

import pytest

from paper_2608_02134_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gmc.h")


def _declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(gmc_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        pytest.fail("libgmc.so is not built; run __graft_entry__.build()")
    return B.lib()


def test_every_declared_symbol_is_exported(lib):
    names = _declared_functions()
    assert len(names) >= 12
    for name in names:
        assert hasattr(lib, name), name
        assert name in B.SIGNATURES, f"binding lacks {name}"


def test_config_layout_round_trips_defaults(lib):
    c = B.gmc_config_default()
    assert c.probe_rank == 4 and c.dtype == B.GMC_BF16 and c.max_batch == 1
    assert c.tau_v == pytest.approx(0.2) and c.tau_s == pytest.approx(0.02)
    assert c.beta_app == pytest.approx(0.5) and c.beta_spa == pytest.approx(0.25)
    assert c.batch_b == 16 and c.pool_mult == 4 and c.tau_r == pytest.approx(0.1)
    assert c.gate_t == pytest.approx(0.08) and c.gate_p == pytest.approx(8.0)
    assert c.amb_margin == pytest.approx(0.05) and c.pop_strength == pytest.approx(0.5)
    assert c.max_head_clusters == 4 and c.disp_eps == pytest.approx(0.05)
    assert c.terminal_q_weight == pytest.approx(2.0)
    assert c.bounded_threshold_n == 4096 and c.app_rank == 128
    assert c.app_max_clients == 4096 and c.batch_b_bounded == 512  # last field: layout intact
    assert c.value_probe is None and c.app_projection is None
    assert c.value_probe_bias is None   # appended last: optional, zero by default


def test_header_constants_match_binding():
    src = open(HEADER).read()
    consts = dict((k, int(v)) for k, v in re.findall(r"#define\s+(GMC_[A-Z0-9_]+)\s+\(?(-?\d+)\)?", src))
    assert consts["GMC_STATS"] == B.GMC_STATS
    assert (consts["GMC_OK"], consts["GMC_ERR_ARG"], consts["GMC_ERR_CAPACITY"], consts["GMC_ERR_STATE"],
            consts["GMC_ERR_HIP"]) == (B.GMC_OK, B.GMC_ERR_ARG, B.GMC_ERR_CAPACITY, B.GMC_ERR_STATE, B.GMC_ERR_HIP)
    assert (consts["GMC_F32"], consts["GMC_BF16"]) == (B.GMC_F32, B.GMC_BF16)
    assert consts["GMC_MAX_GATHER_TENSORS"] == B.GMC_MAX_GATHER_TENSORS


@pytest.mark.parametrize("n,k,want", [(10, 20, 10), (10, 0, 1), (10, -4, 1), (10, 3, 3), (0, 5, 0)])
def test_realized_budget(lib, n, k, want):
    assert B.gmc_realized_k(n, k) == want


def _valid_cfg():
    c = B.gmc_config_default()
    c.d, c.n_q_heads, c.n_kv_heads, c.head_dim = 512, 8, 2, 64
    c.max_n, c.max_t, c.dtype = 256, 16, B.GMC_F32
    c.value_probe = 0x1000
    return c


@pytest.mark.parametrize("field,value", [
    ("d", 0), ("d", 100), ("d", 96), ("n_q_heads", 0), ("n_q_heads", 33), ("n_kv_heads", 3),
    ("head_dim", 48), ("head_dim", 512), ("probe_rank", 0), ("probe_rank", 9), ("dtype", 7),
    ("max_batch", 0), ("max_n", 0), ("max_n", 40000), ("max_t", -1), ("max_k", 300),
    ("value_probe", None), ("tau_v", 0.0), ("g_form", 3), ("batch_b", 0), ("landmarks", 0),
])
def test_init_rejects_bad_config(lib, field, value):
    c = _valid_cfg()
    setattr(c, field, value)
    assert B.gmc_init(c) == B.GMC_ERR_ARG
    assert B.gmc_last_error()


def test_bounded_capacity_needs_projection(lib):
    c = _valid_cfg()
    c.max_n = 5000
    assert B.gmc_init(c) == B.GMC_ERR_ARG
    assert "app_projection" in B.gmc_last_error()


def test_null_config(lib):
    assert lib.gmc_init(None) == B.GMC_ERR_ARG


def test_calls_without_context(lib):
    B.gmc_free()
    B.gmc_free()                                   # idempotent
    assert lib.gmc_prune(None, None, None, None, 4, 1, 1, None, None, None) == B.GMC_ERR_STATE
    assert lib.gmc_prune_ex(1, None, None, None, None, 4, 1, 1, None, None, None, None, None) == B.GMC_ERR_STATE
    assert B.gmc_set_stream(0) == B.GMC_ERR_STATE
    assert lib.gmc_timing_enable(1) == B.GMC_ERR_STATE
    assert B.gmc_workspace_bytes() == 0
    with pytest.raises(B.GmcError):
        B.gmc_trace_dims(10, 1, 2)
    assert B.gmc_compact_sequence(1, 10, 2, 4, 2, 0x1000, None, None, None, None, None, 0, None,
                                  None) == B.GMC_ERR_STATE
    assert B.gmc_gather_rows([0x1000], [0x2000], 1, 1, 10, 8, 16, 0x3000) == B.GMC_ERR_STATE


def test_init_without_device_reports_hip_error(lib):
    try:
        import torch
        has_gpu = torch.cuda.is_available()
    except Exception:  # pragma: no cover
        has_gpu = False
    if has_gpu:
        pytest.skip("a device is present")
    assert B.gmc_init(_valid_cfg()) == B.GMC_ERR_HIP
    assert "device" in B.gmc_last_error()


def test_header_is_plain_c(tmp_path):
    # the boundary header must stay a C header (no C++ or HIP types)
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "use.c"
    src.write_text('#include "gmc.h"\nint main(void) { gmc_config c; gmc_trace t; gmc_config_default(&c);\n'
                   '  (void)t; return gmc_realized_k(4, 2) == 2 ? 0 : 1; }\n')
    r = subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror", "-fsyntax-only",
                        "-I", os.path.dirname(HEADER), str(src)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_new_header_constants_match_binding():
    src = open(HEADER).read()
    consts = dict((k, int(v)) for k, v in re.findall(r"#define\s+(GMC_[A-Z0-9_]+)\s+\(?(-?\d+)u?\)?", src))
    assert (consts["GMC_ERR_DEVICE"], consts["GMC_ERR_NONFINITE"]) == (B.GMC_ERR_DEVICE, B.GMC_ERR_NONFINITE)
    assert (consts["GMC_STATUS_SELECT_TIMEOUT"], consts["GMC_STATUS_BANK_TIMEOUT"],
            consts["GMC_STATUS_NONFINITE"]) == (B.GMC_STATUS_SELECT_TIMEOUT, B.GMC_STATUS_BANK_TIMEOUT,
                                                B.GMC_STATUS_NONFINITE)
    assert (consts["GMC_DIAG_CERT"], consts["GMC_DIAG_FINITE"]) == (B.GMC_DIAG_CERT, B.GMC_DIAG_FINITE)
    assert consts["GMC_CERT_MAX_ROUNDS"] == B.GMC_CERT_MAX_ROUNDS
    for name in ("GMC_STATUS_INPUT", "GMC_MAX_HIST_VIEWS", "GMC_MAX_IMAGES", "GMC_AUDIT_ROW", "GMC_AUDIT_OUT"):
        assert consts[name] == getattr(B, name), name


def test_struct_layouts_match_the_c_compiler(tmp_path):
    # sizes and field offsets of every struct the binding mirrors, as the C
    # compiler lays them out
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    structs = {"gmc_config": B.GmcConfig, "gmc_trace": B.GmcTrace, "gmc_diag": B.GmcDiag}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "gmc.h"', 'int main(void) {']
    for cname, py in structs.items():
        lines.append(f'  printf("{cname} size %zu\\n", sizeof({cname}));')
        for fname, _ in py._fields_:
            lines.append(f'  printf("{cname} {fname} %zu\\n", offsetof({cname}, {fname}));')
    lines += ['  return 0;', '}']
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    r = subprocess.run([cc, "-std=c99", "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split("\n")
    got = {}
    for ln in out:
        if ln:
            a, b, c = ln.split()
            got[(a, b)] = int(c)
    for cname, py in structs.items():
        assert got[(cname, "size")] == ctypes.sizeof(py), cname
        for fname, _ in py._fields_:
            assert got[(cname, fname)] == getattr(py, fname).offset, (cname, fname)


def test_diag_entry_points_without_context(lib):
    B.gmc_free()
    assert B.gmc_set_diag(B.GMC_DIAG_CERT) == B.GMC_ERR_STATE
    code, _ = B.gmc_get_diag(0)
    assert code == B.GMC_ERR_STATE
    assert B.gmc_audit_message(1, 8, 2, 4, *([None] * 11)) == B.GMC_ERR_STATE


def _cpu_cfg():
    c = B.gmc_config_default()
    c.d, c.n_q_heads, c.n_kv_heads, c.head_dim = 64, 4, 2, 32
    return c


def test_wrapper_rejects_mismatched_inputs():
    torch = pytest.importorskip("torch")
    cfg = _cpu_cfg()
    f32 = torch.float32
    h = torch.zeros((2, 10, 64))
    q = torch.zeros((2, 3, 4, 32))
    k = torch.zeros((2, 10, 2, 32))
    pos = torch.zeros((2, 10, 3), dtype=torch.int32)
    bad = [
        (torch.zeros((2, 10, 32)), q, k, pos, None, "hidden"),
        (h, torch.zeros((2, 3, 4, 16)), k, pos, None, "text_q"),
        (h, torch.zeros((1, 3, 4, 32)), k, pos, None, "text_q"),
        (h, q, torch.zeros((2, 10, 4, 32)), pos, None, "vis_k"),
        (h, q, torch.zeros((2, 9, 2, 32)), pos, None, "vis_k"),
        (h, q, k, pos.to(torch.int64), None, "pos3d"),
        (h, q, k, torch.zeros((2, 10, 2), dtype=torch.int32), None, "pos3d"),
        (h.to(torch.bfloat16), q, k, pos, None, "dtype"),
        (h, q, k, pos, torch.zeros((2, 4, 2)), "nonvis_lse"),
        (h, q, k, pos, torch.zeros((2, 4, 3), dtype=torch.float64), "nonvis_lse"),
        (h.transpose(0, 1).contiguous().transpose(0, 1), q, k, pos, None, "contiguous"),
        (h, q, k, pos, None, "GPU"),          # valid shapes, but host tensors
    ]
    for hh, qq, kk, pp, nv, what in bad:
        with pytest.raises(ValueError) as ei:
            B.check_prune_inputs(cfg, f32, hh, qq, kk, pp, nv)
        assert what in str(ei.value), (what, str(ei.value))


def test_gather_and_compact_wrappers_reject_mismatched_inputs():
    torch = pytest.importorskip("torch")
    c = torch.zeros((4, 10, 8), dtype=torch.bfloat16)
    keep = torch.zeros((4, 6), dtype=torch.int32)
    with pytest.raises(ValueError, match="leading shape"):
        B.check_gather_inputs([c, torch.zeros((4, 9, 8), dtype=torch.bfloat16)], keep, 1)
    with pytest.raises(ValueError, match="bytes"):
        B.check_gather_inputs([c, torch.zeros((4, 10, 8), dtype=torch.float32)], keep, 1)
    with pytest.raises(ValueError, match="int32"):
        B.check_gather_inputs([c], keep.to(torch.int64), 1)
    with pytest.raises(ValueError, match="sequences"):
        B.check_gather_inputs([c], keep, 2)
    with pytest.raises(ValueError, match="GPU"):
        B.check_gather_inputs([c], keep, 1)
    idx = torch.zeros((2, 3), dtype=torch.int32)
    rows = torch.zeros((2, 12, 8))
    vis = torch.zeros((2, 3, 8))
    pos = torch.zeros((2, 12, 3), dtype=torch.int32)
    with pytest.raises(ValueError, match="int32"):
        B.check_compact_inputs(idx.to(torch.int64), 5, rows, vis, pos, 12)
    with pytest.raises(ValueError, match="K <= N"):
        B.check_compact_inputs(idx, 2, rows, vis, pos, 12)
    with pytest.raises(ValueError, match="dtype and row size"):
        B.check_compact_inputs(idx, 5, rows, vis.to(torch.bfloat16), pos, 12)
    with pytest.raises(ValueError, match="seq_pos"):
        B.check_compact_inputs(idx, 5, rows, vis, pos[:, :11], 12)
    with pytest.raises(ValueError, match="GPU"):
        B.check_compact_inputs(idx, 5, rows, vis, pos, 12)
