"""The C-ABI library on a machine without a GPU: it loads, exports every
declared entry point, the binding's structs match the header's layout, and
argument errors are reported before any device work."""
import ctypes as C
import os
import re
import subprocess

import pytest

from paper_2205_04702_amd import scratchpipe as sp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "scratchpipe.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sp_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("sp_create", "sp_plan", "sp_forward", "sp_backward_update", "sp_flush",
              "sp_get_stats", "sp_debug_plan", "sp_destroy", "sp_last_error",
              "sp_host_alloc", "sp_host_free"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = sp.load()
    for n in declared_functions():
        assert hasattr(lib, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", sp.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r" T (sp_\w+)", out))
    assert set(declared_functions()) <= exported


def test_struct_layouts_match_header(tmp_path):
    src = tmp_path / "layout.c"
    src.write_text("""
#include <stdio.h>
#include <stddef.h>
#include "scratchpipe.h"
#define P(T, f) printf(#T "." #f " %zu\\n", offsetof(T, f))
int main(void) {
  printf("sp_config %zu\\nsp_batch %zu\\nsp_stats %zu\\nsp_plan_dump %zu\\n",
         sizeof(sp_config), sizeof(sp_batch), sizeof(sp_stats), sizeof(sp_plan_dump));
  P(sp_config, max_ids); P(sp_config, flags); P(sp_config, device); P(sp_config, host_tables);
  P(sp_config, policy); P(sp_config, hold_past); P(sp_config, seed); P(sp_config, max_table_ids);
  P(sp_batch, nnz); P(sp_batch, on_device); P(sp_stats, ms_forward); P(sp_stats, timed_fill);
  P(sp_stats, timed_query); P(sp_stats, host_ms_inputs);
  P(sp_plan_dump, hit); P(sp_plan_dump, nnz); P(sp_config, prefetch); P(sp_config, fill);
  P(sp_stats, prefetched); P(sp_stats, host_ms_gather); P(sp_stats, timed_h2d);
  return 0; }
""")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)], check=True)
    lines = dict(l.rsplit(" ", 1) for l in subprocess.run([str(exe)], capture_output=True,
                                                          text=True).stdout.split("\n") if l)
    assert int(lines["sp_config"]) == C.sizeof(sp.sp_config)
    assert int(lines["sp_batch"]) == C.sizeof(sp.sp_batch)
    assert int(lines["sp_stats"]) == C.sizeof(sp.sp_stats)
    assert int(lines["sp_plan_dump"]) == C.sizeof(sp.sp_plan_dump)
    for key, val in lines.items():
        if "." in key:
            struct, field = key.split(".")
            assert getattr(getattr(sp, struct), field).offset == int(val), key


def _cfg(**over):
    rows = (C.c_int64 * 2)(100, 200)
    slots = (C.c_int64 * 2)(10, 20)
    tabs = (C.c_void_p * 2)(0x1000, 0x2000)
    kw = dict(num_tables=2, rows=rows, dim=16, slots=slots, lookahead=2, host_tables=tabs,
              max_batch=8, max_ids=64, flags=0, device=0)
    kw.update(over)
    return sp.sp_config(**kw), (rows, slots, tabs)


@pytest.mark.parametrize("over,needle", [
    (dict(num_tables=0), "num_tables"),
    (dict(num_tables=65), "num_tables"),
    (dict(dim=12), "dim"),
    (dict(dim=512), "dim"),
    (dict(lookahead=-1), "lookahead"),
    (dict(lookahead=16), "lookahead"),
    (dict(max_ids=-5), "max_"),
    (dict(flags=0x80), "flags"),
    (dict(policy=3), "policy"),
    (dict(policy=-1), "policy"),
    (dict(hold_past=-1), "hold_past"),
    (dict(hold_past=5), "hold_past"),
    (dict(lookahead=12, hold_past=4), "hold_past"),
    (dict(max_table_ids=-1), "max_table_ids"),
    (dict(dim=256, max_batch=1 << 21), "4 GiB"),  # gradients addressed with 32-bit offsets
    (dict(lookahead=8, prefetch=5), "prefetch"),   # above SP_MAX_PREFETCH
    (dict(prefetch=-1), "prefetch"),
    (dict(fill=2), "fill"),
    (dict(fill=-1), "fill"),
])
def test_create_rejects_bad_configs(over, needle):
    cfg, keep = _cfg(**over)
    h = C.c_void_p()
    st = sp.load().sp_create(C.byref(cfg), C.byref(h))
    assert st == sp.SP_ERR_INVALID_ARG and not h.value
    assert needle in sp.sp_last_error(None)


def test_create_rejects_unaligned_tables():
    cfg, keep = _cfg()
    keep[2][1] = 0x2004
    h = C.c_void_p()
    assert sp.load().sp_create(C.byref(cfg), C.byref(h)) == sp.SP_ERR_INVALID_ARG
    assert "aligned" in sp.sp_last_error(None)


def test_create_rejects_bad_table_sizes():
    cfg, keep = _cfg()
    keep[1][0] = 101  # slots > rows
    h = C.c_void_p()
    assert sp.load().sp_create(C.byref(cfg), C.byref(h)) == sp.SP_ERR_INVALID_ARG
    assert "slots[0]" in sp.sp_last_error(None)
    keep[1][0] = 10
    keep[0][1] = (1 << 25) + 1
    assert sp.load().sp_create(C.byref(cfg), C.byref(h)) == sp.SP_ERR_INVALID_ARG
    assert "rows[1]" in sp.sp_last_error(None)


def test_null_handle_calls_report_state_error():
    L = sp.load()
    b = sp.sp_batch()
    t = C.c_int64()
    assert L.sp_plan(None, C.byref(b), 1, C.byref(t)) == sp.SP_ERR_STATE
    assert L.sp_forward(None, 0, None, None) == sp.SP_ERR_STATE
    assert L.sp_backward_update(None, 0, None, C.c_float(0.1), None) == sp.SP_ERR_STATE
    assert L.sp_flush(None) == sp.SP_ERR_STATE
    assert L.sp_sync(None) == sp.SP_ERR_STATE
    assert L.sp_set_flags(None, 0) == sp.SP_ERR_STATE
    L.sp_destroy(None)


def test_worst_case_storage_helper_matches_paper():
    """Sec. VI-D: (8 x 20 x 2048 x 128 x 4 B) x 6 = 960 MiB."""
    assert sp.worst_case_scratchpad_bytes(8, 20, 2048, 128, 6) == 960 * 2 ** 20


@pytest.mark.parametrize("huge", [True, False])
def test_pageable_tables_for_the_staged_fill(huge):
    """Ordinary host tables for the staged fill (in mappings advised for huge pages,
    or plain arrays): fp32, row-major, writable, 16-byte aligned as sp_create requires,
    each table its own allocation, and closing them twice is harmless."""
    import numpy as np
    t = sp.PageableTables([5, 1000, 1], 12, huge_pages=huge)
    assert len(t) == 3
    for i, rows in enumerate([5, 1000, 1]):
        a = t[i]
        assert a.shape == (rows, 12) and a.dtype == np.float32
        assert a.flags.c_contiguous and a.flags.writeable
        assert t.ptrs[i] == a.ctypes.data and t.ptrs[i] % 16 == 0
        a[:] = i + 0.5
    assert float(t[1].sum()) == 1.5 * 1000 * 12 and float(t[0][4, 11]) == 0.5
    t.close()
    t.close()
    assert len(t) == 0


def test_header_constants_match_the_binding():
    """Every integer #define of include/scratchpipe.h that the Python binding also
    names has the same value there, and every SP_FLAG_* and SP_ERR_* is named."""
    hdr = open(os.path.join(ROOT, "include", "scratchpipe.h")).read()
    consts = {m.group(1): int(m.group(2), 0)
              for m in re.finditer(r"^#define (SP_[A-Z_]+) \(?(-?(?:0x)?[0-9a-fA-F]+)u?\)?", hdr,
                                   re.M)}
    assert len(consts) >= 20
    policies = {f"SP_POLICY_{k.upper()}": v for k, v in sp.POLICIES.items()}
    for name, val in consts.items():
        if name.startswith("SP_POLICY_"):
            assert policies[name] == val, name
        elif name.startswith(("SP_FLAG_", "SP_ERR_")) or hasattr(sp, name):
            assert getattr(sp, name) == val, name
