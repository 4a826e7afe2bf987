"""The C-ABI library loads and exports every function include/cora.h declares, and its
host-side argument validation rejects malformed calls (no GPU work is issued)."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "cora.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(cora_[a-z_]+)\s*\(", src)))


def _lib():
    from paper_2608_11235_amd import _lib as L
    if not os.path.exists(L.LIB_PATH):
        pytest.fail("libcora.so is not built (run __graft_entry__.build())")
    return L.load(), L


def test_every_declared_symbol_is_exported():
    lib, L = _lib()
    names = _declared()
    assert len(names) >= 10
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(L.EXPORTS), "binding and header disagree"


def test_struct_layouts_match_header(tmp_path):
    """ctypes mirrors must have the C compiler's sizes and field offsets."""
    _, L = _lib()
    structs = {"cora_model_cfg": L.ModelCfg, "cora_sched_cfg": L.SchedCfg,
               "cora_gate_cfg": L.GateCfg, "cora_state": L.State}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "cora.h"', "int main(void){"]
    for cname, py in structs.items():
        lines.append(f'printf("{cname} size %zu\\n", sizeof({cname}));')
        for f, _ in py._fields_:
            lines.append(f'printf("{cname} {f} %zu\\n", offsetof({cname}, {f}));')
    lines.append("return 0;}")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.check_call(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)])
    out = subprocess.check_output([str(exe)], text=True).split("\n")
    got = {tuple(l.split()[:2]): int(l.split()[2]) for l in out if l}
    for cname, py in structs.items():
        assert got[(cname, "size")] == ctypes.sizeof(py), cname
        for f, _ in py._fields_:
            assert got[(cname, f)] == getattr(py, f).offset, (cname, f)


def _cfg(L, **kw):
    base = dict(n_layers=1, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64, ffn_dim=688,
                vocab=2048, mask_id=2047, qkv_bias=0, rms_eps=1e-5, rope_theta=1e4,
                logit_scale=1.0, init_std=0.02)
    base.update(kw)
    return L.ModelCfg(**base)


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=96), -2), (dict(n_kv_heads=3), -2), (dict(d_model=200), -2),
    (dict(mask_id=2048), -1), (dict(vocab=1, mask_id=0), -1), (dict(rms_eps=0.0), -1),
])
def test_create_rejects_bad_config(kw, status):
    lib, L = _lib()
    cfg = _cfg(L, **kw)
    h = ctypes.c_void_p()
    st = lib.cora_model_create(ctypes.byref(cfg), 0, 1, 64, None, ctypes.byref(h))
    assert st == status
    assert h.value is None
    assert lib.cora_last_error()


@pytest.mark.parametrize("max_batch,max_seq", [(1 << 20, 64), (4096, 4096)])
def test_create_rejects_oversized_workspace(max_batch, max_seq):
    """Activation matrices beyond 2 GB (32-bit operand offsets) are refused before any
    device call."""
    lib, L = _lib()
    cfg = _cfg(L)
    h = ctypes.c_void_p()
    st = lib.cora_model_create(ctypes.byref(cfg), 0, max_batch, max_seq, None, ctypes.byref(h))
    assert st == -2
    assert h.value is None
    assert b"2 GB" in lib.cora_last_error()


def test_vocab_gate_rejects_bad_arguments():
    lib, L = _lib()
    sc, gt = L.SchedCfg(32, 16), L.GateCfg(0.65, 1, 1, 0)
    st = L.State()
    assert lib.cora_vocab_gate(None, 32, -1, 100, 5, ctypes.byref(st), -1, ctypes.byref(sc),
                               ctypes.byref(gt), None) == -1
    bad_sched = L.SchedCfg(512, 16)
    assert lib.cora_vocab_gate(None, 32, -1, 100, 5, ctypes.byref(st), -1,
                               ctypes.byref(bad_sched), ctypes.byref(gt), None) == -2
    bad_gate = L.GateCfg(0.65, 1, 1, 2)   # persist_scope: 0 BLOCK, 1 GLOBAL, else unsupported
    assert lib.cora_vocab_gate(None, 32, -1, 100, 5, ctypes.byref(st), -1, ctypes.byref(sc),
                               ctypes.byref(bad_gate), None) == -2
