"""The C ABI on the host: libaecct.so loads, exports every function include/aecct.h
declares, and rejects bad arguments before any GPU work (no GPU is needed)."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from workloads import build_workload, random_weights
from workloads.configs import CONFIGS, parity_check

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "aecct.h")


@pytest.fixture(scope="module")
def P():
    import paper_2410_05911_amd as P
    P.lib()
    return P


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(aecct_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol(P):
    names = _declared()
    assert "aecct_create" in names and "aecct_decode" in names
    lib = C.CDLL(P.LIB_PATH)
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing


def test_status_strings(P):
    for s in range(6):
        assert P.lib().aecct_status_string(s)
    assert P.lib().aecct_status_string(99) == b"unknown status"


def _create(P, H, w, d=None, n_layers=None, heads=None, path=0, hf=None, dff=None, eps=None, attention=0):
    H = np.ascontiguousarray(H, np.uint8)
    m, n = H.shape
    keep = []

    def f32(a):
        if a is None:
            return None
        a = np.ascontiguousarray(a, np.float32)
        keep.append(a)
        return a.ctypes.data_as(C.POINTER(C.c_float))

    def i8(a):
        a = np.ascontiguousarray(a, np.int8)
        keep.append(a)
        return a.ctypes.data_as(C.POINTER(C.c_int8))
    st = P.Weights()
    st.embed, st.pos = f32(w.embed), f32(w.pos)
    st.w_q, st.w_k, st.w_v, st.w_o = (i8(w.w[k]) for k in ("q", "k", "v", "o"))
    st.w_ff1, st.w_ff2 = i8(w.w["ff1"]), i8(w.w["ff2"])
    st.scale = f32(w.scale)
    st.b_q, st.b_k, st.b_v, st.b_o = (f32(w.b[k]) for k in ("q", "k", "v", "o"))
    st.b_ff1, st.b_ff2 = f32(w.b["ff1"]), f32(w.b["ff2"])
    st.ln1_g, st.ln1_b, st.ln2_g, st.ln2_b = f32(w.ln1_g), f32(w.ln1_b), f32(w.ln2_g), f32(w.ln2_b)
    st.head_w1, st.head_b1 = f32(w.head_w1), float(w.head_b1)
    st.head_wo, st.head_bo = f32(w.head_wo), f32(w.head_bo)
    opt = P.Options(w.first_ring_heads if hf is None else hf, w.d_ff if dff is None else dff,
                    w.ln_eps if eps is None else eps, path, attention)
    h = C.c_void_p()
    rc = P.lib().aecct_create(H.ctypes.data_as(C.POINTER(C.c_uint8)), m, n, C.byref(st),
                              w.d if d is None else d, w.n_layers if n_layers is None else n_layers,
                              w.heads if heads is None else heads, C.byref(opt), C.byref(h))
    if rc == 0:
        P.lib().aecct_destroy(h)
    return rc


def _gpu_present():
    import torch
    return torch.cuda.device_count() > 0


def test_create_validation_before_device(P):
    cfg, H, G, w, y, x = build_workload(1, batch=1)
    INV, UNS = P.ERR_INVALID_ARG, P.ERR_UNSUPPORTED
    bad = H.copy()
    bad[0, 0] = 2
    assert _create(P, bad, w) == INV                       # non-binary H
    zc = H.copy()
    zc[:, 6] = 0
    assert _create(P, zc, w) == INV                        # variable node with no check
    zr = H.copy()
    zr[2] = 0
    assert _create(P, zr, w) == INV                        # check node with no variable
    w2 = random_weights(7, 3, 32, 2, 8, seed=1)
    w2.w["ff1"] = w2.w["ff1"].copy()
    w2.w["ff1"][1, 3, 4] = 2
    assert _create(P, H, w2) == INV                        # non-ternary weight
    w3 = random_weights(7, 3, 32, 2, 8, seed=1)
    w3.ln2_b = w3.ln2_b.copy()
    w3.ln2_b[0, 0] = np.nan
    assert _create(P, H, w3) == INV                        # non-finite parameter
    assert _create(P, H, w, heads=5) == INV                # d % heads != 0
    assert _create(P, H, w, hf=9) == INV                   # more first-ring heads than heads
    assert _create(P, H, w, path=7) == INV
    assert _create(P, H, w, attention=2) == INV            # neither HPSA nor CASA
    w4 = random_weights(7, 3, 32, 2, 4, seed=1)            # d_h = 8: supported
    w5 = random_weights(7, 3, 32, 2, 1, seed=1)            # d_h = 32: not supported
    assert _create(P, H, w5) == UNS
    w6 = random_weights(7, 3, 32, 2, 8, seed=1, d_ff=64)
    assert _create(P, H, w6) == UNS                        # d_ff != 4 d
    h = C.c_void_p()
    assert P.lib().aecct_create(None, 3, 7, None, 32, 2, 8, None, C.byref(h)) == INV
    if not _gpu_present():
        # valid model: validation passes and the first HIP call reports the missing device
        assert _create(P, H, w) == P.ERR_DEVICE
        assert _create(P, H, w4) == P.ERR_DEVICE


def test_null_model_calls(P):
    L = P.lib()
    sz = C.c_size_t()
    assert L.aecct_workspace_size(None, 4, C.byref(sz)) == P.ERR_INVALID_ARG
    assert L.aecct_decode(None, None, 4, None, None, None, 0, None) == P.ERR_INVALID_ARG
    assert L.aecct_stage_embed(None, None, 1, None, None, None, None) == P.ERR_INVALID_ARG
    assert L.aecct_ternary_gemm(None, 0, 0, None, 1, None, None) == P.ERR_INVALID_ARG
    L.aecct_destroy(None)


def test_struct_layouts_match_the_header(P, tmp_path):
    """Every struct the binding mirrors has the C compiler's size and field offsets (a field the
    header lacks, or one out of order, would pass the wrong values silently)."""
    import subprocess
    structs = {"aecct_weights": P.Weights, "aecct_options": P.Options, "aecct_model_info": P.ModelInfo,
               "aecct_spe_params": P.SpeParams, "aecct_train_params": P.TrainParams,
               "aecct_train_grads": P.TrainGrads}
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "aecct.h"', "int main(void) {"]
    for cname, cls in structs.items():
        lines.append(f'  printf("{cname} size %zu\\n", sizeof({cname}));')
        for fname, _ in cls._fields_:
            lines.append(f'  printf("{cname} {fname} %zu\\n", offsetof({cname}, {fname}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c11", "-Wall", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                   check=True)
    got = {}
    for line in subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.splitlines():
        cname, field, val = line.split()
        got[(cname, field)] = int(val)
    for cname, cls in structs.items():
        assert got[(cname, "size")] == C.sizeof(cls), cname
        for fname, _ in cls._fields_:
            assert got[(cname, fname)] == getattr(cls, fname).offset, (cname, fname)
