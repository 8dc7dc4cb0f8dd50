"""MI355X (gfx950) AECCT inference: Python binding of libaecct.so.

Argument marshalling only: every step of a decode runs in the library's HIP kernels.
PyTorch provides device memory and streams.  Importing this package loads the built
library and raises if it is missing; there is no CPU fallback.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libaecct.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_OUT_OF_MEMORY, ERR_DEVICE, ERR_WORKSPACE_TOO_SMALL = range(6)
PATH_AUTO, PATH_LAYERED, PATH_FUSED = 0, 1, 2
ATTN_HPSA, ATTN_CASA = 0, 1
LAYERED_ATTN_AUTO, LAYERED_ATTN_UNFUSED, LAYERED_ATTN_LDS_F32, LAYERED_ATTN_LDS_I16, LAYERED_ATTN_LDS_SPLIT = -1, 0, 1, 2, 3
ACT_SCALE_TOKEN, ACT_SCALE_WORD = 0, 1
LIN_Q, LIN_K, LIN_V, LIN_O, LIN_FF1, LIN_FF2 = range(6)

_vp = C.c_void_p
_i8p = C.POINTER(C.c_int8)
_f32p = C.POINTER(C.c_float)
_u8p = C.POINTER(C.c_uint8)


class Weights(C.Structure):
    _fields_ = [("embed", _f32p), ("pos", _f32p), ("w_q", _i8p), ("w_k", _i8p), ("w_v", _i8p), ("w_o", _i8p),
                ("w_ff1", _i8p), ("w_ff2", _i8p), ("scale", _f32p), ("b_q", _f32p), ("b_k", _f32p), ("b_v", _f32p),
                ("b_o", _f32p), ("b_ff1", _f32p), ("b_ff2", _f32p), ("ln1_g", _f32p), ("ln1_b", _f32p),
                ("ln2_g", _f32p), ("ln2_b", _f32p), ("head_w1", _f32p), ("head_b1", C.c_float),
                ("head_wo", _f32p), ("head_bo", _f32p)]


class Options(C.Structure):
    _fields_ = [("first_ring_heads", C.c_int32), ("d_ff", C.c_int32), ("ln_eps", C.c_float), ("path", C.c_int32),
                ("attention", C.c_int32), ("layered_attention", C.c_int32), ("act_scale_mode", C.c_int32)]


class ModelInfo(C.Structure):
    _fields_ = [("n", C.c_int32), ("m", C.c_int32), ("L", C.c_int32), ("d", C.c_int32), ("n_layers", C.c_int32),
                ("heads", C.c_int32), ("first_ring_heads", C.c_int32), ("d_ff", C.c_int32), ("path", C.c_int32),
                ("nnz_first_ring", C.c_int64), ("nnz_second_ring", C.c_int64), ("device_bytes", C.c_size_t),
                ("attention", C.c_int32), ("layered_attention", C.c_int32), ("act_scale_mode", C.c_int32),
                ("device", C.c_int32), ("compute_units", C.c_int32), ("lds_bytes", C.c_int64)]


class SpeParams(C.Structure):
    _fields_ = [("d_pe", C.c_int32), ("heads", C.c_int32), ("w_in", _f32p), ("b_in", _f32p),
                ("w_q", _f32p), ("w_k", _f32p), ("w_v", _f32p), ("w_o", _f32p),
                ("b_q", _f32p), ("b_k", _f32p), ("b_v", _f32p), ("b_o", _f32p),
                ("w_red", _f32p), ("b_red", C.c_float)]


_TRAIN_FIELDS = ["embed", "pos", "w_q", "w_k", "w_v", "w_o", "w_ff1", "w_ff2", "delta", "b_q", "b_k", "b_v", "b_o",
                 "b_ff1", "b_ff2", "ln1_g", "ln1_b", "ln2_g", "ln2_b", "head_w1", "head_b1", "head_wo", "head_bo"]


class TrainParams(C.Structure):
    _fields_ = [(f, _vp) for f in _TRAIN_FIELDS]


class TrainGrads(C.Structure):
    _fields_ = [(f, _vp) for f in _TRAIN_FIELDS if f != "pos"]


class AecctError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {lib().aecct_status_string(status).decode()} (status {status})")


_lib = None


def lib():
    """The loaded libaecct.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2410_05911_amd/build.py "
                              "(or __graft_entry__.build()); there is no fallback path")
        L = C.CDLL(LIB_PATH)
        L.aecct_status_string.restype = C.c_char_p
        L.aecct_status_string.argtypes = [C.c_int]
        L.aecct_create.restype = C.c_int
        L.aecct_create.argtypes = [_u8p, C.c_int32, C.c_int32, C.POINTER(Weights), C.c_int32, C.c_int32, C.c_int32,
                                   C.POINTER(Options), C.POINTER(_vp)]
        L.aecct_destroy.restype = None
        L.aecct_destroy.argtypes = [_vp]
        L.aecct_get_info.restype = C.c_int
        L.aecct_get_info.argtypes = [_vp, C.POINTER(ModelInfo)]
        L.aecct_workspace_size.restype = C.c_int
        L.aecct_workspace_size.argtypes = [_vp, C.c_int64, C.POINTER(C.c_size_t)]
        L.aecct_decode.restype = C.c_int
        L.aecct_decode.argtypes = [_vp, _vp, C.c_int64, _vp, _vp, _vp, C.c_size_t, _vp]
        L.aecct_decode_static.restype = C.c_int
        L.aecct_decode_static.argtypes = [_vp, _vp, C.c_int64, _vp, _vp, _vp]
        L.aecct_stage_embed.restype = C.c_int
        L.aecct_stage_embed.argtypes = [_vp, _vp, C.c_int64, _vp, _vp, _vp, _vp]
        L.aecct_stage_qkv.restype = C.c_int
        L.aecct_stage_qkv.argtypes = [_vp, C.c_int32, _vp, _vp, C.c_int64, _vp, _vp]
        L.aecct_stage_attention.restype = C.c_int
        L.aecct_stage_attention.argtypes = [_vp, _vp, C.c_int64, _vp, _vp, _vp, _vp]
        L.aecct_stage_oproj_ln.restype = C.c_int
        L.aecct_stage_oproj_ln.argtypes = [_vp, C.c_int32, _vp, _vp, _vp, C.c_int64, _vp, _vp, _vp, _vp]
        L.aecct_stage_ffn1.restype = C.c_int
        L.aecct_stage_ffn1.argtypes = [_vp, C.c_int32, _vp, _vp, C.c_int64, _vp, _vp, _vp]
        L.aecct_stage_ffn2_ln.restype = C.c_int
        L.aecct_stage_ffn2_ln.argtypes = [_vp, C.c_int32, _vp, _vp, _vp, C.c_int64, _vp, _vp, _vp, _vp]
        L.aecct_stage_head.restype = C.c_int
        L.aecct_stage_head.argtypes = [_vp, _vp, _vp, C.c_int64, _vp, _vp, _vp]
        L.aecct_ternary_gemm.restype = C.c_int
        L.aecct_ternary_gemm.argtypes = [_vp, C.c_int32, C.c_int32, _vp, C.c_int64, _vp, _vp]
        L.aecct_aap_ternarize.restype = C.c_int
        L.aecct_aap_ternarize.argtypes = [_f32p, C.c_int64, C.c_float, C.c_float, C.c_float, _i8p, _f32p]
        _f64p = C.POINTER(C.c_double)
        L.aecct_tanner_spectrum.restype = C.c_int
        L.aecct_tanner_spectrum.argtypes = [_u8p, C.c_int32, C.c_int32, _f64p, _f64p]
        L.aecct_spe_table_from_spectrum.restype = C.c_int
        L.aecct_spe_table_from_spectrum.argtypes = [_f64p, _f64p, C.c_int32, C.POINTER(SpeParams), C.c_int32,
                                                    _f32p]
        L.aecct_spe_table.restype = C.c_int
        L.aecct_spe_table.argtypes = [_u8p, C.c_int32, C.c_int32, C.POINTER(SpeParams), C.c_int32, _f32p]
        L.aecct_train_create.restype = C.c_int
        L.aecct_train_create.argtypes = [_u8p, C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                         C.POINTER(Options), C.c_float, C.POINTER(_vp)]
        L.aecct_train_destroy.restype = None
        L.aecct_train_destroy.argtypes = [_vp]
        L.aecct_train_workspace_size.restype = C.c_int
        L.aecct_train_workspace_size.argtypes = [_vp, C.c_int64, C.POINTER(C.c_size_t)]
        L.aecct_train_grad.restype = C.c_int
        L.aecct_train_grad.argtypes = [_vp, C.POINTER(TrainParams), _vp, _vp, C.c_int64, C.POINTER(TrainGrads), _vp,
                                       _vp, C.c_size_t, _vp]
        L.aecct_check_device_arith.restype = C.c_int
        L.aecct_check_device_arith.argtypes = [C.POINTER(C.c_uint64)]
        _lib = L
    return _lib


def aap_ternarize(w, percentile: float = 0.5, delta: float = 1.0, eps: float = 1e-8):
    """AAP import of one trained fp32 weight matrix (Section 4.1, Eq. 1) by the library:
    returns (ternary int8 array of w's shape, weight scale gamma*delta as np.float32)."""
    w = np.ascontiguousarray(w, dtype=np.float32)
    t = np.zeros(w.shape, np.int8)
    sc = C.c_float(0.0)
    _check(lib().aecct_aap_ternarize(w.ctypes.data_as(_f32p), w.size, float(np.float32(percentile)),
                                     float(np.float32(delta)), float(np.float32(eps)), t.ctypes.data_as(_i8p),
                                     C.byref(sc)), "aecct_aap_ternarize")
    return t, np.float32(sc.value)


def tanner_spectrum(H):
    """Laplacian spectrum of the Tanner graph of H by the library (host, float64): returns
    (eigenvalues ascending [L], eigenvectors [L, L] with ROW i the canonical vector i)."""
    H = np.ascontiguousarray(H, dtype=np.uint8)
    m, n = H.shape
    lam = np.zeros(n + m, np.float64)
    vec = np.zeros((n + m, n + m), np.float64)
    _check(lib().aecct_tanner_spectrum(H.ctypes.data_as(_u8p), m, n, lam.ctypes.data_as(C.POINTER(C.c_double)),
                                       vec.ctypes.data_as(C.POINTER(C.c_double))), "aecct_tanner_spectrum")
    return lam, vec


def _spe_struct(p: dict, L: int):
    keep = {k: _host(p.get(k), np.float32) for k in ("w_in", "b_in", "w_q", "w_k", "w_v", "w_o", "b_q", "b_k",
                                                     "b_v", "b_o", "w_red")}
    if keep["w_red"] is not None and keep["w_red"].size != L:
        raise ValueError(f"w_red must have {L} entries")
    s = SpeParams(d_pe=int(p["d_pe"]), heads=int(p["heads"]), b_red=float(np.float32(p.get("b_red", 0.0))))
    for k, a in keep.items():
        setattr(s, k, _p32(a))
    return s, keep


def _p32(a):
    return a.ctypes.data_as(_f32p) if a is not None else None


def spe_table_from_spectrum(lam, vec_rows, p: dict, d: int):
    """Positional table [L, d] fp32 from a spectrum (ROW i of vec_rows = eigenvector i) and
    the SPE parameters (Section 4.3); the attention runs on the current GPU."""
    lam = np.ascontiguousarray(lam, dtype=np.float64)
    vec = np.ascontiguousarray(vec_rows, dtype=np.float64)
    L = lam.size
    s, keep = _spe_struct(p, L)
    out = np.zeros((L, d), np.float32)
    _check(lib().aecct_spe_table_from_spectrum(lam.ctypes.data_as(C.POINTER(C.c_double)),
                                               vec.ctypes.data_as(C.POINTER(C.c_double)), L, C.byref(s), d,
                                               out.ctypes.data_as(_f32p)), "aecct_spe_table_from_spectrum")
    return out


def spe_table(H, p: dict, d: int):
    """The whole SPE construction (spectrum, then attention) for H: positional table [L, d]."""
    H = np.ascontiguousarray(H, dtype=np.uint8)
    m, n = H.shape
    s, keep = _spe_struct(p, n + m)
    out = np.zeros((n + m, d), np.float32)
    _check(lib().aecct_spe_table(H.ctypes.data_as(_u8p), m, n, C.byref(s), d, out.ctypes.data_as(_f32p)),
           "aecct_spe_table")
    return out


def check_device_arith():
    """Counts of fp32 operands where the device's fract/floor split, softmax reciprocal and
    127/alpha differ from their IEEE definitions (all 0 on a conforming GPU)."""
    counts = (C.c_uint64 * 3)()
    _check(lib().aecct_check_device_arith(counts), "aecct_check_device_arith")
    return tuple(int(c) for c in counts)


def _check(status: int, what: str):
    if status != OK:
        raise AecctError(status, what)


def _host(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


def _ptr(t):
    """Device address of a torch tensor (or None)."""
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t.data_ptr()


def _stream_ptr(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


class Decoder:
    """An AECCT model on the current GPU.

    `H` is the (n-k) x n parity-check matrix (0/1) and `w` carries the model parameters
    with the attribute names of `workloads.ModelWeights` (embed, pos, w[kind], b[kind], scale,
    ln1_g, ..., head_wo, head_bo, and optionally attention = "hpsa" | "casa" and
    act_scale = "token" | "word").  `path` and `layered_attention` choose the kernels
    (aecct_path, aecct_layered_attention; -1 = automatic).
    """

    def __init__(self, H, w, path: int = PATH_AUTO, layered_attention: int = LAYERED_ATTN_AUTO):
        H = _host(H, np.uint8)
        m, n = H.shape
        self._keep = [H]

        def f32(a):
            a = _host(a, np.float32)
            self._keep.append(a)
            return None if a is None else a.ctypes.data_as(_f32p)

        def i8(a):
            a = _host(a, np.int8)
            self._keep.append(a)
            return a.ctypes.data_as(_i8p)

        st = Weights()
        st.embed, st.pos = f32(w.embed), f32(w.pos)
        st.w_q, st.w_k, st.w_v, st.w_o = (i8(w.w[k]) for k in ("q", "k", "v", "o"))
        st.w_ff1, st.w_ff2 = i8(w.w["ff1"]), i8(w.w["ff2"])
        st.scale = f32(w.scale)
        st.b_q, st.b_k, st.b_v, st.b_o = (f32(w.b[k]) for k in ("q", "k", "v", "o"))
        st.b_ff1, st.b_ff2 = f32(w.b["ff1"]), f32(w.b["ff2"])
        st.ln1_g, st.ln1_b, st.ln2_g, st.ln2_b = f32(w.ln1_g), f32(w.ln1_b), f32(w.ln2_g), f32(w.ln2_b)
        st.head_w1, st.head_b1 = f32(w.head_w1), float(np.float32(w.head_b1))
        st.head_wo, st.head_bo = f32(w.head_wo), f32(w.head_bo)
        attention = {"hpsa": ATTN_HPSA, "casa": ATTN_CASA}[getattr(w, "attention", "hpsa")]
        act = {"token": ACT_SCALE_TOKEN, "word": ACT_SCALE_WORD}[getattr(w, "act_scale", "token")]
        opt = Options(int(w.first_ring_heads), int(w.d_ff), float(w.ln_eps), int(path), attention,
                      int(layered_attention), act)
        h = _vp()
        _check(lib().aecct_create(H.ctypes.data_as(_u8p), m, n, C.byref(st), int(w.d), int(w.n_layers),
                                  int(w.heads), C.byref(opt), C.byref(h)), "aecct_create")
        self._h = h
        self._keep = None
        info = ModelInfo()
        _check(lib().aecct_get_info(h, C.byref(info)), "aecct_get_info")
        self.info = info
        self.n, self.m, self.L, self.d = info.n, info.m, info.L, info.d
        self.n_layers, self.d_ff, self.path = info.n_layers, info.d_ff, info.path
        self._ws = None

    def close(self):
        if getattr(self, "_h", None):
            lib().aecct_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ------------------------------------------------------------------ decode
    def workspace_size(self, batch: int) -> int:
        sz = C.c_size_t()
        _check(lib().aecct_workspace_size(self._h, int(batch), C.byref(sz)), "aecct_workspace_size")
        return sz.value

    def workspace(self, batch: int, device=None):
        """A cached uint8 device tensor large enough for `batch` words."""
        import torch
        need = self.workspace_size(batch)
        if need == 0:
            return None
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(need, dtype=torch.uint8, device=device or "cuda")
        return self._ws

    def decode(self, y, bits=None, logits=None, workspace=None, stream=None, with_logits: bool = True):
        """y: fp32 CUDA tensor [B, n].  Returns (bits uint8 [B, n], logits fp32 [B, n] or None)."""
        import torch
        B = y.shape[0]
        if bits is None:
            bits = torch.empty((B, self.n), dtype=torch.uint8, device=y.device)
        if logits is None and with_logits:
            logits = torch.empty((B, self.n), dtype=torch.float32, device=y.device)
        ws = workspace if workspace is not None else self.workspace(B, y.device)
        _check(lib().aecct_decode(self._h, _ptr(y), B, _ptr(bits), _ptr(logits), _ptr(ws),
                                  0 if ws is None else ws.numel(), _stream_ptr(stream)), "aecct_decode")
        return bits, logits

    def decode_static(self, y, bits=None, logits=None, stream=None, with_logits: bool = True):
        """aecct_decode_static: the same decode with the library's static device scratch (no
        workspace, no allocation by the library)."""
        import torch
        B = y.shape[0]
        if bits is None:
            bits = torch.empty((B, self.n), dtype=torch.uint8, device=y.device)
        if logits is None and with_logits:
            logits = torch.empty((B, self.n), dtype=torch.float32, device=y.device)
        _check(lib().aecct_decode_static(self._h, _ptr(y), B, _ptr(bits), _ptr(logits), _stream_ptr(stream)),
               "aecct_decode_static")
        return bits, logits

    # ------------------------------------------------------------------ stages
    def stage_embed(self, y, stream=None):
        import torch
        W = y.shape[0]
        R = W * self.L
        x = torch.empty((R, self.d), dtype=torch.float32, device=y.device)
        xq = torch.empty((R, self.d), dtype=torch.int8, device=y.device)
        ax = torch.empty((R,), dtype=torch.float32, device=y.device)
        _check(lib().aecct_stage_embed(self._h, _ptr(y), W, _ptr(x), _ptr(xq), _ptr(ax), _stream_ptr(stream)),
               "aecct_stage_embed")
        return x, xq, ax

    def stage_qkv(self, layer, xq, ax, stream=None):
        import torch
        W = xq.shape[0] // self.L
        qkv = torch.empty((xq.shape[0], 3 * self.d), dtype=torch.float32, device=xq.device)
        _check(lib().aecct_stage_qkv(self._h, layer, _ptr(xq), _ptr(ax), W, _ptr(qkv), _stream_ptr(stream)),
               "aecct_stage_qkv")
        return qkv

    def stage_attention(self, qkv, with_o: bool = True, stream=None):
        import torch
        R = qkv.shape[0]
        W = R // self.L
        o = torch.empty((R, self.d), dtype=torch.float32, device=qkv.device) if with_o else None
        oq = torch.empty((R, self.d), dtype=torch.int8, device=qkv.device)
        ao = torch.empty((R,), dtype=torch.float32, device=qkv.device)
        _check(lib().aecct_stage_attention(self._h, _ptr(qkv), W, _ptr(o), _ptr(oq), _ptr(ao), _stream_ptr(stream)),
               "aecct_stage_attention")
        return o, oq, ao

    def stage_oproj_ln(self, layer, oq, ao, x, stream=None):
        import torch
        R = oq.shape[0]
        x1 = torch.empty((R, self.d), dtype=torch.float32, device=oq.device)
        x1q = torch.empty((R, self.d), dtype=torch.int8, device=oq.device)
        a1 = torch.empty((R,), dtype=torch.float32, device=oq.device)
        _check(lib().aecct_stage_oproj_ln(self._h, layer, _ptr(oq), _ptr(ao), _ptr(x), R // self.L, _ptr(x1),
                                          _ptr(x1q), _ptr(a1), _stream_ptr(stream)), "aecct_stage_oproj_ln")
        return x1, x1q, a1

    def stage_ffn1(self, layer, x1q, a1, stream=None):
        import torch
        R = x1q.shape[0]
        gq = torch.empty((R, self.d_ff), dtype=torch.int8, device=x1q.device)
        ag = torch.empty((R,), dtype=torch.float32, device=x1q.device)
        _check(lib().aecct_stage_ffn1(self._h, layer, _ptr(x1q), _ptr(a1), R // self.L, _ptr(gq), _ptr(ag),
                                      _stream_ptr(stream)), "aecct_stage_ffn1")
        return gq, ag

    def stage_ffn2_ln(self, layer, gq, ag, x1, stream=None):
        import torch
        R = gq.shape[0]
        x = torch.empty((R, self.d), dtype=torch.float32, device=gq.device)
        xq = torch.empty((R, self.d), dtype=torch.int8, device=gq.device)
        ax = torch.empty((R,), dtype=torch.float32, device=gq.device)
        _check(lib().aecct_stage_ffn2_ln(self._h, layer, _ptr(gq), _ptr(ag), _ptr(x1), R // self.L, _ptr(x),
                                         _ptr(xq), _ptr(ax), _stream_ptr(stream)), "aecct_stage_ffn2_ln")
        return x, xq, ax

    def stage_head(self, x, y, stream=None):
        import torch
        W = y.shape[0]
        bits = torch.empty((W, self.n), dtype=torch.uint8, device=y.device)
        logits = torch.empty((W, self.n), dtype=torch.float32, device=y.device)
        _check(lib().aecct_stage_head(self._h, _ptr(x), _ptr(y), W, _ptr(bits), _ptr(logits), _stream_ptr(stream)),
               "aecct_stage_head")
        return bits, logits

    def ternary_gemm(self, layer, kind, a, stream=None):
        import torch
        rows = a.shape[0]
        n_out = self.d_ff if kind == LIN_FF1 else self.d
        acc = torch.empty((rows, n_out), dtype=torch.int32, device=a.device)
        _check(lib().aecct_ternary_gemm(self._h, layer, kind, _ptr(a), rows, _ptr(acc), _stream_ptr(stream)),
               "aecct_ternary_gemm")
        return acc


_TRAIN_KINDS = ("q", "k", "v", "o", "ff1", "ff2")


class Trainer:
    """The quantisation-aware training step (Section 6, second phase) on the current GPU for the
    code of H: forward with Eq. 1 / Eq. 2 straight-through quantisation, the loss of the
    multiplicative noise and every parameter's gradient, in the library's kernels.

    Parameters and gradients are dicts of contiguous fp32 CUDA tensors with the keys of
    `workloads.random_qat_params` (w and b are dicts by map kind; head_b1 a one-element tensor).
    """

    def __init__(self, H, d: int, n_layers: int, heads: int = 8, first_ring_heads: int = -1,
                 attention: str = "hpsa", ln_eps: float = 1e-5, aap_eps: float = 1e-8):
        H = _host(H, np.uint8)
        m, n = H.shape
        self.n, self.m, self.L, self.d, self.n_layers = n, m, n + m, d, n_layers
        opt = Options(int(first_ring_heads), -1, float(ln_eps), PATH_AUTO,
                      {"hpsa": ATTN_HPSA, "casa": ATTN_CASA}[attention], LAYERED_ATTN_AUTO, ACT_SCALE_TOKEN)
        h = _vp()
        _check(lib().aecct_train_create(H.ctypes.data_as(_u8p), m, n, int(d), int(n_layers), int(heads), C.byref(opt),
                                        float(np.float32(aap_eps)), C.byref(h)), "aecct_train_create")
        self._h = h
        self._ws = None

    def close(self):
        if getattr(self, "_h", None):
            lib().aecct_train_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def workspace_size(self, batch: int) -> int:
        sz = C.c_size_t()
        _check(lib().aecct_train_workspace_size(self._h, int(batch), C.byref(sz)), "aecct_train_workspace_size")
        return sz.value

    @staticmethod
    def _flat(d: dict):
        out = {}
        for k, v in d.items():
            if k in ("w", "b"):
                for kind in _TRAIN_KINDS:
                    out[f"{k}_{kind}"] = v[kind]
            else:
                out[k] = v
        return out

    def grad(self, params: dict, y, xs=None, stream=None):
        """One step on the words y [B, n] (xs: transmitted +-1 words, None = all-zero codeword).
        Returns (loss one-element tensor, gradients dict shaped like params, without pos)."""
        import torch
        B = y.shape[0]
        flat = self._flat(params)
        tp = TrainParams(**{f: _ptr(flat.get(f)) for f in _TRAIN_FIELDS})
        grads = {k: (torch.empty_like(v) if k not in ("w", "b") else {kk: torch.empty_like(vv) for kk, vv in v.items()})
                 for k, v in params.items() if k != "pos" and v is not None}
        gflat = self._flat(grads)
        tg = TrainGrads(**{f: _ptr(gflat[f]) for f, _ in TrainGrads._fields_})
        need = self.workspace_size(B)
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(need, dtype=torch.uint8, device=y.device)
        loss = torch.empty(1, dtype=torch.float32, device=y.device)
        _check(lib().aecct_train_grad(self._h, C.byref(tp), _ptr(y), _ptr(xs), B, C.byref(tg), _ptr(loss),
                                      _ptr(self._ws), self._ws.numel(), _stream_ptr(stream)), "aecct_train_grad")
        return loss, grads
