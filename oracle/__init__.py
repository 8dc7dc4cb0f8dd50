"""CPU oracle of the AECCT inference path -- TEST INFRASTRUCTURE ONLY.

ctypes binding of liboracle.so (plain C, see aecct_oracle.c).  Only the test suite,
the package smoke check and the benchmark's CPU-baseline leg may import this module;
the product path never does.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

from .build import LIB, build_oracle

_lib = None

_f32p = C.POINTER(C.c_float)
_f64p = C.POINTER(C.c_double)
_u8p = C.POINTER(C.c_uint8)
_i8p = C.POINTER(C.c_int8)
_i32p = C.POINTER(C.c_int32)


class _Model(C.Structure):
    _fields_ = [("n", C.c_int32), ("m", C.c_int32), ("d", C.c_int32), ("n_layers", C.c_int32),
                ("heads", C.c_int32), ("first_ring_heads", C.c_int32), ("d_ff", C.c_int32),
                ("ln_eps", C.c_float), ("H", _u8p), ("embed", _f32p), ("pos", _f32p),
                ("w", _i8p * 6), ("scale", _f32p), ("bias", _f32p * 6),
                ("ln1_g", _f32p), ("ln1_b", _f32p), ("ln2_g", _f32p), ("ln2_b", _f32p),
                ("head_w1", _f32p), ("head_b1", C.c_float), ("head_wo", _f32p), ("head_bo", _f32p),
                ("attention", C.c_int32), ("act_scale_mode", C.c_int32)]


class _Taps(C.Structure):
    _fields_ = [("x_in", _f32p), ("xq", _i8p), ("ax", _f32p), ("qkv", _f32p),
                ("o", _f32p), ("oq", _i8p), ("ao", _f32p), ("acc_o", _i32p),
                ("x1", _f32p), ("x1q", _i8p), ("a1", _f32p), ("acc_ff1", _i32p),
                ("gq", _i8p), ("ag", _f32p), ("acc_ff2", _i32p), ("x_out", _f32p), ("z", _f32p)]


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build_oracle()
        L = C.CDLL(LIB)
        L.oracle_tree_sum.restype = C.c_float
        L.oracle_tree_sum.argtypes = [_f32p, C.c_int32]
        L.oracle_exp2.restype = C.c_float
        L.oracle_exp2.argtypes = [C.c_float]
        L.oracle_rsqrt.restype = C.c_float
        L.oracle_rsqrt.argtypes = [C.c_float]
        L.oracle_query_scale.restype = C.c_float
        L.oracle_query_scale.argtypes = [C.c_int32]
        L.oracle_masks.argtypes = [_u8p, C.c_int32, C.c_int32, _u8p, _u8p]
        L.oracle_preprocess.argtypes = [_u8p, C.c_int32, C.c_int32, _f32p, _f32p]
        L.oracle_quant_rows.argtypes = [_f32p, C.c_int64, C.c_int32, _i8p, _f32p]
        L.oracle_quant_word.argtypes = [_f32p, C.c_int64, C.c_int32, _i8p, _f32p]
        L.oracle_linear_rows.argtypes = [_i8p, _f32p, C.c_int64, _i8p, C.c_int32, C.c_int32, C.c_float,
                                         _f32p, _f32p, _i32p]
        L.oracle_layernorm_rows.argtypes = [_f32p, C.c_int64, C.c_int32, _f32p, _f32p, C.c_float, _f32p]
        L.oracle_attention_word.restype = C.c_int
        L.oracle_attention_word.argtypes = [C.POINTER(_Model), _u8p, _u8p, _f32p, _f32p]
        L.oracle_attention_dense_f64.restype = C.c_int
        L.oracle_attention_dense_f64.argtypes = [C.POINTER(_Model), _u8p, _u8p, _f64p, C.c_double, _f64p]
        L.oracle_head_word.argtypes = [C.POINTER(_Model), _f32p, _f32p, _f32p, _u8p, _f32p]
        L.oracle_decode.restype = C.c_int
        L.oracle_decode.argtypes = [C.POINTER(_Model), _f32p, C.c_int64, _u8p, _f32p, C.c_int32]
        L.oracle_decode_taps.restype = C.c_int
        L.oracle_decode_taps.argtypes = [C.POINTER(_Model), _f32p, _u8p, _f32p, C.POINTER(_Taps)]
        L.oracle_aap_ternarize.restype = C.c_int
        L.oracle_aap_ternarize.argtypes = [_f32p, C.c_int64, C.c_float, C.c_float, C.c_float, _i8p, _f32p]
        L.oracle_decode_ref64.restype = C.c_int
        L.oracle_decode_ref64.argtypes = [C.POINTER(_Model), _f32p, C.c_int64, _u8p, _f64p, C.c_int32]
        L.oracle_decode_ref64_word.restype = C.c_int
        L.oracle_decode_ref64_word.argtypes = [C.POINTER(_Model), _f32p, _u8p, _f64p, _i8p, _i8p, C.c_double,
                                               C.POINTER(C.c_int64)]
        _lib = L
    return _lib


def _p(a, t):
    return a.ctypes.data_as(t) if a is not None else None


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


KINDS = ("q", "k", "v", "o", "ff1", "ff2")
ATTENTION = {"hpsa": 0, "casa": 1}
ACT_SCALE = {"token": 0, "word": 1}


class OracleModel:
    """Holds contiguous copies of a ModelWeights and the H matrix for the C oracle."""

    def __init__(self, H, w):
        self.H = _c(H, np.uint8)
        self.w = w
        self.n, self.m, self.d = w.n, w.m, w.d
        self.L = w.n + w.m
        self._keep = []

        def keep(a, dt):
            a = None if a is None else _c(a, dt)
            self._keep.append(a)
            return a
        st = _Model()
        st.n, st.m, st.d, st.n_layers = w.n, w.m, w.d, w.n_layers
        st.heads, st.first_ring_heads, st.d_ff, st.ln_eps = w.heads, w.first_ring_heads, w.d_ff, w.ln_eps
        st.H = _p(self.H, _u8p)
        st.embed = _p(keep(w.embed, np.float32), _f32p)
        st.pos = _p(keep(w.pos, np.float32), _f32p)
        for i, k in enumerate(KINDS):
            st.w[i] = _p(keep(w.w[k], np.int8), _i8p)
            st.bias[i] = _p(keep(w.b[k], np.float32), _f32p)
        st.scale = _p(keep(w.scale, np.float32), _f32p)
        st.ln1_g = _p(keep(w.ln1_g, np.float32), _f32p)
        st.ln1_b = _p(keep(w.ln1_b, np.float32), _f32p)
        st.ln2_g = _p(keep(w.ln2_g, np.float32), _f32p)
        st.ln2_b = _p(keep(w.ln2_b, np.float32), _f32p)
        st.head_w1 = _p(keep(w.head_w1, np.float32), _f32p)
        st.head_b1 = w.head_b1
        st.head_wo = _p(keep(w.head_wo, np.float32), _f32p)
        st.head_bo = _p(keep(w.head_bo, np.float32), _f32p)
        st.attention = ATTENTION[getattr(w, "attention", "hpsa")]
        st.act_scale_mode = ACT_SCALE[getattr(w, "act_scale", "token")]
        self.st = st

    # ------------------------------------------------------------ whole decode
    def decode(self, y, n_threads: int = 1):
        y = _c(y, np.float32)
        B = y.shape[0]
        bits = np.zeros((B, self.n), np.uint8)
        f = np.zeros((B, self.n), np.float32)
        rc = lib().oracle_decode(C.byref(self.st), _p(y, _f32p), B, _p(bits, _u8p), _p(f, _f32p), n_threads)
        if rc:
            raise RuntimeError("oracle_decode failed")
        return bits, f

    def decode_ref64(self, y, n_threads: int = 1):
        y = _c(y, np.float32)
        B = y.shape[0]
        bits = np.zeros((B, self.n), np.uint8)
        f = np.zeros((B, self.n), np.float64)
        rc = lib().oracle_decode_ref64(C.byref(self.st), _p(y, _f32p), B, _p(bits, _u8p), _p(f, _f64p),
                                       n_threads)
        if rc:
            raise RuntimeError("oracle_decode_ref64 failed")
        return bits, f

    def decode_ref64_word(self, y_word, force=None, margin: float = 0.0):
        """One word in the fp64 reference mode: (bits, f float64, codes dict, stats) where codes
        holds the word's int8 activation codes per layer: xq [N, L, d], oq, x1q [N, L, d],
        gq [N, L, d_ff] (the same quantisation points as the canonical taps).  `force`, a dict of
        such codes (e.g. canonical taps), decides codes whose fp64 value lies within `margin` of
        a rounding tie; stats = (codes so decided against the fp64 choice, codes of `force` that
        differ from the fp64 choice away from a tie)."""
        w = self.w
        N, L, d, dff = w.n_layers, self.L, w.d, w.d_ff
        y = _c(y_word, np.float32).reshape(-1)
        codes = np.zeros((N, L * (3 * d + dff)), np.int8)
        fc = None
        if force is not None:
            fc = np.ascontiguousarray(np.concatenate(
                [np.asarray(force[k], np.int8).reshape(N, -1) for k in ("xq", "oq", "x1q", "gq")], 1))
            assert fc.shape == codes.shape
        bits = np.zeros(self.n, np.uint8)
        f = np.zeros(self.n, np.float64)
        stats = np.zeros(2, np.int64)
        if lib().oracle_decode_ref64_word(C.byref(self.st), _p(y, _f32p), _p(bits, _u8p), _p(f, _f64p),
                                          _p(codes, _i8p), _p(fc, _i8p), float(margin),
                                          stats.ctypes.data_as(C.POINTER(C.c_int64))):
            raise RuntimeError("oracle_decode_ref64_word failed")
        c = {"xq": codes[:, :L * d].reshape(N, L, d), "oq": codes[:, L * d:2 * L * d].reshape(N, L, d),
             "x1q": codes[:, 2 * L * d:3 * L * d].reshape(N, L, d), "gq": codes[:, 3 * L * d:].reshape(N, L, dff)}
        return bits, f, c, (int(stats[0]), int(stats[1]))

    def decode_taps(self, y_word):
        """One word; returns (bits, f, taps dict of per-layer arrays)."""
        w = self.w
        N, L, d, dff = w.n_layers, self.L, w.d, w.d_ff
        y = _c(y_word, np.float32).reshape(-1)
        t = dict(
            x_in=np.zeros((N, L, d), np.float32), xq=np.zeros((N, L, d), np.int8), ax=np.zeros((N, L), np.float32),
            qkv=np.zeros((N, L, 3 * d), np.float32), o=np.zeros((N, L, d), np.float32),
            oq=np.zeros((N, L, d), np.int8), ao=np.zeros((N, L), np.float32), acc_o=np.zeros((N, L, d), np.int32),
            x1=np.zeros((N, L, d), np.float32), x1q=np.zeros((N, L, d), np.int8), a1=np.zeros((N, L), np.float32),
            acc_ff1=np.zeros((N, L, dff), np.int32), gq=np.zeros((N, L, dff), np.int8),
            ag=np.zeros((N, L), np.float32), acc_ff2=np.zeros((N, L, d), np.int32),
            x_out=np.zeros((N, L, d), np.float32), z=np.zeros((L,), np.float32))
        st = _Taps()
        for name, typ in _Taps._fields_:
            setattr(st, name, t[name].ctypes.data_as(typ))
        bits = np.zeros(self.n, np.uint8)
        f = np.zeros(self.n, np.float32)
        rc = lib().oracle_decode_taps(C.byref(self.st), _p(y, _f32p), _p(bits, _u8p), _p(f, _f32p), C.byref(st))
        if rc:
            raise RuntimeError("oracle_decode_taps failed")
        return bits, f, t

    # ------------------------------------------------------------ stages
    def masks(self):
        return masks(self.H)

    def attention(self, qkv, M1=None, M2=None):
        if M1 is None:
            M1, M2 = masks(self.H)
        qkv = _c(qkv, np.float32)
        o = np.zeros((self.L, self.d), np.float32)
        if lib().oracle_attention_word(C.byref(self.st), _p(M1, _u8p), _p(M2, _u8p), _p(qkv, _f32p), _p(o, _f32p)):
            raise RuntimeError("empty attention row")
        return o

    def attention_dense_f64(self, qkv, score_scale, M1=None, M2=None):
        """softmax(score_scale * q.k) attention in fp64 over the dense masks."""
        if M1 is None:
            M1, M2 = masks(self.H)
        qkv = _c(qkv, np.float64)
        o = np.zeros((self.L, self.d), np.float64)
        if lib().oracle_attention_dense_f64(C.byref(self.st), _p(M1, _u8p), _p(M2, _u8p), _p(qkv, _f64p),
                                            float(score_scale), _p(o, _f64p)):
            raise RuntimeError("empty attention row")
        return o

    def head(self, X, y_word):
        X = _c(X, np.float32)
        y = _c(y_word, np.float32).reshape(-1)
        f = np.zeros(self.n, np.float32)
        bits = np.zeros(self.n, np.uint8)
        z = np.zeros(self.L, np.float32)
        lib().oracle_head_word(C.byref(self.st), _p(X, _f32p), _p(y, _f32p), _p(f, _f32p), _p(bits, _u8p),
                               _p(z, _f32p))
        return f, bits, z


# ---------------------------------------------------------------- free functions

def tree_sum(v) -> np.float32:
    v = _c(v, np.float32)
    return np.float32(lib().oracle_tree_sum(_p(v, _f32p), v.size))


def exp2(x) -> np.float32:
    return np.float32(lib().oracle_exp2(float(np.float32(x))))


def rsqrt(v) -> np.float32:
    return np.float32(lib().oracle_rsqrt(float(np.float32(v))))


def query_scale(dh: int) -> np.float32:
    return np.float32(lib().oracle_query_scale(int(dh)))


def masks(H):
    H = _c(H, np.uint8)
    m, n = H.shape
    L = n + m
    M1 = np.zeros((L, L), np.uint8)
    M2 = np.zeros((L, L), np.uint8)
    lib().oracle_masks(_p(H, _u8p), m, n, _p(M1, _u8p), _p(M2, _u8p))
    return M1, M2


def preprocess(H, y_word):
    H = _c(H, np.uint8)
    m, n = H.shape
    y = _c(y_word, np.float32).reshape(-1)
    t = np.zeros(n + m, np.float32)
    lib().oracle_preprocess(_p(H, _u8p), m, n, _p(y, _f32p), _p(t, _f32p))
    return t


def quant_rows(x):
    x = _c(x, np.float32)
    rows, K = x.shape
    q = np.zeros((rows, K), np.int8)
    r = np.zeros(rows, np.float32)
    lib().oracle_quant_rows(_p(x, _f32p), rows, K, _p(q, _i8p), _p(r, _f32p))
    return q, r


def quant_word(x):
    """Eq. 2 with one alpha over all rows of x (a word): (codes, alpha per row, all equal)."""
    x = _c(x, np.float32)
    rows, K = x.shape
    q = np.zeros((rows, K), np.int8)
    r = np.zeros(rows, np.float32)
    lib().oracle_quant_word(_p(x, _f32p), rows, K, _p(q, _i8p), _p(r, _f32p))
    return q, r


def linear_rows(q, r, T, s, b):
    """AAP linear rows with weight scale s (gamma*delta); the oracle takes fp32(s / 127)."""
    q = _c(q, np.int8)
    r = _c(r, np.float32)
    T = _c(T, np.int8)
    b = _c(b, np.float32)
    rows, K = q.shape
    n_out = T.shape[1]
    out = np.zeros((rows, n_out), np.float32)
    acc = np.zeros((rows, n_out), np.int32)
    sq = np.float32(s) / np.float32(127.0)
    lib().oracle_linear_rows(_p(q, _i8p), _p(r, _f32p), rows, _p(T, _i8p), K, n_out, float(sq),
                             _p(b, _f32p), _p(out, _f32p), _p(acc, _i32p))
    return out, acc


def layernorm_rows(R, g, b, eps=1e-5):
    R = _c(R, np.float32)
    rows, d = R.shape
    out = np.zeros_like(R)
    lib().oracle_layernorm_rows(_p(R, _f32p), rows, d, _p(_c(g, np.float32), _f32p), _p(_c(b, np.float32), _f32p),
                                float(np.float32(eps)), _p(out, _f32p))
    return out


def aap_ternarize(w, p=0.5, delta=1.0, eps=1e-8):
    """AAP import of one fp32 weight matrix (Eq. 1): (ternary int8 of w's shape, scale gamma*delta)."""
    w = _c(w, np.float32)
    t = np.zeros(w.shape, np.int8)
    sc = np.zeros(1, np.float32)
    rc = lib().oracle_aap_ternarize(_p(w, _f32p), w.size, float(np.float32(p)), float(np.float32(delta)),
                                    float(np.float32(eps)), _p(t, _i8p), _p(sc, _f32p))
    if rc:
        raise ValueError("oracle_aap_ternarize: invalid arguments")
    return t, sc[0]
