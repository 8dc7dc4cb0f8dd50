"""Seeded random AECCT weights with the shapes of the inference model.

Shapes follow the encoder of Section 4: per layer six in-block linear maps
(query, key, value, attention output, FFN in, FFN out) whose weights are ternary
{-1, 0, +1} with one fp32 scale per matrix (Section 4.1, Eq. 1 and Eq. 3), fp32
biases, two LayerNorms (Post-LN, Section 6), a per-position embedding table of the
2n-k input scalars (Section 3), and the two output projections W_{d->1} and W_o.
The values are random: trained weights are not available, and throughput does not
depend on them.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

#: order of the six in-block linear maps, used by every array indexed by "kind"
LINEAR_KINDS = ("q", "k", "v", "o", "ff1", "ff2")


@dataclass
class ModelWeights:
    n: int                 # code length
    m: int                 # parity checks (rows of H)
    d: int                 # model width
    n_layers: int
    heads: int
    first_ring_heads: int
    d_ff: int
    ln_eps: float
    embed: np.ndarray      # [L, d] fp32
    pos: np.ndarray | None  # [L, d] fp32 fixed positional table or None
    w: dict                # kind -> int8 [N, in, out] in {-1,0,1}
    scale: np.ndarray      # [N, 6] fp32, per-matrix weight scale (gamma * delta)
    b: dict                # kind -> fp32 [N, out]
    ln1_g: np.ndarray      # [N, d]
    ln1_b: np.ndarray
    ln2_g: np.ndarray
    ln2_b: np.ndarray
    head_w1: np.ndarray    # [d]
    head_b1: float
    head_wo: np.ndarray    # [L, n]
    head_bo: np.ndarray    # [n]
    extra: dict = field(default_factory=dict)
    attention: str = "hpsa"   # "hpsa": heads split over the two rings; "casa": every head over both
    act_scale: str = "token"  # Eq. 2 scale alpha per "token" (row) or per "word" (all of its tokens)

    @property
    def L(self) -> int:
        return self.n + self.m

    def linear_shape(self, kind: str) -> tuple[int, int]:
        if kind == "ff1":
            return self.d, self.d_ff
        if kind == "ff2":
            return self.d_ff, self.d
        return self.d, self.d


def random_weights(n: int, m: int, d: int, n_layers: int, heads: int = 8, *, p_zero: float = 0.5,
                   seed: int = 0, first_ring_heads: int | None = None, d_ff: int | None = None,
                   ln_eps: float = 1e-5, with_pos: bool = False, zero_linear: bool = False,
                   attention: str = "hpsa", act_scale: str = "token") -> ModelWeights:
    """Draw a model.  Ternary entries are i.i.d. with P(0) = p_zero, P(+1) = P(-1) = (1-p_zero)/2,
    every weight scale is fp32(1/sqrt(d)), embeddings are N(0,1), biases and LayerNorm offsets
    N(0, 0.1^2), LayerNorm gains 1 + N(0, 0.1^2), W_{d->1} ~ N(0, 1/d), W_o ~ N(0, 1/L).

    The draw order is fixed (embedding, then per kind the ternary tensors, biases, then the
    LayerNorm and head parameters) so that a seed names one model.
    """
    rng = np.random.default_rng(seed)
    L = n + m
    hf = heads // 2 if first_ring_heads is None else first_ring_heads
    dff = 4 * d if d_ff is None else d_ff
    embed = rng.standard_normal((L, d)).astype(np.float32)
    pos = rng.standard_normal((L, d)).astype(np.float32) * np.float32(0.5) if with_pos else None
    w, b = {}, {}
    pm = (1.0 - p_zero) / 2.0
    for kind in LINEAR_KINDS:
        kin, kout = (d, dff) if kind == "ff1" else (dff, d) if kind == "ff2" else (d, d)
        t = rng.choice(np.array([-1, 0, 1], dtype=np.int8), size=(n_layers, kin, kout), p=[pm, p_zero, pm])
        w[kind] = np.zeros_like(t) if zero_linear else t
        b[kind] = (rng.standard_normal((n_layers, kout)) * 0.1).astype(np.float32)
    scale = np.full((n_layers, 6), np.float32(1.0 / np.sqrt(d)), dtype=np.float32)
    ln1_g = (1.0 + 0.1 * rng.standard_normal((n_layers, d))).astype(np.float32)
    ln1_b = (0.1 * rng.standard_normal((n_layers, d))).astype(np.float32)
    ln2_g = (1.0 + 0.1 * rng.standard_normal((n_layers, d))).astype(np.float32)
    ln2_b = (0.1 * rng.standard_normal((n_layers, d))).astype(np.float32)
    head_w1 = (rng.standard_normal(d) / np.sqrt(d)).astype(np.float32)
    head_b1 = float(np.float32(0.1 * rng.standard_normal()))
    head_wo = (rng.standard_normal((L, n)) / np.sqrt(L)).astype(np.float32)
    head_bo = (0.1 * rng.standard_normal(n)).astype(np.float32)
    return ModelWeights(n=n, m=m, d=d, n_layers=n_layers, heads=heads, first_ring_heads=hf, d_ff=dff,
                        ln_eps=ln_eps, embed=embed, pos=pos, w=w, scale=scale, b=b,
                        ln1_g=ln1_g, ln1_b=ln1_b, ln2_g=ln2_g, ln2_b=ln2_b,
                        head_w1=head_w1, head_b1=head_b1, head_wo=head_wo, head_bo=head_bo,
                        attention=attention, act_scale=act_scale)


def random_spe_params(L: int, d_pe: int, heads: int, *, seed: int = 0) -> dict:
    """Seeded parameters of the spectral positional encoding network (Section 4.3), fp32.

    W_{2->d_PE} ~ N(0, 1); the attention's W_q, W_k, W_v, W_o ~ N(0, 1/d_PE), all stored
    [in][out]; biases N(0, 0.1^2); the reduction over the L eigen-rows w_red ~ N(0, 1/L) with
    bias b_red ~ N(0, 0.1^2).  Random: trained parameters are not available.
    """
    rng = np.random.default_rng(seed)
    f = lambda a: np.ascontiguousarray(a, dtype=np.float32)
    p = {"d_pe": int(d_pe), "heads": int(heads),
         "w_in": f(rng.standard_normal((2, d_pe))), "b_in": f(0.1 * rng.standard_normal(d_pe))}
    for name in ("q", "k", "v", "o"):
        p["w_" + name] = f(rng.standard_normal((d_pe, d_pe)) / np.sqrt(d_pe))
        p["b_" + name] = f(0.1 * rng.standard_normal(d_pe))
    p["w_red"] = f(rng.standard_normal(L) / np.sqrt(L))
    p["b_red"] = float(np.float32(0.1 * rng.standard_normal()))
    return p


def with_positional_table(w: ModelWeights, table: np.ndarray, d_pe: int) -> ModelWeights:
    """The model with `table` as its positional table and the last d_pe embedding columns zeroed,
    so that the embedded token is the concatenation of the scaled embedding and the table row."""
    from dataclasses import replace
    embed = w.embed.copy()
    embed[:, w.d - d_pe:] = 0.0
    return replace(w, embed=embed, pos=np.ascontiguousarray(table, dtype=np.float32))


def random_qat_params(n: int, m: int, d: int, n_layers: int, *, seed: int = 0, d_ff: int | None = None,
                      latent_std: float | None = None, delta_spread: float = 0.05) -> dict:
    """Seeded parameters of the quantisation-aware training phase (Section 6): latent fp32 weights
    of the six in-block maps per layer ~ N(0, latent_std^2) (default latent_std = 1/sqrt(d), so that
    Eq. 1's scale gamma*delta, about 0.67/sqrt(d), is of the size of the inference weights' scale),
    the learnable factors delta
    = 1 + N(0, delta_spread^2) (the paper initialises them to one), and the other parameters drawn
    as in random_weights.  fp32 arrays in a dict: embed, pos (None), w[kind], delta [N, 6],
    b[kind], ln1_g, ln1_b, ln2_g, ln2_b, head_w1, head_b1, head_wo, head_bo."""
    rng = np.random.default_rng(seed)
    L = n + m
    dff = 4 * d if d_ff is None else d_ff
    sd = (1.0 / np.sqrt(d)) if latent_std is None else latent_std
    f = lambda a: np.ascontiguousarray(a, dtype=np.float32)
    p = {"embed": f(rng.standard_normal((L, d))), "pos": None, "w": {}, "b": {}}
    for kind in LINEAR_KINDS:
        kin, kout = (d, dff) if kind == "ff1" else (dff, d) if kind == "ff2" else (d, d)
        p["w"][kind] = f(rng.standard_normal((n_layers, kin, kout)) * sd)
        p["b"][kind] = f(0.1 * rng.standard_normal((n_layers, kout)))
    p["delta"] = f(1.0 + delta_spread * rng.standard_normal((n_layers, 6)))
    p["ln1_g"] = f(1.0 + 0.1 * rng.standard_normal((n_layers, d)))
    p["ln1_b"] = f(0.1 * rng.standard_normal((n_layers, d)))
    p["ln2_g"] = f(1.0 + 0.1 * rng.standard_normal((n_layers, d)))
    p["ln2_b"] = f(0.1 * rng.standard_normal((n_layers, d)))
    p["head_w1"] = f(rng.standard_normal(d) / np.sqrt(d))
    p["head_b1"] = float(np.float32(0.1 * rng.standard_normal()))
    p["head_wo"] = f(rng.standard_normal((L, n)) / np.sqrt(L))
    p["head_bo"] = f(0.1 * rng.standard_normal(n))
    return p
