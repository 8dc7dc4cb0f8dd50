"""GPU parity: the HIP path against the CPU oracle, through the C ABI.

Every floating-point value is compared bit for bit: both sides follow the same
evaluation order (pairwise feature sums, ascending neighbour and token sums, the same
exp), so the required tolerance (1e-3 on logits, identical bits where |logit| > 1e-3)
is met with margin 0.  Integer work (syndromes, int8 codes, int32 accumulators) is
compared exactly.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from workloads import CONFIGS, build_workload  # noqa: E402

LOGIT_TOL = 1e-3


@pytest.fixture(scope="module")
def P():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2410_05911_amd as P
    P.lib()
    return P


_cache = {}


def _setup(P, c, batch, path):
    key = (c, batch, path)
    if key not in _cache:
        cfg, H, G, w, y, x = build_workload(c, batch=batch)
        dec = P.Decoder(H, w, path=path)
        _cache[key] = (cfg, H, G, w, y, x, dec)
    return _cache[key]


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _np(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def _assert_logits(f_gpu, f_ref, bits_gpu, bits_ref, y):
    """Bit-exact expectation, with the tolerance rule checked explicitly as well."""
    diff = np.abs(f_gpu.astype(np.float64) - f_ref.astype(np.float64))
    assert diff.max() <= LOGIT_TOL, diff.max()
    sure = np.abs(f_ref) > LOGIT_TOL
    assert (bits_gpu[sure] == bits_ref[sure]).all()
    nbad = int((f_gpu != f_ref).sum())
    assert nbad == 0, f"{nbad} logits differ (max |diff| {diff.max():.3g})"
    assert (bits_gpu == bits_ref).all()


# ------------------------------------------------------------------------------ ternary GEMM
@pytest.mark.parametrize("c", [1, 2, 3, 4, 5])
def test_ternary_gemm_teacher_forced(P, c):
    """int8 x ternary accumulators (Eq. 3) exactly equal an int64 matmul, for every map,
    with a ragged number of rows (not a multiple of the 16-row MFMA tile)."""
    print(f"[gemm] config {c}", flush=True)
    cfg, H, G, w, y, x, dec = _setup(P, c, 4, P.PATH_LAYERED)
    rng = np.random.default_rng(100 + c)
    rows = 16 * 37 + 5
    for layer in sorted({0, w.n_layers - 1}):
        for kind, name in enumerate(("q", "k", "v", "o", "ff1", "ff2")):
            T = w.w[name][layer]
            a = rng.integers(-127, 128, (rows, T.shape[0])).astype(np.int8)
            a[3] = 127
            a[4] = -127
            acc = _np(dec.ternary_gemm(layer, kind, _dev(a)))
            ref = a.astype(np.int64) @ T.astype(np.int64)
            assert (acc == ref).all(), (layer, name)
    assert _np(dec.ternary_gemm(0, 0, _dev(np.zeros((0, w.d), np.int8)))).shape == (0, w.d)


# ------------------------------------------------------------------------------ stages
def _oracle_taps(om, ys):
    taps = []
    for yw in ys:
        bits, f, t = om.decode_taps(yw)
        t["bits"], t["f"] = bits, f
        taps.append(t)
    return {k: np.stack([t[k] for t in taps]) for k in taps[0]}


@pytest.mark.parametrize("c,words", [(1, 5), (2, 3), (3, 2), (4, 1), (5, 1)])
def test_stages_teacher_forced(P, oracle_mod, c, words):
    """Each layered-path stage, fed the oracle's own inputs for that stage, reproduces the
    oracle's outputs bit for bit (fp32 values, int8 codes and per-row scales)."""
    print(f"[stages] config {c} words {words}", flush=True)
    cfg, H, G, w, y, x, dec = _setup(P, c, 8, P.PATH_LAYERED)
    om = oracle_mod.OracleModel(H, w)
    ys = y[:words]
    T = _oracle_taps(om, ys)
    L, d, N = om.L, w.d, w.n_layers

    def rows(a):          # [words, N?, L, ...] per-layer slice -> [words*L, ...]
        return np.ascontiguousarray(a.reshape((words * L,) + a.shape[2:]))

    xg, xqg, axg = dec.stage_embed(_dev(ys))
    assert (_np(xg) == rows(T["x_in"][:, 0])).all()
    assert (_np(xqg) == rows(T["xq"][:, 0])).all()
    assert (_np(axg) == rows(T["ax"][:, 0])).all()
    for l in range(N):
        qkv = dec.stage_qkv(l, _dev(rows(T["xq"][:, l])), _dev(rows(T["ax"][:, l])))
        assert (_np(qkv) == rows(T["qkv"][:, l])).all(), ("qkv", l)
        o, oq, ao = dec.stage_attention(_dev(rows(T["qkv"][:, l])))
        assert (_np(o) == rows(T["o"][:, l])).all(), ("o", l)
        assert (_np(oq) == rows(T["oq"][:, l])).all(), ("oq", l)
        assert (_np(ao) == rows(T["ao"][:, l])).all(), ("ao", l)
        x1, x1q, a1 = dec.stage_oproj_ln(l, _dev(rows(T["oq"][:, l])), _dev(rows(T["ao"][:, l])),
                                         _dev(rows(T["x_in"][:, l])))
        assert (_np(x1) == rows(T["x1"][:, l])).all(), ("x1", l)
        assert (_np(x1q) == rows(T["x1q"][:, l])).all(), ("x1q", l)
        assert (_np(a1) == rows(T["a1"][:, l])).all(), ("a1", l)
        gq, ag = dec.stage_ffn1(l, _dev(rows(T["x1q"][:, l])), _dev(rows(T["a1"][:, l])))
        assert (_np(gq) == rows(T["gq"][:, l])).all(), ("gq", l)
        assert (_np(ag) == rows(T["ag"][:, l])).all(), ("ag", l)
        xo, xoq, axo = dec.stage_ffn2_ln(l, _dev(rows(T["gq"][:, l])), _dev(rows(T["ag"][:, l])),
                                         _dev(rows(T["x1"][:, l])))
        assert (_np(xo) == rows(T["x_out"][:, l])).all(), ("x_out", l)
        if l + 1 < N:
            assert (_np(xoq) == rows(T["xq"][:, l + 1])).all(), ("xq", l + 1)
            assert (_np(axo) == rows(T["ax"][:, l + 1])).all(), ("ax", l + 1)
    bits, logits = dec.stage_head(_dev(rows(T["x_out"][:, N - 1])), _dev(ys))
    assert (_np(logits) == T["f"]).all()
    assert (_np(bits) == T["bits"]).all()


# ------------------------------------------------------------------------------ end to end
# oracle sample sizes per workload (whole words the CPU oracle decodes in seconds), spread over
# the batch: every persistent block's share and every workspace chunk of the layered path
_SAMPLE = {1: 1024, 2: 768, 3: 96, 4: 64, 5: 32}


@pytest.mark.parametrize("c", [1, 2, 3, 4, 5])
def test_decode_full_batch_against_oracle(P, oracle_mod, c):
    """Full configured batch through aecct_decode; the oracle recomputes a spread sample of
    the words (all of them for Hamming(7,4))."""
    cfg = CONFIGS[c]
    print(f"[e2e] config {c} batch {cfg.batch}", flush=True)
    cfg, H, G, w, y, x, dec = _setup(P, c, cfg.batch, P.PATH_AUTO)
    bits, logits = dec.decode(_dev(y))
    bits, logits = _np(bits), _np(logits)
    k = min(_SAMPLE[c], cfg.batch)
    idx = np.unique(np.linspace(0, cfg.batch - 1, k).astype(np.int64))
    om = oracle_mod.OracleModel(H, w)
    bo, fo = om.decode(y[idx], n_threads=16)
    _assert_logits(logits[idx], fo, bits[idx], bo, y[idx])


@pytest.mark.parametrize("c", [1, 2, 3])
def test_decode_edge_batches(P, oracle_mod, c):
    """batch 0 (no-op), 1, and ragged batches; per-word results do not depend on the batch."""
    print(f"[edge] config {c}", flush=True)
    cfg, H, G, w, y, x, dec = _setup(P, c, 67, P.PATH_AUTO)
    om = oracle_mod.OracleModel(H, w)
    bo, fo = om.decode(y, n_threads=16)
    for B in (1, 2, 3, 17, 67):
        bits, logits = dec.decode(_dev(y[:B]))
        _assert_logits(_np(logits), fo[:B], _np(bits), bo[:B], y[:B])
    e = torch.empty((0, cfg.n), dtype=torch.float32, device="cuda")
    b0, l0 = dec.decode(e)
    assert b0.shape == (0, cfg.n)
    # noiseless all-zero codeword: |y| = 1 and zero syndrome; y = -0.0 counts as bit 0
    z = np.ones((2, cfg.n), np.float32)
    z[1] = -0.0
    bits, logits = dec.decode(_dev(z))
    bo, fo = om.decode(z)
    _assert_logits(_np(logits), fo, _np(bits), bo, z)


def test_workspace_too_small_and_bad_args(P):
    cfg, H, G, w, y, x, dec = _setup(P, 3, 4, P.PATH_LAYERED)
    yd = _dev(y)
    need = dec.workspace_size(4)
    assert need > 0
    ws = torch.empty(need - 1, dtype=torch.uint8, device="cuda")
    with pytest.raises(P.AecctError) as ei:
        dec.decode(yd, workspace=ws)
    assert ei.value.status == P.ERR_WORKSPACE_TOO_SMALL
    with pytest.raises(P.AecctError) as ei:
        dec.stage_qkv(w.n_layers, torch.zeros((dec.L * 4, w.d), dtype=torch.int8, device="cuda"),
                      torch.zeros(dec.L * 4, device="cuda"))
    assert ei.value.status == P.ERR_INVALID_ARG


def test_deterministic_and_stream(P):
    cfg, H, G, w, y, x, dec = _setup(P, 2, 2048, P.PATH_AUTO)
    yd = _dev(y)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        b1, l1 = dec.decode(yd, stream=s)
    s.synchronize()
    b2, l2 = dec.decode(yd)
    assert torch.equal(l1, l2) and torch.equal(b1, b2)


# ------------------------------------------------------------------------------ fused path
@pytest.mark.parametrize("c", [1, 2])
def test_fused_and_layered_paths_agree(P, c):
    """The single-launch fused kernel and the per-stage layered kernels give identical bits
    and logits (same evaluation order), on a ragged batch."""
    print(f"[paths] config {c}", flush=True)
    cfg, H, G, w, y, x = build_workload(c, batch=4099)
    fused = P.Decoder(H, w, path=P.PATH_FUSED)
    layered = P.Decoder(H, w, path=P.PATH_LAYERED)
    assert fused.path == P.PATH_FUSED and layered.path == P.PATH_LAYERED
    assert P.Decoder(H, w).path == P.PATH_FUSED       # the automatic choice takes the fused kernel
    yd = _dev(y)
    bf, lf = fused.decode(yd)
    bl, ll = layered.decode(yd)
    assert torch.equal(lf, ll) and torch.equal(bf, bl)


@pytest.mark.parametrize("hf,with_pos", [(2, False), (6, True), (0, False), (8, True)])
def test_fused_head_split_and_positional_table(P, oracle_mod, hf, with_pos):
    """Other first/second-ring head splits (Table 4 of the paper ablates 2/6, 4/4, 6/2) and
    a fixed positional table (the inference form of the spectral encoding) on BCH(31,16)."""
    from workloads import random_weights
    from workloads.configs import parity_check
    from workloads.channel import awgn_words
    from workloads.codes import generator_from_parity
    print(f"[variants] hf {hf} pos {with_pos}", flush=True)
    H = parity_check(CONFIGS[2])
    m, n = H.shape
    w = random_weights(n, m, 32, 3, 8, seed=40 + hf, first_ring_heads=hf, with_pos=with_pos)
    y, x, _ = awgn_words(generator_from_parity(H), 333, (3.0, 5.0), seed=7)
    om = oracle_mod.OracleModel(H, w)
    bo, fo = om.decode(y, n_threads=16)
    for path in (P.PATH_FUSED, P.PATH_LAYERED):
        dec = P.Decoder(H, w, path=path)
        bits, logits = dec.decode(_dev(y))
        _assert_logits(_np(logits), fo, _np(bits), bo, y)


@pytest.mark.parametrize("hf", [2, 6])
def test_fused_with_fewer_words_in_flight(P, oracle_mod, hf):
    """BCH(31,16), 6 layers, with a head group that mixes both rings: its neighbour tables are
    padded to the group's longest list and leave LDS for 11 words per block instead of 12; the
    automatic choice must still be the fused kernel, run with fewer wavefronts."""
    from workloads import build_workload
    print(f"[waves] hf {hf}", flush=True)
    cfg, H, G, w, y, x = build_workload(2, batch=517, first_ring_heads=hf)
    om = oracle_mod.OracleModel(H, w)
    bo, fo = om.decode(y, n_threads=16)
    dec = P.Decoder(H, w)
    assert dec.path == P.PATH_FUSED
    bits, logits = dec.decode(_dev(y))
    _assert_logits(_np(logits), fo, _np(bits), bo, y)


@pytest.mark.parametrize("d", [32, 64])
@pytest.mark.parametrize("regime", ["mixed", "overflow", "underflow", "zero_values"])
def test_softmax_shifted_rows(P, oracle_mod, regime, d):
    """Attention rows whose unshifted weight sum leaves [2^-64, 2^64] take the max-shifted
    form on every path (d = 32: fused and layered; d = 64: the layered projection + attention
    kernel): query/key scales blown up (scores of hundreds: about 5 % of the rows, or nearly
    all, overflow), or query and key biases of opposite sign (every score far below -64).
    "zero_values": a zero value map makes every attention output row 0, so its Eq. 2 scale is 0
    (codes 0, dequantisation scale 0)."""
    from workloads import random_weights
    from workloads.configs import parity_check
    from workloads.channel import awgn_words
    from workloads.codes import generator_from_parity
    print(f"[softmax] regime {regime} d {d}", flush=True)
    H = parity_check(CONFIGS[2])
    m, n = H.shape
    w = random_weights(n, m, d, 2, 8, seed=77)
    if regime == "mixed":
        w.scale[:, 0:2] *= np.float32(5.0)
    elif regime == "overflow":
        w.scale[:, 0:2] *= np.float32(40.0)
    elif regime == "underflow":
        w.b["q"][:] = np.float32(6.0)
        w.b["k"][:] = np.float32(-6.0)
    else:
        w.scale[:, 2] = np.float32(0.0)
        w.b["v"][:] = np.float32(0.0)
    y, x, _ = awgn_words(generator_from_parity(H), 129, (3.0, 5.0), seed=8)
    om = oracle_mod.OracleModel(H, w)
    bo, fo = om.decode(y, n_threads=16)
    assert np.isfinite(fo).all()
    for path in ((P.PATH_FUSED, P.PATH_LAYERED) if d == 32 else (P.PATH_LAYERED,)):
        dec = P.Decoder(H, w, path=path)
        bits, logits = dec.decode(_dev(y))
        _assert_logits(_np(logits), fo, _np(bits), bo, y)


def test_decode_with_aap_imported_weights(P, oracle_mod):
    """A model whose six in-block maps come from fp32 matrices through the library's AAP import
    (Eq. 1) decodes like the oracle model whose maps come from the oracle's import."""
    import copy
    from workloads import random_weights
    from workloads.configs import parity_check
    from workloads.channel import awgn_words
    from workloads.codes import generator_from_parity
    H = parity_check(CONFIGS[2])
    m, n = H.shape
    base = random_weights(n, m, 32, 2, 8, seed=91)
    rng = np.random.default_rng(92)
    w_lib, w_orc = copy.deepcopy(base), copy.deepcopy(base)
    for kind_i, kind in enumerate(("q", "k", "v", "o", "ff1", "ff2")):
        for layer in range(base.n_layers):
            W = rng.standard_normal(base.w[kind][layer].shape).astype(np.float32) * 0.05
            delta = np.float32(1.0 + 0.1 * layer + 0.05 * kind_i)
            t_l, s_l = P.aap_ternarize(W, 0.5, delta, 1e-8)
            t_o, s_o = oracle_mod.aap_ternarize(W, p=0.5, delta=delta, eps=1e-8)
            w_lib.w[kind][layer], w_lib.scale[layer, kind_i] = t_l, s_l
            w_orc.w[kind][layer], w_orc.scale[layer, kind_i] = t_o, s_o
    y, x, _ = awgn_words(generator_from_parity(H), 200, (3.0, 5.0), seed=93)
    bo, fo = oracle_mod.OracleModel(H, w_orc).decode(y, n_threads=16)
    for path in (P.PATH_FUSED, P.PATH_LAYERED):
        bits, logits = P.Decoder(H, w_lib, path=path).decode(_dev(y))
        _assert_logits(_np(logits), fo, _np(bits), bo, y)


@pytest.mark.parametrize("c", [1, 2, 3])
def test_casa_decode_against_oracle(P, oracle_mod, c):
    """The CASA variant (Section 3: the ECCT mask on every head) on every path that takes the
    shape, against the oracle on a sample of a ragged batch."""
    print(f"[casa] config {c}", flush=True)
    cfg, H, G, w, y, x = build_workload(c, batch=1027, attention="casa")
    k = {1: 1027, 2: 256, 3: 24}[c]
    idx = np.unique(np.linspace(0, 1026, k).astype(np.int64))
    bo, fo = oracle_mod.OracleModel(H, w).decode(y[idx], n_threads=16)
    paths = (P.PATH_FUSED, P.PATH_LAYERED) if c in (1, 2) else (P.PATH_LAYERED,)
    for path in paths:
        dec = P.Decoder(H, w, path=path)
        assert dec.info.attention == P.ATTN_CASA and dec.path == path
        bits, logits = dec.decode(_dev(y))
        _assert_logits(_np(logits)[idx], fo, _np(bits)[idx], bo, y[idx])


def _random_parity_check(m, n, seed, col_weight=3):
    """A random 0/1 parity-check matrix with no empty row or column (not a designed code)."""
    rng = np.random.default_rng(seed)
    H = np.zeros((m, n), np.uint8)
    for i in range(n):
        H[rng.choice(m, size=col_weight, replace=False), i] = 1
    for j in range(m):
        if not H[j].any():
            H[j, rng.integers(n)] = 1
    return H


@pytest.mark.parametrize("d,m,n,hf,attention", [(64, 21, 47, 4, "hpsa"), (64, 13, 30, 2, "hpsa"),
                                                 (128, 25, 51, 4, "hpsa"), (128, 9, 20, 6, "casa"),
                                                 (64, 40, 90, 0, "hpsa"), (128, 37, 70, 8, "hpsa"),
                                                 (64, 100, 201, 4, "hpsa"), (64, 131, 263, 2, "casa"),
                                                 (128, 150, 299, 4, "hpsa"), (128, 200, 401, 4, "hpsa"),
                                                 (128, 255, 510, 6, "hpsa")])
def test_layered_wide_models_odd_token_counts(P, oracle_mod, d, m, n, hf, attention):
    """d = 64 and 128 on token counts L = n + m that are not multiples of 16 (partial token
    tiles in the fused projection/attention kernels), several head splits and CASA.  Words of up
    to 256 (d = 64) or 512 (d = 128) tokens keep keys and values in LDS as fp32 (at d = 128 up to
    384 tokens with O written as Eq. 2 codes, one row per lane pair, and L = 449 with fp32 O and
    a second row on some lane pairs); the longer ones
    (L = 301, 394, 601, 765) as int16 accumulators, or (d = 128 with head partitioning) one node
    type's rows at a time with the other type's keys and values in LDS as fp32, whose token tiles
    straddle the variable/check boundary when n is not a multiple of 16."""
    from workloads import random_weights
    print(f"[wide] d {d} m {m} n {n} hf {hf} {attention}", flush=True)
    H = _random_parity_check(m, n, seed=m * 131 + n)
    w = random_weights(n, m, d, 2, 8, seed=d + m + n, first_ring_heads=hf, attention=attention)
    rng = np.random.default_rng(5)
    y = (1.0 - 2.0 * rng.integers(0, 2, (37, n)) + 0.6 * rng.standard_normal((37, n))).astype(np.float32)
    bo, fo = oracle_mod.OracleModel(H, w).decode(y, n_threads=16)
    dec = P.Decoder(H, w)
    assert dec.path == P.PATH_LAYERED
    long_word = m + n > (256 if d == 64 else 512)
    split = d == 128 and attention == "hpsa"
    assert dec.info.layered_attention == (P.LAYERED_ATTN_LDS_I16 if long_word else P.LAYERED_ATTN_LDS_F32)
    bits, logits = dec.decode(_dev(y))
    _assert_logits(_np(logits), fo, _np(bits), bo, y)
    if long_word and split:                  # rows one node type at a time on the same words
        dec = P.Decoder(H, w, layered_attention=P.LAYERED_ATTN_LDS_SPLIT)
        bits, logits = dec.decode(_dev(y))
        _assert_logits(_np(logits), fo, _np(bits), bo, y)


@pytest.mark.parametrize("d,with_pos", [(64, False), (64, True), (128, False), (128, True)])
def test_layered_single_layer(P, oracle_mod, d, with_pos):
    """One layer: its token block is both the first (X rebuilt from t_i and the embedding rows, with
    or without a positional table) and the last (the head's z per token instead of X)."""
    from workloads import random_weights
    print(f"[one layer] d {d} pos {with_pos}", flush=True)
    m, n = 30, 61
    H = _random_parity_check(m, n, seed=5 * d + int(with_pos))
    w = random_weights(n, m, d, 1, 8, seed=d + 3, with_pos=with_pos)
    rng = np.random.default_rng(13)
    y = (1.0 - 2.0 * rng.integers(0, 2, (300, n)) + 0.6 * rng.standard_normal((300, n))).astype(np.float32)
    idx = np.unique(np.linspace(0, 299, 40).astype(np.int64))
    bo, fo = oracle_mod.OracleModel(H, w).decode(y[idx], n_threads=16)
    dec = P.Decoder(H, w)
    assert dec.path == P.PATH_LAYERED
    bits, logits = dec.decode(_dev(y))
    _assert_logits(_np(logits)[idx], fo, _np(bits)[idx], bo, y[idx])


@pytest.mark.parametrize("m,n,hf,words", [(25, 51, 8, 37), (40, 90, 5, 300), (60, 121, 11, 9)])
def test_layered_d128_sixteen_heads(P, oracle_mod, m, n, hf, words):
    """d = 128 with sixteen 8-dimension heads (two per head group): the fused projection +
    attention with one row per thread, its neighbour lists staged in LDS and the next word's tiles
    read during the last group's rows; several words per block (300 words) so the read-ahead
    crosses word boundaries, and first-ring head counts that split a group between the rings."""
    from workloads import random_weights
    print(f"[d128 h16] m {m} n {n} hf {hf} words {words}", flush=True)
    H = _random_parity_check(m, n, seed=3 * m + n)
    w = random_weights(n, m, 128, 2, 16, seed=m + 7 * n, first_ring_heads=hf)
    rng = np.random.default_rng(11)
    y = (1.0 - 2.0 * rng.integers(0, 2, (words, n)) + 0.6 * rng.standard_normal((words, n))).astype(np.float32)
    k = min(words, 40)
    idx = np.unique(np.linspace(0, words - 1, k).astype(np.int64))
    bo, fo = oracle_mod.OracleModel(H, w).decode(y[idx], n_threads=16)
    dec = P.Decoder(H, w)
    assert dec.path == P.PATH_LAYERED and dec.info.layered_attention == P.LAYERED_ATTN_LDS_F32
    bits, logits = dec.decode(_dev(y))
    _assert_logits(_np(logits)[idx], fo, _np(bits)[idx], bo, y[idx])


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("regime", ["mixed", "underflow", "zero_values"])
def test_long_words_shifted_softmax(P, oracle_mod, regime, d):
    """The long-word forms (L = 601: int16 values, and at d = 128 rows one node type at a time) with
    rows that take the max-shifted softmax (some or all), and with a zero value map (O = 0, Eq. 2
    scale 0)."""
    from workloads import random_weights
    print(f"[long softmax] d {d} {regime}", flush=True)
    m, n = 200, 401
    H = _random_parity_check(m, n, seed=17)
    w = random_weights(n, m, d, 2, 8, seed=23)
    if regime == "mixed":
        w.scale[:, 0:2] *= np.float32(5.0)
    elif regime == "underflow":
        w.b["q"][:] = np.float32(6.0)
        w.b["k"][:] = np.float32(-6.0)
    else:
        w.scale[:, 2] = np.float32(0.0)
        w.b["v"][:] = np.float32(0.0)
    rng = np.random.default_rng(6)
    y = (1.0 - 2.0 * rng.integers(0, 2, (21, n)) + 0.6 * rng.standard_normal((21, n))).astype(np.float32)
    bo, fo = oracle_mod.OracleModel(H, w).decode(y, n_threads=16)
    assert np.isfinite(fo).all()
    dec = P.Decoder(H, w)
    assert dec.info.layered_attention == P.LAYERED_ATTN_LDS_I16
    bits, logits = dec.decode(_dev(y))
    _assert_logits(_np(logits), fo, _np(bits), bo, y)
    if d == 128:
        dec = P.Decoder(H, w, layered_attention=P.LAYERED_ATTN_LDS_SPLIT)
        bits, logits = dec.decode(_dev(y))
        _assert_logits(_np(logits), fo, _np(bits), bo, y)


@pytest.mark.parametrize("regime", ["plain", "mixed"])
def test_long_words_int16_keys(P, oracle_mod, regime):
    """d = 128 words of 1700 tokens: too long for fp32 keys beside int16 values in LDS, so keys
    and values both stay int16 accumulators; plain rows and rows that take the max-shifted
    softmax."""
    from workloads import random_weights
    print(f"[long int16 keys] {regime}", flush=True)
    m, n = 567, 1133
    H = _random_parity_check(m, n, seed=41)
    w = random_weights(n, m, 128, 2, 8, seed=43)
    if regime == "mixed":
        w.scale[:, 0:2] *= np.float32(5.0)
    rng = np.random.default_rng(9)
    y = (1.0 - 2.0 * rng.integers(0, 2, (9, n)) + 0.6 * rng.standard_normal((9, n))).astype(np.float32)
    bo, fo = oracle_mod.OracleModel(H, w).decode(y, n_threads=16)
    dec = P.Decoder(H, w)
    assert dec.info.layered_attention == P.LAYERED_ATTN_LDS_I16
    bits, logits = dec.decode(_dev(y))
    _assert_logits(_np(logits), fo, _np(bits), bo, y)


def test_layered_attention_forms_of_the_workloads(P):
    """LDPC(128,64) and LDPC(256,128) run keys and values in LDS as fp32, LDPC(1024,512) (1536
    tokens) as int16 accumulators."""
    for c, form in ((3, P.LAYERED_ATTN_LDS_F32), (4, P.LAYERED_ATTN_LDS_F32), (5, P.LAYERED_ATTN_LDS_I16)):
        cfg, H, G, w, y, x, dec = _setup(P, c, 4, P.PATH_LAYERED)
        assert dec.info.layered_attention == form, c
        print(f"[forms] config {c}: device {dec.info.device}, {dec.info.compute_units} CUs, "
              f"{dec.info.lds_bytes} LDS bytes per workgroup", flush=True)
        assert dec.info.compute_units > 0 and dec.info.lds_bytes >= 64 * 1024


@pytest.mark.parametrize("c", [3, 4, 5])
def test_layered_attention_forms_agree_on_the_whole_batch(P, c):
    """The full configured batch through every Q/K/V + attention form the shape allows: the
    production kernels (fp32 K and V in LDS with lane pairs on LDPC(256,128), fp32 keys beside
    int16 values on LDPC(1024,512)), the int16 forms, the node-type split (one node type's rows at
    a time, that type's keys and values in LDS as fp32), and the unfused GEMM + attention kernels
    that the stage entry points run; all bit-identical."""
    cfg = CONFIGS[c]
    print(f"[forms e2e] config {c} batch {cfg.batch}", flush=True)
    cfg, H, G, w, y, x = build_workload(c)
    yd = _dev(y)
    ref = None
    forms = {3: (P.LAYERED_ATTN_AUTO, P.LAYERED_ATTN_LDS_I16, P.LAYERED_ATTN_UNFUSED),
             4: (P.LAYERED_ATTN_AUTO, P.LAYERED_ATTN_LDS_I16, P.LAYERED_ATTN_LDS_SPLIT, P.LAYERED_ATTN_UNFUSED),
             5: (P.LAYERED_ATTN_AUTO, P.LAYERED_ATTN_LDS_SPLIT, P.LAYERED_ATTN_UNFUSED)}[c]
    for form in forms:
        dec = P.Decoder(H, w, layered_attention=form)
        if form != P.LAYERED_ATTN_AUTO:
            assert dec.info.layered_attention == form
        bits, logits = dec.decode(yd)
        torch.cuda.synchronize()
        if ref is None:
            ref = (bits, logits)
        else:
            nb = int((logits != ref[1]).sum())
            assert nb == 0 and torch.equal(bits, ref[0]), (form, nb)
        dec.close()
    if c == 5:
        with pytest.raises(P.AecctError) as ei:
            P.Decoder(H, w, layered_attention=P.LAYERED_ATTN_LDS_F32)   # 1536 tokens: no room in LDS
        assert ei.value.status == P.ERR_UNSUPPORTED


@pytest.mark.parametrize("m,n,hf,attention,with_pos", [
    (6, 14, 4, "hpsa", False),     # L = 20: two token tiles
    (9, 23, 2, "hpsa", True),      # L = 32: two full tiles
    (11, 22, 4, "casa", False),    # L = 33: three tiles, one token in the last
    (20, 40, 6, "hpsa", False),    # L = 60: four tiles
    (22, 42, 4, "hpsa", True),     # L = 64: four full tiles, the largest the kernel takes
    (30, 34, 0, "hpsa", False),    # L = 64, n = 34 variables, all heads second-ring
    (3, 5, 8, "hpsa", False),      # L = 8: one partial tile, all heads first-ring
])
def test_fused_kernel_tile_counts(P, oracle_mod, m, n, hf, attention, with_pos):
    """The single-wave kernel at every token-tile count it instantiates (1 to 4 tiles of 16),
    on random parity-check matrices, against the oracle; the layered path must agree too."""
    from workloads import random_weights
    print(f"[tiles] m {m} n {n} hf {hf} {attention} pos {with_pos}", flush=True)
    H = _random_parity_check(m, n, seed=7 * m + n, col_weight=min(3, m))
    w = random_weights(n, m, 32, 3, 8, seed=m + 3 * n, first_ring_heads=hf, attention=attention,
                       with_pos=with_pos)
    rng = np.random.default_rng(m * n)
    y = (1.0 - 2.0 * rng.integers(0, 2, (301, n)) + 0.7 * rng.standard_normal((301, n))).astype(np.float32)
    bo, fo = oracle_mod.OracleModel(H, w).decode(y, n_threads=16)
    fused = P.Decoder(H, w, path=P.PATH_FUSED)
    assert fused.path == P.PATH_FUSED
    for dec in (fused, P.Decoder(H, w, path=P.PATH_LAYERED)):
        bits, logits = dec.decode(_dev(y))
        _assert_logits(_np(logits), fo, _np(bits), bo, y)


def test_device_arithmetic_matches_ieee_definitions(P):
    """The fract/floor split of 2^x, the softmax reciprocal and 127/alpha, computed with gfx950
    instructions, equal their IEEE definitions (the oracle's) on every fp32 operand of the ranges
    the kernels use."""
    fract_floor, recip, inv127 = P.check_device_arith()
    assert (fract_floor, recip, inv127) == (0, 0, 0)


@pytest.mark.parametrize("d,m,n,layers", [(64, 700, 1301, 2), (128, 700, 1301, 1), (64, 1365, 2731, 1)])
def test_layered_unfused_attention_long_words(P, oracle_mod, d, m, n, layers):
    """Words too long for a head group's keys and values in LDS (L = 2001, and L = 4096, the
    largest token count the library accepts): the Q/K/V GEMM, attention rows gathered from device
    memory with Eq. 2 of O on the way out, then the token block reading the int8 codes of O."""
    from workloads import random_weights
    print(f"[unfused long] d {d} L {m + n}", flush=True)
    H = _random_parity_check(m, n, seed=29)
    w = random_weights(n, m, d, layers, 8, seed=31)
    rng = np.random.default_rng(8)
    y = (1.0 - 2.0 * rng.integers(0, 2, (3, n)) + 0.7 * rng.standard_normal((3, n))).astype(np.float32)
    bo, fo = oracle_mod.OracleModel(H, w).decode(y, n_threads=16)
    dec = P.Decoder(H, w)
    assert dec.info.layered_attention == P.LAYERED_ATTN_UNFUSED
    bits, logits = dec.decode(_dev(y))
    _assert_logits(_np(logits), fo, _np(bits), bo, y)
