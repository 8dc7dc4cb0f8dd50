"""aecct_decode_static (no workspace, no allocation: the library's static device scratch)
against aecct_decode through the C ABI, bit for bit, on two calls in a row, the second with a
smaller batch (the scratch keeps the first call's contents)."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from workloads import build_workload  # noqa: E402


@pytest.fixture(scope="module")
def P():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2410_05911_amd as P
    P.lib()
    return P


@pytest.mark.parametrize("c,act_scale,batches", [
    (1, "token", (300, 5)),        # fused path: no scratch at all
    (2, "token", (4099, 17)),      # fused path
    (2, "word", (700, 50)),        # layered, one alpha per word: the extra fp32 regions
    (3, "token", (900, 33)),       # layered, fp32 keys and values in LDS
    (4, "token", (500, 17)),       # layered: the 256 MiB array takes about 190 words per chunk
    (5, "token", (120, 3)),        # layered, int16 values: about 47 words per chunk
])
def test_static_scratch_decode_matches_decode(P, c, act_scale, batches):
    print(f"[no-alloc] config {c} alpha per {act_scale} batches {batches}", flush=True)
    cfg, H, G, w, y, x = build_workload(c, batch=batches[0], act_scale=act_scale)
    dec = P.Decoder(H, w)
    for B in batches:
        yd = torch.from_numpy(np.ascontiguousarray(y[:B])).cuda()
        b_ref, l_ref = dec.decode(yd)
        b_st, l_st = dec.decode_static(yd)
        torch.cuda.synchronize()
        assert torch.equal(l_st, l_ref) and torch.equal(b_st, b_ref), (c, B)
    e = torch.empty((0, cfg.n), dtype=torch.float32, device="cuda")
    b0, l0 = dec.decode_static(e)                  # batch 0: a no-op
    assert b0.shape == (0, cfg.n)
    with pytest.raises(P.AecctError) as ei:        # NULL y
        P._check(P.lib().aecct_decode_static(dec._h, None, 4, b_ref.data_ptr(), None, None), "decode_static")
    assert ei.value.status == P.ERR_INVALID_ARG
    dec.close()
