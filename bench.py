"""Throughput of the AECCT decode on one MI355X.

Workload: BCH(31,16) (cyclic H from the t = 3 generator polynomial), d = 32, N = 6 layers,
8 heads (4 first-ring, 4 second-ring), ternary weights with P(0) = 0.5, a batch of 65536
BPSK/AWGN words at Eb/N0 in {4, 5, 6, 7} dB, seeded synthetic data and random weights.
One step = one aecct_decode of the whole batch (pre-processing, every layer, head and hard
decision); y is resident in device memory before timing starts.

Prints one JSON line: words/s, the roofline of the dominant kernel (algorithmic fp32 ALU
operations per launch over its HIP-event duration, against one fp32 VALU operation per lane
per clock), and the CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

WORKLOAD = 2                      # BCH(31,16), batch 65536
PEAK_ALU_OPS = 256 * 4 * 16 * 2.4e9   # CUs x SIMDs x lanes x clock: fp32 VALU ops/s, non-packed
PEAK_INT8 = 5.0e15                # dense int8 MFMA ops/s
PEAK_HBM = 8.0e12


def algorithmic_counts(H, w, attention: str = "hpsa"):
    """Per-word work of the method as the paper writes it (not as executed).

    fp32/ALU operations: every scalar operation of Sections 3-4 counts once, with each
    multiply-accumulate of a dot product, of the attention-weighted value sum, of the
    dequantisation plus bias and of the LayerNorm affine map counted as one operation (one
    fused instruction); exp, division, square root and rounding count once each.  The
    ternary x int8 products are MFMA work, counted separately as int8 MACs.
      quantisation of a K-wide row (Eq. 2): max|x|, multiply, round per value + Q_b/alpha
      dequant (Eq. 3): one multiply-add per output + alpha * scale per row and map
      LayerNorm: sum, subtract, square-accumulate, normalise, affine per value + 5 per row
      attention pair: d_h multiply-adds (q.k), scale, max, subtract, exp, sum, d_h (p v)
      attention row and head: 1/S and d_h products
    """
    m, n = H.shape
    L, d, N, dff, heads = n + m, w.d, w.n_layers, w.d_ff, w.heads
    dh, hf = d // heads, w.first_ring_heads
    A = np.zeros((L, L), np.int64)
    A[:n, n:] = H.T
    A[n:, :n] = H
    nnz1 = int((A != 0).sum())
    nnz2 = int(((A @ A) != 0).sum())
    quant = lambda K: 3 * K + 1
    token_layer = (3 * quant(d) + quant(dff)          # inputs of the QKV, O, FF1, FF2 maps
                   + (3 * d + d + dff + d) + 4        # dequant + bias, 4 row scales
                   + 2 * d                            # two residual adds
                   + 2 * (5 * d + 5)                  # two LayerNorms
                   + dff)                             # ReLU
    pair = 2 * dh + 5
    row_head = dh + 1
    # HPSA: h_f heads over the first ring, the rest over the second; CASA: every head over both
    pairs = heads * (nnz1 + nnz2) if attention == "casa" else hf * nnz1 + (heads - hf) * nnz2
    layer = L * token_layer + pairs * pair + L * heads * row_head
    embed = L * (d + 1) + int(H.sum())                # t * E_i rows, |y| / sign, syndrome XORs
    head = L * (d + 1) + n * (L + 1 + 2)              # z_i, f_o, hard decision
    alu = embed + N * layer + head
    macs = N * L * (3 * d * d + d * d + 2 * d * dff)
    hbm = 4 * n + n + 4 * n                           # y in, bits and logits out
    return dict(alu_ops=alu, int8_macs=macs, hbm_bytes=hbm, pairs_per_layer=pairs)


def kernel_source_hash():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2410_05911_amd", "csrc")
    # the fused kernel, its device helpers and table layout, and the host code that packs its tables
    for f in ("kernel_fused.hip", "device_common.h", "fused_layout.h", "host_fused.h", "host_fused.cpp"):
        h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(kernel, workload):
    """HBM bytes per launch from the committed rocprofv3 counter summary (lines
    `source_hash: ...` and `hbm_bytes_per_launch: ...`), if it was taken on the current
    kernel sources; otherwise None."""
    p = os.path.join(ROOT, "profiles", f"{kernel}__{workload}__hbm_counters.md")
    if not os.path.exists(p):
        return None
    rec = {}
    for ln in open(p):
        if ":" in ln and ln.strip().startswith(("source_hash", "hbm_bytes_per_launch")):
            k, v = ln.split(":", 1)
            rec[k.strip()] = v.strip().strip("`")
    if rec.get("source_hash") != kernel_source_hash():
        return None
    return float(rec["hbm_bytes_per_launch"]) if "hbm_bytes_per_launch" in rec else None


def copy_calibration(mib: int = 512):
    """A plain device-to-device copy of a known size (the scale for the HBM counters)."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read": n * 4, "copy_calibration_bytes_written": n * 4}))


def cpu_model() -> str:
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_rate(om, y, threads, budget_s):
    """Words/s of the oracle at `threads` OpenMP threads on the first k words of y, k sized from a
    probe so that the timed run takes about budget_s."""
    probe = 64 if threads == 1 else 512
    t0 = time.perf_counter()
    om.decode(y[:probe], n_threads=threads)
    t1 = time.perf_counter() - t0
    k = int(min(y.shape[0], max(probe, probe * budget_s / max(t1, 1e-6))))
    t0 = time.perf_counter()
    om.decode(y[:k], n_threads=threads)
    dt = time.perf_counter() - t0
    return k / dt, k, dt


def cpu_baseline(H, w, y, budget_s=10.0):
    """The oracle (canonical fp32, as committed) on the host: at the host's thread share (at most
    16, the CPU share of one GPU on these machines) and at one thread."""
    import oracle
    nproc = os.cpu_count() or 1
    threads = min(nproc, 16)
    om = oracle.OracleModel(H, w)
    v, k, dt = _oracle_rate(om, y, threads, budget_s)
    v1, k1, dt1 = _oracle_rate(om, y, 1, budget_s / 2)
    return {"value": v, "unit": "codewords/s", "cores": threads, "kind": "oracle",
            "sample": f"first {k} of {y.shape[0]} words of the same workload, canonical fp32 oracle, "
                      f"{threads} OpenMP threads, {dt:.1f} s",
            "cpu_model": cpu_model(), "host_nproc": nproc,
            "one_thread": {"value": v1, "unit": "codewords/s", "cores": 1,
                           "sample": f"first {k1} words, 1 thread, {dt1:.1f} s"}}


def aap_import_bench(repeats: int = 5):
    """AAP weight import (Eq. 1, a host step of model creation) for every in-block map of a
    d = 128, 10-layer model (the LDPC(256,128) shape): 60 fp32 matrices, 1.97 M weights."""
    import paper_2410_05911_amd as P
    rng = np.random.default_rng(4242)
    d, N = 128, 10
    mats = []
    for _ in range(N):
        mats += [rng.standard_normal((d, d)).astype(np.float32) * 0.05 for _ in range(4)]
        mats += [rng.standard_normal((d, 4 * d)).astype(np.float32) * 0.05,
                 rng.standard_normal((4 * d, d)).astype(np.float32) * 0.05]
    total = sum(m.size for m in mats)
    P.aap_ternarize(mats[0])
    best = float("inf")
    for _ in range(repeats):
        t0 = time.perf_counter()
        for m in mats:
            P.aap_ternarize(m)
        best = min(best, time.perf_counter() - t0)
    out = {"metric": "AAP weight import (Eq. 1) throughput, host", "value": total / best, "unit": "weights/s",
           "higher_is_better": True, "ms_per_model": best * 1e3,
           "config": {"workload": "aap_import_d128_N10", "matrices": len(mats), "weights": total,
                      "percentile": 0.5, "delta": 1.0, "eps": 1e-8}}
    import oracle
    t0 = time.perf_counter()
    for m in mats:
        oracle.aap_ternarize(m)
    dt = time.perf_counter() - t0
    out["cpu_baseline"] = {"value": total / dt, "unit": "weights/s", "cores": 1, "kind": "oracle",
                           "sample": "the same 60 matrices, one pass, full sort per matrix"}
    print(json.dumps(out), flush=True)


def spe_bench(c: int, repeats: int = 3):
    """Spectral positional encoding (Section 4.3, a create-time step) for workload c's code:
    the Laplacian spectrum on the host, then the table (per-node attention on the GPU)."""
    import paper_2410_05911_amd as P
    from workloads import CONFIGS, random_spe_params
    from workloads.configs import parity_check
    cfg = CONFIGS[c]
    H = parity_check(cfg)
    m, n = H.shape
    L = n + m
    d = cfg.d
    d_pe, heads = d // 4, 4
    p = random_spe_params(L, d_pe, heads, seed=123)
    t0 = time.perf_counter()
    lam, vec = P.tanner_spectrum(H)
    t_spec = time.perf_counter() - t0
    P.spe_table_from_spectrum(lam, vec, p, d)
    best = float("inf")
    for _ in range(repeats):
        t0 = time.perf_counter()
        P.spe_table_from_spectrum(lam, vec, p, d)
        best = min(best, time.perf_counter() - t0)
    pairs = L * heads * L * L            # (node, head, row, key)
    import oracle.spe as ospe
    k = 4
    t0 = time.perf_counter()
    ospe.spe_table_from_spectrum(lam, vec.T, p, d, nodes=list(range(k)))
    dt = time.perf_counter() - t0
    print(json.dumps({"metric": "SPE table construction (Section 4.3), create time", "value": best * 1e3,
                      "unit": "ms (table from spectrum, incl. copies)", "higher_is_better": False,
                      "spectrum_host_s": t_spec, "score_pairs": pairs, "pairs_per_s": pairs / best,
                      "config": {"workload": f"spe_{cfg.name}", "tokens": L, "d": d, "d_pe": d_pe,
                                 "heads": heads},
                      "cpu_baseline": {"value": dt / k * L * 1e3, "unit": "ms (table from spectrum)", "cores": 1,
                                       "kind": "oracle", "sample": f"{k} of {L} nodes, float64 numpy, "
                                       f"{dt:.1f} s, scaled to all nodes"}}), flush=True)


def train_bench(c: int, batch: int, steps: int, warmup: int):
    """The quantisation-aware training step (Section 6, second phase) of workload c's shape on the
    GPU: Eq. 1 on every latent matrix, forward, loss and every gradient (no optimiser update)."""
    import torch
    import paper_2410_05911_amd as P
    from workloads import CONFIGS, random_qat_params
    from workloads.configs import parity_check
    from workloads.channel import awgn_words
    from workloads.codes import generator_from_parity
    cfg = CONFIGS[c]
    H = parity_check(cfg)
    m, n = H.shape
    L, d, N = n + m, cfg.d, cfg.n_layers
    p = random_qat_params(n, m, d, N, seed=7)
    y, x, _ = awgn_words(generator_from_parity(H), batch, (3.0, 4.0, 5.0, 6.0, 7.0), seed=8)
    y = (y * (1 - 2 * x.astype(np.float32))).astype(np.float32)       # all-zero codeword, as the paper trains
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    pd = {k: ({kk: dev(vv) for kk, vv in v.items()} if k in ("w", "b") else
              (dev(np.array([v], np.float32)) if k == "head_b1" else (None if v is None else dev(v))))
          for k, v in p.items()}
    tr = P.Trainer(H, d, N)
    yd = dev(y)
    for _ in range(warmup):
        tr.grad(pd, yd)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        loss, g = tr.grad(pd, yd)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    # fp32 multiply-adds of the step's GEMMs (forward, input gradients, weight gradients) and head
    R = batch * L
    lin = N * (4 * d * d + 2 * d * 4 * d)
    fma = 3 * R * lin + 3 * batch * L * n
    import oracle.qat as Q
    k = 2
    t0 = time.perf_counter()
    Q.forward_backward(H, p, y[:k])
    dt = time.perf_counter() - t0
    print(json.dumps({"metric": "QAT training step (forward + every gradient), words/s", "value": batch / (ms * 1e-3),
                      "unit": "codewords/s", "ms_per_step": ms, "steps": steps, "warmup": warmup,
                      "higher_is_better": True, "loss": loss.item(),
                      "config": {"workload": f"qat_{cfg.name}_batch{batch}", "tokens": L, "d": d, "layers": N,
                                 "batch": batch},
                      "gemm_fma_per_step": fma, "gemm_fma_rate_T": fma / (ms * 1e-3) / 1e12,
                      # the step's products as fp32 work against the fp32 MFMA peak: every GEMM flop
                      # over the whole step time (a lower bound of the GEMM kernels' own rate; the
                      # products with a ternary operand run on the bf16 matrix cores, three exact
                      # bf16 products per fp32 one, at d and d_ff multiples of 64)
                      "roofline": {"bound": "mfma", "kernel": "k_gemm_tern + k_gemm_mfma (all step GEMMs, whole-step time)",
                                   "achieved": 2 * fma / (ms * 1e-3) / 1e12, "peak": 157.3, "unit": "TFLOP/s",
                                   "frac": 2 * fma / (ms * 1e-3) / 1e12 / 157.3, "traffic": None},
                      "cpu_baseline": {"value": k / dt, "unit": "codewords/s", "cores": 1, "kind": "oracle",
                                       "sample": f"{k} words, float64 numpy oracle, {dt:.2f} s"}}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=20, help="untimed steps; the clocks settle over the first ~20")
    ap.add_argument("--path", type=int, default=0, help="0 auto, 1 layered, 2 fused")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--workload", type=int, default=WORKLOAD)
    ap.add_argument("--attention", choices=("hpsa", "casa"), default="hpsa",
                    help="head-partitioned masks (the method) or the ECCT mask on every head")
    ap.add_argument("--first-ring-heads", type=int, default=None,
                    help="h_f, heads on the first-ring mask (default heads / 2; HPSA only)")
    ap.add_argument("--act-scale", choices=("token", "word"), default="token",
                    help="Eq. 2 scale per token (default) or per word")
    ap.add_argument("--layered-attention", type=int, default=-1,
                    help="layered path's Q/K/V + attention form: -1 auto, 0 unfused, 1 fp32 in LDS, 2 int16 in LDS, 3 one node type at a time")
    ap.add_argument("--train", action="store_true",
                    help="only time the QAT training step of --workload's shape (batch --train-batch)")
    ap.add_argument("--train-batch", type=int, default=128, help="words per training step (the paper: 128)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 512 MiB device copy (HBM counter calibration)")
    ap.add_argument("--aap-import", action="store_true",
                    help="only time the AAP weight import (Eq. 1) of a d = 128, 10-layer model")
    ap.add_argument("--spe", action="store_true",
                    help="only time the spectral positional encoding of --workload's code")
    args = ap.parse_args()
    if args.spe:
        spe_bench(args.workload)
        return
    if args.train:
        train_bench(args.workload, args.train_batch, args.steps, args.warmup)
        return
    if args.copy_calibration:
        copy_calibration()
        return
    if args.aap_import:
        aap_import_bench()
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (the decode shards over words with no exchange); "
              f"--gpus {args.gpus} is not supported", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2410_05911_amd as P
    from workloads import build_workload

    if args.first_ring_heads is not None and args.attention != "hpsa":
        print("--first-ring-heads applies to the head-partitioned masks only", file=sys.stderr)
        sys.exit(2)
    cfg, H, G, w, y, x = build_workload(args.workload, attention=args.attention,
                                        first_ring_heads=args.first_ring_heads, act_scale=args.act_scale)
    default_split = args.attention == "hpsa" and w.first_ring_heads == cfg.heads // 2
    wl_name = cfg.name if default_split else (cfg.name + "_casa" if args.attention == "casa"
                                              else f"{cfg.name}_hf{w.first_ring_heads}")
    if args.act_scale == "word":
        wl_name += "_alpha_per_word"
    if args.layered_attention != -1:
        wl_name += f"_lattn{args.layered_attention}"
    default_split = default_split and args.act_scale == "token" and args.layered_attention == -1
    B = cfg.batch
    dev = torch.device("cuda:0")
    dec = P.Decoder(H, w, path=args.path, layered_attention=args.layered_attention)
    yd = torch.from_numpy(y).to(dev)
    bits = torch.empty((B, cfg.n), dtype=torch.uint8, device=dev)
    logits = torch.empty((B, cfg.n), dtype=torch.float32, device=dev)
    ws = dec.workspace(B, dev)
    stream = torch.cuda.current_stream(dev)

    for _ in range(args.warmup):
        dec.decode(yd, bits, logits, ws, stream)
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        dec.decode(yd, bits, logits, ws, stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    ms = ev0.elapsed_time(ev1) / args.steps
    value = B / (ms * 1e-3)

    cnt = algorithmic_counts(H, w, args.attention)
    path = "fused" if dec.path == P.PATH_FUSED else "layered"
    kernel = "k_fused_decode" if path == "fused" else "layered_decode"
    launch_s = ms * 1e-3                        # fused: one launch per step
    achieved = cnt["alu_ops"] * B / launch_s
    roofline = {
        "bound": "alu",
        "kernel": kernel,
        "achieved": achieved / 1e12,
        "peak": PEAK_ALU_OPS / 1e12,
        "unit": "Top/s (fp32 VALU ops, one per lane per clock)",
        "frac": achieved / PEAK_ALU_OPS,
        "traffic": measured_traffic(kernel, cfg.name) if default_split else None,
        "alu_ops_per_word": cnt["alu_ops"],
        "int8_mfma_frac": 2 * cnt["int8_macs"] * B / launch_s / PEAK_INT8,
        "hbm_alg_frac": cnt["hbm_bytes"] * B / launch_s / PEAK_HBM,
    }
    out = {
        "metric": "decoded codewords/sec (1 GPU) + % of int8-MFMA/HBM roofline",
        "value": value,
        "unit": "codewords/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8xternary->int32, fp32",
        "data": "synthetic: seeded BPSK/AWGN words, random ternary weights",
        "config": {"workload": wl_name, "code": "BCH(31,16)" if cfg.code == "bch" else cfg.code,
                   "n": cfg.n, "tokens": dec.L, "d": cfg.d, "layers": cfg.n_layers, "heads": cfg.heads,
                   "first_ring_heads": w.first_ring_heads if args.attention == "hpsa" else None,
                   "attention": args.attention, "act_scale": args.act_scale, "batch": B, "path": path,
                   "layered_attention": dec.info.layered_attention,
                   "wall_s_timed": t_wall},
        "roofline": roofline,
    }
    # outside the timed region: the same decode with y copied in from pinned host memory and the
    # bits and logits copied back, all on the decode stream (context for callers holding host data)
    yh = torch.from_numpy(y).pin_memory()
    bh = torch.empty((B, cfg.n), dtype=torch.uint8).pin_memory()
    lh = torch.empty((B, cfg.n), dtype=torch.float32).pin_memory()
    n_host = max(3, min(args.steps, 20))
    torch.cuda.synchronize()
    h0 = torch.cuda.Event(enable_timing=True)
    h1 = torch.cuda.Event(enable_timing=True)
    h0.record(stream)
    for _ in range(n_host):
        yd.copy_(yh, non_blocking=True)
        dec.decode(yd, bits, logits, ws, stream)
        bh.copy_(bits, non_blocking=True)
        lh.copy_(logits, non_blocking=True)
    h1.record(stream)
    torch.cuda.synchronize()
    ms_host = h0.elapsed_time(h1) / n_host
    out["host_inclusive"] = {"value": B / (ms_host * 1e-3), "unit": "codewords/s", "ms_per_step": ms_host,
                             "steps": n_host, "what": "y host-to-device from pinned memory, decode, bits and "
                                                      "logits device-to-host, one stream"}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(H, w, y)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
