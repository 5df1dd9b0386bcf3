"""Benchmark of the attention hot path on one MI355X.

One step = one pass over the whole path on resident synthetic inputs:
  * the fused causal attention forward on the prefill workload
    (causal MHA B=4 H=16 S=2048 D=128 bf16 by default), then
  * the split-KV decode (split kernel + LSE merge) on the ragged decode
    batch (B=64 Hq=32 Hkv=8 D=128, lengths in [512, 4096]), alternating
    between two copies of the cache so the 256 MB last-level cache cannot
    hand the previous step's cache to the next one.

Kernel durations are taken with HIP events recorded on the stream the
kernels are launched on (torch's current stream), around every launch of
the timed steps.  Prints ONE JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6  # dense bf16 MFMA, 256 CU x 4096 FLOP/clk x 2.4 GHz
PEAK_HBM_GBS = 8000.0      # HBM3E


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_digest() -> str:
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_04523_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, name), "rb") as fh:
            h.update(name.encode() + b"\0" + fh.read())
    return h.hexdigest()[:16]


def read_traffic(summary_name: str, digest: str):
    """HBM bytes per launch from a committed rocprofv3 counter summary,
    or None when absent or taken on a different kernel source."""
    path = os.path.join(ROOT, "profiles", summary_name)
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_d = re.search(r"kernel_source_digest:\s*([0-9a-f]+)", text)
    m_t = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m_d or not m_t or m_d.group(1) != digest:
        return None
    return float(m_t.group(1))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--prefill", default="c2_mha_s2k")
    ap.add_argument("--decode", default="c5_decode_b64")
    ap.add_argument("--split", type=int, default=0, help="decode keys per split (0 = default)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=96,
                    help="query rows per head timed for the CPU oracle baseline")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run one plain device copy of this size (counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the path shards by kv-head groups across GPUs, see DESIGN.md)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2609_04523_amd as mk
    import workloads

    if not os.path.exists(mk.LIB_PATH):
        from paper_2609_04523_amd import build as hip_build
        hip_build.build()
    mk.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    pcfg = workloads.CONFIGS[args.prefill]
    dcfg = workloads.CONFIGS[args.decode]
    log(f"[bench] inputs: prefill {pcfg.name}, decode {dcfg.name}")
    q, k, v = workloads.config_inputs(pcfg)
    q, k, v = q.to(dev), k.to(dev), v.to(dev)
    o = torch.empty(q.shape, device=dev, dtype=torch.float32 if pcfg.out_fp32 else torch.bfloat16)
    lse = torch.empty(q.shape[:3], device=dev, dtype=torch.float32)
    qd, kc, vc, lens = workloads.config_inputs(dcfg)
    caches = [(kc.to(dev), vc.to(dev)), (kc.to(dev).clone(), vc.to(dev).clone())]
    del kc, vc
    qd = qd.to(dev)
    lens_d = lens.to(dev)
    B, Hq, D = qd.shape
    Hkv, Smax = dcfg.Hkv, dcfg.Smax
    ws_bytes = mk.mk_attn_decode_workspace_bytes(B, Hq, Smax, D, args.split)
    ws = torch.empty(ws_bytes, device=dev, dtype=torch.uint8)
    od = torch.empty((B, Hq, D), device=dev, dtype=torch.bfloat16)
    lsed = torch.empty((B, Hq), device=dev, dtype=torch.float32)
    torch.cuda.synchronize()

    fwd_entry = mk.mk_attn_fwd_o32 if pcfg.out_fp32 else mk.mk_attn_fwd
    stream = torch.cuda.current_stream()

    def prefill():
        fwd_entry(q, k, v, o, lse, pcfg.B, pcfg.Hq, pcfg.Hkv, pcfg.S, pcfg.S, pcfg.D, 1,
                  pcfg.scale, None, stream)

    def decode(i):
        kcc, vcc = caches[i & 1]
        mk.mk_attn_decode(qd, kcc, vcc, od, lsed, B, Hq, Hkv, Smax, D, dcfg.scale, lens_d,
                          args.split, ws, ws_bytes, stream)

    if args.calib_copy_mib:
        n = args.calib_copy_mib << 20
        src = torch.empty(n, device=dev, dtype=torch.uint8).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] calibration copy of {n} bytes done")
        del src, dst

    log(f"[bench] warmup {args.warmup}")
    for i in range(args.warmup):
        prefill()
        decode(i)
    torch.cuda.synchronize()

    K = args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
    log(f"[bench] timing {K} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(K):
        e = ev[i]
        e[0].record(stream)
        prefill()
        e[1].record(stream)
        e[2].record(stream)
        decode(i)
        e[3].record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / K
    t_pre = [e[0].elapsed_time(e[1]) for e in ev]   # ms
    t_dec = [e[2].elapsed_time(e[3]) for e in ev]
    pre_ms = sum(t_pre) / K
    dec_ms = sum(t_dec) / K
    flops = pcfg.flops
    tflops = flops / (pre_ms * 1e-3) / 1e12
    sum_l = int(lens.clamp(0, Smax).sum())
    dec_bytes = 4 * D * Hkv * sum_l + (B * Hq * D * 2) * 2 + B * Hq * 4  # K+V, q, o, lse
    dec_gbs = dec_bytes / (dec_ms * 1e-3) / 1e9
    log(f"[bench] prefill {pre_ms * 1e3:.1f} us ({tflops:.1f} TFLOP/s), "
        f"decode {dec_ms * 1e3:.1f} us ({dec_gbs:.1f} GB/s), step {ms_step:.3f} ms")

    digest = kernel_source_digest()
    traffic_pre = read_traffic(f"fwd_kernel_{pcfg.name}_counters.md", digest)
    traffic_dec = read_traffic(f"dec_split_kernel_{dcfg.name}_counters.md", digest)

    result = {
        "metric": "attention fwd TFLOP/s and % bf16 MFMA peak (prefill); HBM GB/s (decode)",
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16, generated on the host, resident in HBM)",
        "config": {
            "workload": (f"{pcfg.name}: causal attention fwd B={pcfg.B} Hq={pcfg.Hq} "
                         f"Hkv={pcfg.Hkv} S={pcfg.S} D={pcfg.D} bf16 in, "
                         f"{'fp32' if pcfg.out_fp32 else 'bf16'} O + fp32 LSE; then "
                         f"{dcfg.name}: decode B={B} Hq={Hq} Hkv={Hkv} D={D} "
                         f"lengths U[{dcfg.lmin},{dcfg.lmax}] split-KV + LSE merge"),
            "prefill_flops_per_step": flops,
            "decode_bytes_per_step": dec_bytes,
            "decode_sum_kv_len": sum_l,
            "kernel_source_digest": digest,
        },
        "prefill_us": round(pre_ms * 1e3, 2),
        "roofline": {
            "bound": "mfma",
            "achieved": round(tflops, 2),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(tflops / PEAK_BF16_TFLOPS, 4),
            "traffic": traffic_pre,
        },
        "decode": {
            "value": round(dec_gbs, 1),
            "unit": "GB/s",
            "us": round(dec_ms * 1e3, 2),
            "roofline": {
                "bound": "hbm",
                "achieved": round(dec_gbs, 1),
                "peak": PEAK_HBM_GBS,
                "unit": "GB/s",
                "frac": round(dec_gbs / PEAK_HBM_GBS, 4),
                "traffic": traffic_dec,
            },
        },
        "cpu_baseline": None,
    }

    if not args.no_cpu_baseline:
        from oracle import oracle as orc  # timed CPU baseline only
        nrows = min(args.cpu_rows, pcfg.S)
        rows = workloads.sample_rows(pcfg.B, pcfg.Hq, pcfg.S, nrows, seed=pcfg.seed + 7)
        qh, kh, vh = workloads.config_inputs(pcfg)
        qb, kb, vb = workloads.bits(qh), workloads.bits(kh), workloads.bits(vh)
        threads = orc.default_threads()
        log(f"[bench] cpu oracle baseline: {nrows} rows/head on {threads} threads")
        c0 = time.perf_counter()
        orc.attn_fwd(qb, kb, vb, causal=True, scale=pcfg.scale, rows=rows.numpy(),
                     threads=threads)
        c1 = time.perf_counter()
        pairs = int((rows.long() + 1).sum())  # row i sees i+1 keys
        cpu_tflops = 4 * pcfg.D * pairs / (c1 - c0) / 1e12
        result["cpu_baseline"] = {
            "value": cpu_tflops,
            "unit": "TFLOP/s",
            "cores": threads,
            "kind": "oracle",
            "sample": (f"{nrows} seeded query rows per head of {pcfg.name} "
                       f"({pairs} query-key pairs, {c1 - c0:.2f} s)"),
        }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
