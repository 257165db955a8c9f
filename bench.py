"""Benchmark: triadic GDN forward + backward on one MI355X.

One step is the whole hot path on one batch: a training-mode chunkwise
forward (tla_fwd with a `saved` buffer) followed by the backward (tla_bwd),
at B=4, H=8, T=4096, K=V=128, E=8, chunk 64, bf16 operands with fp32
accumulation (the 1.3B-model head shape of the paper's efficiency study at
batch 4).  Inputs are seeded synthetic tensors with the paper's distributions,
resident in HBM before timing starts.

Prints one JSON line: throughput in tokens/s (B*T per step), the roofline of
the dominant kernel (algorithmic FLOPs or bytes per launch over its average
HIP-event duration inside the timed region), and the fp64 CPU oracle timed
on a bounded sample of the same workload.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def algorithmic(cfg):
    """Per token-head algorithmic FLOPs / bytes of each kernel (GDN).  FLOPs
    count the method's own contractions (not split-operand or recompute
    work); bytes count each kernel's compulsory HBM reads and writes."""
    K, V, E, C = cfg.K, cfg.V, cfg.E, cfg.chunk
    ckpt = 2.0 * E * K * V / C          # one bf16 chunk state per token-head
    return {
        "prep": {"flops": 4 * C * K + C * C / 3.0},
        "fwd_recurrent": {"flops": 6 * K * V * E + 4 * C * V,
                          "bytes": 2 * (2 * K + V) + 2 * V + ckpt + 8 * V},
        "bwd_recurrent": {"flops": 6 * K * V * E + 4 * C * V,
                          "bytes": 2 * (2 * K + V) + ckpt + 8 * V},
        "bwd_state": {"flops": 6 * K * V * E,
                      "bytes": 2 * ckpt + 2 * V + 8 * V + 4 * K + 8 * K},
        "bwd_chunk": {"flops": 6 * C * K + 4 * C * V + 2 * C * C / 3.0},
        "total_flops": 18 * K * V * E + 12 * C * K + 12 * C * V + C * C,
    }


def cpu_baseline(cfg, inp, dO, nb=2):
    """The fp64 oracle (token-by-token recurrence + reverse mode, OpenMP over
    heads) on the first `nb` batch entries, all heads, full T."""
    import oracle
    from paper_2609_36529_amd import synth
    sl = lambda x: None if x is None else synth.to64(x[:nb])
    args = [sl(inp[n]) for n in ("q", "k", "v", "q2", "k2", "g", "beta", "s0")]
    d = sl(dO)
    t0 = time.perf_counter()
    oracle.fwd(cfg.variant, *args)
    oracle.bwd(cfg.variant, *args, d)
    dt = time.perf_counter() - t0
    tokens = nb * cfg.T
    return {"value": tokens / dt, "unit": "tokens/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"GDN fwd+bwd (fp64 oracle: forward, then reverse-mode backward "
                      f"with its own recompute) on {nb} of {cfg.B} batch entries x {cfg.H} heads, "
                      f"full T={cfg.T}: {tokens} tokens in {dt:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the operator's work shards over batch, heads "
              "and value tiles with no exchange, so per-GPU throughput at N GPUs is the N=1 "
              "figure; multi-GPU runs are not part of this build.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2609_36529_amd as tla
    from paper_2609_36529_amd import synth

    dev = torch.device("cuda:0")
    cfg = synth.CONFIGS["gdn_bf16"]
    inp = synth.make_inputs(cfg)
    dO = synth.make_dO(cfg)
    d = {k: (None if v is None else v.to(dev)) for k, v in inp.items()}
    dO_d = dO.to(dev)
    B, T, H, K, V, E, C = cfg.B, cfg.T, cfg.H, cfg.K, cfg.V, cfg.E, cfg.chunk
    out_dt = torch.bfloat16
    desc = tla.describe(cfg.variant, d["q"], d["v"], d["q2"], C, out_dt)
    ws_f = torch.empty(tla.workspace_bytes(desc, tla.OP_FWD), dtype=torch.uint8, device=dev)
    ws_b = torch.empty(tla.workspace_bytes(desc, tla.OP_BWD), dtype=torch.uint8, device=dev)
    saved = torch.empty(tla.saved_bytes(desc), dtype=torch.uint8, device=dev)
    o = torch.empty((B, T, H, V), dtype=out_dt, device=dev)
    sf = torch.empty((B, H, E, K, V), dtype=torch.float32, device=dev)
    grads = {
        "dq": torch.empty_like(d["q"], dtype=out_dt), "dk": torch.empty_like(d["k"], dtype=out_dt),
        "dv": torch.empty_like(d["v"], dtype=out_dt), "dq2": torch.empty_like(d["q2"], dtype=out_dt),
        "dk2": torch.empty_like(d["k2"], dtype=out_dt),
        "dg": torch.empty((B, T, H, E), dtype=torch.float32, device=dev),
        "dbeta": torch.empty((B, T, H), dtype=torch.float32, device=dev),
        "ds0": torch.empty((B, H, E, K, V), dtype=torch.float32, device=dev),
    }

    def step():
        tla.fwd(cfg.variant, d["q"], d["k"], d["v"], d["q2"], d["k2"], d["g"], d["beta"], d["s0"],
                chunk=C, out_dtype=out_dt, training=True, o=o, s_final=sf, ws=ws_f, saved=saved)
        tla.bwd(cfg.variant, d["q"], d["k"], d["v"], d["q2"], d["k2"], d["g"], d["beta"], d["s0"],
                dO_d, saved, chunk=C, out_dtype=out_dt, ws=ws_b, grads=grads)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    tla.prof_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    prof = tla.prof_read()
    tla.prof_enable(False)

    ms_per_step = 1e3 * elapsed / args.steps
    tokens = B * T
    alg = algorithmic(cfg)
    token_heads = B * T * H
    kernels = {}
    for name, (tot, n) in prof.items():
        if n == 0:
            continue
        avg_ms = tot / n
        entry = {"avg_ms": round(avg_ms, 4), "launches": n}
        a = alg.get(name, {})
        if "flops" in a:
            entry["tflops"] = round(a["flops"] * token_heads / (avg_ms * 1e-3) / 1e12, 2)
        if "bytes" in a:
            entry["gbs"] = round(a["bytes"] * token_heads / (avg_ms * 1e-3) / 1e9, 1)
        kernels[name] = entry
    dom = max(kernels, key=lambda k: kernels[k]["avg_ms"] * kernels[k]["launches"])
    a = alg[dom]
    if dom == "bwd_state":
        roof = {"bound": "hbm", "achieved": kernels[dom]["gbs"], "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    else:
        roof = {"bound": "mfma", "achieved": kernels[dom]["tflops"], "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof["traffic"] = None
    roof["kernel"] = dom
    step_tflops = alg["total_flops"] * token_heads / (ms_per_step * 1e-3) / 1e12

    result = {
        "metric": "fwd+bwd tokens/s, triadic GDN H=8 K=V=128 E=8 T=4096",
        "value": round(tokens / (ms_per_step * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "triadic GDN fwd+bwd (training step of the operator)",
                   "B": B, "T": T, "H": H, "K": K, "V": V, "E": E, "chunk": C,
                   "operands": "bf16, fp32 accumulation, fp32 state", "outputs": "bf16",
                   "seed": cfg.seed},
        "mfma_frac_of_bf16_peak": round(step_tflops / PEAK_BF16_TFLOPS, 4),
        "step_tflops": round(step_tflops, 2),
        "kernels": kernels,
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(cfg, inp, dO)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
