"""Benchmark: triadic GDN forward + backward on one MI355X.

One step is the whole hot path on one batch: a training-mode chunkwise
forward (tla_fwd with a `saved` buffer) followed by the backward (tla_bwd),
at B=4, H=8, T=4096, K=V=128, E=8, chunk 64, bf16 operands with fp32
accumulation (the 1.3B-model head shape of the paper's efficiency study at
batch 4).  Inputs are seeded synthetic tensors with the paper's distributions,
resident in HBM before timing starts.

Prints one JSON line: throughput in tokens/s (B*T per step), every kernel's
average HIP-event time with its algorithmic FLOP and byte rates, the
roofline of the dominant kernel, and the fp64 CPU oracle timed on a bounded
sample of the same workload.

`--decode` times the recurrent decode step instead (N=256, H=16, E=16) and
prints its own JSON line; `--forward NAME` times the inference forward of
one of the other workloads (sgla_bf16: sGLA B4 H8 T4096 E8; gdn_bf16: GDN,
same shape; gdn_long_bf16: GDN B1 H16 T65536 E16) with its own JSON line.

Helper modes for the HBM-traffic measurement (run under rocprofv3 --pmc):
  --copy-calibration     a plain fp32 copy kernel of known size
  --pmc-summary R W CR CW  reduce four rocprofv3 counter directories (bench
                         and copy kernel, each with the L2-to-memory read
                         request counters TCC_EA0_RDREQ_32B/64B/128B and the
                         write request counters TCC_EA0_WRREQ/_64B) to
                         per-kernel bytes per launch, written to
                         profiles/hbm_traffic.json with the hash of each
                         kernel's sources (bench.py reports it only while the
                         sources are unchanged)
"""
import argparse
import csv
import glob
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
TRAFFIC_JSON = os.path.join(ROOT, "profiles", "hbm_traffic.json")
CSRC = os.path.join(ROOT, "paper_2609_36529_amd", "csrc")
KERNEL_SOURCES = {
    "prep": "tla_fwd.hip", "fwd_recurrent": "tla_fwd.hip", "bwd_recurrent": "tla_bwd.hip",
    "bwd_state": "tla_bwd.hip", "bwd_chunk": "tla_bwd.hip", "step": "tla_step.hip",
}
KERNEL_SYMBOLS = {  # rocprofv3 kernel-name prefix -> timing slot
    "tla::k_prep<": "prep", "tla::k_fwd<": "fwd_recurrent", "tla::k_fwd_dual<": "fwd_recurrent",
    "tla::k_bwd_rec<": "bwd_recurrent",
    "tla::k_bwd_state<": "bwd_state", "tla::k_bwd_chunk<": "bwd_chunk", "tla::k_step<": "step",
}
COPY_BYTES = 1 << 28         # copy-calibration buffer (fp32)


def source_hash(kind):
    h = hashlib.sha256()
    for f in (KERNEL_SOURCES[kind], "tla_common.hpp", "tla_internal.hpp"):
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def algorithmic(cfg):
    """Per token-head algorithmic FLOPs and HBM bytes of each kernel (GDN,
    bf16 operands and outputs).  FLOPs count the method's own contractions
    (dense, no split-operand or recompute work).  Bytes count only the
    operator's inputs and outputs that the kernel reads or writes, and the
    bf16 chunk-boundary states (the chunk-start states the forward stores for
    the backward, Appendix A "Kernels", and the backward's chunk-end state
    gradients), every tensor once; this design's other intermediates (the
    prep results, U, V - W, dU, dW, partial sums) are not counted."""
    K, V, E, C = cfg.K, cfg.V, cfg.E, cfg.chunk
    ckpt = 2.0 * E * K * V / C          # one bf16 chunk state per token-head
    qkv = 2 * (2 * K + V)               # q, k and v (or dO), bf16
    return {
        # Grams A_qk, A_kk and the (I + L) solve; reads q, k, q2, k2, g, beta
        "prep": {"flops": 4 * C * K + C * C / 3.0, "bytes": 2 * 2 * K + 2 * 2 * E + 4 * E + 4},
        # W, Q S_e, K^T diag(c) U over E slices, Tu (V - W), M U; reads q, k,
        # v, writes o and the chunk-start state
        "fwd_recurrent": {"flops": 6 * K * V * E + 4 * C * V, "bytes": qkv + 2 * V + ckpt},
        # K dS', M^T dO, Tu^T dU, Q^T diag(b) dO, K^T diag(a) dW; reads q, k,
        # dO, writes the chunk-end state gradient
        "bwd_recurrent": {"flops": 6 * K * V * E + 4 * C * V, "bytes": qkv + ckpt},
        # dO S^T, dW S^T, U dS'^T per slice; reads both chunk-boundary tensors, q, k, dO
        "bwd_state": {"flops": 6 * K * V * E, "bytes": 2 * ckpt + qkv},
        # Grams, dM, dTu, dq / dk products; reads q, k, v, q2, k2, g, beta, dO,
        # writes every input gradient
        "bwd_chunk": {"flops": 10 * C * K + 4 * C * V + 2 * C * C / 3.0,
                      "bytes": 2 * (2 * K + 2 * V + 2 * E) + 4 * E + 4
                      + 2 * (2 * K + V + 2 * E) + 4 * E + 4},
        "total_flops": 18 * K * V * E + 14 * C * K + 12 * C * V + 2 * C * C,
    }


# The chunkwise kernels whose work is the method's dense bf16 contractions
# (the recurrent forward and backward, the chunk-parallel state contractions,
# the intra-chunk Grams): they are placed on the bf16 MFMA roofline.
MFMA_KERNELS = ("prep", "fwd_recurrent", "bwd_recurrent", "bwd_state")


def bound_of(name, a):
    """'mfma' for the contraction kernels, else whichever roofline time is
    longer for the kernel's algorithmic counts."""
    if name in MFMA_KERNELS:
        return "mfma"
    t_f = a.get("flops", 0.0) / (PEAK_BF16_TFLOPS * 1e12)
    t_b = a.get("bytes", 0.0) / (PEAK_HBM_GBS * 1e9)
    return "mfma" if t_f >= t_b else "hbm"


def cpu_baseline(cfg, inp, dO, min_seconds=10.0):
    """The fp64 oracle (token-by-token recurrence + reverse mode, OpenMP over
    heads) on the whole workload (all batch entries and heads, full T),
    repeated until at least `min_seconds` have elapsed."""
    import oracle
    from paper_2609_36529_amd import synth
    args = [synth.to64(inp[n]) if inp[n] is not None else None
            for n in ("q", "k", "v", "q2", "k2", "g", "beta", "s0")]
    d = synth.to64(dO)
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.fwd(cfg.variant, *args)
        oracle.bwd(cfg.variant, *args, d)
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    tokens = reps * cfg.B * cfg.T
    return {"value": round(tokens / dt, 1), "unit": "tokens/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"GDN fwd+bwd of the whole workload ({cfg.B} x {cfg.T} tokens x {cfg.H} "
                      f"heads; fp64 oracle: forward, then reverse-mode backward with its own "
                      f"recompute), {reps} repetition(s) in {dt:.1f} s"}


def traffic_for(kind, alg_bytes, token_heads):
    """Measured HBM bytes per launch of `kind` from profiles/hbm_traffic.json,
    or None when absent or taken from different kernel sources."""
    try:
        with open(TRAFFIC_JSON) as fh:
            rec = json.load(fh)["kernels"][kind]
    except (OSError, KeyError, ValueError):
        return None, None
    if rec.get("source_hash") != source_hash(kind):
        return None, None
    t = rec["fetch_bytes"] + rec["write_bytes"]
    return t, round(t / (alg_bytes * token_heads), 3)


def copy_calibration():
    import torch
    n = COPY_BYTES // 4
    x = torch.rand(n, device="cuda")
    y = torch.empty_like(x)
    for _ in range(5):
        torch.mul(x, 1.0, out=y)   # reads and writes COPY_BYTES each
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": COPY_BYTES, "launches": 5}), flush=True)


def _pmc_table(d, counter):
    """{kernel slot: average counter value per dispatch} from a rocprofv3 dir."""
    sums, disp = {}, {}
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] != counter:
                continue
            name = r["Kernel_Name"]
            slot = next((v for k, v in KERNEL_SYMBOLS.items() if k in name), None)
            if slot is None:
                slot = "copy" if ("mul" in name.lower() or "elementwise" in name.lower()) else None
            if slot is None:
                continue
            sums[slot] = sums.get(slot, 0.0) + float(r["Counter_Value"])
            disp.setdefault(slot, set()).add(r["Dispatch_Id"])
    return {k: sums[k] / len(disp[k]) for k in sums}


def _hbm_bytes(d, kind):
    """{kernel slot: HBM bytes per dispatch} from the L2-to-memory request
    counters of a rocprofv3 directory: reads are TCC_EA0_RDREQ_32B / _64B /
    _128B (32, 64, 128 bytes each), writes TCC_EA0_WRREQ_64B (64 bytes) and
    the remaining TCC_EA0_WRREQ (32 bytes)."""
    if kind == "read":
        parts = {"TCC_EA0_RDREQ_32B_sum": 32, "TCC_EA0_RDREQ_64B_sum": 64,
                 "TCC_EA0_RDREQ_128B_sum": 128}
        tabs = {c: _pmc_table(d, c) for c in parts}
        return {k: sum(parts[c] * tabs[c].get(k, 0.0) for c in parts) for k in tabs["TCC_EA0_RDREQ_32B_sum"]}
    wr, wr64 = _pmc_table(d, "TCC_EA0_WRREQ_sum"), _pmc_table(d, "TCC_EA0_WRREQ_64B_sum")
    return {k: 64 * wr64.get(k, 0.0) + 32 * (wr[k] - wr64.get(k, 0.0)) for k in wr}


def pmc_summary(read_dir, write_dir, copy_read_dir, copy_write_dir):
    """Per-kernel HBM bytes per launch from two counter passes over the bench
    (read requests, write requests) and the same passes over a plain copy
    kernel of known size, whose ratio of true to counted bytes scales each
    direction."""
    fe, wr = _hbm_bytes(read_dir, "read"), _hbm_bytes(write_dir, "write")
    cf, cw = _hbm_bytes(copy_read_dir, "read"), _hbm_bytes(copy_write_dir, "write")
    f_scale = COPY_BYTES / cf["copy"]
    w_scale = COPY_BYTES / cw["copy"]
    out = {"units": "bytes per launch", "counters": "TCC_EA0_RDREQ_{32B,64B,128B}, TCC_EA0_WRREQ{,_64B}",
           "read_scale": f_scale, "write_scale": w_scale,
           "copy_read_counted": cf["copy"], "copy_write_counted": cw["copy"], "kernels": {}}
    for kind in sorted(set(fe) & set(wr)):
        if kind == "copy":
            continue
        out["kernels"][kind] = {"read_counted": fe[kind], "write_counted": wr[kind],
                                "fetch_bytes": fe[kind] * f_scale,
                                "write_bytes": wr[kind] * w_scale,
                                "source_hash": source_hash(kind)}
    os.makedirs(os.path.dirname(TRAFFIC_JSON), exist_ok=True)
    with open(TRAFFIC_JSON, "w") as fh:
        json.dump(out, fh, indent=1)
    print(f"copy kernel: counted {cf['copy'] / 2**20:.1f} MiB read, {cw['copy'] / 2**20:.1f} MiB "
          f"written per launch for {COPY_BYTES >> 20} MiB each way -> scale {f_scale:.4f} / {w_scale:.4f}")
    print("| kernel | read (counted) MB | write (counted) MB | HBM bytes per launch (scaled) |")
    print("|---|---|---|---|")
    for kind, r in out["kernels"].items():
        print(f"| {kind} | {r['read_counted'] / 1e6:.1f} | {r['write_counted'] / 1e6:.1f} | "
              f"{r['fetch_bytes'] + r['write_bytes']:.4g} |")


def _warm_up(call, n, min_seconds=0.1):
    """n untimed calls, then more (in tens) until at least min_seconds of
    work have run: the part needs about 70 ms of work before its clocks
    settle, and a short call (0.2 ms) would otherwise be timed on the way up."""
    import torch
    for _ in range(n):
        call()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < min_seconds:
        for _ in range(10):
            call()
        torch.cuda.synchronize()


def decode_bench(steps, warmup, emit=True):
    """The recurrent decode step (tla_step) at N=256 sequences, H=16, E=16,
    K=V=128, bf16 token inputs, fp32 state [N,H,E,K,V] (4 GiB) updated in
    place; 8 pre-generated tokens are cycled so no input generation is timed.
    HBM-bound: one read and one write of the state per step."""
    import torch
    import paper_2609_36529_amd as tla
    from paper_2609_36529_amd import synth
    N, H, E, K, V = 256, 16, 16, 128, 128
    state = synth.make_decode_state(N, H, E, K, V).cuda()
    toks = []
    for i in range(8):
        t = synth.make_decode_token(N, H, K, V, E, dtype="bf16", seed=900 + i)
        toks.append({k: v.cuda() for k, v in t.items()})
    o = torch.empty((N, H, V), dtype=torch.bfloat16, device="cuda")

    def one(i):
        t = toks[i % len(toks)]
        tla.step(tla.GDN, t["q"], t["k"], t["v"], t["q2"], t["k2"], t["g"], t["beta"], state,
                 out_dtype=torch.bfloat16, o=o)
    cnt = [0]

    def next_call():
        one(cnt[0])
        cnt[0] += 1
    _warm_up(next_call, warmup)
    tla.prof_enable(True)
    t0 = time.perf_counter()
    for i in range(steps):
        one(i)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    tot, n = tla.prof_read()["step"]
    tla.prof_enable(False)
    avg_ms = tot / n
    state_bytes = 2.0 * N * H * E * K * V * 4
    gbs = state_bytes / (avg_ms * 1e-3) / 1e9
    res = {
        "metric": "decode tokens/s, triadic GDN tla_step N=256 H=16 E=16 K=V=128",
        "value": round(N / (elapsed / steps), 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": steps, "warmup": warmup, "ms_per_step": round(1e3 * elapsed / steps, 4),
        "higher_is_better": True, "dtype": "f32 state, bf16 tokens", "data": "synthetic",
        "config": {"workload": "GDN decode step", "N": N, "H": H, "E": E, "K": K, "V": V},
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                     "kernel": "step", "algorithmic_bytes_per_launch": state_bytes,
                     "avg_ms": round(avg_ms, 4)}}
    if emit:
        print(json.dumps(res), flush=True)
    return res


def forward_bench(name, steps, warmup, emit=True):
    """Inference forward (tla_fwd without `saved`) of a named workload: prep +
    recurrent forward, bf16 operands, bf16 output, final state returned.
    MFMA-bound by its algorithmic counts (inputs and outputs only move about
    1.2-1.6 KB per token-head against 0.56-1.6 MFLOP)."""
    import torch
    import paper_2609_36529_amd as tla
    from paper_2609_36529_amd import synth
    cfg = synth.CONFIGS[name]
    inp = synth.make_inputs(cfg)
    d = {k: (None if v is None else v.cuda()) for k, v in inp.items()}
    del inp
    B, T, H, K, V, E, C = cfg.B, cfg.T, cfg.H, cfg.K, cfg.V, cfg.E, cfg.chunk
    desc = tla.describe(cfg.variant, d["q"], d["v"], d["q2"], C, torch.bfloat16)
    ws = torch.empty(tla.workspace_bytes(desc, tla.OP_FWD), dtype=torch.uint8, device="cuda")
    o = torch.empty((B, T, H, V), dtype=torch.bfloat16, device="cuda")
    sf = torch.empty((B, H, E, K, V), dtype=torch.float32, device="cuda")

    def one():
        tla.fwd(cfg.variant, d["q"], d["k"], d["v"], d["q2"], d["k2"], d["g"], d["beta"], d["s0"],
                chunk=C, out_dtype=torch.bfloat16, o=o, s_final=sf, ws=ws)
    _warm_up(one, warmup)
    tla.prof_enable(True)
    t0 = time.perf_counter()
    for _ in range(steps):
        one()
    torch.cuda.synchronize()
    elapsed = (time.perf_counter() - t0) / steps
    prof = tla.prof_read()
    tla.prof_enable(False)
    if cfg.variant == 1:   # GDN: 6KVE + 4CK + 4CV + C^2/3 per token-head
        flops = 6 * K * V * E + 4 * C * K + 4 * C * V + C * C / 3.0
    else:                  # sGLA: 4KVE + 2CK + 2CV
        flops = 4 * K * V * E + 2 * C * K + 2 * C * V
    th = B * T * H
    tflops = flops * th / elapsed / 1e12
    kern = {k: round(v[0] / v[1], 4) for k, v in prof.items() if v[1]}
    res = {
        "metric": f"forward tokens/s, {name}", "value": round(B * T / elapsed, 1),
        "unit": "tokens/s", "n_gpus": 1, "steps": steps, "warmup": warmup,
        "ms_per_step": round(1e3 * elapsed, 4), "higher_is_better": True, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{'GDN' if cfg.variant == 1 else 'sGLA'} inference forward",
                   "B": B, "T": T, "H": H, "K": K, "V": V, "E": E, "chunk": C, "seed": cfg.seed},
        "kernels_ms": kern,
        "roofline": {"bound": "mfma", "achieved": round(tflops, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(tflops / PEAK_BF16_TFLOPS, 4),
                     "kernel": "prep + fwd_recurrent"}}
    if emit:
        print(json.dumps(res), flush=True)
    return res


def other_workloads(steps=10, warmup=20):
    """The inference forwards and the decode step, timed after the training
    step and reported beside it: throughput, time per call and the roofline
    fraction of each (each after at least 100 ms of untimed calls, see
    _warm_up: its inputs are generated on the host while the part idles)."""
    out = {}
    for name in ("sgla_bf16", "gdn_bf16", "gdn_long_bf16"):
        r = forward_bench(name, steps, warmup, emit=False)
        out[name + "_forward"] = {"value": r["value"], "unit": r["unit"],
                                  "ms_per_step": r["ms_per_step"], "config": r["config"],
                                  "mfma_frac": r["roofline"]["frac"]}
    r = decode_bench(steps, warmup, emit=False)
    out["gdn_decode_N256H16E16"] = {"value": r["value"], "unit": r["unit"],
                                    "ms_per_step": r["ms_per_step"], "config": r["config"],
                                    "hbm_frac": r["roofline"]["frac"]}
    return out


def gate_bench(steps, warmup):
    """The mixer's output side (RMSNorm times a sigmoid gate) forward and
    backward on the forward's output at the metric shape: B4 T4096 H8 V128
    rows, bf16.  HBM-bound; algorithmic bytes per element: forward 3 x 2 (o,
    z read, y written), backward 5 x 2 (o, z, dy read, d_o, dz written), plus
    the fp32 gain-gradient partials (1024 workgroups x V floats, written and
    read once)."""
    import torch
    import paper_2609_36529_amd as tla
    B, T, H, V = 4, 4096, 8, 128
    rows = B * T * H
    g = torch.Generator().manual_seed(17)
    o = torch.randn(rows, V, generator=g).to(torch.bfloat16).cuda()
    z = (2.0 * torch.randn(rows, V, generator=g)).to(torch.bfloat16).cuda()
    dy = torch.randn(rows, V, generator=g).to(torch.bfloat16).cuda()
    w = (1.0 + 0.5 * torch.randn(V, generator=g)).float().cuda()

    def one():
        tla.out_gate_fwd(o, z, w)
        tla.out_gate_bwd(o, z, w, dy)
    for _ in range(warmup):
        one()
    torch.cuda.synchronize()
    tla.prof_enable(True)
    t0 = time.perf_counter()
    for _ in range(steps):
        one()
    torch.cuda.synchronize()
    elapsed = (time.perf_counter() - t0) / steps
    prof = tla.prof_read()
    tla.prof_enable(False)
    kern = {k: round(v[0] / v[1], 4) for k, v in prof.items() if v[1]}
    part = 1024 * V * 4
    bytes_fwd, bytes_bwd = 6 * rows * V, 10 * rows * V + part
    gbs_f = bytes_fwd / (kern["out_gate_fwd"] * 1e-3) / 1e9
    gbs_b = bytes_bwd / (kern["out_gate_bwd"] * 1e-3) / 1e9
    print(json.dumps({
        "metric": "output gate fwd+bwd tokens/s, B4 T4096 H8 V128", "value": round(B * T / elapsed, 1),
        "unit": "tokens/s", "n_gpus": 1, "steps": steps, "warmup": warmup,
        "ms_per_step": round(1e3 * elapsed, 4), "higher_is_better": True, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "RMSNorm x sigmoid gate, forward and backward", "rows": rows, "V": V},
        "kernels_ms": kern,
        "roofline": {"bound": "hbm", "achieved": round(gbs_b, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(gbs_b / PEAK_HBM_GBS, 4), "kernel": "out_gate_bwd",
                     "forward_gbs": round(gbs_f, 1), "forward_frac": round(gbs_f / PEAK_HBM_GBS, 4)}}),
          flush=True)


def heads_bench(steps, warmup):
    """The mixer's gate heads (log forget gate g = -exp(A) softplus(x + b) per
    key slice, write strength beta = sigmoid(x_beta)) forward and backward at
    the metric shape: B4 T4096 H8 E8, bf16 pre-activations.  HBM-bound;
    algorithmic bytes per (token, head, slice): forward 2 + 4 (x read, g
    written), backward 2 + 4 + 2 (x, dg read, dx written); per (token, head):
    forward 2 + 4, backward 2 + 4 + 2; plus the backward's fp32 partials of
    dA, db (2 per column per 64 tokens, written and read once)."""
    import torch
    import paper_2609_36529_amd as tla
    B, T, H, E = 4, 4096, 8, 8
    n = B * T
    gen = torch.Generator().manual_seed(19)
    x = torch.randn(n, H, E, generator=gen).to(torch.bfloat16).cuda()
    xb = torch.randn(n, H, generator=gen).to(torch.bfloat16).cuda()
    A = torch.log(1.0 + 15.0 * torch.rand(H, E, generator=gen)).float().cuda()
    b = (-4.0 + torch.rand(H, E, generator=gen)).float().cuda()
    dg = torch.randn(n, H, E, generator=gen).float().cuda()
    dbeta = torch.randn(n, H, generator=gen).float().cuda()

    def one():
        tla.gate_heads_fwd(x, xb, A, b)
        tla.gate_heads_bwd(x, xb, A, b, dg, dbeta)
    for _ in range(warmup):
        one()
    torch.cuda.synchronize()
    tla.prof_enable(True)
    t0 = time.perf_counter()
    for _ in range(steps):
        one()
    torch.cuda.synchronize()
    elapsed = (time.perf_counter() - t0) / steps
    prof = tla.prof_read()
    tla.prof_enable(False)
    kern = {k: round(v[0] / v[1], 4) for k, v in prof.items() if v[1]}
    part = 2 * 2 * ((n + 63) // 64) * H * E * 4
    bytes_fwd = 6 * n * H * E + 6 * n * H
    bytes_bwd = 8 * n * H * E + 8 * n * H + part
    gbs_f = bytes_fwd / (kern["gate_heads_fwd"] * 1e-3) / 1e9
    gbs_b = bytes_bwd / (kern["gate_heads_bwd"] * 1e-3) / 1e9
    print(json.dumps({
        "metric": "gate heads fwd+bwd tokens/s, B4 T4096 H8 E8", "value": round(n / elapsed, 1),
        "unit": "tokens/s", "n_gpus": 1, "steps": steps, "warmup": warmup,
        "ms_per_step": round(1e3 * elapsed, 4), "higher_is_better": True, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "forget gate and write strength heads, forward and backward",
                   "tokens": n, "H": H, "E": E},
        "kernels_ms": kern,
        "roofline": {"bound": "hbm", "achieved": round(gbs_b, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(gbs_b / PEAK_HBM_GBS, 4), "kernel": "gate_heads_bwd",
                     "forward_gbs": round(gbs_f, 1), "forward_frac": round(gbs_f / PEAK_HBM_GBS, 4)}}),
          flush=True)


def conv_bench(steps, warmup):
    """The mixer's input side after the projection GEMM (causal depthwise
    convolution of width 4, SiLU / softplus, L2 normalisation) forward and
    backward at the metric shape: B4 T4096 H8 K=V=128 E=8, bf16, Ctot = 3200
    channels per token.  HBM-bound; algorithmic bytes per token and channel:
    forward 2 + 2 (y read, output written), backward 2 + 2 + 2 (y and the
    output gradient read, dy written), plus the fp32 tap-gradient partials
    (written and read once)."""
    import torch
    import paper_2609_36529_amd as tla
    B, T, H, K, V, E, W = 4, 4096, 8, 128, 128, 8, 4
    C = H * (2 * K + V + 2 * E)
    gen = torch.Generator().manual_seed(23)
    y = torch.randn(B, T, C, generator=gen).to(torch.bfloat16).cuda()
    w = ((torch.rand(W, C, generator=gen) * 2 - 1) / W ** 0.5).float().cuda()
    grads = tuple(torch.randn(B, T, H, d, generator=gen).to(torch.bfloat16).cuda() for d in (K, K, V, E, E))

    def one():
        tla.conv_in_fwd(y, w, H, K, V, E)
        tla.conv_in_bwd(y, w, H, K, V, E, grads)
    for _ in range(warmup):
        one()
    torch.cuda.synchronize()
    tla.prof_enable(True)
    t0 = time.perf_counter()
    for _ in range(steps):
        one()
    torch.cuda.synchronize()
    elapsed = (time.perf_counter() - t0) / steps
    prof = tla.prof_read()
    tla.prof_enable(False)
    kern = {k: round(v[0] / v[1], 4) for k, v in prof.items() if v[1]}
    n = B * T
    parts = (B * ((T + 31) // 32) + 3) // 4
    bytes_fwd = 4 * n * C
    bytes_bwd = 6 * n * C + 2 * parts * W * C * 4
    gbs_f = bytes_fwd / (kern["conv_in_fwd"] * 1e-3) / 1e9
    gbs_b = bytes_bwd / (kern["conv_in_bwd"] * 1e-3) / 1e9
    print(json.dumps({
        "metric": "input side fwd+bwd tokens/s, B4 T4096 H8 K=V=128 E=8 W4", "value": round(n / elapsed, 1),
        "unit": "tokens/s", "n_gpus": 1, "steps": steps, "warmup": warmup,
        "ms_per_step": round(1e3 * elapsed, 4), "higher_is_better": True, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "causal depthwise conv + SiLU/softplus + L2 norm, forward and backward",
                   "tokens": n, "channels": C, "taps": W},
        "kernels_ms": kern,
        "roofline": {"bound": "hbm", "achieved": round(gbs_b, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(gbs_b / PEAK_HBM_GBS, 4), "kernel": "conv_in_bwd",
                     "forward_gbs": round(gbs_f, 1), "forward_frac": round(gbs_f / PEAK_HBM_GBS, 4)}}),
          flush=True)


def proj_bench(steps, warmup):
    """The mixer's input projection with its epilogue fused (section "Input
    projections", Alg. 2) at d_model 2048 (the 1.3B block) for this bench's
    8 heads, B4 T4096 K=V=128 E=8 W4: forward tla_proj_in_fwd (GEMM u Wp^T
    into the convolution, activations and norms, keeping y for the backward)
    and backward tla_proj_in_bwd (input-side backward, transposes, the du and
    dWp GEMMs).  MFMA-bound; algorithmic FLOP: forward 2 n Ctot Dm (the
    16-row halo that each 256-token tile recomputes is not counted),
    backward twice that."""
    import torch
    import paper_2609_36529_amd as tla
    B, T, Dm, H, K, V, E, W = 4, 4096, 2048, 8, 128, 128, 8, 4
    C = H * (2 * K + V + 2 * E)
    gen = torch.Generator().manual_seed(29)
    u = torch.randn(B, T, Dm, generator=gen).to(torch.bfloat16).cuda()
    Wp = (torch.randn(C, Dm, generator=gen) / Dm ** 0.5).to(torch.bfloat16).cuda()
    w = ((torch.rand(W, C, generator=gen) * 2 - 1) / W ** 0.5).float().cuda()
    grads = tuple(torch.randn(B, T, H, d, generator=gen).to(torch.bfloat16).cuda() for d in (K, K, V, E, E))

    def one():
        outs = tla.proj_in_fwd(u, Wp, w, H, K, V, E, keep_y=True)
        tla.proj_in_bwd(u, Wp, w, outs[5], H, K, V, E, grads)
    for _ in range(warmup):
        one()
    torch.cuda.synchronize()
    tla.prof_enable(True)
    t0 = time.perf_counter()
    for _ in range(steps):
        one()
    torch.cuda.synchronize()
    elapsed = (time.perf_counter() - t0) / steps
    prof = tla.prof_read()
    tla.prof_enable(False)
    kern = {k: round(v[0] / v[1], 4) for k, v in prof.items() if v[1]}
    n = B * T
    flop_fwd = 2.0 * n * C * Dm
    tf_f = flop_fwd / (kern["proj_in_fwd"] * 1e-3) / 1e12
    tf_g = 2 * flop_fwd / (kern["proj_gemm"] * 1e-3) / 1e12

    # context only: the library GEMM that PyTorch calls for the same three
    # products (plain 2-D products of resident bf16 tensors, no epilogue)
    def lib_gemm_ms(a, b_t):
        for _ in range(5):
            torch.matmul(a, b_t)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            torch.matmul(a, b_t)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps
    u2, dy2 = u.reshape(n, Dm), torch.randn(n, C, generator=gen).to(torch.bfloat16).cuda()
    lib = {"u Wp^T (16384 x 3200 x 2048)": lib_gemm_ms(u2, Wp.t().contiguous()),
           "dy Wp (16384 x 2048 x 3200)": lib_gemm_ms(dy2, Wp),
           "dy^T u (3200 x 2048 x 16384)": lib_gemm_ms(dy2.t(), u2)}
    lib = {k: round(v, 4) for k, v in lib.items()}
    print(json.dumps({
        "metric": "input projection fwd+bwd tokens/s, B4 T4096 d_model 2048 H8 K=V=128 E=8 W4",
        "value": round(n / elapsed, 1), "unit": "tokens/s", "n_gpus": 1, "steps": steps,
        "warmup": warmup, "ms_per_step": round(1e3 * elapsed, 4), "higher_is_better": True,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "projection GEMM with fused conv + SiLU/softplus + L2 norm, forward and backward",
                   "tokens": n, "d_model": Dm, "channels": C, "taps": W},
        "kernels_ms": kern,
        "roofline": {"bound": "mfma", "achieved": round(tf_f, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(tf_f / PEAK_BF16_TFLOPS, 4), "kernel": "proj_in_fwd",
                     "backward_gemm_tflops": round(tf_g, 1),
                     "backward_gemm_frac": round(tf_g / PEAK_BF16_TFLOPS, 4)},
        "library_gemm_ms_context": lib}),
          flush=True)


def mfma_peak_bench(steps, warmup):
    """Measured side of the MFMA roofline's peak: back-to-back bf16 MFMAs on
    register accumulators (no memory traffic), 16x16x32 and 32x32x16, at one
    and two waves per SIMD (256 and 512 workgroups of four waves on the 256
    compute units), timed with HIP events on the launch stream."""
    import torch
    import paper_2609_36529_amd as tla
    sink = torch.empty(512 * 256, dtype=torch.float32, device="cuda")
    iters = 4000
    res = []
    for shape, name in ((0, "16x16x32"), (1, "32x32x16")):
        for blocks in (256, 512):
            for _ in range(max(warmup, 3)):
                tla.mfma_rate(shape, blocks, iters, sink)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            flop = 0
            for _ in range(steps):
                flop += tla.mfma_rate(shape, blocks, iters, sink)
            b.record()
            torch.cuda.synchronize()
            tf = flop / (a.elapsed_time(b) * 1e-3) / 1e12
            res.append({"mfma": name, "waves_per_simd": blocks // 256, "tflops": round(tf, 1),
                        "frac_of_datasheet": round(tf / PEAK_BF16_TFLOPS, 4)})
    best = max(r["tflops"] for r in res)
    print(json.dumps({
        "metric": "bf16 MFMA rate, register accumulators", "value": best, "unit": "TFLOP/s", "n_gpus": 1,
        "steps": steps, "warmup": warmup, "higher_is_better": True, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "back-to-back MFMAs on independent accumulators, no memory traffic"},
        "datasheet_peak": PEAK_BF16_TFLOPS, "runs": res}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    # (the part needs about 70 ms of work before its clocks settle: with 3
    # warm-up steps the timed training steps ran about 5% slower)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the inference forwards and decode reported beside the training step")
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--pmc-summary", nargs=4, metavar="DIR")
    ap.add_argument("--decode", action="store_true",
                    help="time the decode step instead (its own JSON line)")
    ap.add_argument("--gate", action="store_true",
                    help="time the output gate (RMSNorm x sigmoid) forward and backward")
    ap.add_argument("--heads", action="store_true",
                    help="time the gate heads (forget gate, write strength) forward and backward")
    ap.add_argument("--conv", action="store_true",
                    help="time the input side (short convolution, activations, L2 norm) forward and backward")
    ap.add_argument("--mfma-peak", action="store_true",
                    help="measure the bf16 MFMA rate with no memory traffic (the roofline's measured peak)")
    ap.add_argument("--proj", action="store_true",
                    help="time the fused input projection (GEMM + input side) forward and backward")
    ap.add_argument("--forward", metavar="NAME",
                    help="time the inference forward of sgla_bf16, gdn_bf16 or gdn_long_bf16")
    args = ap.parse_args()
    if args.pmc_summary:
        pmc_summary(*args.pmc_summary)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the operator's work shards over batch, heads "
              "and value tiles with no exchange, so per-GPU throughput at N GPUs is the N=1 "
              "figure; it takes no multi-GPU runs.", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return
    if args.decode:
        decode_bench(args.steps, args.warmup)
        return
    if args.gate:
        gate_bench(args.steps, args.warmup)
        return
    if args.heads:
        heads_bench(args.steps, args.warmup)
        return
    if args.conv:
        conv_bench(args.steps, args.warmup)
        return
    if args.proj:
        proj_bench(args.steps, args.warmup)
        return
    if args.mfma_peak:
        mfma_peak_bench(args.steps, args.warmup)
        return
    if args.forward:
        forward_bench(args.forward, args.steps, args.warmup)
        return

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
    stream = torch.cuda.current_stream(dev)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev[0].record(stream)
    for i in range(args.steps):
        step()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    prof = tla.prof_read()
    tla.prof_enable(False)
    warm = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps))
    # cold cache: a 512 MiB write between steps evicts the inputs, states
    # and intermediates from the 256 MB last-level cache; each step alone is
    # timed with events on the launch stream
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    cold = []
    for _ in range(args.steps):
        flush.fill_(1)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        step()
        b.record(stream)
        b.synchronize()
        cold.append(a.elapsed_time(b))
    cold.sort()
    del flush

    ms_per_step = 1e3 * elapsed / args.steps
    tokens = B * T
    alg = algorithmic(cfg)
    token_heads = B * T * H
    kernels = {}
    for name, (tot, n) in prof.items():
        if n == 0:
            continue
        avg_ms = tot / n
        a = alg[name]
        entry = {"avg_ms": round(avg_ms, 4), "launches": n, "bound": bound_of(name, a),
                 "tflops": round(a["flops"] * token_heads / (avg_ms * 1e-3) / 1e12, 2),
                 "gbs": round(a["bytes"] * token_heads / (avg_ms * 1e-3) / 1e9, 1)}
        entry["frac"] = round(entry["tflops"] / PEAK_BF16_TFLOPS if entry["bound"] == "mfma"
                              else entry["gbs"] / PEAK_HBM_GBS, 4)
        kernels[name] = entry
    dom = max(kernels, key=lambda k: kernels[k]["avg_ms"] * kernels[k]["launches"])
    kd = kernels[dom]
    if kd["bound"] == "hbm":
        roof = {"bound": "hbm", "achieved": kd["gbs"], "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    else:
        roof = {"bound": "mfma", "achieved": kd["tflops"], "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof["traffic"], roof["traffic_over_algorithmic"] = traffic_for(dom, alg[dom]["bytes"],
                                                                    token_heads)
    roof["kernel"] = dom
    roof["algorithmic_per_launch"] = {"flops": alg[dom]["flops"] * token_heads,
                                      "bytes": alg[dom]["bytes"] * token_heads}
    step_tflops = alg["total_flops"] * token_heads / (ms_per_step * 1e-3) / 1e12

    result = {
        "metric": "fwd+bwd tokens/s and MFMA % of bf16 peak, triadic GDN H=8 K=V=128 E=8 T=4096",
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
        "ms_per_step_median": round(warm[len(warm) // 2], 4),
        "ms_per_step_min": round(warm[0], 4),
        "cold_cache": {"ms_per_step_median": round(cold[len(cold) // 2], 4),
                       "ms_per_step_min": round(cold[0], 4),
                       "flush": "512 MiB device write before each step"},
        "step_tflops": round(step_tflops, 2),
        "mfma_pct_of_bf16_peak": round(100.0 * step_tflops / PEAK_BF16_TFLOPS, 2),
        "kernels": kernels,
        "roofline": roof,
    }
    if not args.no_extras:
        del ws_f, ws_b, saved, grads
        torch.cuda.empty_cache()
        result["other_workloads"] = other_workloads()
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(cfg, inp, dO)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
