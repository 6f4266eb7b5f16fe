"""Benchmark of the RateQuant hot path on one MI355X.

One step = one pass of the whole path over the Llama-3-8B shaped workload
(32 layers, batch 16, 8 kv-heads, 32 query heads, head_dim 128, bf16,
KIVI g32 with a 32-token window, bits {1..4} at 2.5 average):

  1. distortion sweep at 1..4 bits over 512 calibration tokens of every
     key and value component (512 components), with the least-squares fit;
  2. bit allocation for the 512 components (greedy + continuous optimum);
  3. bit table -> cache layout;
  4. prefill quantization of 8191 tokens per sequence, all layers;
  5. one decode step: append the 8192nd token (one 32-token block leaves
     the window and is quantized), all layers;
  6. decode attention over the 8192 cached tokens, all layers.

Inputs are seeded synthetic tensors already resident in HBM.  The printed
JSON line reports decode-attention effective HBM bandwidth (algorithmic
bytes / time) as `value`, KV-quantize tokens/s, the roofline of the
dominant kernel measured live with HIP events, and the numpy oracle timed on
a bounded sample on the host.
"""
import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=5)
    p.add_argument("--warmup", type=int, default=2)
    p.add_argument("--workload", default="llama3-8b-kv-b16-t8192-kivi-2.5b")
    p.add_argument("--cpu-seconds", type=float, default=15.0,
                   help="budget of the oracle CPU-baseline sample")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--calib-tokens", type=int, default=512)
    return p.parse_args()


def attention_bytes(wl, bits_table, T):
    """Algorithmic bytes one layer of decode attention must move."""
    R = wl.residual
    nq = max(0, ((T - R) // 32) * 32)
    B, H, Hq = wl.batch, wl.n_kv_heads, wl.n_q_heads
    total = 0
    for l in range(bits_table.shape[0]):
        codes = sum(B * nq * 128 * int(b) // 8 for b in bits_table[l].reshape(-1))
        per_blk = 512 if wl.family == 0 else 64
        meta = B * H * 2 * (nq // 32) * per_blk
        resid = B * H * 2 * (T - nq) * 128 * 2
        qo = B * Hq * 128 * (2 + 4)
        total += codes + meta + resid + qo
    return total


def quantize_bytes(wl, bits_table, T):
    """Algorithmic bytes of quantizing T tokens of every layer: 16-bit K
    and V read once, codes + metadata written, window written."""
    B, H = wl.batch, wl.n_kv_heads
    R = wl.residual
    nq = max(0, ((T - R) // 32) * 32)
    per_blk = 512 if wl.family == 0 else 64
    total = 0
    for l in range(bits_table.shape[0]):
        rd = 2 * B * H * T * 128 * 2
        codes = sum(B * nq * 128 * int(b) // 8 for b in bits_table[l].reshape(-1))
        meta = B * H * 2 * (nq // 32) * per_blk
        win = B * H * 2 * (T - nq) * 128 * 2
        total += rd + codes + meta + win
    return total


def cpu_baseline(wl, bits_table, seconds):
    """The oracle (numpy), as it stands, on a bounded sample of the same
    workload: whole (layer, batch entry, kv-head) units, each quantized
    and packed by the oracle (its cache builder), then decode attention read
    back from the packed codes (unpack + dequantize + fp64 attention).  Units
    are added until the time budget is spent.  Reports the attention rate in
    the metric's unit (algorithmic bytes / oracle attention time) and the
    quantize rate in whole-model tokens per second."""
    from threadpoolctl import threadpool_limits

    import workloads
    from oracle import attention as oatt
    from oracle import cache as ocache
    from oracle import quant as oq

    T = wl.context
    R = wl.residual
    nq = max(0, ((T - R) // 32) * 32)
    G = wl.group
    att_bytes, t_att, t_q, units = 0, 0.0, 0.0, 0
    with threadpool_limits(limits=1):
        for l, b in ((l, b) for l in range(wl.n_layers)
                     for b in range(wl.batch)):
            if t_att + t_q >= seconds:
                break
            q16 = workloads.q_cpu(wl, l)
            k16, v16 = workloads.kv_cpu(wl, l, b, T)
            for h in range(wl.n_kv_heads):
                k = workloads.u16_to_f32(k16[h], wl.dtype)
                v = workloads.u16_to_f32(v16[h], wl.dtype)
                bk, bv = int(bits_table[l, h, 0]), int(bits_table[l, h, 1])
                q = workloads.u16_to_f32(q16[b, h * G:(h + 1) * G], wl.dtype)
                t0 = time.perf_counter()
                u = ocache.Unit(wl.family, k, v, bk, bv, R)   # quantize + pack
                t1 = time.perf_counter()
                kc = ocache.unpack_keys(u.k_words, bk)
                vc = ocache.unpack_values(u.v_words, bv)
                ks = np.concatenate([oq.kivi_dequant_keys(
                    kc, *_kivi_meta_keys(u.k_meta)), u.k_res])
                vs = np.concatenate([oq.kivi_dequant_values(
                    vc, *_kivi_meta_values(u.v_meta)), u.v_res])
                oatt.decode_attention(q, ks, vs)
                t2 = time.perf_counter()
                t_q += t1 - t0
                t_att += t2 - t1
                units += 1
                att_bytes += (nq * 128 * (bk + bv) // 8 + 2 * (nq // 32) * 512
                              + 2 * (T - nq) * 256 + G * 128 * 6)
    # a whole-model token is one token of every (layer, kv-head)
    q_tok_s = units * T / (wl.n_layers * wl.n_kv_heads) / t_q
    return {"value": round(att_bytes / t_att / 1e9, 4), "unit": "GB/s",
            "cores": 1, "kind": "oracle",
            "quantize_tok_s": round(q_tok_s, 1),
            "sample": f"{units} (layer, batch, kv-head) units, {T} tokens "
                      f"each: oracle quantize + pack ({t_q:.1f} s), then "
                      f"unpack + dequantize + fp64 decode attention "
                      f"({t_att:.1f} s); single thread"}


TRAFFIC = os.path.join(ROOT, "profiles", "hbm_traffic.json")


def kernel_sources_digest(name):
    """sha256 over the sources a kernel is built from: counters taken on
    an older build no longer describe it."""
    import glob
    import hashlib
    csrc = os.path.join(ROOT, "paper_2605_06675_amd", "csrc")
    pats = {"quantize_kernel": ["rq_quant.hip"],
            "attn_kernel": ["rq_attn*.hip", "rq_attn_impl.h"]}[name]
    files = sorted(f for p in pats + ["rq_device.h", "rq_internal.h"]
                   for f in glob.glob(os.path.join(csrc, p)))
    h = hashlib.sha256()
    for f in files:
        with open(f, "rb") as fh:
            h.update(os.path.basename(f).encode() + b"\0" + fh.read())
    return h.hexdigest()


def measured_traffic(name):
    """HBM bytes per launch from the committed rocprofv3 FETCH_SIZE and
    WRITE_SIZE passes (scaled by the copy-kernel calibration), or None when
    none were taken or the kernel's sources changed since."""
    try:
        with open(TRAFFIC) as f:
            rec = json.load(f).get(name)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("sources_sha256") != kernel_sources_digest(name):
        return None
    return int(rec["fetch_bytes"] * rec["fetch_factor"]
               + rec["write_bytes"] * rec["write_factor"])


def _kivi_meta_keys(m):
    from oracle import fmt
    s = fmt.from_pair_order(m[:, :, 0, :]).reshape(m.shape[0], 128)
    z = fmt.from_pair_order(m[:, :, 1, :]).reshape(m.shape[0], 128)
    return s, z


def _kivi_meta_values(m):
    from oracle import fmt
    nb = m.shape[0]
    s = fmt.from_pair_order(m[:, :, 0, :]).transpose(0, 2, 1).reshape(nb * 32, 4)
    z = fmt.from_pair_order(m[:, :, 1, :]).transpose(0, 2, 1).reshape(nb * 32, 4)
    return s, z


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus must "
                          "be 1 (the path shards by kv-head/batch with no "
                          "exchange, see the design notes)"}))
        sys.exit(2)
    import torch

    import paper_2605_06675_amd as rq
    import workloads

    rq.lib()
    wl = workloads.WORKLOADS[args.workload]
    if wl.family != workloads.KIVI:
        raise SystemExit("bench drives the KIVI workloads")
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    L, B, H, Hq, T = wl.n_layers, wl.batch, wl.n_kv_heads, wl.n_q_heads, wl.context
    lo, hi = min(wl.bit_set), max(wl.bit_set)
    n_comp = wl.n_comp

    # ---- inputs, resident in HBM before timing
    w, alpha_p, beta_p = workloads.allocation_inputs(wl)
    bits0, _, _ = rq.rq_allocate_bits(w, alpha_p, beta_p, wl.avg_bits, lo, hi)
    table = bits0.reshape(L, H, 2)
    KV = [workloads.kv_device(wl, l) for l in range(L)]
    Q = [workloads.q_device(wl, l) for l in range(L)]
    calib = workloads.calib_cpu(n_comp, args.calib_tokens, wl.dtype)
    td = workloads.torch_dtype(wl.dtype)
    calib_k = torch.from_numpy(calib[: n_comp // 2].view(np.int16)).view(td).to(dev)
    calib_v = torch.from_numpy(calib[n_comp // 2:].view(np.int16)).view(td).to(dev)
    cal_bits = [1, 2, 3, 4]
    cal_ws = torch.empty(rq.rq_calibrate_workspace(n_comp // 2,
                                                   args.calib_tokens, 4),
                         dtype=torch.uint8, device=dev)
    kvc = rq.KVCache(wl.family, wl.dtype, L, B, H, Hq, T, wl.residual, table,
                     device=dev)
    ws = kvc.workspace(T)
    outs = [torch.empty((B, Hq, 128), dtype=torch.float32, device=dev)
            for _ in range(L)]
    torch.cuda.synchronize()

    ev = lambda: torch.cuda.Event(enable_timing=True)
    phases = ("calib", "quantize", "append", "attention")

    # the slices k[:, :, :T-1] are views; the library needs contiguous
    # inputs, so keep contiguous copies of the prefill part and the last
    # token (setup, untimed)
    KV = [(k[:, :, : T - 1].contiguous(), v[:, :, : T - 1].contiguous(),
           k[:, :, T - 1:].contiguous(), v[:, :, T - 1:].contiguous())
          for (k, v) in KV]

    def step(rec):
        e = {p: (ev(), ev()) for p in phases}
        t_host = {}
        e["calib"][0].record()
        r1 = rq.rq_calibrate_distortion(wl.family, wl.dtype, calib_k, 0,
                                        cal_bits, ws=cal_ws)
        r2 = rq.rq_calibrate_distortion(wl.family, wl.dtype, calib_v, 1,
                                        cal_bits, ws=cal_ws)
        e["calib"][1].record()
        t0 = time.perf_counter()
        bits, cont, J = rq.rq_allocate_bits(w, alpha_p, beta_p, wl.avg_bits,
                                            lo, hi)
        assert np.array_equal(bits, bits0)
        rq.rq_cache_sizes(kvc.desc)
        t_host["alloc"] = time.perf_counter() - t0
        e["quantize"][0].record()
        for l in range(L):
            rq.rq_quantize_kv(kvc.desc, l, 0, KV[l][0], KV[l][1])
        e["quantize"][1].record()
        e["append"][0].record()
        for l in range(L):
            rq.rq_quantize_kv(kvc.desc, l, T - 1, KV[l][2], KV[l][3])
        e["append"][1].record()
        e["attention"][0].record()
        for l in range(L):
            rq.rq_decode_attention(kvc.desc, l, T, Q[l], outs[l], ws)
        e["attention"][1].record()
        rec.append((e, t_host, (r1, r2)))

    for _ in range(args.warmup):
        step([])
    torch.cuda.synchronize()
    rec = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(rec)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    ms = {p: float(np.mean([r[0][p][0].elapsed_time(r[0][p][1]) for r in rec]))
          for p in phases}
    alloc_ms = float(np.mean([r[1]["alloc"] for r in rec])) * 1e3
    att_bytes = attention_bytes(wl, table, T)
    q_bytes = quantize_bytes(wl, table, T - 1)
    att_gbs = att_bytes / (ms["attention"] * 1e-3) / 1e9
    # KV quantize tok/s: B * T tokens through all L layers' K and V
    q_tok_s = B * (T - 1) / (ms["quantize"] * 1e-3)
    q_gbs = q_bytes / (ms["quantize"] * 1e-3) / 1e9
    # per-launch figures: the phases are L back-to-back launches on the
    # stream the events were recorded on
    kernels = {
        "quantize_kernel": {
            "call": "rq_quantize_kv prefill of one layer (quantize_kernel; "
                    "ring_kernel writes the window)",
            "bytes": q_bytes / L, "us": ms["quantize"] * 1e3 / L},
        "attn_kernel": {
            "call": "rq_decode_attention of one layer (attn_kernel)",
            "bytes": att_bytes / L, "us": ms["attention"] * 1e3 / L},
    }
    rooflines = {}
    for name, k in kernels.items():
        ach = k["bytes"] / (k["us"] * 1e-6) / 1e9
        rooflines[name] = {
            "bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
            "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4),
            "traffic": measured_traffic(name), "kernel": name,
            "call": k["call"], "bytes_per_launch": int(k["bytes"]),
            "avg_launch_us": round(k["us"], 2)}
    # the kernel that takes the most time in a step
    dom = max(kernels, key=lambda n: kernels[n]["us"])
    roofline = rooflines[dom]
    r1, r2 = rec[-1][2]
    beta_fit = np.concatenate([r1[2], r2[2]])
    line = {
        "metric": "mixed-bit decode attention effective HBM GB/s (% of peak); "
                  "KV quantize tok/s",
        "value": round(att_gbs, 1),
        "unit": "GB/s",
        "pct_of_peak": round(100 * att_gbs / PEAK_HBM_GBS, 2),
        "quantize_tok_s": round(q_tok_s, 0),
        "quantize_gbs": round(q_gbs, 1),
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 3),
        "phase_ms": {**{p: round(v, 3) for p, v in ms.items()},
                     "alloc_host": round(alloc_ms, 3)},
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        # inputs are 16-bit; quantization runs in fp32, attention on fp16
        # matrix-core operands with fp32 accumulation and softmax
        "dtype": "f16/f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "layers": L, "batch": B,
                   "kv_heads": H, "q_heads": Hq, "head_dim": 128,
                   "context": T, "residual_window": wl.residual,
                   "avg_bits": wl.avg_bits, "bit_set": list(wl.bit_set),
                   "attention_bytes_per_step": att_bytes,
                   "quantize_bytes_per_step": q_bytes,
                   "fitted_beta_median": round(float(np.median(beta_fit)), 3)},
        "roofline": roofline,
        "roofline_by_kernel": rooflines,
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl, table, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
