"""Benchmark of the RateQuant hot path on one MI355X.

One step = one pass of the whole path over one workload (default: the
Llama-3-8B shaped one -- 32 layers, batch 16, 8 kv-heads, 32 query heads,
head_dim 128, bf16, KIVI g32 with a 32-token window, bits {1..4} at 2.5
average):

  1. distortion sweep over 512 calibration tokens of every key and value
     component at the workload's bit-widths, with the least-squares fit;
  2. bit allocation for all components (greedy + continuous optimum);
  3. bit table -> cache layout;
  4. prefill quantization of the context (less the decode steps), all
     layers;
  5. the decode steps (one for most workloads; 64 for the long-context
     one): append one token per layer (a 32-token block leaves the window
     and is quantized when due) and decode attention over the whole cache,
     all layers.

Inputs are seeded synthetic tensors already resident in HBM.  The printed
JSON line reports decode-attention effective HBM bandwidth (algorithmic
bytes / time) as `value`, KV-quantize tokens/s, the roofline of the kernel
that takes the most time in a step (HIP events on the stream the library
launches on), and the oracle timed on a bounded sample on the host.
"""
import argparse
import glob
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
TRAFFIC = os.path.join(ROOT, "profiles", "hbm_traffic.json")
DEFAULT = "llama3-8b-kv-b16-t8192-kivi-2.5b"
# decode steps per workload (the long-context workload runs 64)
STEPS = {"qwen3-32b-kv-b1-t131072-kivi-2b": 64}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default=DEFAULT)
    p.add_argument("--cpu-seconds", type=float, default=8.0,
                   help="budget of each oracle CPU-baseline sample (one core, "
                        "then all cores)")
    p.add_argument("--cpu-workers", type=int, default=0,
                   help="processes of the all-core sample (0: the cores this "
                        "process may run on, at most 16)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-extras", action="store_true",
                   help="skip the measurements outside the step (sensitivity, "
                        "stream ceiling, uniform and fused comparisons), e.g. "
                        "under counter collection")
    p.add_argument("--calib-tokens", type=int, default=512)
    return p.parse_args()


def meta_pair_bytes(family):
    """Metadata bytes of one 32-token block of K plus one of V: 512 for a
    KIVI-style side (scale and zero point per group), 64 for a per-token
    side (one fp16 scale or norm per token)."""
    k = 512 if family in (0, 4) else 64
    v = 512 if family == 0 else 64
    return k + v


def n_quantized(T, R):
    return max(0, ((T - R) // 32) * 32)


def attention_bytes(wl, bits_table, T):
    """Algorithmic bytes of decode attention over T tokens, all layers:
    codes at their widths, metadata, the 16-bit window, queries, outputs."""
    nq = n_quantized(T, wl.residual)
    B, H, Hq = wl.batch, wl.n_kv_heads, wl.n_q_heads
    total = 0
    for l in range(bits_table.shape[0]):
        codes = sum(B * nq * 128 * int(b) // 8 for b in bits_table[l].reshape(-1))
        meta = B * H * (nq // 32) * meta_pair_bytes(wl.family)
        resid = B * H * 2 * (T - nq) * 128 * 2
        qo = B * Hq * 128 * (2 + 4)
        total += codes + meta + resid + qo
    return total


def quantize_bytes(wl, bits_table, T):
    """Algorithmic bytes of quantizing T tokens of every layer: 16-bit K
    and V read once, codes + metadata written, window written."""
    B, H = wl.batch, wl.n_kv_heads
    nq = n_quantized(T, wl.residual)
    total = 0
    for l in range(bits_table.shape[0]):
        rd = 2 * B * H * T * 128 * 2
        codes = sum(B * nq * 128 * int(b) // 8 for b in bits_table[l].reshape(-1))
        meta = B * H * (nq // 32) * meta_pair_bytes(wl.family)
        win = B * H * 2 * (T - nq) * 128 * 2
        total += rd + codes + meta + win
    return total


def _oracle_units(job):
    """The kv-heads of one (layer, batch entry) through the oracle, one unit
    at a time: quantize + pack (its cache builder), then unpack + dequantize
    + fp64 decode attention from the packed codes.  Inputs are generated
    first and not timed.  Returns [(quantize s, attention s, algorithmic
    attention bytes)] and the process id."""
    import workloads
    from oracle import attention as oatt
    from oracle import cache as ocache
    from oracle import fmt
    from oracle import quant as oq
    wname, l, b, heads = job
    wl = workloads.WORKLOADS[wname]
    T, R, G = wl.context, wl.residual, wl.group
    nq = n_quantized(T, R)
    mb = meta_pair_bytes(wl.family)
    q16 = workloads.q_cpu(wl, l)
    k16, v16 = workloads.kv_cpu(wl, l, b, T)
    out = []
    for h, bk, bv in heads:
        k = workloads.u16_to_f32(k16[h], wl.dtype)
        v = workloads.u16_to_f32(v16[h], wl.dtype)
        q = workloads.u16_to_f32(q16[b, h * G:(h + 1) * G], wl.dtype)
        rot = None
        if wl.family == workloads.TURBO:
            rot = workloads.u16_to_f32(workloads.turbo_rotation(42, l, h),
                                       workloads.BF16).astype(np.float64)
        t0 = time.perf_counter()
        u = ocache.Unit(wl.family, k, v, bk, bv, R, rotation=rot)
        t1 = time.perf_counter()
        kc = ocache.unpack_keys(u.k_words, bk)
        vc = ocache.unpack_values(u.v_words, bv)
        if wl.family == workloads.KIVI:
            kh = oq.kivi_dequant_keys(kc, *_kivi_meta_keys(u.k_meta))
            vh = oq.kivi_dequant_values(vc, *_kivi_meta_values(u.v_meta))
        elif wl.family == workloads.KIVI_RTN:
            kh = oq.kivi_dequant_keys(kc, *_kivi_meta_keys(u.k_meta))
            nv = fmt.from_pair_order(u.v_meta).reshape(-1)
            vh = oq.rtn_dequant(vc, nv, bv)
        else:
            nk = fmt.from_pair_order(u.k_meta).reshape(-1)
            nv = fmt.from_pair_order(u.v_meta).reshape(-1)
            if wl.family == workloads.QUAROT:
                kh, vh = oq.quarot_dequant(kc, nk, bk), oq.quarot_dequant(vc, nv, bv)
            elif wl.family == workloads.RTN:
                kh, vh = oq.rtn_dequant(kc, nk, bk), oq.rtn_dequant(vc, nv, bv)
            else:
                kh = oq.turbo_dequant(kc, nk, rot, bk)
                vh = oq.turbo_dequant(vc, nv, rot, bv)
        oatt.decode_attention(q, np.concatenate([kh, u.k_res]),
                              np.concatenate([vh, u.v_res]))
        t2 = time.perf_counter()
        nbytes = (nq * 128 * (bk + bv) // 8 + (nq // 32) * mb
                  + 2 * (T - nq) * 256 + G * 128 * 6)
        out.append((t1 - t0, t2 - t1, nbytes))
    return out, os.getpid()


def _pool_init():
    from threadpoolctl import threadpool_limits
    global _LIMITS
    _LIMITS = threadpool_limits(limits=1)


def _cpu_jobs(wl, bits_table):
    for l in range(wl.n_layers):
        for b in range(wl.batch):
            yield (wl.name, l, b, [(h, int(bits_table[l, h, 0]), int(bits_table[l, h, 1]))
                                   for h in range(wl.n_kv_heads)])


def _cpu_rates(res, busy, wl):
    """Attention GB/s and whole-model quantize tok/s: the sample's bytes
    and tokens over the oracle time of the busiest process (busy: its
    (quantize s, attention s); the sums themselves on one core)."""
    nb = sum(r[2] for r in res)
    tok = len(res) * wl.context / (wl.n_layers * wl.n_kv_heads)
    return nb / busy[1] / 1e9, tok / busy[0]


def cpu_baseline(wl, bits_table, seconds, workers):
    """The oracle (numpy), as it stands, on bounded samples of the same
    workload: whole (layer, batch entry, kv-head) units, first on one core
    (one (layer, batch) row of units after another until about `seconds`
    of oracle time), then on every allowed core (one single-threaded
    process per core, the sample about `seconds` per process).  Only the
    oracle's work is timed, not the input generation.  Runs before the GPU
    is touched, so the worker processes are plain forks.  Reports the
    attention rate in the metric's unit (algorithmic bytes / oracle
    attention time) and the quantize rate in whole-model tokens per
    second."""
    import multiprocessing as mp
    import platform
    from threadpoolctl import threadpool_limits

    model = platform.processor() or "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    allowed = len(os.sched_getaffinity(0))
    n = workers or min(16, allowed)
    one, spent = [], 0.0
    with threadpool_limits(limits=1):
        for job in _cpu_jobs(wl, bits_table):
            res, _ = _oracle_units(job)
            one += res
            spent = sum(r[0] + r[1] for r in one)
            if spent >= seconds:
                break
    tq1, ta1 = sum(r[0] for r in one), sum(r[1] for r in one)
    a1, q1 = _cpu_rates(one, (tq1, ta1), wl)
    # all cores: about `seconds` of oracle work per process
    per_row = spent / (len(one) / wl.n_kv_heads)
    rows = max(n, int(round(seconds / per_row)) * n)
    batch = [j for _, j in zip(range(rows), _cpu_jobs(wl, bits_table))]
    ctx = mp.get_context("fork")
    t1 = time.perf_counter()
    with ctx.Pool(n, initializer=_pool_init) as pool:
        outs = pool.map(_oracle_units, batch, chunksize=1)
    wall = time.perf_counter() - t1
    many = [r for res, _ in outs for r in res]
    per_pid = {}
    for res, pid in outs:
        q, a = per_pid.get(pid, (0.0, 0.0))
        per_pid[pid] = (q + sum(r[0] for r in res), a + sum(r[1] for r in res))
    busy = (max(v[0] for v in per_pid.values()), max(v[1] for v in per_pid.values()))
    an, qn = _cpu_rates(many, busy, wl)
    return {"value": round(an, 4), "unit": "GB/s", "cores": len(per_pid),
            "kind": "oracle", "quantize_tok_s": round(qn, 1),
            "single_core": {"value": round(a1, 4), "unit": "GB/s",
                            "quantize_tok_s": round(q1, 1), "units": len(one),
                            "oracle_seconds": round(tq1 + ta1, 2)},
            "cpu_model": model, "nproc": os.cpu_count(), "allowed_cpus": allowed,
            "sample": f"{len(many)} (layer, batch, kv-head) units of "
                      f"{wl.context} tokens on {len(per_pid)} processes (busiest "
                      f"process {busy[0] + busy[1]:.1f} s of oracle time, {wall:.1f} s "
                      f"wall with input generation); single core: {len(one)} units, "
                      f"{tq1 + ta1:.1f} s: oracle quantize + pack, then unpack + "
                      f"dequantize + fp64 decode attention"}


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


# the mixed family quantizes its keys and its values with two kernels
QUANT_KERNEL = {0: "kivi_quant_kernel", 1: "sym_quant_kernel",
                2: "turbo_quant_kernel", 3: "sym_quant_kernel",
                4: "kivi_quant_kernel+sym_quant_kernel"}
KERNEL_SOURCES = {"kivi_quant_kernel": ["rq_quant.hip"],
                  "sym_quant_kernel": ["rq_quant.hip"],
                  "kivi_quant_kernel+sym_quant_kernel": ["rq_quant.hip"],
                  "turbo_quant_kernel": ["rq_quant_turbo.hip"],
                  "attn_kernel": ["rq_attn*.hip", "rq_attn_impl.h"]}


def kernel_sources_digest(name):
    """sha256 over the sources a kernel is built from: counters taken on
    an older build no longer describe it."""
    csrc = os.path.join(ROOT, "paper_2605_06675_amd", "csrc")
    files = sorted(f for p in KERNEL_SOURCES[name] + ["rq_device.h", "rq_internal.h"]
                   for f in glob.glob(os.path.join(csrc, p)))
    h = hashlib.sha256()
    for f in files:
        with open(f, "rb") as fh:
            h.update(os.path.basename(f).encode() + b"\0" + fh.read())
    return h.hexdigest()


def measured_traffic(workload, name):
    """HBM bytes per launch from the committed rocprofv3 FETCH_SIZE and
    WRITE_SIZE passes (scaled by the copy-kernel calibration), or None when
    none were taken or the kernel's sources changed since."""
    try:
        with open(TRAFFIC) as f:
            rec = json.load(f).get(workload, {}).get(name)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("sources_sha256") != kernel_sources_digest(name):
        return None
    return int(rec["fetch_bytes"] * rec["fetch_factor"]
               + rec["write_bytes"] * rec["write_factor"])


def sensitivity_rate(args, wl, dev):
    """Stage-1 sensitivity (outside the step: it runs once, offline, on
    gradients of a calibration set): rq_sensitivity over fp32 gradients of
    16 sequences x calib_tokens positions for every component of the model,
    timed per call (kernel, reduction, the copy of w and the wait) with HIP
    events, median of 5 after one warm-up."""
    import torch

    import paper_2605_06675_amd as rq
    S, T, n = 16, args.calib_tokens, wl.n_comp
    g = torch.Generator(device=dev).manual_seed(7)
    grad = torch.randn((S, n, T, 128), generator=g, device=dev,
                       dtype=torch.float32)
    ws = torch.empty(rq.rq_sensitivity_workspace(rq.RQ_F32, S, n, T),
                     dtype=torch.uint8, device=dev)
    rq.rq_sensitivity(rq.RQ_F32, grad, ws=ws)
    times = []
    for _ in range(5):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        rq.rq_sensitivity(rq.RQ_F32, grad, ws=ws)
        b.record()
        torch.cuda.synchronize()
        times.append(a.elapsed_time(b) * 1e3)
    us = float(np.median(times))
    nbytes = grad.numel() * 4
    del grad
    gbs = nbytes / (us * 1e-6) / 1e9
    return {"call": f"rq_sensitivity over fp32 gradients [{S}][{n}][{T}][128]",
            "kernel": "sens_kernel", "bound": "hbm", "bytes": nbytes,
            "us": round(us, 2), "achieved": round(gbs, 1), "unit": "GB/s",
            "peak": PEAK_HBM_GBS, "frac": round(gbs / PEAK_HBM_GBS, 4)}


def stream_ceiling(dev, gib=4, reps=10):
    """The device's streaming-read rate: rq_read_probe (a plain kernel of
    16-byte non-temporal loads) over a 4 GiB buffer, median of 10 calls."""
    import torch

    import paper_2605_06675_amd as rq
    buf = torch.empty(gib << 30, dtype=torch.uint8, device=dev)
    n_blocks = 4096
    sink = torch.empty(n_blocks, dtype=torch.int32, device=dev)
    rq.rq_read_probe(buf, sink, n_blocks)
    ts = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        rq.rq_read_probe(buf, sink, n_blocks)
        b.record()
        torch.cuda.synchronize()
        ts.append(a.elapsed_time(b) * 1e-3)
    del buf
    gbs = (gib << 30) / float(np.median(ts)) / 1e9
    return {"kernel": "read_probe_kernel", "bytes": gib << 30,
            "achieved": round(gbs, 1), "unit": "GB/s",
            "frac_of_peak": round(gbs / PEAK_HBM_GBS, 4)}


def fused_comparison(wl, kvc, prefill, Q, outs, table, T0, dev, D=8, reps=5):
    """Decode steps through rq_decode_step (per layer and step: the flush
    launch when a block leaves the window, then one launch that appends the
    token and attends) against rq_quantize_kv + rq_decode_attention per
    layer, over D steps after a prefill of T0 - D tokens (the decode tokens
    are the prefill's last D), all layers in model order; ms per decode
    step, median of `reps` runs of each."""
    import torch

    import paper_2605_06675_amd as rq
    L = table.shape[0]
    Tp = T0 - D
    toks = [[(prefill[l][0][:, :, Tp + s:Tp + s + 1].contiguous(),
              prefill[l][1][:, :, Tp + s:Tp + s + 1].contiguous()) for s in range(D)]
            for l in range(L)]
    # the window, and with it the workspace, varies over the steps
    ws = torch.zeros(max(rq.rq_decode_workspace(kvc.desc, Tp + s + 1) for s in range(D)),
                     dtype=torch.uint8, device=dev)

    def run(fused):
        for l in range(L):
            rq.rq_quantize_kv(kvc.desc, l, 0, prefill[l][0][:, :, :Tp].contiguous(),
                              prefill[l][1][:, :, :Tp].contiguous())
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for s in range(D):
            for l in range(L):
                k, v = toks[l][s]
                if fused:
                    rq.rq_decode_step(kvc.desc, l, Tp + s, k, v, Q[l][0], outs[l], ws)
                else:
                    rq.rq_quantize_kv(kvc.desc, l, Tp + s, k, v)
                    rq.rq_decode_attention(kvc.desc, l, Tp + s + 1, Q[l][0], outs[l], ws)
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / D

    t_sep, t_fus = [], []
    for _ in range(reps):
        t_sep.append(run(False))
        t_fus.append(run(True))
    sep, fus = float(np.median(t_sep)), float(np.median(t_fus))
    return {"steps": D, "layers": L, "separate_ms_per_step": round(sep, 3),
            "fused_ms_per_step": round(fus, 3), "speedup": round(sep / fus, 4),
            "calls": "rq_quantize_kv + rq_decode_attention vs rq_decode_step, "
                     "per layer in model order"}


def uniform_comparison(wl, kvc, prefill, dec, Q, outs, table, T0, nsteps,
                       rot, dev, reps=10):
    """The paper's zero-overhead claim (Appendix "Runtime Analysis"): decode
    attention over a cache with every head at the same width and the same
    average (K at floor, V at ceil of the average) against the mixed
    allocation, both over the whole cache after the decode steps, all
    layers, median of `reps`; the ratio compares time per algorithmic
    byte (1.0 = no overhead from mixing widths)."""
    import torch

    import paper_2605_06675_amd as rq
    L, H = table.shape[0], table.shape[1]
    T = T0 + nsteps
    ut = np.empty_like(table)
    ut[..., 0] = int(np.floor(wl.avg_bits))
    ut[..., 1] = int(np.ceil(wl.avg_bits))
    ukv = rq.KVCache(wl.family, wl.dtype, L, wl.batch, H, wl.n_q_heads,
                     wl.context, wl.residual, ut, device=dev, rotation=rot)
    for l in range(L):
        ukv.append(l, prefill[l][0], prefill[l][1])
        for s in range(nsteps):
            ukv.append(l, dec[l][0][s], dec[l][1][s])
    ws = torch.zeros(max(rq.rq_decode_workspace(c.desc, T) for c in (kvc, ukv)),
                     dtype=torch.uint8, device=dev)

    def timed(c):
        ts = []
        for r in range(reps + 1):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for l in range(L):
                rq.rq_decode_attention(c.desc, l, T, Q[l][nsteps - 1], outs[l], ws)
            b.record()
            torch.cuda.synchronize()
            if r:
                ts.append(a.elapsed_time(b) * 1e3 / L)
        return float(np.median(ts))

    us_m, us_u = timed(kvc), timed(ukv)
    by_m = attention_bytes(wl, table, T) / L
    by_u = attention_bytes(wl, ut, T) / L
    del ukv
    torch.cuda.empty_cache()
    return {"uniform_bits_kv": [int(ut[0, 0, 0]), int(ut[0, 0, 1])],
            "mixed_us_per_layer": round(us_m, 2), "uniform_us_per_layer": round(us_u, 2),
            "mixed_gbs": round(by_m / us_m / 1e3, 1),
            "uniform_gbs": round(by_u / us_u / 1e3, 1),
            "time_ratio_mixed_over_uniform": round(us_m / us_u, 4),
            "per_byte_ratio_mixed_over_uniform": round((us_m / by_m) / (us_u / by_u), 4)}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus must "
                          "be 1 (the path shards by kv-head/batch with no "
                          "exchange, see the design notes)"}))
        sys.exit(2)
    import workloads
    from oracle import alloc as oalloc

    wl = workloads.WORKLOADS[args.workload]
    L, H = wl.n_layers, wl.n_kv_heads
    lo, hi = min(wl.bit_set), max(wl.bit_set)
    w, alpha_p, beta_p = workloads.allocation_inputs(wl)
    cpu = None
    if not args.no_cpu_baseline:
        # the oracle's own allocation picks the sample's units; the host
        # samples run before the GPU is initialised (the pool forks)
        t_or = oalloc.greedy(w, alpha_p, beta_p,
                             oalloc.budget(wl.n_comp, wl.avg_bits), lo, hi)
        cpu = cpu_baseline(wl, np.asarray(t_or).reshape(L, H, 2),
                           args.cpu_seconds, args.cpu_workers)
        cpu["allocation_matches_library"] = None

    import torch

    import paper_2605_06675_amd as rq

    rq.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    B, Hq, T = wl.batch, wl.n_q_heads, wl.context
    n_comp = wl.n_comp
    nsteps = STEPS.get(wl.name, 1)
    T0 = T - nsteps                      # prefill length
    td = workloads.torch_dtype(wl.dtype)

    # ---- inputs, resident in HBM before timing
    bits0, _, _ = rq.rq_allocate_bits(w, alpha_p, beta_p, wl.avg_bits, lo, hi)
    table = bits0.reshape(L, H, 2)
    if cpu is not None:
        cpu["allocation_matches_library"] = bool(np.array_equal(
            np.asarray(t_or).reshape(-1), bits0))
    rot = None
    if wl.family == workloads.TURBO:
        r16 = workloads.turbo_rotations(wl)
        rot = torch.from_numpy(r16.view(np.int16)).view(torch.bfloat16).to(dev)
    prefill, dec = [], []
    for l in range(L):
        k, v = workloads.kv_device(wl, l)
        prefill.append((k[:, :, :T0].contiguous(), v[:, :, :T0].contiguous()))
        # decode tokens: [step][B][H][1][128], each step contiguous
        dec.append((k[:, :, T0:].permute(2, 0, 1, 3).unsqueeze(3).contiguous(),
                    v[:, :, T0:].permute(2, 0, 1, 3).unsqueeze(3).contiguous()))
        del k, v
    Q = [[workloads.q_device(wl, l, step=s) for s in range(nsteps)]
         for l in range(L)]
    calib = workloads.calib_cpu(n_comp, args.calib_tokens, wl.dtype)
    calib_k = torch.from_numpy(calib[: n_comp // 2].view(np.int16)).view(td).to(dev)
    calib_v = torch.from_numpy(calib[n_comp // 2:].view(np.int16)).view(td).to(dev)
    cal_bits = list(wl.bit_set)
    cal_ws = torch.empty(rq.rq_calibrate_workspace(n_comp // 2, args.calib_tokens,
                                                   len(cal_bits)),
                         dtype=torch.uint8, device=dev)
    cal_rot = rot.reshape(L * H, 128, 128) if rot is not None else None
    kvc = rq.KVCache(wl.family, wl.dtype, L, B, H, Hq, T, wl.residual, table,
                     device=dev, rotation=rot)
    # the window, and with it the workspace, varies over the decode steps
    ws = torch.zeros(max(rq.rq_decode_workspace(kvc.desc, T0 + s + 1)
                         for s in range(nsteps)), dtype=torch.uint8, device=dev)
    outs = [torch.empty((B, Hq, 128), dtype=torch.float32, device=dev)
            for _ in range(L)]
    torch.cuda.synchronize()

    ev = lambda: torch.cuda.Event(enable_timing=True)

    def step(rec):
        e = {"calib": (ev(), ev()), "quantize": (ev(), ev())}
        e_app = [(ev(), ev()) for _ in range(nsteps)]
        e_att = [(ev(), ev()) for _ in range(nsteps)]
        e["calib"][0].record()
        r1 = rq.rq_calibrate_distortion(wl.family, wl.dtype, calib_k, 0, cal_bits,
                                        ws=cal_ws, rotation=cal_rot,
                                        codebook=kvc.codebook)
        r2 = rq.rq_calibrate_distortion(wl.family, wl.dtype, calib_v, 1, cal_bits,
                                        ws=cal_ws, rotation=cal_rot,
                                        codebook=kvc.codebook)
        e["calib"][1].record()
        t0 = time.perf_counter()
        bits, cont, J = rq.rq_allocate_bits(w, alpha_p, beta_p, wl.avg_bits, lo, hi)
        assert np.array_equal(bits, bits0)
        rq.rq_cache_sizes(kvc.desc)
        t_alloc = time.perf_counter() - t0
        e["quantize"][0].record()
        for l in range(L):
            rq.rq_quantize_kv(kvc.desc, l, 0, prefill[l][0], prefill[l][1])
        e["quantize"][1].record()
        for s in range(nsteps):
            e_app[s][0].record()
            for l in range(L):
                rq.rq_quantize_kv(kvc.desc, l, T0 + s, dec[l][0][s], dec[l][1][s])
            e_app[s][1].record()
            e_att[s][0].record()
            for l in range(L):
                rq.rq_decode_attention(kvc.desc, l, T0 + s + 1, Q[l][s], outs[l], ws)
            e_att[s][1].record()
        rec.append((e, e_app, e_att, t_alloc, (r1, r2)))

    for _ in range(args.warmup):
        step([])
    torch.cuda.synchronize()
    rec = []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(rec)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    sens = ceiling = uniform = fused = None
    if not args.no_extras:
        sens = sensitivity_rate(args, wl, dev)
        ceiling = stream_ceiling(dev)
        uniform = uniform_comparison(wl, kvc, prefill, dec, Q, outs, table, T0,
                                     nsteps, rot, dev)
    if not args.no_extras:
        fused = fused_comparison(wl, kvc, prefill, Q, outs, table, T0, dev,
                                 D=max(8, nsteps))

    # stage times: medians over the timed steps
    el = lambda p: p[0].elapsed_time(p[1])
    ms = {"calib": float(np.median([el(r[0]["calib"]) for r in rec])),
          "quantize": float(np.median([el(r[0]["quantize"]) for r in rec])),
          "append": float(np.median([sum(el(x) for x in r[1]) for r in rec])),
          "attention": float(np.median([sum(el(x) for x in r[2]) for r in rec]))}
    alloc_ms = float(np.median([r[3] for r in rec])) * 1e3
    att_bytes = sum(attention_bytes(wl, table, T0 + s + 1) for s in range(nsteps))
    q_bytes = quantize_bytes(wl, table, T0)
    att_gbs = att_bytes / (ms["attention"] * 1e-3) / 1e9
    # KV quantize tok/s: B * T0 tokens through all L layers' K and V
    q_tok_s = B * T0 / (ms["quantize"] * 1e-3)
    q_gbs = q_bytes / (ms["quantize"] * 1e-3) / 1e9
    qk = QUANT_KERNEL[wl.family]
    # per launch: the phase time over its launches (back to back on the
    # stream, one kernel per call; events around single calls would add the
    # dispatch and drain of each launch, which back-to-back launches overlap)
    kernels = {
        qk: {"call": f"rq_quantize_kv prefill of one layer ({T0} tokens; the "
                     "launch also writes the window)",
             "bytes": q_bytes / L, "us": ms["quantize"] * 1e3 / L},
        "attn_kernel": {"call": "rq_decode_attention of one layer",
                        "bytes": att_bytes / (L * nsteps),
                        "us": ms["attention"] * 1e3 / (L * nsteps)},
    }
    rooflines = {}
    for name, k in kernels.items():
        ach = k["bytes"] / (k["us"] * 1e-6) / 1e9
        rooflines[name] = {
            "bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
            "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4),
            "traffic": measured_traffic(wl.name, name), "kernel": name,
            "call": k["call"], "bytes_per_launch": int(k["bytes"]),
            "avg_launch_us": round(k["us"], 2)}
    # the kernel that takes the most time in a step
    total_us = {qk: ms["quantize"], "attn_kernel": ms["attention"]}
    dom = max(total_us, key=total_us.get)
    r1, r2 = rec[-1][4]
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
        # inputs are 16-bit; quantization runs in fp32 (TurboQuant's rotation
        # on bf16 matrix cores), attention on fp16 matrix-core operands with
        # fp32 accumulation and softmax
        "dtype": "f16/f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "layers": L, "batch": B,
                   "kv_heads": H, "q_heads": Hq, "head_dim": 128,
                   "context": T, "decode_steps": nsteps,
                   "residual_window": wl.residual,
                   "family": ["kivi", "quarot", "turbo", "rtn",
                              "kivi_rtn"][wl.family],
                   "avg_bits": wl.avg_bits, "bit_set": list(wl.bit_set),
                   "attention_bytes_per_step": att_bytes,
                   "quantize_bytes_per_step": q_bytes,
                   "fitted_beta_median": round(float(np.nanmedian(beta_fit)), 3)},
        "roofline": rooflines[dom],
        "roofline_by_kernel": rooflines,
        "stream_ceiling": ceiling,
        "uniform_vs_mixed": uniform,
        "decode_step_fused": fused,
        "sensitivity": sens,
    }
    for name, r in rooflines.items():
        if ceiling:
            r["frac_of_stream_ceiling"] = round(r["achieved"] / ceiling["achieved"], 4)
    if cpu is not None:
        line["cpu_baseline"] = cpu
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
