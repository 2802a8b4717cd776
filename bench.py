#!/usr/bin/env python3
"""Benchmark of the paged-KV attention hot path on one MI355X.

Headline workload (the one `value` is quoted on): batched single-token decode over 64
conversations with cached contexts uniform in [8192, 32768] tokens, 32 query / 8 KV heads,
head_dim 128, bf16 K/V with per-KV-head scales in [0.5, 2], 16-token pages placed at random,
one layer. One step = one `attn_decode_batch` call (split-K kernel + merge kernel) with all
inputs already resident in HBM. `value` = algorithmic bytes of a step (K and V read once,
Q, O, page-table entries) / measured step time.

Extra components (same JSON line, "components"): extend-prefill of 16 conversations
(prefix U[16384, 65536], chunk log-normal median 1024 in [128, 4096]), turn-1 prefill of 8
conversations (L U[32768, 131072]) and its one-time KV transfer (pack + unpack), and KV append.

Usage: python bench.py [--gpus 1] [--steps 20] [--warmup 3] [--skip-components]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from synth import values as sv  # noqa: E402
from synth.traces import (DecodeBatch, ExtendBatch, MixedTrace, PrefillTransfer, KIND_K,  # noqa: E402
                          KIND_Q, KIND_V, pages_for)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA, TFLOP/s
METRIC = "decode-attn HBM GB/s + extend/prefill TFLOP/s, each as % of MI355X peak"
PROFILES = os.path.join(ROOT, "profiles")
# The sources each kernel is built from: counters committed under profiles/ apply only while these
# are unchanged (their SHA-256 is stored with the counters).
KERNEL_SOURCES = {
    "decode_split": ["paper_2606_01839_amd/csrc/decode.hip", "paper_2606_01839_amd/csrc/decode_split.hpp",
                     "paper_2606_01839_amd/csrc/device_common.hpp"],
    "attn_fwd": ["paper_2606_01839_amd/csrc/attn_fwd.hip", "paper_2606_01839_amd/csrc/decode_split.hpp",
                 "paper_2606_01839_amd/csrc/device_common.hpp"],
    "kv_move": ["paper_2606_01839_amd/csrc/kv_move.hip", "paper_2606_01839_amd/csrc/device_common.hpp"],
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def gen_kv(seed, conv, start, n, hkv, d, sk=None, sv_=None, device="cuda"):
    per = hkv * d
    k = sv.bf16_tensor(sv.mix_key(seed, conv, KIND_K, 0), (n, hkv, d), head_scale=sk,
                       start=start * per, device=device)
    v = sv.bf16_tensor(sv.mix_key(seed, conv, KIND_V, 0), (n, hkv, d), head_scale=sv_,
                       start=start * per, device=device)
    return k, v


def gen_q(seed, conv, start, n, hq, d, device="cuda"):
    return sv.bf16_tensor(sv.mix_key(seed, conv, KIND_Q, 0), (n, hq, d), start=start * hq * d,
                          device=device)


def source_hash(group: str) -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[group]:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def kernel_counters(name: str, workload: str, group: str, alg_bytes=None) -> dict:
    """Figures from the committed rocprofv3 counters of a kernel (profiles/<name>_counters.json):
    HBM traffic per launch (FETCH_SIZE and WRITE_SIZE, each calibrated on a 1 GiB device copy in
    the same run) and, for the attention kernel, its matrix-core busy fraction, sustained clock and
    LDS bank-conflict cycles. Only when the file was taken on this workload and on the kernel's
    current sources; otherwise traffic is None."""
    try:
        with open(os.path.join(PROFILES, f"{name}_counters.json")) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return {"traffic": None}
    if t.get("source_sha256") != source_hash(group) or t.get("workload") != workload:
        return {"traffic": None, "counters_note": f"profiles/{name}_counters.json was taken on other "
                                                  "sources or another workload"}
    out = {"traffic": t.get("traffic_bytes_per_launch"), "counters_file": f"profiles/{name}_counters.json"}
    if alg_bytes and out["traffic"]:
        out["traffic_over_algorithmic"] = out["traffic"] / alg_bytes
    for k in ("mfma_busy", "sustained_clock_ghz", "lds_bank_conflict_cycles_per_launch"):
        if k in t:
            out[k] = t[k]
    return out


def energy_run(fn, seconds=8.0):
    """Run fn back to back for about `seconds` and read the GPU's energy accumulator (amdsmi)
    before and after: joules, the firmware's own time base, average watts and the call count.
    None where the counter is unavailable. Power is sampled, not controlled."""
    try:
        import amdsmi
        amdsmi.amdsmi_init()
        h = amdsmi.amdsmi_get_processor_handles()[0]
        read = lambda: amdsmi.amdsmi_get_energy_count(h)
        read()
    except Exception:
        return None
    fn()
    torch.cuda.synchronize()
    e0 = read()
    t0 = time.perf_counter()
    n = 0
    while time.perf_counter() - t0 < seconds:
        fn()
        n += 1
        if n % 4 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    e1 = read()
    joules = (e1["energy_accumulator"] - e0["energy_accumulator"]) * e1["counter_resolution"] * 1e-6
    fw_s = (e1["timestamp"] - e0["timestamp"]) * 1e-9
    watts = joules / fw_s if fw_s > 0 else None
    return {"calls": n, "wall_s": wall, "joules": joules, "counter_s": fw_s, "avg_watts": watts}


def timed(fn, steps, warmup):
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        fn()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) / steps * 1e3


def profiled(pool, fn, steps):
    pool.profile_start()
    for _ in range(steps):
        fn()
    return pool.profile_stop()


def blas_threads() -> int:
    try:
        from threadpoolctl import threadpool_info
        n = [i.get("num_threads", 0) for i in threadpool_info() if i.get("user_api") == "blas"]
        if n:
            return int(max(n))
    except Exception:
        pass
    return len(os.sched_getaffinity(0))


def host_info() -> dict:
    """CPU model, usable cores and the BLAS library numpy calls (the CPU baseline's machine)."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = None
    try:
        from threadpoolctl import threadpool_info
        for i in threadpool_info():
            if i.get("user_api") == "blas":
                blas = {"library": i.get("internal_api"), "version": i.get("version"),
                        "threads": i.get("num_threads"), "architecture": i.get("architecture")}
                break
    except Exception:
        pass
    return {"cpu_model": model, "usable_cores": len(os.sched_getaffinity(0)), "blas": blas}


def device_block() -> dict:
    """hipDeviceProp figures of the GPU and a streaming-read probe: 4 GiB read once with the
    non-temporal 16-byte loads of the decode and pack kernels, 8 workgroups per CU (median of 10
    after 3 warm-ups, HIP events on the probe's stream)."""
    from paper_2606_01839_amd import device_info, probe_stream_read
    info = device_info(0)
    buf = torch.empty(4 << 30, dtype=torch.uint8, device="cuda")
    buf.fill_(1)
    sink = torch.zeros(4, dtype=torch.uint8, device="cuda")
    for _ in range(3):
        probe_stream_read(buf, sink)
    ts = []
    for _ in range(10):
        a_, b_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a_.record()
        probe_stream_read(buf, sink)
        b_.record()
        torch.cuda.synchronize()
        ts.append(a_.elapsed_time(b_))
    ms = float(np.median(ts))
    del buf, sink
    torch.cuda.empty_cache()
    return {"name": info["name"], "arch": info["arch"], "cu_count": info["cu_count"],
            "clock_mhz": info["clock_khz"] / 1e3, "memory_clock_mhz": info["memory_clock_khz"] / 1e3,
            "memory_bus_width_bits": info["memory_bus_width_bits"],
            "lds_per_cu_kib": info["lds_per_cu_bytes"] / 1024, "l2_mib": info["l2_bytes"] / 2**20,
            "hbm_gib": info["total_mem_bytes"] / 2**30,
            "stream_read_probe": {"bytes": 4 << 30, "ms": ms, "gbs": (4 << 30) / (ms * 1e-3) / 1e9,
                                  "frac_of_peak": (4 << 30) / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS}}


def sample_rows(n: int, seed: int, k: int = 4):
    """Query rows 0 .. n-1 to check and time: first and last, rows around the 16-token page and
    64-row tile boundaries nearest the middle, and k seeded random rows (sorted, distinct)."""
    mid = n // 2
    rows = {0, n - 1, (mid // 16) * 16, (mid // 16) * 16 - 1, (mid // 64) * 64 + 63}
    rows |= set(int(x) for x in np.random.default_rng(seed).integers(0, n, size=k))
    return sorted(r for r in rows if 0 <= r < n)


def oracle_rows(kv, q_rows, out_rows, pos, hq, d):
    """The fp64 oracle on sampled query rows of one conversation (inputs already fp64 on the
    host): (max abs error of the GPU rows, oracle seconds, algorithmic FLOPs of those rows)."""
    from oracle.attention import attend_rows
    qf = sv.bf16_to_f64(q_rows)
    t = time.perf_counter()
    ref = attend_rows(qf, pos, kv[0], kv[1])
    secs = time.perf_counter() - t
    err = float(np.abs(sv.bf16_to_f64(out_rows) - ref).max())
    return err, secs, sum(4 * d * hq * (int(p) + 1) for p in pos)


def oracle_baseline(flops, secs, total_flops, sample):
    rate = flops / secs
    return {"value": rate / 1e12, "unit": "TFLOP/s", "cores": blas_threads(), "kind": "oracle",
            "sample": sample, "full_batch_s_extrapolated": total_flops / rate, **host_info()}


# ------------------------------------------------------------------------------------------------
# workload construction (shared with tests/test_gpu_fullsize.py)
# ------------------------------------------------------------------------------------------------
def make_decode_case(tr=None):
    """Decode batch pool: every conversation's K/V appended; returns (pool, convs, lens,
    [(k, v)] device inputs per conversation, q [B][Hq][d] for each last position)."""
    from paper_2606_01839_amd import KVPool
    tr = tr or DecodeBatch()
    sh = tr.shape
    hq, hkv, d = sh.n_q_heads, sh.n_kv_heads, sh.head_dim
    lens = tr.lengths().astype(np.int64)
    sk, svs = tr.head_scales()
    n_pages = int(sum(pages_for(L) for L in lens) * 1.1)
    pool = KVPool(1, hq, hkv, d, n_pages=n_pages, max_convs=tr.batch,
                  max_pages_per_conv=pages_for(tr.hi), placement_seed=tr.seed + 1)
    convs, kv_dev = [], []
    for b, L in enumerate(lens):
        c = pool.conv_create()
        k, v = gen_kv(tr.seed, b, 0, int(L), hkv, d, sk, svs)
        pool.kv_append(c, k[None], v[None])
        convs.append(c)
        kv_dev.append((k, v))
    q = torch.cat([gen_q(tr.seed, b, int(L) - 1, 1, hq, d) for b, L in enumerate(lens)])
    return pool, convs, lens, kv_dev, q


def make_extend_case(tr=None):
    """Extend batch: prefixes appended; returns (pool, convs, prefix, chunk, k_new, v_new, q) with
    the turn's new K/V ([1][sum chunk][Hkv][d], not yet appended) and q [sum chunk][Hq][d]."""
    from paper_2606_01839_amd import KVPool
    tr = tr or ExtendBatch()
    sh = tr.shape
    hq, hkv, d = sh.n_q_heads, sh.n_kv_heads, sh.head_dim
    prefix, chunk = tr.lengths()
    total = prefix + chunk
    pool = KVPool(1, hq, hkv, d, n_pages=int(sum(pages_for(L) for L in total)) + 64,
                  max_convs=tr.n_convs, max_pages_per_conv=pages_for(int(total.max())),
                  placement_seed=tr.seed + 1)
    convs = []
    for b in range(tr.n_convs):
        c = pool.conv_create()
        k, v = gen_kv(tr.seed, b, 0, int(prefix[b]), hkv, d)
        pool.kv_append(c, k[None], v[None])
        convs.append(c)
        del k, v
    new_kv = [gen_kv(tr.seed, b, int(prefix[b]), int(chunk[b]), hkv, d) for b in range(tr.n_convs)]
    kcat = torch.cat([k for k, _ in new_kv])[None].contiguous()
    vcat = torch.cat([v for _, v in new_kv])[None].contiguous()
    q = torch.cat([gen_q(tr.seed, b, int(prefix[b]), int(chunk[b]), hq, d) for b in range(tr.n_convs)])
    return pool, convs, prefix, chunk, kcat, vcat, q


def make_prefill_case(tr=None):
    """Turn-1 prefill batch: prompts appended; returns (pool, convs, lens, q [sum L][Hq][d])."""
    from paper_2606_01839_amd import KVPool
    tr = tr or PrefillTransfer()
    sh = tr.shape
    hq, hkv, d = sh.n_q_heads, sh.n_kv_heads, sh.head_dim
    lens = tr.lengths().astype(np.int64)
    npg = int(sum(pages_for(L) for L in lens)) + 64
    pool = KVPool(1, hq, hkv, d, n_pages=npg, max_convs=tr.n_convs,
                  max_pages_per_conv=pages_for(tr.hi), placement_seed=tr.seed + 1)
    convs = []
    for b, L in enumerate(lens):
        c = pool.conv_create()
        k, v = gen_kv(tr.seed, b, 0, int(L), hkv, d)
        pool.kv_append(c, k[None], v[None])
        convs.append(c)
        del k, v
    q = torch.cat([gen_q(tr.seed, b, 0, int(L), hq, d) for b, L in enumerate(lens)])
    return pool, convs, lens, q


# ------------------------------------------------------------------------------------------------
# headline: decode batch
# ------------------------------------------------------------------------------------------------
def bench_decode(args):
    tr = DecodeBatch()
    sh = tr.shape
    hq, hkv, d = sh.n_q_heads, sh.n_kv_heads, sh.head_dim
    t0 = time.perf_counter()
    pool, convs, lens, kv_dev, q = make_decode_case(tr)
    sk, svs = tr.head_scales()
    out = torch.empty_like(q)
    torch.cuda.synchronize()
    log(f"decode: filled {len(lens)} conversations ({lens.sum()} tokens) in {time.perf_counter() - t0:.1f}s")

    step = lambda: pool.attn_decode_batch(convs, 0, q, out)
    ms = timed(step, args.steps, args.warmup)
    # per-step distribution: events on the stream the pool launches on (torch's current stream)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    for a_, b_ in evs:
        a_.record()
        step()
        b_.record()
    torch.cuda.synchronize()
    step_ms = np.array([a_.elapsed_time(b_) for a_, b_ in evs])
    prof = profiled(pool, step, args.steps)
    en = energy_run(step) if args.energy else None
    split_ms = prof["decode_split"][0] / max(1, prof["decode_split"][1])
    merge_ms = prof["decode_merge"][0] / max(1, prof["decode_merge"][1])

    kv_bytes = int(lens.sum()) * 2 * hkv * d * 2
    q_bytes = len(lens) * hq * d * 2
    pt_bytes = int(sum(pages_for(L) for L in lens)) * 4
    step_bytes = kv_bytes + 2 * q_bytes + pt_bytes
    split_bytes = kv_bytes + q_bytes + pt_bytes
    out_host = out.cpu()

    # parity of every conversation against the oracle, and the oracle's own time (CPU baseline)
    from oracle.attention import attend_rows
    max_abs, num, den = 0.0, 0.0, 0.0
    cpu_s = 0.0
    # the device-generated inputs are the seeded generator's values: check two against the host
    for b in (int(np.argmin(lens)), int(np.argmax(lens))):
        L = int(lens[b])
        kh, vh = gen_kv(tr.seed, b, 0, min(L, 4096), hkv, d, sk, svs, device="cpu")
        assert torch.equal(kh, kv_dev[b][0][:min(L, 4096)].cpu()) and torch.equal(vh, kv_dev[b][1][:min(L, 4096)].cpu())
    host = [(sv.bf16_to_f64(kv_dev[b][0]), sv.bf16_to_f64(kv_dev[b][1]), sv.bf16_to_f64(q[b:b + 1]))
            for b in range(len(lens))]
    for b, L in enumerate(lens):
        kf, vf, qf = host[b]
        t = time.perf_counter()
        ref = attend_rows(qf, [int(L) - 1], kf, vf)
        cpu_s += time.perf_counter() - t
        diff = sv.bf16_to_f64(out_host[b:b + 1]) - ref
        max_abs = max(max_abs, float(np.abs(diff).max()))
        num += float((diff ** 2).sum())
        den += float((ref ** 2).sum())
    rel_l2 = math.sqrt(num / den)
    # the oracle's timing: whole decode steps repeated until about 10 s of CPU work
    passes = 1
    while cpu_s < 10.0 and passes < 16:
        t = time.perf_counter()
        for b, L in enumerate(lens):
            kf, vf, qf = host[b]
            attend_rows(qf, [int(L) - 1], kf, vf)
        cpu_s += time.perf_counter() - t
        passes += 1
    del host
    workload = (f"decode batch: {len(lens)} conversations, context U[{tr.lo},{tr.hi}] (sum "
                f"{int(lens.sum())} tokens), {hq}q/{hkv}kv heads, head_dim {d}, bf16 K/V x per-head "
                f"scale U[{tr.scale_lo},{tr.scale_hi}], 16-token pages randomly placed, 1 layer")
    counters = kernel_counters("decode_split", workload, "decode_split", split_bytes)
    res = {
        "ms_per_step": ms,
        "step_ms_p10_p50_p90": [float(np.percentile(step_ms, x)) for x in (10, 50, 90)],
        "value_gbs": step_bytes / (ms * 1e-3) / 1e9,
        "split_ms": split_ms,
        "merge_ms": merge_ms,
        "split_bytes": split_bytes,
        "step_bytes": step_bytes,
        "workload": workload,
        "counters": counters,
        "energy": None if not en or not en["avg_watts"] else {
            **en, "tokens_per_joule": en["calls"] * len(lens) / en["wall_s"] / en["avg_watts"],
            "gb_per_joule": en["calls"] * step_bytes / 1e9 / en["wall_s"] / en["avg_watts"]},
        "parity": {"convs": len(lens), "max_abs": max_abs, "rel_l2": rel_l2,
                   "ok": bool(max_abs <= 1e-2 and rel_l2 <= 3e-3)},
        "cpu": {"value": passes * step_bytes / cpu_s / 1e9, "unit": "GB/s", "cores": blas_threads(),
                "kind": "oracle", **host_info(),
                "sample": f"fp64 oracle over all {len(lens)} conversations x {hq} heads of the same "
                          f"decode step (inputs already in host memory as fp64), {passes} passes "
                          f"in {cpu_s:.1f} s"},
    }
    pool.close()
    del kv_dev
    torch.cuda.empty_cache()
    return res


# ------------------------------------------------------------------------------------------------
# components: extend-prefill, turn-1 prefill + transfer, append
# ------------------------------------------------------------------------------------------------
def attn_flops(prefix, n, hq, d):
    pairs = sum(int(nn) * int(P) + int(nn) * (int(nn) + 1) // 2 for P, nn in zip(prefix, n))
    return 4 * d * hq * pairs


def bench_extend(args):
    tr = ExtendBatch()
    sh = tr.shape
    hq, hkv, d = sh.n_q_heads, sh.n_kv_heads, sh.head_dim
    pool, convs, prefix, chunk, kcat, vcat, q = make_extend_case(tr)
    total = prefix + chunk
    torch.cuda.synchronize()
    pool.profile_start()
    pool.kv_append_batch(convs, chunk, kcat, vcat)
    app = pool.profile_stop()["append"]
    out = torch.empty_like(q)
    step = lambda: pool.attn_extend(convs, chunk, 0, q, out)
    reps = max(3, args.steps // 4)
    ms = timed(step, reps, 1)
    prof = profiled(pool, step, reps)
    fwd_ms = prof["attn_fwd"][0] / max(1, prof["attn_fwd"][1])
    flops = attn_flops(prefix, chunk, hq, d)
    app_bytes = 2 * int(chunk.sum()) * 2 * hkv * d * 2    # read + write of the new K and V
    # parity on sampled rows of the first and last conversations, and the oracle's time on them
    err, secs, s_flops, n_rows = 0.0, 0.0, 0, 0
    for b in (0, tr.n_convs - 1):
        L, P, n = int(total[b]), int(prefix[b]), int(chunk[b])
        kv = tuple(sv.bf16_to_f64(t) for t in gen_kv(tr.seed, b, 0, L, hkv, d, device="cpu"))
        r0 = int(chunk[:b].sum())
        rows = sample_rows(n, tr.seed + b)
        e, t, f = oracle_rows(kv, q[[r0 + i for i in rows]], out[[r0 + i for i in rows]],
                              [P + i for i in rows], hq, d)
        err, secs, s_flops, n_rows = max(err, e), secs + t, s_flops + f, n_rows + len(rows)
        del kv
    ok = err <= 1e-2
    cpu = oracle_baseline(s_flops, secs, flops, f"fp64 oracle on {n_rows} sampled query rows (all {hq} "
                          f"heads) of conversations 0 and {tr.n_convs - 1}, {secs:.1f} s; the full "
                          f"batch time is extrapolated at that rate")
    pool.close()
    del kcat, vcat
    torch.cuda.empty_cache()
    workload = (f"extend-prefill: {tr.n_convs} conversations, prefix U[{tr.prefix_lo},{tr.prefix_hi}], chunk "
                f"logN(median {tr.chunk_median}) in [{tr.chunk_lo},{tr.chunk_hi}] (sum {int(chunk.sum())}), "
                f"{hq}q/{hkv}kv, d {d}")
    app_workload = f"kv_append of the {int(chunk.sum())} new tokens of the extend batch (1 layer)"
    return {
        "extend": {"workload": workload,
                   "ms": ms, "kernel_ms": fwd_ms, "flops": flops,
                   "tflops": flops / (ms * 1e-3) / 1e12,
                   "roofline": {"bound": "mfma", "achieved": flops / (fwd_ms * 1e-3) / 1e12,
                                "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                                "frac": flops / (fwd_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS,
                                **kernel_counters("attn_fwd_extend", workload, "attn_fwd")},
                   "spot_parity_ok": bool(ok), "spot_max_abs": err, "cpu_oracle": cpu},
        "append": {"workload": app_workload,
                   "kernel_ms": app[0], "bytes": app_bytes,
                   "gbs": app_bytes / (app[0] * 1e-3) / 1e9,
                   "roofline": {"bound": "hbm", "achieved": app_bytes / (app[0] * 1e-3) / 1e9,
                                "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                "frac": app_bytes / (app[0] * 1e-3) / 1e9 / HBM_PEAK_GBS,
                                **kernel_counters("kv_append_extend", app_workload, "kv_move", app_bytes)}},
    }


def bench_append(args):
    """kv_append in a decoder pool of the mixed trace's shape (32 layers, 32q/8kv, d 128): 64
    conversations with cached contexts U[1000, 3000] (so most last pages are partly filled) receive
    (a) one decoded token each for every layer -- the append of a decode step, 20 steps in a row --
    and (b) one extend chunk each, 16 of them with logN(median 1024) lengths in [128, 4096].
    Algorithmic bytes: the new K and V read once and written once (2 x 4096 B per token and layer)."""
    from paper_2606_01839_amd import KVPool
    NL, hq, hkv, d, seed, B, steps = 32, 32, 8, 128, 1008, 64, 20
    rng = np.random.default_rng(seed)
    lens = rng.integers(1000, 3001, size=B)
    chunks = np.clip(np.exp(rng.normal(math.log(1024), 0.7, size=16)).astype(np.int64), 128, 4096)
    tok_bytes = NL * 2 * hkv * d * 2                     # K + V of one token, all layers
    pool = KVPool(NL, hq, hkv, d, n_pages=int(sum(pages_for(int(L) + steps + 4096) for L in lens)) + 64,
                  max_convs=B, max_pages_per_conv=pages_for(3000 + steps + 4096), placement_seed=seed)
    convs = [pool.conv_create() for _ in range(B)]
    for b0 in range(0, B, 16):                           # untimed fill (zeros: the bytes do not matter)
        n = [int(L) for L in lens[b0:b0 + 16]]
        z = torch.zeros((NL, sum(n), hkv, d), dtype=torch.bfloat16, device="cuda")
        pool.kv_append_batch(convs[b0:b0 + 16], n, z, z)
        del z
    kd = [sv.bf16_tensor(sv.mix_key(seed, s_, KIND_K, 0), (NL, B, hkv, d), device="cuda") for s_ in range(steps)]
    vd = [sv.bf16_tensor(sv.mix_key(seed, s_, KIND_V, 0), (NL, B, hkv, d), device="cuda") for s_ in range(steps)]
    torch.cuda.synchronize()
    pool.profile_start()
    for s_ in range(steps):
        pool.kv_append_batch(convs, [1] * B, kd[s_], vd[s_])
    dec = pool.profile_stop()["append"]
    sel = convs[:16]
    kc = sv.bf16_tensor(sv.mix_key(seed, 99, KIND_K, 0), (NL, int(chunks.sum()), hkv, d), device="cuda")
    vc = sv.bf16_tensor(sv.mix_key(seed, 99, KIND_V, 0), (NL, int(chunks.sum()), hkv, d), device="cuda")
    torch.cuda.synchronize()
    pool.profile_start()
    pool.kv_append_batch(sel, [int(c) for c in chunks], kc, vc)
    ext = pool.profile_stop()["append"]
    # bit-exactness of the last decode step's token and of the chunks, read back through the pool
    ok = True
    view = pool.kv_view()
    for b in (0, B - 1):
        pages = pool.conv_pages(convs[b])
        L = int(lens[b]) + steps - 1                      # position of the last decoded token
        blk = view[:, int(pages[L // 16])].cpu()          # [NL][Hkv][16 * 2 * d]
        t = L % 16
        k_got = blk[:, :, :16 * d].view(NL, hkv, d // 32, 16, 32)[:, :, :, t, :].reshape(NL, hkv, d)
        v_got = blk[:, :, 16 * d:].view(NL, hkv, d, 16)[:, :, :, t]
        ok = ok and torch.equal(k_got, kd[-1][:, b].cpu().view(torch.int16)) and \
            torch.equal(v_got, vd[-1][:, b].cpu().view(torch.int16))
    pool.close()
    del kd, vd, kc, vc
    torch.cuda.empty_cache()
    dec_bytes = 2 * B * tok_bytes
    ext_bytes = 2 * int(chunks.sum()) * tok_bytes
    gbs = lambda b, ms: b / (ms * 1e-3) / 1e9
    wl_dec = f"kv_append of one decoded token for each of {B} conversations (context U[1000,3000]), {NL} layers, {hkv} kv heads, d {d}"
    wl_ext = (f"kv_append of 16 extend chunks logN(median 1024) in [128,4096] (sum {int(chunks.sum())}) into "
              f"conversations of context U[1000,3000], {NL} layers, {hkv} kv heads, d {d}")
    return {"append_decode_step": {
                "workload": wl_dec, "launches": dec[1], "kernel_ms_per_step": dec[0] / dec[1],
                "bytes_per_step": dec_bytes, "gbs": gbs(dec_bytes, dec[0] / dec[1]),
                "last_token_bit_exact": bool(ok),
                "roofline": {"bound": "hbm", "achieved": gbs(dec_bytes, dec[0] / dec[1]), "peak": HBM_PEAK_GBS,
                             "unit": "GB/s", "frac": gbs(dec_bytes, dec[0] / dec[1]) / HBM_PEAK_GBS,
                             **kernel_counters("kv_append_decode", wl_dec, "kv_move", dec_bytes)}},
            "append_chunks": {
                "workload": wl_ext, "kernel_ms": ext[0], "bytes": ext_bytes, "gbs": gbs(ext_bytes, ext[0]),
                "roofline": {"bound": "hbm", "achieved": gbs(ext_bytes, ext[0]), "peak": HBM_PEAK_GBS,
                             "unit": "GB/s", "frac": gbs(ext_bytes, ext[0]) / HBM_PEAK_GBS,
                             **kernel_counters("kv_append_chunks", wl_ext, "kv_move", ext_bytes)}}}


def chunked_prefill(tr, lens, q, out_one_shot, mk, chunk=8192):
    """The same turn-1 prefill batch done the way a prefiller with chunked prefill runs it
    (Section 5.1: 8192-token chunks): every round appends the next chunk of each unfinished
    conversation and attends it against the conversation's cached prefix (cs_attn_extend). Inputs
    of each round are staged before timing. Reports the attention and append kernel time, the
    wall time, and whether the output equals the one-shot prefill bit for bit (with 64-aligned
    chunks the query tiles sweep the same key tiles in the same order)."""
    sh = tr.shape
    hq, hkv, d = sh.n_q_heads, sh.n_kv_heads, sh.head_dim
    pool = mk(tr.seed + 7)
    convs = [pool.conv_create() for _ in lens]
    row0 = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64)
    rounds = []
    for s0 in range(0, int(lens.max()), chunk):
        act = [b for b in range(len(lens)) if lens[b] > s0]
        n = [int(min(chunk, lens[b] - s0)) for b in act]
        ks, vs = [], []
        for b, nb in zip(act, n):
            k, v = gen_kv(tr.seed, b, s0, nb, hkv, d)
            ks.append(k)
            vs.append(v)
        qc = torch.cat([q[int(row0[b]) + s0:int(row0[b]) + s0 + nb] for b, nb in zip(act, n)])
        rounds.append((act, n, s0, torch.cat(ks)[None], torch.cat(vs)[None], qc, torch.empty_like(qc)))
        del ks, vs
    torch.cuda.synchronize()
    pool.profile_start()
    t0 = time.perf_counter()
    for act, n, s0, k, v, qc, oc in rounds:
        pool.kv_append_batch([convs[b] for b in act], n, k, v)
        pool.attn_extend([convs[b] for b in act], n, 0, qc, oc)
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3
    prof = pool.profile_stop()
    same = True
    for act, n, s0, k, v, qc, oc in rounds:
        r = 0
        for b, nb in zip(act, n):
            ref = out_one_shot[int(row0[b]) + s0:int(row0[b]) + s0 + nb]
            same = same and torch.equal(oc[r:r + nb], ref)
            r += nb
    flops = attn_flops([0] * len(lens), lens, hq, d)
    fwd_ms, app_ms = prof["attn_fwd"][0], prof["append"][0]
    pool.close()
    del rounds
    torch.cuda.empty_cache()
    return {"chunk_tokens": chunk, "rounds": int(-(-int(lens.max()) // chunk)),
            "attn_launches": prof["attn_fwd"][1], "attn_kernel_ms": fwd_ms,
            "append_kernel_ms": app_ms, "wall_ms": wall_ms, "flops": flops,
            "attn_tflops": flops / (fwd_ms * 1e-3) / 1e12,
            "frac": flops / (fwd_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS,
            "bitwise_equal_to_one_shot": bool(same)}


def bench_prefill_transfer(args, parts=("prefill", "chunked", "transfer")):
    """Turn-1 prefill batch: the one-shot prefill ("prefill"), the same batch in 8192-token chunks
    ("chunked") and the one-time transfer of every conversation ("transfer"); `parts` picks which
    run (a profiler run of one part then sees only that part's kernels)."""
    from paper_2606_01839_amd import KVPool
    tr = PrefillTransfer()
    sh = tr.shape
    hq, hkv, d = sh.n_q_heads, sh.n_kv_heads, sh.head_dim
    pre, convs, lens, q = make_prefill_case(tr)
    npg = pre.desc.n_pages
    mk = lambda seed: KVPool(1, hq, hkv, d, n_pages=npg, max_convs=tr.n_convs,
                             max_pages_per_conv=pages_for(tr.hi), placement_seed=seed)
    res = {}
    if "prefill" in parts or "chunked" in parts:
        res.update(_prefill_parts(args, tr, pre, convs, lens, q, mk, parts))
    if "transfer" in parts:
        res.update(_transfer_part(tr, pre, convs, lens, mk))
    pre.close()
    del q
    torch.cuda.empty_cache()
    return res


def _prefill_parts(args, tr, pre, convs, lens, q, mk, parts):
    sh = tr.shape
    hq, hkv, d = sh.n_q_heads, sh.n_kv_heads, sh.head_dim
    out = torch.empty_like(q)
    step = lambda: pre.attn_prefill_turn1(convs, lens, 0, q, out)
    reps = 2
    ms = timed(step, reps, 1)
    prof = profiled(pre, step, reps)
    fwd_ms = prof["attn_fwd"][0] / max(1, prof["attn_fwd"][1])
    flops = attn_flops([0] * len(lens), lens, hq, d)
    en = energy_run(step) if args.energy else None
    # parity on sampled rows of the two shortest conversations, and the oracle's time on them
    row0 = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64)
    err, secs, s_flops, n_rows = 0.0, 0.0, 0, 0
    picks = [int(b) for b in np.argsort(lens, kind="stable")[:2]]
    for b in picks:
        L = int(lens[b])
        kv = tuple(sv.bf16_to_f64(t) for t in gen_kv(tr.seed, b, 0, L, hkv, d, device="cpu"))
        rows = sample_rows(L, tr.seed + b)
        e, t, f = oracle_rows(kv, q[[int(row0[b]) + i for i in rows]], out[[int(row0[b]) + i for i in rows]],
                              rows, hq, d)
        err, secs, s_flops, n_rows = max(err, e), secs + t, s_flops + f, n_rows + len(rows)
        del kv
    cpu = oracle_baseline(s_flops, secs, flops, f"fp64 oracle on {n_rows} sampled query rows (all {hq} "
                          f"heads) of conversations {picks[0]} and {picks[1]} (the two shortest), "
                          f"{secs:.1f} s; the full batch time is extrapolated at that rate")
    workload = f"turn-1 prefill: {tr.n_convs} conversations, L U[{tr.lo},{tr.hi}] (sum {int(lens.sum())}), {hq}q/{hkv}kv, d {d}"
    res = {
        "prefill": {"workload": workload,
                    "ms": ms, "kernel_ms": fwd_ms, "flops": flops,
                    "tflops": flops / (ms * 1e-3) / 1e12,
                    "roofline": {"bound": "mfma", "achieved": flops / (fwd_ms * 1e-3) / 1e12,
                                 "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                                 "frac": flops / (fwd_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS,
                                 **kernel_counters("attn_fwd_prefill", workload, "attn_fwd")},
                    "spot_parity_ok": bool(err <= 1e-2), "spot_max_abs": err, "cpu_oracle": cpu},
        "prefill_energy": None if not en or not en["avg_watts"] else {
            **en, "tokens_per_joule": en["calls"] * int(lens.sum()) / en["wall_s"] / en["avg_watts"],
            "tflop_per_joule": en["calls"] * flops / 1e12 / en["wall_s"] / en["avg_watts"]},
    }
    if "chunked" in parts:
        res["prefill_chunked"] = chunked_prefill(tr, lens, q, out, mk)
    del out
    return res


def _transfer_part(tr, pre, convs, lens, mk):
    """Pack every conversation of the prefill batch, unpack into a pool with another placement,
    and check pack -> unpack -> pack is bit-exact."""
    sh = tr.shape
    hkv, d = sh.n_kv_heads, sh.head_dim
    dst = mk(tr.dst_seed)
    wires = [torch.empty(pre.kv_pack_size(c), dtype=torch.uint8, device="cuda") for c in convs]
    pre.profile_start()
    for c, w in zip(convs, wires):
        pre.kv_pack(c, w)
    pk = pre.profile_stop()["pack"]
    dst.profile_start()
    dconvs = [dst.kv_unpack(w, int(L)) for w, L in zip(wires, lens)]
    up = dst.profile_stop()["unpack"]
    ok = True
    for c, w in zip(dconvs, wires):
        ok = ok and torch.equal(dst.kv_pack(c), w)
    torch.cuda.synchronize()
    move = 2 * int(lens.sum()) * 2 * hkv * d * 2          # read + write of every valid token's K, V
    dst.close()
    del wires
    torch.cuda.empty_cache()
    gbs = lambda b, t: b / (t * 1e-3) / 1e9
    workload = (f"one-time transfer of the turn-1 prefill batch: {tr.n_convs} conversations, L U[{tr.lo},"
                f"{tr.hi}] (sum {int(lens.sum())}), {hkv} kv heads, d {d}, 1 layer")
    return {
        "pack": {"workload": workload, "kernel_ms": pk[0], "launches": pk[1], "bytes": move,
                 "gbs": gbs(move, pk[0]),
                 "roofline": {"bound": "hbm", "achieved": gbs(move, pk[0]), "peak": HBM_PEAK_GBS,
                              "unit": "GB/s", "frac": gbs(move, pk[0]) / HBM_PEAK_GBS,
                              **kernel_counters("kv_pack", workload, "kv_move", move / pk[1])}},
        "unpack": {"workload": workload, "kernel_ms": up[0], "launches": up[1], "bytes": move,
                   "gbs": gbs(move, up[0]),
                   "roofline": {"bound": "hbm", "achieved": gbs(move, up[0]), "peak": HBM_PEAK_GBS,
                                "unit": "GB/s", "frac": gbs(move, up[0]) / HBM_PEAK_GBS,
                                **kernel_counters("kv_unpack", workload, "kv_move", move / up[1])},
                   "round_trip_bit_exact": bool(ok)},
    }


# ------------------------------------------------------------------------------------------------
# prefill latency curve (the placement layer's admission signal, Section 3.1 / 4.2)
# ------------------------------------------------------------------------------------------------
def bench_prefill_curve(args):
    """Turn-1 prefill time of one conversation against its length (32q/8kv, d 128, one layer), the
    quadratic least-squares fit the scheduler reads at admission (cs_prefill_curve_fit) and its
    R^2. The paper profiles the same curve offline on its prefiller and finds it quadratic with
    R^2 = 1.0 (Section 3.1)."""
    from paper_2606_01839_amd import KVPool, prefill_curve_fit
    hq, hkv, d, seed = 32, 8, 128, 1006
    lens = [2048, 4096, 8192, 16384, 32768, 65536, 131072]
    pool = KVPool(1, hq, hkv, d, n_pages=pages_for(max(lens)) + 8, max_convs=2,
                  max_pages_per_conv=pages_for(max(lens)), placement_seed=seed)
    ms = []
    for L in lens:
        c = pool.conv_create()
        k, v = gen_kv(seed, 0, 0, L, hkv, d)
        pool.kv_append(c, k[None], v[None])
        q = gen_q(seed, 0, 0, L, hq, d)
        out = torch.empty_like(q)
        step = lambda: pool.attn_prefill_turn1([c], [L], 0, q, out)
        step()
        prof = profiled(pool, step, 2)
        ms.append(prof["attn_fwd"][0] / prof["attn_fwd"][1])
        pool.conv_destroy(c)
        del k, v, q, out
    pool.close()
    torch.cuda.empty_cache()
    coef, r2 = prefill_curve_fit(lens, [m * 1e-3 for m in ms])
    return {"prefill_curve": {
        "workload": "turn-1 prefill of one conversation, 32q/8kv, d 128, 1 layer, L in " + str(lens),
        "lengths": lens, "kernel_ms": ms, "coef_s": list(coef), "r2": r2,
        "tflops": [attn_flops([0], [L], hq, d) / (m * 1e-3) / 1e12 for L, m in zip(lens, ms)]}}


def bench_gqa_shapes(args):
    """The same attention kernel at the GQA shape of the paper's served model (Qwen3-0.6B: 16 query
    heads, 8 KV heads, head_dim 128; Section 5.1), the Llama-3-8B shape (32/8/128) and a group of 8
    (64/8/128): turn-1 prefill of 4 conversations of 32k-64k tokens, one layer."""
    from paper_2606_01839_amd import KVPool
    res = {}
    lens = np.array([32768, 65536, 49152, 40960])
    for hq, hkv in [(16, 8), (32, 8), (64, 8)]:
        d, seed = 128, 1007
        pool = KVPool(1, hq, hkv, d, n_pages=int(sum(pages_for(int(L)) for L in lens)) + 16,
                      max_convs=len(lens), max_pages_per_conv=pages_for(int(lens.max())),
                      placement_seed=seed)
        convs = []
        for b, L in enumerate(lens):
            c = pool.conv_create()
            k, v = gen_kv(seed, b, 0, int(L), hkv, d)
            pool.kv_append(c, k[None], v[None])
            convs.append(c)
            del k, v
        q = torch.cat([gen_q(seed, b, 0, int(L), hq, d) for b, L in enumerate(lens)])
        out = torch.empty_like(q)
        step = lambda: pool.attn_prefill_turn1(convs, lens, 0, q, out)
        step()
        prof = profiled(pool, step, 2)
        ms = prof["attn_fwd"][0] / prof["attn_fwd"][1]
        fl = attn_flops([0] * len(lens), lens, hq, d)
        res[f"{hq}q/{hkv}kv"] = {"kernel_ms": ms, "tflops": fl / (ms * 1e-3) / 1e12,
                                 "frac": fl / (ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS}
        pool.close()
        del q, out
        torch.cuda.empty_cache()
    return {"gqa_shapes": {"workload": "turn-1 prefill, 4 conversations of 32k-64k tokens, d 128, 1 layer",
                           **res}}


def bench_transfer_overlap(args):
    """The decoder receiving a transferred conversation while it decodes (Section 4: the turn-1 KV
    arrives once, then stays): the decode batch (64 conversations, 8k-32k) runs 20 steps on one
    stream while another stream unpacks a 65,536-token conversation of a 32-layer Llama-3-8B-shaped
    model (8 GiB wire) into a second pool, back to back. Reports each kernel's event-timed rate
    alone and under the overlap."""
    from paper_2606_01839_amd import KVPool
    tr = DecodeBatch()
    sh = tr.shape
    hq, hkv, d = sh.n_q_heads, sh.n_kv_heads, sh.head_dim
    pool, convs, lens, kv_dev, q = make_decode_case(tr)
    del kv_dev
    out = torch.empty_like(q)
    NL, L, seed = 32, 65536, 1008
    mk = lambda s: KVPool(NL, hq, hkv, d, n_pages=pages_for(L) + 8, max_convs=2,
                          max_pages_per_conv=pages_for(L) + 8, placement_seed=s)
    src, dst = mk(seed), mk(seed + 1)
    c = src.conv_create()
    for l0 in range(0, L, 8192):
        k = torch.stack([sv.bf16_tensor(sv.mix_key(seed, 0, KIND_K, l), (8192, hkv, d), start=l0 * hkv * d,
                                        device="cuda") for l in range(NL)])
        v = torch.stack([sv.bf16_tensor(sv.mix_key(seed, 0, KIND_V, l), (8192, hkv, d), start=l0 * hkv * d,
                                        device="cuda") for l in range(NL)])
        src.kv_append(c, k, v)
        del k, v
    wire = src.kv_pack(c)
    src.close()
    torch.cuda.synchronize()
    dec_bytes = int(lens.sum()) * 2 * hkv * d * 2 + len(lens) * hq * d * 2 + int(sum(pages_for(int(x)) for x in lens)) * 4
    move = 2 * L * NL * hkv * d * 2 * 2

    def unpack_once():
        h = dst.kv_unpack(wire, L)
        dst.conv_destroy(h)

    def run(decode_steps, unpacks):
        sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
        pool.profile_start()
        dst.profile_start()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        with torch.cuda.stream(sb):
            for _ in range(unpacks):
                unpack_once()
        with torch.cuda.stream(sa):
            for _ in range(decode_steps):
                pool.attn_decode_batch(convs, 0, q, out)
        torch.cuda.synchronize()
        wall = (time.perf_counter() - t0) * 1e3
        pd, pu = pool.profile_stop(), dst.profile_stop()
        res = {"wall_ms": wall,
               "hbm_gbs": (decode_steps * dec_bytes + unpacks * move) / (wall * 1e-3) / 1e9}
        if decode_steps:
            ms = pd["decode_split"][0] / pd["decode_split"][1]
            res["decode_split_ms"], res["decode_split_gbs"] = ms, dec_bytes / (ms * 1e-3) / 1e9
        if unpacks:
            ms = pu["unpack"][0] / unpacks
            res["unpack_ms"], res["unpack_gbs"] = ms, move / (ms * 1e-3) / 1e9
        return res

    run(2, 1)
    alone_dec, alone_up = run(20, 0), run(0, 4)
    both = run(20, 4)
    pool.close()
    dst.close()
    del wire, q, out
    torch.cuda.empty_cache()
    return {"transfer_overlap": {
        "workload": "decode batch (64 conversations, 8k-32k, 1 layer) on one stream; unpack of a "
                    "65536-token 32-layer 32q/8kv d128 conversation (8 GiB wire) on another",
        "decode_alone": alone_dec, "unpack_alone": alone_up, "overlapped": both,
        "note": "per-kernel rates use each kernel's own event-timed duration, which includes the "
                "time the two streams share the GPU; hbm_gbs = all algorithmic bytes / wall time"}}


def bench_decode_curve(args):
    """Decode step time against the batch's active KV tokens (Section 3.2: decode is memory-bound,
    gated by KV-cache bandwidth; the paper finds iteration latency set by decode at 262,144 active
    tokens): 32 conversations of equal length, 32q/8kv d128, one layer, active tokens 32k..2M.
    A least-squares line t = a + b * tokens gives the fixed cost a and the marginal bandwidth
    4096 B / b."""
    from paper_2606_01839_amd import KVPool
    hq, hkv, d, seed, B = 32, 8, 128, 1009, 32
    per = [1024, 2048, 4096, 8192, 16384, 32768, 65536]
    pool = KVPool(1, hq, hkv, d, n_pages=B * pages_for(max(per)) + 16, max_convs=B,
                  max_pages_per_conv=pages_for(max(per)), placement_seed=seed)
    convs = [pool.conv_create() for _ in range(B)]
    have = 0
    pts = []
    for L in per:
        for b, c in enumerate(convs):
            k, v = gen_kv(seed, b, have, L - have, hkv, d)
            pool.kv_append(c, k[None], v[None])
        have = L
        q = torch.cat([gen_q(seed, b, L - 1, 1, hq, d) for b in range(B)])
        out = torch.empty_like(q)
        step = lambda: pool.attn_decode_batch(convs, 0, q, out)
        ms = timed(step, 20, 3)
        pts.append((B * L, ms))
    pool.close()
    torch.cuda.empty_cache()
    x = np.array([p[0] for p in pts], dtype=np.float64)
    y = np.array([p[1] for p in pts], dtype=np.float64)
    b_, a_ = np.polyfit(x, y, 1)
    return {"decode_curve": {
        "workload": f"decode step, {B} conversations of equal length, 32q/8kv d128, 1 layer",
        "active_tokens": [int(v) for v in x], "step_ms": [float(v) for v in y],
        "fixed_ms": float(a_), "marginal_gbs": 4096 / (b_ * 1e-3) / 1e9}}


# ------------------------------------------------------------------------------------------------
# mixed agentic trace (256 conversations, 32 layers, Llama-3-8B attention shape)
# ------------------------------------------------------------------------------------------------
class _Live:
    __slots__ = ("tr", "h", "turn", "phase", "left", "length", "order", "host", "pending")

    def __init__(self, tr, h, length, order, phase="decode"):
        self.tr, self.h, self.turn, self.length, self.order = tr, h, 0, length, order
        self.phase, self.left, self.host = phase, tr.decodes[0], None
        self.pending = tr.turn1 if phase == "prefill" else 0   # prompt tokens still to prefill


# Turn-1 prefill curve of one layer (32q/8kv, d 128) measured on MI355X by bench_prefill_curve;
# the scheduler's admission reads it, scaled to the 32 layers of the mixed trace.
PREFILL_CURVE_1L = (1.57e-5, 4.94e-9, 6.81e-12)
ADMIT_WATERMARK = 0.8    # bind only while the decoder's pages after the transfer stay below this


COLLOCATED_BUDGET = 2944   # tokens per step of the paper's collocated replicas (Section 5.1)


def bench_mixed(args, collocated=False, trace_cfg=None, pool_pages=None):
    """Serve the synthetic agentic trace on one decoder pool (Section 4: after the one-time
    transfer a conversation's later turns run on its decoder).

    Placement follows the paper's reactive scheduler through the library (Section 4.2): a waiting
    conversation is admitted with cs_sched_admit (its expected turn-1 prefill time read off the
    quadratic curve) and bound with cs_sched_bind, which reads the decoder pool's current
    occupancy -- no knowledge of how long a conversation will grow. Binding also keeps the pool
    below an 80% high-water mark so live conversations have room to grow. At admission the turn-1
    prompt is prefilled on a separate prefiller pool (all layers), packed, unpacked into the
    decoder pool and released from the prefiller -- the one-time transfer. Every step, each live
    conversation either appends its pending turn chunk (extend; whole chunks, at most 8192 extend
    tokens per step, the first always) or decodes one token; finished conversations are destroyed
    and new ones admitted between steps. When a step's new tokens do not fit in the pool, extend
    chunks wait, then the most recently admitted conversation is swapped out (kv_pack to host
    memory, destroyed) and later swapped back in (kv_unpack) before anything new is admitted.

    With --mixed-to-completion the run continues until every conversation has completed, in the
    layer-ordered form of the step (a model forward pass) except every 25th step, which runs in the
    overlapped order with per-kernel timing events, sampling oracle parity every 2000 steps;
    otherwise `args.mixed_steps` timed steps alternate between the two orders of cs_mixed_step.

    collocated=True is the paper's collocated baseline instead (Section 5.1): no prefiller; a new
    conversation's turn-1 prompt is prefilled on the decoder itself in chunks, batched with the
    decodes under a budget of COLLOCATED_BUDGET tokens per step (decode tokens first, then prompt
    and append chunks in admission order, split as the budget allows), layer-ordered steps.

    trace_cfg (a synth.traces.MixedTrace) and pool_pages (decoder pool size in pages) replace the
    256-conversation trace and the HBM-sized pool, for small runs of the same serving loop."""
    from paper_2606_01839_amd import KVPool, Scheduler
    tr = trace_cfg if trace_cfg is not None else MixedTrace()
    sh = tr.shape
    NL, hq, hkv, d = sh.n_layers, sh.n_q_heads, sh.n_kv_heads, sh.head_dim
    trace = tr.conversations()
    to_completion = bool(getattr(args, "mixed_to_completion", False))
    page_bytes = NL * hkv * 2 * 16 * d * 2                       # one page, all layers
    import gc
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()                                     # earlier components' cached blocks
    free, _ = torch.cuda.mem_get_info()
    max_t1 = max(c.turn1 for c in trace)
    reserve = 3 * pages_for(max_t1) * page_bytes + (24 << 30)    # prefiller, wire, step buffers
    n_pages = int((0.85 * free - reserve) // page_bytes) if pool_pages is None else int(pool_pages)
    max_final = max(c.final_len() for c in trace)
    dec = KVPool(NL, hq, hkv, d, n_pages=n_pages, max_convs=tr.n_convs,
                 max_pages_per_conv=pages_for(max_final), placement_seed=tr.seed + 1)
    pre = KVPool(NL, hq, hkv, d, n_pages=pages_for(max_t1) + 16, max_convs=2,
                 max_pages_per_conv=pages_for(max_t1) + 16, placement_seed=tr.seed + 2)
    sched = Scheduler(tuple(NL * c for c in PREFILL_CURVE_1L), 1e9, [dec])
    # Values: rows of two seeded tables made once with the counter-based generator (K and V rows of
    # Hkv*d values, Q rows of Hq*d values, 2^20 and 2^19 rows, N(0,1)-like bf16). Token `pos` of
    # conversation c, kind and layer reads row (offset(c, kind, layer) + pos) mod rows: a gather per
    # step instead of hashing every element of the step's inputs, and the oracle checks read the
    # same rows back.
    kv_rows, q_rows_n = 1 << 20, 1 << 19
    t_kv = sv.bf16_tensor(sv.mix_key(tr.seed, 7001), (kv_rows, hkv * d), device="cuda")
    t_q = sv.bf16_tensor(sv.mix_key(tr.seed, 7002), (q_rows_n, hq * d), device="cuda")
    offs = {}

    def conv_offs(c, kind):
        o = offs.get((c, kind))
        if o is None:
            o = offs[(c, kind)] = np.array([sv.mix_key(tr.seed, c, kind, l) & ((1 << 40) - 1)
                                            for l in range(NL)], dtype=np.int64)
        return o

    def gather(kind, items, layers, H):
        """[len(layers)][sum n][H][d] device tensor of the tokens (conv, start, n) of each layer."""
        table, rows_n = (t_q, q_rows_n) if kind == KIND_Q else (t_kv, kv_rows)
        counts = np.array([n for _, _, n in items], dtype=np.int64)
        pos = np.concatenate([p0 + np.arange(n, dtype=np.int64) for _, p0, n in items])
        base = np.stack([conv_offs(c, kind)[layers] for c, _, _ in items], axis=1)      # [layers][items]
        idx = (np.repeat(base, counts, axis=1) + pos[None, :]) & (rows_n - 1)
        out = table.index_select(0, torch.from_numpy(idx.reshape(-1)).cuda())
        return out.view(len(layers), int(counts.sum()), H, d)

    def rows(kind, items, layer, H, device="cuda"):
        """Values of tokens (conv, start, n) for one layer: [sum n][H][d]."""
        out = gather(kind, items, [layer], H)[0]
        return out.cpu() if device == "cpu" else out

    def rows_all(kind, items, H):
        """The same for every layer: [NL][sum n][H][d]."""
        return gather(kind, items, list(range(NL)), H)

    stats = {"prefill_flops": 0, "prefill_ms": 0.0, "pack_ms": 0.0, "unpack_ms": 0.0, "move_bytes": 0,
             "admitted": 0, "completed": 0, "swapped_out": 0, "swapped_in": 0, "turn1_tokens": 0,
             "admission_expected_s": 0.0}
    live, queue, swapped = [], list(trace), []
    t_run = time.perf_counter()
    order = [0]

    def used_free():
        return dec.occupancy()

    def swap_in():
        while swapped:
            lc = swapped[0]
            used, fr = used_free()
            if used + pages_for(lc.length) > ADMIT_WATERMARK * n_pages:
                return False
            swapped.pop(0)
            lc.h = dec.kv_unpack(lc.host.cuda(), lc.length)
            lc.host = None
            live.append(lc)
            stats["swapped_in"] += 1
        return True

    def swap_out(lc):
        host = dec.kv_pack(lc.h).cpu()                           # synchronous copy to host memory
        dec.conv_destroy(lc.h)
        lc.host, lc.h = host, None
        live.remove(lc)
        swapped.append(lc)
        stats["swapped_out"] += 1

    def admit():
        if not swap_in():                                        # swapped conversations come first
            return
        while queue:
            c = queue[0]
            L = c.turn1
            used, _ = used_free()
            # prompts still to be prefilled on the decoder (collocated) count as taken
            used += sum(pages_for(x.length + x.pending) - pages_for(x.length) for x in live if x.phase == "prefill")
            if used + pages_for(L) > ADMIT_WATERMARK * n_pages:
                return
            if sched.bind(L) < 0:                                # cs_sched_bind: occupancy now
                return
            queue.pop(0)
            if collocated:                                       # prefilled in chunks on the decoder
                stats["admitted"] += 1
                order[0] += 1
                live.append(_Live(c, dec.conv_create(), 0, order[0], phase="prefill"))
                continue
            start, done = sched.admit(L, time.perf_counter() - t_run)   # cs_sched_admit
            stats["admission_expected_s"] += done - start
            h = pre.conv_create()
            k = rows_all(KIND_K, [(c.cid, 0, L)], hkv)
            v = rows_all(KIND_V, [(c.cid, 0, L)], hkv)
            pre.kv_append(h, k, v)
            del k, v
            qs = rows_all(KIND_Q, [(c.cid, 0, L)], hq)
            out = torch.empty_like(qs[0])
            torch.cuda.synchronize()
            pre.profile_start()
            for l in range(NL):
                pre.attn_prefill_turn1([h], [L], l, qs[l], out)
            wire = pre.kv_pack(h)
            pp = pre.profile_stop()
            dec.profile_start()
            hd = dec.kv_unpack(wire, L)
            up = dec.profile_stop()
            pre.conv_destroy(h)
            del qs, out, wire
            stats["prefill_ms"] += pp["attn_fwd"][0]
            stats["pack_ms"] += pp["pack"][0]
            stats["unpack_ms"] += up["unpack"][0]
            stats["prefill_flops"] += attn_flops([0], [L], hq, d) * NL
            stats["move_bytes"] += 2 * L * NL * hkv * d * 2 * 2
            stats["admitted"] += 1
            stats["turn1_tokens"] += L
            order[0] += 1
            live.append(_Live(c, hd, L, order[0]))

    t0 = time.perf_counter()
    admit()
    log(f"mixed: decoder pool {n_pages} pages; admitted {len(live)} conversations "
        f"in {time.perf_counter() - t0:.1f}s")
    mk_tot = lambda: {"wall_s": 0.0, "tokens": 0, "dec_bytes": 0, "ext_flops": 0, "split_ms": 0.0,
                      "merge_ms": 0.0, "fwd_ms": 0.0, "append_ms": 0.0, "append_bytes": 0, "steps": 0,
                      "dec_tokens": 0, "ext_tokens": 0}
    tot, tot_ord = mk_tot(), mk_tot()
    parity = {}
    samples = []
    steplog = []     # layer-ordered timed steps: (seconds, decode tokens, prompt chunk tokens, append tokens)
    want_check = False
    check_every = int(getattr(args, "mixed_check_every", 2000))
    sample_every = 25
    max_steps = 10 ** 7 if to_completion else args.mixed_steps + 1
    max_s = getattr(args, "mixed_max_s", None)
    stop = [False]
    import signal
    old_term = signal.signal(signal.SIGTERM, lambda *a: stop.__setitem__(0, True))
    step = 0
    while step < max_steps and (live or swapped or queue) and not stop[0]:
        if max_s and time.perf_counter() - t_run > max_s:
            break
        if not live:                                             # nothing resident: admit / swap in
            admit()
            if not live:
                raise RuntimeError("mixed trace: no conversation fits the decoder pool")
        dcs = [lc for lc in live if lc.phase == "decode"]
        ext = []
        if collocated:
            budget = COLLOCATED_BUDGET - len(dcs)
            for lc in sorted((x for x in live if x.phase in ("prefill", "append")), key=lambda x: x.order):
                if budget <= 0:
                    break
                n = min(lc.pending, budget)
                ext.append((lc, n))
                budget -= n
        else:
            budget = 8192
            for lc in live:
                if lc.phase == "append":
                    n = lc.pending
                    if not ext or sum(x[1] for x in ext) + n <= budget:
                        ext.append((lc, n))
        # the step's new tokens must fit: extend chunks wait while other work can run, then the
        # most recently admitted conversation swaps out
        while True:
            need = sum(pages_for(lc.length + n) - pages_for(lc.length) for lc, n in ext) + \
                   sum(pages_for(lc.length + 1) - pages_for(lc.length) for lc in dcs)
            if need <= used_free()[1]:
                break
            if len(ext) > 1 or (ext and dcs):
                ext.pop()
                continue
            victims = [lc for lc in live if lc.length > 0 and not (ext and lc is ext[0][0])]
            if not victims:
                raise RuntimeError("mixed trace: one conversation's turn does not fit the decoder pool")
            swap_out(max(victims, key=lambda x: x.order))
            dcs = [lc for lc in live if lc.phase == "decode"]
        if not ext and not dcs:
            step += 1
            continue
        items_new = [(lc.tr.cid, lc.length, n) for lc, n in ext] + [(lc.tr.cid, lc.length, 1) for lc in dcs]
        k = rows_all(KIND_K, items_new, hkv)
        v = rows_all(KIND_V, items_new, hkv)
        qe = rows_all(KIND_Q, items_new[:len(ext)], hq) if ext else None
        qd = rows_all(KIND_Q, items_new[len(ext):], hq) if dcs else None
        torch.cuda.synchronize()
        timed_step = step > 0                                      # step 0 warms up
        # to completion: every sample_every-th step runs in the overlapped order with per-kernel
        # timing events, which samples the decode and extend rates over the whole run
        if to_completion:
            ordered = step % sample_every != 0
        else:
            ordered = True if collocated else step % 2 == 0
        acc = tot_ord if ordered else tot
        if timed_step and not ordered:
            dec.profile_start()
        ts = time.perf_counter()
        oe, od = dec.mixed_step([lc.h for lc, _ in ext], [n for _, n in ext], [lc.h for lc in dcs], k, v, qe, qd,
                                layer_ordered=ordered)
        torch.cuda.synchronize()
        te = time.perf_counter()
        if timed_step:
            pr = dec.profile_stop() if not ordered else None
            n_ext = sum(n for _, n in ext)
            acc["wall_s"] += te - ts
            acc["tokens"] += n_ext + len(dcs)
            acc["ext_tokens"] += n_ext
            acc["dec_tokens"] += len(dcs)
            acc["dec_bytes"] += NL * (sum(lc.length + 1 for lc in dcs) * 2 * hkv * d * 2
                                      + 2 * len(dcs) * hq * d * 2
                                      + sum(pages_for(lc.length + 1) for lc in dcs) * 4)
            acc["ext_flops"] += NL * attn_flops([lc.length for lc, _ in ext], [n for _, n in ext], hq, d)
            if pr is not None:
                acc["split_ms"] += pr["decode_split"][0]
                acc["merge_ms"] += pr["decode_merge"][0]
                acc["fwd_ms"] += pr["attn_fwd"][0]
                acc["append_ms"] += pr["append"][0]
                acc["append_bytes"] += 2 * NL * (n_ext + len(dcs)) * hkv * d * 2 * 2
            acc["steps"] += 1
            if ordered:
                steplog.append((te - ts, len(dcs), sum(n for lc, n in ext if lc.phase == "prefill"),
                                sum(n for lc, n in ext if lc.phase == "append")))
        mode = "layer_ordered" if ordered else "overlapped"
        if to_completion and step > 0 and step % check_every == 0:
            want_check = True
        check = (mode not in parity) if not to_completion else want_check
        if check and dcs and ext:
            want_check = False
            # oracle check: shortest decoding and shortest extending conversation, first and last layer
            from oracle.attention import attend_rows
            errs = []
            lcd = min(dcs, key=lambda x: x.length)
            i_d = dcs.index(lcd)
            i_e = min(range(len(ext)), key=lambda i: ext[i][0].length)
            lce, ne = ext[i_e]
            row_e = sum(n for _, n in ext[:i_e + 1]) - 1
            for layer in (0, NL - 1):
                for lc, qrow, outrow, pos in ((lcd, qd[layer, i_d], od[layer, i_d], lcd.length),
                                              (lce, qe[layer, row_e], oe[layer, row_e], lce.length + ne - 1)):
                    kk = rows(KIND_K, [(lc.tr.cid, 0, pos + 1)], layer, hkv, device="cpu")
                    vv = rows(KIND_V, [(lc.tr.cid, 0, pos + 1)], layer, hkv, device="cpu")
                    ref = attend_rows(sv.bf16_to_f64(qrow[None]), [pos], sv.bf16_to_f64(kk), sv.bf16_to_f64(vv))
                    errs.append(float(np.abs(sv.bf16_to_f64(outrow[None]) - ref).max()))
            parity[mode] = {"samples": len(errs), "max_abs": max(errs), "ok": bool(max(errs) <= 1e-2)}
            samples.append({"step": step, "max_abs": max(errs)})
        del k, v, qe, qd, oe, od
        # advance the trace
        for lc, n in ext:
            lc.length += n
            lc.pending -= n
            if lc.pending == 0:
                lc.phase, lc.left = "decode", lc.tr.decodes[lc.turn]
        finished = []
        for lc in dcs:
            lc.length += 1
            lc.left -= 1
            if lc.left == 0:
                lc.turn += 1
                if lc.turn == lc.tr.turns:
                    finished.append(lc)
                else:
                    lc.phase, lc.pending = "append", lc.tr.appends[lc.turn - 1]
        for lc in finished:
            live.remove(lc)
            dec.conv_destroy(lc.h)
            stats["completed"] += 1
        if finished or swapped:
            admit()
        step += 1
        if to_completion and step % 1000 == 0:
            log(f"mixed: step {step}, {stats['completed']} completed, {len(live)} live, "
                f"{len(swapped)} swapped, {len(queue)} waiting, {time.perf_counter() - t_run:.0f}s")
    run_s = time.perf_counter() - t_run
    # a handler installed outside Python (a profiler's, for one) reads back as None: restore the
    # default then
    signal.signal(signal.SIGTERM, old_term if old_term is not None else signal.SIG_DFL)
    stopped_early = bool(live or swapped or queue) and to_completion
    used, free_pages = dec.occupancy()
    sched.close()
    dec.close()
    pre.close()
    torch.cuda.empty_cache()
    gbs = lambda b, ms: b / (ms * 1e-3) / 1e9 if ms > 0 else None
    tfs = lambda f, ms: f / (ms * 1e-3) / 1e12 if ms > 0 else None
    roof_s = lambda t: t["dec_bytes"] / (HBM_PEAK_GBS * 1e9) + t["ext_flops"] / (BF16_PEAK_TFLOPS * 1e12)
    workload = (f"mixed agentic trace: {tr.n_convs} conversations, turns U[{tr.turns_lo},{tr.turns_hi}], "
                f"turn-1 logN(median {tr.turn1_median}) <= {tr.turn1_hi}, appends logN(median "
                f"{tr.append_median}), decodes logN(median {tr.decode_median}); {NL} layers "
                f"{hq}q/{hkv}kv d{d}; decoder pool {n_pages} pages ({n_pages * page_bytes / 2**30:.0f} GiB)")
    placement = {"rule": "cs_sched_admit on the prefill curve + cs_sched_bind on the pool's current "
                         f"occupancy, {int(100 * ADMIT_WATERMARK)}% high-water mark; swap out/in "
                         "(kv_pack to host / kv_unpack) when a step's tokens do not fit",
                 "admitted": stats["admitted"], "completed": stats["completed"],
                 "swapped_out": stats["swapped_out"], "swapped_in": stats["swapped_in"],
                 "turn1_prefill_s_expected_by_curve": stats["admission_expected_s"],
                 "turn1_prefill_s_measured": stats["prefill_ms"] * 1e-3}
    def tbt(rows_):
        t_ = np.array([r[0] for r in rows_ if r[1] > 0]) * 1e3
        return [float(np.percentile(t_, 50)), float(np.percentile(t_, 95))] if t_.size else None

    tbt_all = tbt(steplog)
    tbt_prompt = tbt([r for r in steplog if r[2] > 0])
    tbt_no_prompt = tbt([r for r in steplog if r[2] == 0])
    if collocated:
        t = tot_ord
        return {"mixed_collocated": {
            "workload": workload + f"; collocated: turn-1 prompts prefilled on the decoder in chunks, "
                                   f"{COLLOCATED_BUDGET} tokens per step (decode tokens first)",
            "timed_steps": t["steps"], "admitted": stats["admitted"], "completed": stats["completed"],
            "swapped_out": stats["swapped_out"],
            "tokens_per_s": t["tokens"] / t["wall_s"] if t["wall_s"] else None,
            "decode_tokens": t["dec_tokens"], "chunk_tokens": t["ext_tokens"],
            "step_ms": 1e3 * t["wall_s"] / max(1, t["steps"]),
            "tbt_ms_p50_p95": tbt_all, "tbt_ms_p50_p95_steps_with_prompt_chunk": tbt_prompt,
            "tbt_ms_p50_p95_steps_without": tbt_no_prompt,
            "step_roofline": {"frac": roof_s(t) / t["wall_s"] if t["wall_s"] else None},
            "spot_parity": parity}}
    if to_completion:
        t = {k_: tot[k_] + tot_ord[k_] for k_ in tot}            # every timed step, both orders
        return {"mixed_to_completion": {
            "workload": workload, "steps": step, "timed_steps": t["steps"], "run_s": run_s,
            "stopped_early": stopped_early,
            **placement, "live_end": len(live), "swapped_end": len(swapped), "waiting_end": len(queue),
            "decode_tokens": t["dec_tokens"], "extend_tokens": t["ext_tokens"],
            "turn1_tokens": stats["turn1_tokens"],
            "step_tokens_per_s": t["tokens"] / t["wall_s"] if t["wall_s"] else None,
            "run_tokens_per_s": (t["tokens"] + stats["turn1_tokens"]) / run_s,
            "step_ms": 1e3 * t["wall_s"] / max(1, t["steps"]),
            "step_roofline": {"roofline_s": roof_s(t), "measured_step_s": t["wall_s"],
                              "frac": roof_s(t) / t["wall_s"] if t["wall_s"] else None},
            "sampled_kernel_rates": {
                "steps": tot["steps"],
                "note": f"every {sample_every}th step runs in the overlapped order with per-kernel "
                        "timing events (all other steps are layer-ordered, without events); rates "
                        "use each kernel kind's event-timed duration, which includes the time the "
                        "two streams share the GPU",
                "decode_gbs": gbs(tot["dec_bytes"], tot["split_ms"] + tot["merge_ms"]),
                "decode_split_gbs": gbs(tot["dec_bytes"], tot["split_ms"]),
                "extend_tflops": tfs(tot["ext_flops"], tot["fwd_ms"]),
                "append_gbs": gbs(tot["append_bytes"], tot["append_ms"]),
                "step_ms": 1e3 * tot["wall_s"] / max(1, tot["steps"]),
                "step_roofline_frac": roof_s(tot) / tot["wall_s"] if tot["wall_s"] else None},
            "turn1_prefill_tflops": tfs(stats["prefill_flops"], stats["prefill_ms"]),
            "pack_gbs": gbs(stats["move_bytes"], stats["pack_ms"]),
            "unpack_gbs": gbs(stats["move_bytes"], stats["unpack_ms"]),
            "occupancy_end": {"used_pages": used, "free_pages": free_pages},
            "tbt_ms_p50_p95": tbt_all,
            "parity_samples": samples,
            "parity_ok": bool(samples and all(s_["max_abs"] <= 1e-2 for s_ in samples))}}
    return {"mixed": {
        "workload": workload,
        "timed_steps": tot["steps"], "live_convs_end": len(live), **placement,
        "tokens_per_s": tot["tokens"] / tot["wall_s"] if tot["wall_s"] else None,
        "step_ms": 1e3 * tot["wall_s"] / max(1, tot["steps"]),
        "decode_tokens": tot["dec_tokens"], "extend_tokens": tot["ext_tokens"],
        "steps_note": "timed steps alternate between the two orders of the mixed step; tokens_per_s, "
                      "step_ms and step_roofline are over the overlapped steps, layer_ordered over "
                      "the others",
        "layer_ordered": {
            "steps": tot_ord["steps"],
            "tokens_per_s": tot_ord["tokens"] / tot_ord["wall_s"] if tot_ord["wall_s"] else None,
            "step_ms": 1e3 * tot_ord["wall_s"] / max(1, tot_ord["steps"]),
            "frac": roof_s(tot_ord) / tot_ord["wall_s"] if tot_ord["wall_s"] else None,
            "tbt_ms_p50_p95": tbt_all,
            "note": "layer l+1's attention starts after layer l's (extend and decode of one layer "
                    "overlap), as in a model forward pass; no timing events on these steps"},
        "step_roofline": {
            "decode_bytes_per_step": tot["dec_bytes"] / max(1, tot["steps"]),
            "extend_flops_per_step": tot["ext_flops"] / max(1, tot["steps"]),
            "roofline_ms_per_step": 1e3 * roof_s(tot) / max(1, tot["steps"]),
            "frac": roof_s(tot) / tot["wall_s"] if tot["wall_s"] else None,
            "note": "time the step's decode bytes take at 8 TB/s plus its extend FLOPs at 2.5 PFLOP/s, "
                    "over the measured step time (extend runs on a second stream, overlapping the "
                    "decode). Per-kernel rates below use each kernel's own event-timed duration, "
                    "which includes the time it shares the GPU with the other stream."},
        "decode_gbs": gbs(tot["dec_bytes"], tot["split_ms"] + tot["merge_ms"]),
        "decode_split_gbs": gbs(tot["dec_bytes"], tot["split_ms"]),
        "extend_tflops": tfs(tot["ext_flops"], tot["fwd_ms"]),
        "append_gbs": gbs(tot["append_bytes"], tot["append_ms"]),
        "turn1_prefill_tflops": tfs(stats["prefill_flops"], stats["prefill_ms"]),
        "pack_gbs": gbs(stats["move_bytes"], stats["pack_ms"]),
        "unpack_gbs": gbs(stats["move_bytes"], stats["unpack_ms"]),
        "occupancy_end": {"used_pages": used, "free_pages": free_pages},
        "spot_parity": parity}}


def bench_sim(comps):
    """The host simulator (paper_2606_01839_amd/sim.py) timed with the rates this run measured
    (turn-1 prefill curve, decode fixed cost and marginal bandwidth, extend rate, pack/unpack):
    the 256-conversation agentic trace, Poisson arrivals, 1 prefiller + 2 decoders of 116,000 pages
    (85% of HBM at 32 layers), 2 s of tool time between turns. CPU only."""
    from paper_2606_01839_amd.sim import ConvSpec, CostModel, Simulator
    cost = CostModel.from_bench({"components": comps})
    convs = MixedTrace().conversations()
    out = {"workload": "host simulation of the mixed agentic trace (256 conversations) on 1 prefiller + "
                       "2 decoders, Poisson arrivals, 2 s tool time, rates measured in this run",
           "cost_model": {k: getattr(cost, k) for k in ("prefill_curve", "decode_fixed_s", "decode_gbs",
                                                        "extend_tflops", "move_gbs", "link_gbs")}}
    for rate in (0.2, 1.0):
        arr = np.cumsum(np.random.default_rng(7).exponential(1.0 / rate, size=len(convs)))
        spec = [ConvSpec(c.turn1, c.appends, c.decodes, float(a)) for c, a in zip(convs, arr)]
        sim = Simulator(spec, cost, n_decoders=2, pages_per_decoder=116_000, max_wait_s=30.0, tool_s=2.0)
        r = sim.run()
        L = np.array([x[0] for x in r["turn1_ttft"]], dtype=float)
        T = np.array([x[1] for x in r["turn1_ttft"]])
        c = np.polyfit(L, T, 2)
        later = np.array([t for _, _, t in r["later_ttft"]])
        out[f"rate_{rate}"] = {
            "completed": r["completed"], "refusals": r["refusals"], "swaps": r["swaps"],
            "makespan_s": r["makespan_s"], "tokens_per_s": r["tokens_per_s"],
            "decode_tokens_per_s": r["decode_tokens_per_s"],
            "turn1_ttft_s_p50_p95": [float(np.median(T)), float(np.percentile(T, 95))],
            "turn1_ttft_quadratic_r2": float(1 - ((T - np.polyval(c, L)) ** 2).sum() / ((T - T.mean()) ** 2).sum()),
            "later_ttft_s_p50_p95": [float(np.median(later)), float(np.percentile(later, 95))],
            "decode_dominated_share_by_active_kv": [
                {"active_tokens": [lo, hi], "iterations": n, "share": s_}
                for lo, hi, n, s_ in sim.decode_dominance([0, 131072, 262144, 524288, 1048576, 1 << 40]) if n]}
    return {"sim": out}


def copy_calibration():
    """A plain 1 GiB device copy: its FETCH_SIZE / WRITE_SIZE counters calibrate the HBM traffic
    reported for the decode kernel (known 1 GiB read + 1 GiB written)."""
    a = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    del a, b


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--skip-components", action="store_true")
    ap.add_argument("--only", choices=["decode", "extend", "prefill", "prefill1", "transfer", "append", "mixed",
                                       "curve", "shapes", "overlap", "dcurve", "device"], default=None,
                    help="run one component and print only its JSON (for profiling)")
    ap.add_argument("--mixed-steps", type=int, default=400,
                    help="timed steps of the mixed agentic trace component (0 = skip it)")
    ap.add_argument("--mixed-to-completion", action="store_true",
                    help="with --only mixed: serve the whole trace until every conversation completes")
    ap.add_argument("--mixed-max-s", type=float, default=None,
                    help="with --mixed-to-completion: stop (and report) after this many seconds")
    ap.add_argument("--mixed-collocated", action="store_true",
                    help="with --only mixed: the collocated baseline (turn-1 prompts chunked into the "
                         "decoder's steps, 2944 tokens per step)")
    ap.add_argument("--no-energy", dest="energy", action="store_false",
                    help="skip the energy runs (8 s of decode and 8 s of prefill, amdsmi counter)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 1 GiB copy (for counter calibration under rocprofv3)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the hot path shards by conversation with no exchange "
              "on the hot path, and this benchmark runs on a single MI355X (use --gpus 1).", file=sys.stderr)
        sys.exit(2)
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    from paper_2606_01839_amd import load_library
    load_library()
    if args.calibrate_copy:
        copy_calibration()
    if args.only and args.only != "decode":
        fn = {"extend": bench_extend, "prefill": bench_prefill_transfer,
              "mixed": lambda a: bench_mixed(a, collocated=a.mixed_collocated),
              "prefill1": lambda a: bench_prefill_transfer(a, parts=("prefill",)),
              "transfer": lambda a: bench_prefill_transfer(a, parts=("transfer",)),
              "append": bench_append, "device": lambda a: {"device": device_block(), "host": host_info()},
              "curve": bench_prefill_curve, "shapes": bench_gqa_shapes,
              "overlap": bench_transfer_overlap, "dcurve": bench_decode_curve}[args.only]
        print(json.dumps({"component": args.only, **fn(args)}), flush=True)
        return
    device = device_block()
    dec = bench_decode(args)
    comps = {}
    if not args.skip_components and not args.only:
        comps.update(bench_extend(args))
        comps.update(bench_prefill_transfer(args))
        comps.update(bench_append(args))
        comps.update(bench_prefill_curve(args))
        comps.update(bench_gqa_shapes(args))
        comps.update(bench_transfer_overlap(args))
        comps.update(bench_decode_curve(args))
        if args.mixed_steps > 0:
            comps.update(bench_mixed(args))
            comps.update(bench_mixed(args, collocated=True))
        comps.update(bench_sim(comps))
    split_gbs = dec["split_bytes"] / (dec["split_ms"] * 1e-3) / 1e9
    line = {
        "metric": METRIC,
        "value": round(dec["value_gbs"], 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(dec["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded counter-based generator; no dataset)",
        "config": {"workload": dec["workload"], "global_batch": 64, "seq_len": "8192-32768",
                   "parallelism": "none (1 GPU)"},
        "roofline": {"bound": "hbm", "kernel": "decode_split_kernel<128>",
                     "achieved": round(split_gbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(split_gbs / HBM_PEAK_GBS, 4), **dec["counters"],
                     "algorithmic_bytes_per_launch": dec["split_bytes"],
                     "kernel_ms": round(dec["split_ms"], 4), "merge_kernel_ms": round(dec["merge_ms"], 4)},
        "cpu_baseline": dec["cpu"],
        "device": device,
        "parity": dec["parity"],
        "step_ms_p10_p50_p90": dec["step_ms_p10_p50_p90"],
        "energy": dec["energy"],
        "components": comps,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
