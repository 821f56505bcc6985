"""Benchmark of the AATC hot path on one MI355X.

Step (the whole hot path once, Llama-3.1-8B-shaped layer, decode batch 1): one
aatc_append_decode_attention call, which
  1. encodes one new token's keys and values (8 KV heads) into the packed caches (records
     for K, bit-transposed tiles for V) at the last cached position, and
  2. runs decode attention of 32 query heads (GQA 4:1) over the 32768 cached tokens per
     KV head packed at 2.75 bits per channel,
in a single kernel launch.
The cache stays at 32768 tokens: every step rewrites the last token.  To measure HBM
rather than the 256 MB Infinity Cache, the steps rotate over enough cache copies to
exceed 512 MB.  The steps are captured in HIP graphs (one step per cache copy) so the
measurement is of the GPU, not of Python launch overhead.

value = packed-cache bytes read per step (codes + fp16 token scales of K and V) /
wall time per step.  roofline = the same bytes / that kernel's average duration (HIP
events on the launch stream) against 8 TB/s.  Encode throughput of a 65536-token
prefill (8 KV heads, K and V) is reported alongside.  cpu_baseline = the NumPy oracle's
decode attention on a bounded token sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0


def _log(msg):
    print(msg, file=sys.stderr, flush=True)


def bf16_tensor(arr, device="cuda"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).to(device)


def setup_decode(cfg_id=2):
    import torch
    import paper_2608_14191_amd as P
    from kvsynth import workload

    w = workload(cfg_id)
    H, HQ, L, B = w.n_kv_heads, w.n_q_heads, w.n_tokens, w.batch
    avg = w.cfg["avg_bits"][0]
    qw = w.cfg["query_weighted_k"]
    t0 = time.time()
    cal_k = [P.aatc_calibrate(w.calib(h, "k"), avg, q_calib=w.calib_queries(h) if qw else None,
                              q_group=w.group) for h in range(H)]
    cal_v = [P.aatc_calibrate(w.calib(h, "v"), avg) for h in range(H)]
    _log(f"[setup] calibrated {2 * H} tensors in {time.time() - t0:.1f}s")
    pk = torch.from_numpy(P.aatc_params_pack(cal_k)).cuda()
    pv = torch.from_numpy(P.aatc_params_pack(cal_v)).cuda()
    rk, rv = cal_k[0].record_bytes, cal_v[0].record_bytes
    cap = L
    kc = torch.zeros((B, H, cap, rk), dtype=torch.uint8, device="cuda")
    vc = torch.zeros((B, H, cap // 64, 64 * rv), dtype=torch.uint8, device="cuda")
    ka = torch.zeros((B, H, cap), dtype=torch.int16, device="cuda")
    va = torch.zeros((B, H, cap), dtype=torch.int16, device="cuda")
    t0 = time.time()
    last_tok = []
    for b in range(B):
        for kind, codes, alpha, params, layout in (("k", kc, ka, pk, P.LAYOUT_RECORDS),
                                                   ("v", vc, va, pv, P.LAYOUT_TILES)):
            x = bf16_tensor(np.stack([w.cache(b, h, kind) for h in range(H)], axis=1))
            P.aatc_encode(params, H, x, L, H * 128, layout, codes[b], alpha[b], cap, 0)
            last_tok.append(x[L - 1:L].clone())
            del x
    torch.cuda.synchronize()
    _log(f"[setup] encoded the {B}x{H}x{L}-token caches in {time.time() - t0:.1f}s")
    q = bf16_tensor(np.stack([w.queries(b) for b in range(B)]))
    return dict(w=w, P=P, pk=pk, pv=pv, kc=kc, vc=vc, ka=ka, va=va, q=q, cap=cap, L=L,
                rk=rk, rv=rv, last_tok=last_tok, cal_k=cal_k, cal_v=cal_v)


def setup_decode_random_codes(cfg_id, seed=0):
    """Another decode workload for throughput only: the configuration's own calibrations
    (so its record sizes and widths), with caches of uniformly random code bits and token
    scales in [0.5, 2).  The decode kernel reads every byte whatever its value, so the
    timing is that of real codes; parity of these shapes is covered by the GPU tests."""
    import torch
    import paper_2608_14191_amd as P
    from kvsynth import workload

    w = workload(cfg_id)
    H, L, B = w.n_kv_heads, w.n_tokens, w.batch
    avg = w.cfg["avg_bits"][0]
    qw = w.cfg["query_weighted_k"]
    cal_k = [P.aatc_calibrate(w.calib(h, "k"), avg, q_calib=w.calib_queries(h) if qw else None,
                              q_group=w.group) for h in range(H)]
    cal_v = [P.aatc_calibrate(w.calib(h, "v"), avg) for h in range(H)]
    pk = torch.from_numpy(P.aatc_params_pack(cal_k)).cuda()
    pv = torch.from_numpy(P.aatc_params_pack(cal_v)).cuda()
    rk, rv = cal_k[0].record_bytes, cal_v[0].record_bytes
    g = torch.Generator(device="cuda").manual_seed(seed)
    kc = torch.randint(0, 256, (B, H, L, rk), dtype=torch.uint8, device="cuda", generator=g)
    vc = torch.randint(0, 256, (B, H, L // 64, 64 * rv), dtype=torch.uint8, device="cuda",
                       generator=g)

    def scales():
        a = 0.5 + 1.5 * torch.rand((B, H, L), device="cuda", generator=g)
        return a.to(torch.float16).view(torch.int16)
    ka, va = scales(), scales()
    x_last = [bf16_tensor(np.stack([w.cache(0, h, kind, n=1, start=L - 1)[0]
                                    for h in range(H)]))[None] for kind in ("k", "v")]
    q = bf16_tensor(np.stack([w.queries(b) for b in range(B)]))
    return dict(w=w, P=P, pk=pk, pv=pv, kc=kc, vc=vc, ka=ka, va=va, q=q, cap=L, L=L,
                rk=rk, rv=rv, last_tok=x_last, cal_k=cal_k, cal_v=cal_v)


def decode_bytes(s) -> int:
    w = s["w"]
    return w.batch * w.n_kv_heads * s["L"] * (s["rk"] + s["rv"] + 4)


def run_decode_bench(s, steps, warmup):
    """Time exactly `steps` steps, captured in HIP graphs (one step per cache copy)."""
    import torch
    P, w = s["P"], s["w"]
    H, HQ, B, L, cap = w.n_kv_heads, w.n_q_heads, w.batch, s["L"], s["cap"]
    per_copy = sum(t.numel() for t in (s["kc"], s["vc"])) + 2 * (s["ka"].numel() + s["va"].numel())
    n_copies = max(2, math.ceil(512e6 / per_copy))
    copies = [(s["kc"], s["ka"], s["vc"], s["va"])]
    for _ in range(n_copies - 1):
        copies.append(tuple(t.clone() for t in copies[0]))
    lens = torch.full((B,), L, dtype=torch.int32, device="cuda")
    out = torch.zeros((B, HQ, 128), dtype=torch.float32, device="cuda")
    ws = torch.zeros(P.aatc_decode_workspace_bytes(B, HQ, H, cap), dtype=torch.uint8,
                     device="cuda")
    scale = 128 ** -0.5
    xk, xv = s["last_tok"][0], s["last_tok"][1]

    x_new_k = xk.reshape(1, H, 128).expand(B, H, 128).contiguous()
    x_new_v = xv.reshape(1, H, 128).expand(B, H, 128).contiguous()

    def step(i):
        """Append the step's token (position L - 1) to K and V and decode: one launch."""
        kc, ka, vc, va = copies[i % n_copies]
        P.aatc_append_decode_attention(s["pk"], s["pv"], B, HQ, H, s["q"], x_new_k, x_new_v,
                                       kc, ka, vc, va, lens, cap, s["rk"], s["rv"], scale, out,
                                       ws)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for i in range(max(warmup, 1)):
            step(i)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    def capture(n, fn):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(n):
                fn(i)
        return g

    g_full = capture(n_copies, step)
    rest = steps % n_copies
    g_rest = capture(rest, step) if rest else None
    g_full.replay()                    # replay once untimed
    torch.cuda.synchronize()

    t0 = time.perf_counter()
    for _ in range(steps // n_copies):
        g_full.replay()
    if g_rest is not None:
        g_rest.replay()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    # The step's one kernel: HIP events (on the stream the graphs run on) around replays.
    reps = max(1, min(20, steps // n_copies))
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        g_full.replay()
    e1.record()
    torch.cuda.synchronize()
    kern_ms = e0.elapsed_time(e1) / (reps * n_copies)
    return elapsed, kern_ms, n_copies, out


def run_encode_bench(avg_bits, reps=5):
    """Prefill encode of 65536 tokens x 8 KV heads (K records + V tiles)."""
    import torch
    import paper_2608_14191_amd as P
    from kvsynth import workload
    w = workload(4)
    H, L = w.n_kv_heads, w.n_tokens
    cal_k = [P.aatc_calibrate(w.calib(h, "k"), avg_bits) for h in range(H)]
    cal_v = [P.aatc_calibrate(w.calib(h, "v"), avg_bits) for h in range(H)]
    pk = torch.from_numpy(P.aatc_params_pack(cal_k)).cuda()
    pv = torch.from_numpy(P.aatc_params_pack(cal_v)).cuda()
    rk, rv = cal_k[0].record_bytes, cal_v[0].record_bytes
    xk = bf16_tensor(np.stack([w.cache(0, h, "k") for h in range(H)], axis=1))
    xv = bf16_tensor(np.stack([w.cache(0, h, "v") for h in range(H)], axis=1))
    kc = torch.zeros((H, L, rk), dtype=torch.uint8, device="cuda")
    vc = torch.zeros((H, L // 64, 64 * rv), dtype=torch.uint8, device="cuda")
    ka = torch.zeros((H, L), dtype=torch.int16, device="cuda")
    va = torch.zeros((H, L), dtype=torch.int16, device="cuda")

    def once():
        P.aatc_encode(pk, H, xk, L, H * 128, P.LAYOUT_RECORDS, kc, ka, L, 0)
        P.aatc_encode(pv, H, xv, L, H * 128, P.LAYOUT_TILES, vc, va, L, 0)

    once()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        once()
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / reps
    return dict(avg_bits=avg_bits, tokens=L, seconds=dt, tokens_per_s=L / dt,
                bytes=int(L * H * (2 * 128 * 2 + rk + rv + 4)))


GROUP_WORKLOAD = ("llama31_8b_decode_b1_32k_groups: batch 1, 32 q / 8 kv heads in 2 head "
                  "groups of 4 (512 channels each), 32768 tokens, 2.75 bits; step = decode "
                  "attention (query weights, splits, merge)")


def setup_group_decode(gkv=4):
    """The Llama decode shape under head-group transforms: host calibrations of each group's
    concatenated calibration draws, the 32768 tokens of every group encoded on the GPU (the
    group prefill, timed)."""
    import concurrent.futures as cf
    import torch
    import paper_2608_14191_amd as P
    from kvsynth import workload

    w = workload(2)
    H, L = w.n_kv_heads, w.n_tokens
    ng = H // gkv
    avg = w.cfg["avg_bits"][0]
    t0 = time.time()
    xs = [(kind, np.concatenate([w.calib(h, kind) for h in range(g * gkv, (g + 1) * gkv)],
                                axis=1)) for kind in ("k", "v") for g in range(ng)]
    with cf.ThreadPoolExecutor(max_workers=len(xs)) as ex:       # (ctypes drops the GIL)
        cals = list(ex.map(lambda kx: P.aatc_calibrate_group(kx[1], avg), xs))
    cal_k, cal_v = cals[:ng], cals[ng:]
    _log(f"[groups] calibrated {len(cals)} group tensors in {time.time() - t0:.1f}s")
    pk = torch.from_numpy(P.aatc_group_params_pack(cal_k)).cuda()
    pv = torch.from_numpy(P.aatc_group_params_pack(cal_v)).cuda()
    rk, rv = cal_k[0].record_bytes, cal_v[0].record_bytes
    kc = torch.zeros((1, ng, L, rk), dtype=torch.uint8, device="cuda")
    vc = torch.zeros((1, ng, L, rv), dtype=torch.uint8, device="cuda")
    ka = torch.zeros((1, ng, L), dtype=torch.int16, device="cuda")
    va = torch.zeros((1, ng, L), dtype=torch.int16, device="cuda")
    xk = bf16_tensor(np.stack([w.cache(0, h, "k") for h in range(H)], axis=1))
    xv = bf16_tensor(np.stack([w.cache(0, h, "v") for h in range(H)], axis=1))

    def prefill():
        P.aatc_group_encode(pk, ng, gkv, xk, L, H * 128, kc[0], ka[0], L, 0)
        P.aatc_group_encode(pv, ng, gkv, xv, L, H * 128, vc[0], va[0], L, 0)

    prefill()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    prefill()
    e1.record()
    torch.cuda.synchronize()
    enc_ms = e0.elapsed_time(e1)
    del xk, xv
    q = bf16_tensor(w.queries(0)[None])
    return dict(w=w, P=P, pk=pk, pv=pv, kc=kc, vc=vc, ka=ka, va=va, q=q, L=L, rk=rk, rv=rv,
                gkv=gkv, ng=ng, enc_ms=enc_ms)


def run_group_decode_bench(s, steps=40):
    """Group decode steps captured in HIP graphs over rotating cache copies; HIP events
    around the replays give the time of one step's three kernels."""
    import torch
    P, w = s["P"], s["w"]
    H, HQ, L = w.n_kv_heads, w.n_q_heads, s["L"]
    per_copy = sum(t.numel() for t in (s["kc"], s["vc"])) + 2 * (s["ka"].numel() + s["va"].numel())
    n_copies = max(2, math.ceil(512e6 / per_copy))
    copies = [(s["kc"], s["ka"], s["vc"], s["va"])]
    for _ in range(n_copies - 1):
        copies.append(tuple(t.clone() for t in copies[0]))
    lens = torch.full((1,), L, dtype=torch.int32, device="cuda")
    out = torch.zeros((1, HQ, 128), dtype=torch.float32, device="cuda")
    ws = torch.empty(P.aatc_group_decode_workspace_bytes(1, HQ, H, s["gkv"], L),
                     dtype=torch.uint8, device="cuda")

    def step(i):
        kc, ka, vc, va = copies[i % n_copies]
        P.aatc_group_decode_attention(s["pk"], s["pv"], 1, HQ, H, s["gkv"], s["q"], kc, ka, vc,
                                      va, lens, L, s["rk"], s["rv"], 128 ** -0.5, out, ws)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for i in range(3):
            step(i)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(n_copies):
            step(i)
    g.replay()
    torch.cuda.synchronize()
    reps = max(1, steps // n_copies)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    step_ms = e0.elapsed_time(e1) / (reps * n_copies)
    nb = s["ng"] * L * (s["rk"] + s["rv"] + 4)
    tok_s = L / (s["enc_ms"] * 1e-3)
    return {"workload": GROUP_WORKLOAD, "bytes_per_step": nb,
            "kernel_us_per_step": round(step_ms * 1e3, 2),
            "GBps": round(nb / (step_ms * 1e-3) / 1e9, 1),
            "frac": round(nb / (step_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "cache_copies": n_copies,
            "prefill_encode": {"tokens": L, "ms": round(s["enc_ms"], 3),
                               "tokens_per_s": round(tok_s, 1)},
            "data": "synthetic tokens, host calibrations"}


# Dense int8 matrix-core peak of the MI355X (ops/s), for the encode's transform products.
MFMA_I8_PEAK_OPS = 5.0e15


def encode_entry(r):
    """Bench entry of one prefill encode measurement: throughput, its HBM fraction, and the
    matrix-core rate: the transform is 65536 x 8 heads x 128 x 128 multiply-adds per tensor
    (K and V), executed as nine int8 limb products each."""
    macs = 2 * r["tokens"] * 8 * 128 * 128
    return {"workload": f"llama31_8b_prefill_64k at {r['avg_bits']} bits",
            "tokens_per_s": round(r["tokens_per_s"], 1),
            "ms": round(r["seconds"] * 1e3, 3),
            "hbm_bytes": r["bytes"],
            "roofline_frac": round(r["bytes"] / r["seconds"] / 1e9 / HBM_PEAK_GBS, 4),
            "mfma_int8_ops_per_prefill": 2 * 9 * macs,
            "mfma_frac": round(2 * 9 * macs / r["seconds"] / MFMA_I8_PEAK_OPS, 4)}


def cpu_baseline(s, target_seconds=15.0, single_thread_seconds=8.0):
    """The oracle's decode attention over a bounded token sample of the same workload, on
    all host threads and again on one."""
    from oracle import aatc as ora
    from threadpoolctl import threadpool_info, threadpool_limits
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    w = s["w"]
    H = w.n_kv_heads

    def ocal(c):
        bits = c.bits_np
        return ora.Calibration(d=128, budget=c.budget_bits, record_bytes=c.record_bytes,
                               d_active=c.d_active, bits=bits, perm=np.arange(128),
                               T64=c.T.astype(np.float64), T32=c.T, s16=c.s16,
                               sigma2=np.ones(128), weight=np.ones(128), bits_eig=bits)
    ck = [ocal(c) for c in s["cal_k"]]
    cv = [ocal(c) for c in s["cal_v"]]
    n = 8192
    krec = [s["kc"][0, h, :n].cpu().numpy() for h in range(H)]
    vrec = [ora.tiles_to_records(s["vc"][0, h, :n // 64].cpu().numpy(), s["rv"]) for h in range(H)]
    ka = [s["ka"][0, h, :n].cpu().numpy().view(np.float16) for h in range(H)]
    va = [s["va"][0, h, :n].cpu().numpy().view(np.float16) for h in range(H)]
    q32 = w.as_f32(w.queries(0))

    def timed(seconds):
        reps, t_total = 0, 0.0
        while t_total < seconds and reps < 200:
            t0 = time.perf_counter()
            ora.decode_attention(q32, ck, cv, krec, ka, vrec, va, n)
            t_total += time.perf_counter() - t0
            reps += 1
        return reps, t_total / reps

    nbytes = H * n * (s["rk"] + s["rv"] + 4)
    reps, per = timed(target_seconds)
    with threadpool_limits(limits=1):
        reps1, per1 = timed(single_thread_seconds)
    return {"value": nbytes / per / 1e9, "unit": "GB/s", "cores": int(threads), "kind": "oracle",
            "sample": f"oracle decode attention of 32 query heads over the first {n} of the "
                      f"32768 cached tokens (8 KV heads), {reps} runs, {per:.2f} s each; "
                      f"GB/s over the same packed-cache bytes as the GPU metric",
            "single_thread": {"value": nbytes / per1 / 1e9, "unit": "GB/s", "cores": 1,
                              "sample": f"the same sample, {reps1} runs, {per1:.2f} s each"}}


COUNTERS_SUMMARY = os.path.join(ROOT, "profiles", "decode_mfma_llama31_8b_b1_32k_counters.md")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2608_14191_amd", "csrc", f)
                  for f in ("decode.hip", "params.h", "launch.h", "encode_core.h", "abi.cpp",
                            "workspace.h", "exact_dot.h")]


def kernel_source_hash() -> str:
    """sha256 over the decode kernel's sources (identifies the kernel a counter run saw)."""
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def counted_traffic():
    """HBM bytes per decode launch from the committed rocprofv3 --pmc summary, or None if
    there is none or it was taken on other kernel sources."""
    try:
        with open(COUNTERS_SUMMARY) as f:
            fields = dict(line.split(":", 1) for line in f.read().splitlines()
                          if line.startswith(("traffic_bytes_per_launch:", "source_sha256:")))
    except OSError:
        return None
    if fields.get("source_sha256", "").strip() != kernel_source_hash():
        return None
    return int(fields["traffic_bytes_per_launch"].strip())


def counters_run(s, n_decode=6, copy_mib=256):
    """Eager launches for `rocprofv3 --pmc` (one counter per run): decode steps (append +
    decode, one launch each) over rotating cache copies, then a plain device copy of known
    size that calibrates the counters."""
    import torch
    P, w = s["P"], s["w"]
    H, HQ, B, L, cap = w.n_kv_heads, w.n_q_heads, w.batch, s["L"], s["cap"]
    copies = [(s["kc"], s["ka"], s["vc"], s["va"])]
    for _ in range(3):
        copies.append(tuple(t.clone() for t in copies[0]))
    lens = torch.full((B,), L, dtype=torch.int32, device="cuda")
    out = torch.zeros((B, HQ, 128), dtype=torch.float32, device="cuda")
    ws = torch.zeros(P.aatc_decode_workspace_bytes(B, HQ, H, cap), dtype=torch.uint8,
                     device="cuda")
    xk = s["last_tok"][0].reshape(1, H, 128).expand(B, H, 128).contiguous()
    xv = s["last_tok"][1].reshape(1, H, 128).expand(B, H, 128).contiguous()
    for i in range(n_decode):
        kc, ka, vc, va = copies[i % len(copies)]
        P.aatc_append_decode_attention(s["pk"], s["pv"], B, HQ, H, s["q"], xk, xv, kc, ka, vc,
                                       va, lens, cap, s["rk"], s["rv"], 128 ** -0.5, out, ws)
    torch.cuda.synchronize()
    src = torch.ones(copy_mib << 20, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    _log(f"[counters] {n_decode} decodes, 3 copies of {copy_mib} MiB; decode algorithmic "
         f"bytes {decode_bytes(s)}; kernel sources sha256 {kernel_source_hash()}")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-encode", action="store_true")
    ap.add_argument("--no-other-decode", action="store_true",
                    help="skip the Qwen-shape and long-context decode entries")
    ap.add_argument("--counters", action="store_true",
                    help="eager decodes plus a calibration copy, for rocprofv3 --pmc runs")
    ap.add_argument("--encode-only", action="store_true",
                    help="only the prefill encode entries (for rocprofv3 runs of the encode)")
    ap.add_argument("--no-groups", action="store_true",
                    help="skip the head-group decode entry")
    ap.add_argument("--groups-only", action="store_true",
                    help="only the head-group entry (for rocprofv3 runs of the group kernels)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the decode path shards by KV head with no communication; see DESIGN.md)",
              file=sys.stderr)
        sys.exit(2)
    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.encode_only:
        enc = [run_encode_bench(avg) for avg in (2.75, 4.0)]
        print(json.dumps({"encode": [encode_entry(r) for r in enc]}), flush=True)
        return
    if args.groups_only:
        print(json.dumps({"groups": [run_group_decode_bench(setup_group_decode())]}), flush=True)
        return
    s = setup_decode(2)
    if args.counters:
        counters_run(s)
        return
    nbytes = decode_bytes(s)
    elapsed, kern_ms, n_copies, _ = run_decode_bench(s, args.steps, args.warmup)
    ms_per_step = elapsed / args.steps * 1e3
    value = nbytes / (elapsed / args.steps) / 1e9
    achieved = nbytes / (kern_ms * 1e-3) / 1e9
    _log(f"[decode] {ms_per_step * 1e3:.1f} us/step, kernel {kern_ms * 1e3:.1f} us, "
         f"{value:.0f} GB/s step, {achieved:.0f} GB/s kernel ({n_copies} cache copies)")
    enc = []
    if not args.no_encode:
        for avg in (2.75, 4.0):
            r = run_encode_bench(avg)
            enc.append(r)
            _log(f"[encode] {avg} bits: {r['seconds'] * 1e3:.2f} ms, {r['tokens_per_s']:.3e} tok/s, "
                 f"{r['bytes'] / r['seconds'] / 1e9:.0f} GB/s")
    other = []
    if not args.no_other_decode:
        names = {3: "qwen25_7b_decode_b8_16k: batch 8, 28 q / 4 kv heads, 16384 tokens, 2.75 bits",
                 5: "llama31_8b_decode_b4_128k: batch 4, 32 q / 8 kv heads, 131072 tokens, "
                    "2.0 bits, query-weighted keys"}
        for cfg in (3, 5):
            so = setup_decode_random_codes(cfg)
            nb = decode_bytes(so)
            el, km, nc, _ = run_decode_bench(so, 40, 5)
            other.append({"workload": names[cfg], "bytes_per_step": nb,
                          "us_per_step": round(el / 40 * 1e6, 2),
                          "kernel_us": round(km * 1e3, 2),
                          "kernel_GBps": round(nb / (km * 1e-3) / 1e9, 1),
                          "frac": round(nb / (km * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                          "cache_copies": nc, "data": "random code bits, real calibrations"})
            _log(f"[decode cfg {cfg}] kernel {km * 1e3:.1f} us, {nb / (km * 1e-3) / 1e9:.0f} GB/s")
            del so
            torch.cuda.empty_cache()
    groups = []
    if not args.no_groups:
        sg = setup_group_decode()
        groups.append(run_group_decode_bench(sg))
        _log(f"[groups] {groups[-1]['kernel_us_per_step']} us/step, {groups[-1]['GBps']} GB/s")
        del sg
        torch.cuda.empty_cache()
    line = {
        "metric": "decode-attention HBM GB/s (% of peak) on packed KV; encode tokens/sec",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int-codes/f32",
        "data": "synthetic",
        "config": {"workload": "llama31_8b_decode_b1_32k: 1 layer, batch 1, 32 q heads, 8 kv "
                               "heads, head_dim 128, 32768 cached tokens, 2.75 avg bits, bf16 "
                               "q/k/v; step = append 1 token + decode attention",
                   "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
                   "bytes_per_step": nbytes, "cache_copies": n_copies},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": counted_traffic()},
        "encode": [encode_entry(r) for r in enc],
        "decode_other": other,
        "groups": groups,
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(s)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
