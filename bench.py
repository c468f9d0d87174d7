"""Benchmark of the revisit-consistency hot path on one MI355X.

One step = one query chunk through the whole path, all on the device:
pose retrieval over the history bank -> reprojection of the chunk's query
tokens into the retrieved frames -> biased chunk attention, on the
Wan-1.3B history-bank workload (12 heads, D 128, bf16, Lq 4680, Lk 37440,
top-4 retrieval from 200 chunks, reprojection into 12 frames). Inputs are
resident in HBM before the timed region.

Prints one JSON line. ``value`` is the algorithmic attention throughput of
the whole step (4 Lq Lk D H flops per step / step time). ``roofline``
describes the dominant kernel (biased attention) from HIP events recorded on
its launch stream, with the socket power and GFX clock amd-smi reports while
that kernel runs back to back (the chip runs it at its power limit, below
the 2.4 GHz clock the published peaks assume); ``stages`` adds per-stage times, the reprojection
throughput of a batched launch (1024 independent problems, > 2x the 256 MB
last-level cache), retrieval latency, the retrieval bandwidth on a stress
bank, and the cache packing of the step's retrieved chunks for all 30
layers from a store of every bank chunk's keys and values (HBM-bound, not
part of the step), and the streaming driver's per-chunk time for the paper's
cache layout over all 30 layers; ``configs`` times every workload
configuration at its own shape (C1 tiny fp32 reference, C2 plain window with
the bias off, C3 loop closure, C4 the headline's history bank, C5 Wan-14B
720p): attention with the bias on and off, fp8 logits with their deviation
from the bf16 output, and the configuration's correspondence and retrieval,
each next to the fp64 oracle timed on a sample; ``cpu_baseline`` times the
fp64 oracle on a bounded sample of the headline workload on this host.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
"""

from __future__ import annotations

import argparse
import json
import math
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "biased-attention TFLOP/s + MFMA util; reprojection tokens/s (Wan-1.3B shape)"
BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
PEAK_CLOCK_MHZ = 2400.0  # the clock the published peaks are quoted at
FP32_PEAK_TFLOPS = 157.3  # MI355X fp32 (the fp32 attention kernel runs on the fp32 matrix cores)
FP8_BF16_PEAK_TFLOPS = 2.0 / (1.0 / 5000.0 + 1.0 / 2500.0)  # half the flops at the fp8 peak, half at bf16
BENCH_QUERY = 1  # query chunk n = 225: a full top-4 retrieval
PACK_LAYERS = 30  # transformer blocks of the 1.3B backbone: one packing call covers all of them
ROPE_T_PAIRS, ROPE_THETA = 22, 10000.0  # temporal band of the factorised 3-D RoPE at head dim 128
STREAM_CHUNKS, STREAM_CAPACITY, STREAM_TIMED_FROM = 14, 16, 9  # chunks 9..13 retrieve the first lap
REPROJ_BATCH = 1024
PREWARM_S = 0.5  # untimed steps before the warm-up steps, so that the timed steps see the sustained clock


def profiled_counters():
    """HBM traffic of the attention / reprojection / packing kernels as last measured with
    rocprofv3 (profiles/counters.json), valid only while the kernel sources are
    unchanged since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "counters.json")
    if not os.path.exists(path):
        return {}
    with open(path) as f:
        c = json.load(f)
    src = os.path.join(ROOT, "paper_2607_21848_amd", "csrc")
    out = {}
    for key, fname in (("attention", "attention.hip"), ("reproject", "reproject.hip"), ("rotation", "reproject.hip"),
                       ("kvpack", "kvpack.hip")):
        with open(os.path.join(src, fname), "rb") as f:
            sha = hashlib.sha256(f.read()).hexdigest()[:16]
        if c.get(f"{key}_sha") == sha:
            out[key] = c[f"{key}_traffic_bytes"]
    if "attention" in out:
        for key in ("mfma_busy_fraction", "valu_busy_fraction"):
            if key in c:
                out[key] = c[key]
    return out


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def host_info():
    cpu = platform.processor() or ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return cpu


def blas_threads():
    for var in ("OPENBLAS_NUM_THREADS", "OMP_NUM_THREADS"):
        if os.environ.get(var):
            try:
                return min(int(os.environ[var]), len(os.sched_getaffinity(0)))
            except ValueError:
                pass
    return len(os.sched_getaffinity(0))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target oracle time for the CPU baseline")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run a plain device-to-device copy of this many MiB (5 times), the reference "
                         "kernel for scaling HBM byte counters")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the sweep over the five workload configurations (for profiler passes, which "
                         "need only the headline stages)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: the benchmark runs on one GPU only (asked for --gpus {args.gpus}); the path would "
              "shard per head and per query token across GPUs, but no multi-GPU path is implemented", flush=True)
        sys.exit(2)

    import torch

    import paper_2607_21848_amd as rv
    import workloads as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", flush=True)
        sys.exit(1)
    rv.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    def t(a):
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    def tb(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)

    log("generating the Wan-1.3B history-bank workload")
    wl = W.make_c4("bf16")
    r = wl.retrieval
    qs = slice(BENCH_QUERY, BENCH_QUERY + 1)
    # device-resident inputs
    bank_c2w, bank_fd, bank_fc, bank_fk = t(r.bank_c2w), t(r.bank_frame_depth), t(r.bank_frame_c2w), t(r.bank_frame_K)
    q_c2w, q_chunk = t(r.query_c2w[qs]), t(r.query_chunk[qs])
    tgt_d, tgt_c, tgt_k = t(r.query_frame_depth[qs]), t(r.query_frame_c2w[qs]), t(r.query_frame_K[qs])
    q, k, v = tb(wl.q), tb(wl.k), tb(wl.v)
    slot = t(wl.slot)
    # preallocated outputs: the timed loop allocates nothing
    ridx = torch.empty((1, r.k), dtype=torch.int32, device=dev)
    rscore = torch.empty((1, r.k), dtype=torch.float32, device=dev)
    rcount = torch.empty((1,), dtype=torch.int32, device=dev)
    rsel = torch.empty((1, r.k * 3), dtype=torch.int32, device=dev)
    cuv = torch.empty((1, wl.S, wl.Lq, 2), dtype=torch.float32, device=dev)
    cidx = torch.empty((1, wl.S, wl.Lq), dtype=torch.int32, device=dev)
    o = torch.empty_like(q)
    lse = torch.empty((wl.H, wl.Lq), dtype=torch.float32, device=dev)
    # the attention's key-split workspace (the library allocates nothing)
    ws = torch.empty(max(rv.attention_workspace_size(torch.bfloat16, wl.Lq, wl.Lk, wl.H, wl.D),
                         rv.attention_workspace_size(torch.float8_e4m3fn, wl.Lq, wl.Lk, wl.H, wl.D), 16),
                     dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        rv.retrieve_chunks(bank_c2w, q_c2w, q_chunk, E=r.E, w_v=r.w_v, tau_c=r.tau_c, tau_v=r.tau_v, delta=r.delta,
                           first_candidate=r.first_candidate, k=r.k, frames_per_chunk=3,
                           out=(ridx, rscore, rcount, rsel))
        if ev is not None:
            ev[1].record(stream)
        rv.reproject_correspondence(tgt_d, tgt_c, tgt_k, bank_fd, bank_fc, bank_fk, p=wl.p, eps=wl.eps,
                                    src_sel=rsel, out=(cuv, cidx))
        if ev is not None:
            ev[2].record(stream)
        rv.biased_chunk_attention(q, k, v, slot, cuv[0], cidx[0], h=wl.h, w=wl.w, softmax_scale=wl.softmax_scale,
                                  lam=wl.lam, sigma=wl.sigma, out=(o, lse), workspace=ws)
        if ev is not None:
            ev[3].record(stream)

    # bring the GPU to its sustained clock first (the host-side set-up above leaves it idle), untimed
    t_warm = time.perf_counter()
    while time.perf_counter() - t_warm < PREWARM_S:
        for _ in range(20):
            step()
        torch.cuda.synchronize()
    log(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"timing {args.steps} steps")
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = 1e3 * wall / args.steps
    st_ms = np.array([[e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2]), e[2].elapsed_time(e[3])] for e in evs])
    retr_ms, repr_ms, attn_ms = st_ms.mean(axis=0)
    flops = wl.flops
    attn_tflops = flops / (attn_ms * 1e-3) / 1e12
    value = flops / (ms_step * 1e-3) / 1e12
    log(f"step {ms_step:.3f} ms; retrieval {retr_ms * 1e3:.1f} us, reprojection {repr_ms * 1e3:.1f} us, "
        f"attention {attn_ms:.3f} ms = {attn_tflops:.1f} TFLOP/s")

    # sanity: the step produced a full retrieval and finite outputs
    assert int(rcount.item()) == r.k and torch.isfinite(o.float()).all()

    # the chip's power and clock while the headline attention runs back to back
    power = _power_state(lambda: rv.biased_chunk_attention(
        q, k, v, slot, cuv[0], cidx[0], h=wl.h, w=wl.w, softmax_scale=wl.softmax_scale, lam=wl.lam,
        sigma=wl.sigma, out=(o, lse), workspace=ws))
    if power is not None:
        log(f"sustained attention: socket power {power['socket_power_w']:.0f} W, "
            f"GFX clock {power['gfx_clock_mhz']:.0f} MHz, hotspot {power.get('hotspot_c', float('nan')):.0f} C "
            f"({power['samples']} samples)")

    # fp8 logits: the same chunk with q and k in fp8 e4m3 (v, o bf16). Half the flops (Q K^T) run on the
    # fp8 matrix cores, half (P V) on bf16 ones: the time-weighted peak is 2 / (1/5000 + 1/2500) TFLOP/s
    q8, k8 = q.float().to(torch.float8_e4m3fn), k.float().to(torch.float8_e4m3fn)
    o8 = torch.empty_like(o)
    lse8 = torch.empty_like(lse)

    def attn8():
        rv.biased_chunk_attention(q8, k8, v, slot, cuv[0], cidx[0], h=wl.h, w=wl.w, softmax_scale=wl.softmax_scale,
                                  lam=wl.lam, sigma=wl.sigma, out=(o8, lse8), workspace=ws)
    # median rounds after a sustained warm-up, as every stage below: a burst right
    # after the headline steps catches the clock moving to the new load
    a8_ms = _timed_rounds({"fp8": attn8}, args.steps, stream)["fp8"]
    a8_tflops = flops / (a8_ms * 1e-3) / 1e12
    a8_dev = float((o8.float() - o.float()).abs().max().item())
    log(f"attention with fp8 logits {a8_ms:.3f} ms = {a8_tflops:.1f} TFLOP/s; max |O_fp8 - O_bf16| = {a8_dev:.2e}")
    del q8, k8, o8, lse8

    # reprojection throughput: one launch over REPROJ_BATCH independent C3-shaped problems
    log(f"batched reprojection: {REPROJ_BATCH} problems")
    arrs = W.make_reproj_batch(REPROJ_BATCH)
    bt = [t(a) for a in arrs]
    B, Tq, Hd, Wd = arrs[0].shape
    S = arrs[3].shape[1]
    p = 2
    Lq_r = Tq * (Hd // p) * (Wd // p)
    buv = torch.empty((B, S, Lq_r, 2), dtype=torch.float32, device=dev)
    bidx = torch.empty((B, S, Lq_r), dtype=torch.int32, device=dev)
    reps = 20
    rb_ms = _timed_rounds({"general": lambda: rv.reproject_correspondence(*bt, p=p, eps=0.05, out=(buv, bidx))},
                          reps, stream)["general"]
    tokens = B * Lq_r
    # algorithmic bytes per query token: p^2 depth pixels in, S (u^ pair + code) out, and the
    # problem's S source depth maps shared by its Lq_r tokens
    bytes_per_token = p * p * 4 + S * 12 + S * Hd * Wd * 4 / Lq_r
    rb_gbs = tokens * bytes_per_token / (rb_ms * 1e-3) / 1e9
    log(f"batched reprojection {rb_ms:.3f} ms: {tokens / (rb_ms * 1e-3):.3e} tokens/s, {rb_gbs:.0f} GB/s algorithmic")
    # the same problems on token depth pooled once per stored frame (p = 1, intrinsics / p): 4 B of target depth
    # per token instead of 16, and a quarter of the source depth
    pt = rv.pool_token_depth(bt[0].reshape(-1, Hd, Wd), p).reshape(B, Tq, Hd // p, Wd // p)
    ps = rv.pool_token_depth(bt[3].reshape(-1, Hd, Wd), p).reshape(B, S, Hd // p, Wd // p)
    kt, ks = (bt[2].double() / p).float(), (bt[5].double() / p).float()
    pargs_r = (pt, bt[1], kt, ps, bt[4], ks)
    rp_ms = _timed_rounds({"pooled": lambda: rv.reproject_correspondence(*pargs_r, p=1, eps=0.05, out=(buv, bidx))},
                          reps, stream)["pooled"]
    pooled_bytes_per_token = 4 + S * 12 + S * (Hd // p) * (Wd // p) * 4 / Lq_r
    rp_gbs = tokens * pooled_bytes_per_token / (rp_ms * 1e-3) / 1e9
    log(f"batched reprojection on pooled maps {rp_ms:.3f} ms: {tokens / (rp_ms * 1e-3):.3e} tokens/s, "
        f"{rp_gbs:.0f} GB/s algorithmic")
    # rotation-only path: REPROJ_BATCH shared-centre problems (panorama-clip shape), no depth read; the
    # algorithmic bytes are the S (u^ pair + code) written per token
    rarrs = [t(a) for a in W.make_rotation_batch(REPROJ_BATCH)]
    rr_ms = _timed_rounds({"rotation": lambda: rv.reproject_rotation(*rarrs, h=Hd // p, w=Wd // p, p=p, out=(buv, bidx))},
                          reps, stream)["rotation"]
    rot_bytes_per_token = S * 12
    rr_gbs = tokens * rot_bytes_per_token / (rr_ms * 1e-3) / 1e9
    log(f"batched rotation-only correspondence {rr_ms:.3f} ms: {tokens / (rr_ms * 1e-3):.3e} tokens/s, "
        f"{rr_gbs:.0f} GB/s algorithmic")
    # single-call latency at the exact C3 shape (one problem: 3 query frames x 6 sources): median of 50
    # per-call event pairs after 10 warm-up calls
    one = [x[:1] for x in bt]
    for _ in range(10):
        rv.reproject_correspondence(*one, p=p, eps=0.05, out=(buv[:1], bidx[:1]))
    evs1 = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(50)]
    torch.cuda.synchronize()
    for ea, eb in evs1:
        ea.record(stream)
        rv.reproject_correspondence(*one, p=p, eps=0.05, out=(buv[:1], bidx[:1]))
        eb.record(stream)
    torch.cuda.synchronize()
    r1_us = float(np.median([ea.elapsed_time(eb) for ea, eb in evs1])) * 1e3
    log(f"reprojection single call at the C3 shape: {r1_us:.1f} us (median of 50)")
    del bt, buv, bidx, pt, ps, pargs_r, one, rarrs

    # retrieval bandwidth on a stress bank far larger than the configs' (2^23 poses = 512 MiB)
    from workloads.synth import ring_bank
    n_stress = 1 << 23
    log(f"retrieval stress bank: {n_stress} poses")
    srng = np.random.default_rng(23)
    sbank = torch.from_numpy(ring_bank(srng, n_stress, radius=20.0)).to(dev)
    squery = torch.from_numpy(ring_bank(srng, 1, radius=20.0)).to(dev)
    schunk = torch.tensor([n_stress + 5], dtype=torch.int32, device=dev)
    sargs = dict(E=40.0, w_v=0.5, tau_c=0.05, tau_v=float(np.pi / 4), delta=3, first_candidate=1, k=4)
    sws = torch.empty(max(rv.retrieve_workspace_size(n_stress, 1, sargs["k"]), 16), dtype=torch.uint8, device=dev)
    sout = rv.retrieve_chunks(sbank, squery, schunk, **sargs, workspace=sws)
    rs_ms = _timed_rounds({"stress": lambda: rv.retrieve_chunks(sbank, squery, schunk, **sargs, out=(*sout[:3], None),
                                                                 workspace=sws)}, reps, stream)["stress"]
    rs_gbs = n_stress * 64 / (rs_ms * 1e-3) / 1e9
    log(f"retrieval stress {rs_ms * 1e3:.1f} us: {rs_gbs:.0f} GB/s algorithmic (64 B per pose)")
    del sbank, squery, schunk, sout

    # cache packing: the query chunk's retrieved chunks (out_idx of the timed retrieval, on the device)
    # gathered from a history store holding every bank chunk's keys and values for every layer, keys
    # re-rotated to the packed frame positions 3..14 (after the anchor, ending where the recent window begins)
    F_pack, T_pack = 3, 3 * wl.h * wl.w
    pack_layer_bytes = 2 * (int(r.bank_c2w.shape[0]) * T_pack + wl.Lk) * wl.H * wl.D * 2
    free_b = torch.cuda.mem_get_info(dev)[0]
    pack_layers = int(max(1, min(PACK_LAYERS, (free_b - (24 << 30)) // pack_layer_bytes)))
    log(f"cache packing: {pack_layers} layers x {r.k} chunks from a {int(r.bank_c2w.shape[0])}-chunk store "
        f"({pack_layers * pack_layer_bytes / 1e9:.1f} GB allocated)")
    n_bank = int(r.bank_c2w.shape[0])
    store_k = torch.empty((pack_layers, n_bank, T_pack, wl.H, wl.D), dtype=torch.bfloat16, device=dev)
    store_v = torch.empty_like(store_k)
    cache_k = torch.zeros((pack_layers, wl.Lk, wl.H, wl.D), dtype=torch.bfloat16, device=dev)
    cache_v = torch.zeros_like(cache_k)
    gen = torch.Generator(device=dev)
    gen.manual_seed(31)
    psel = ridx[0]
    for j in psel.tolist():  # only the selected chunks are ever read
        store_k[:, j].normal_(generator=gen)
        store_v[:, j].normal_(generator=gen)
    pargs = dict(F=F_pack, h=wl.h, w=wl.w, dst_pos=F_pack, dst_row0=T_pack, rope_t_pairs=ROPE_T_PAIRS,
                 rope_theta=ROPE_THETA)
    pk_ms = _timed_rounds({"pack": lambda: rv.pack_retrieved_kv(store_k, store_v, psel, cache_k, cache_v, **pargs)},
                          reps, stream, rounds=3)["pack"]
    pk_bytes = 2 * pack_layers * r.k * 2 * T_pack * wl.H * wl.D * 2  # K and V, read once and written once
    pk_gbs = pk_bytes / (pk_ms * 1e-3) / 1e9
    log(f"cache packing {pk_ms:.3f} ms: {pk_gbs:.0f} GB/s algorithmic")
    del store_k, store_v, cache_k, cache_v

    torch.cuda.empty_cache()  # hand the packing store back before the stream allocates its ring

    # streaming driver: the paper's cache layout (anchor, 1 retrieved, 2 recent, current) chunk by chunk,
    # all 30 layers, on a 14-chunk loop whose second lap revisits the first; per-chunk device time
    from workloads.stream import make_stream
    log("streaming driver: 14 chunks, 30 layers, history ring of 16 chunks")
    sst = make_stream(n_chunks=STREAM_CHUNKS, h=wl.h, w=wl.w, p=wl.p, H=wl.H, D=wl.D, L=PACK_LAYERS, qkv=False)
    Ts = sst.F * sst.h * sst.w
    drv = rv.StreamDriver(F=sst.F, h=sst.h, w=sst.w, p=sst.p, H=sst.H, D=sst.D, layers=sst.L, dtype=torch.bfloat16,
                          capacity=STREAM_CAPACITY, max_chunks=64, E=sst.E, w_v=sst.w_v, tau_c=sst.tau_c,
                          tau_v=sst.tau_v, delta=sst.delta, eps=sst.eps, lam=sst.lam, sigma=sst.sigma,
                          softmax_scale=sst.softmax_scale, rope_t_pairs=ROPE_T_PAIRS, rope_theta=ROPE_THETA)
    gen.manual_seed(47)
    sq, sk, sv = (torch.randn((sst.L, Ts, sst.H, sst.D), generator=gen, device=dev).to(torch.bfloat16)
                  for _ in range(3))
    so = torch.empty_like(sq)
    slse = torch.empty((sst.L, sst.H, Ts), dtype=torch.float32, device=dev)
    s_in = [(t(c.depth), t(c.c2w), t(c.K)) for c in sst.chunks]
    s_ms, s_lk = [], []
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for n, (d_, c_, k_) in enumerate(s_in):
        e0.record(stream)
        drv.step(d_, c_, k_, sq, sk, sv, out=(so, slse))
        e1.record(stream)
        torch.cuda.synchronize()
        stt = drv.state()
        if n >= STREAM_TIMED_FROM:
            s_ms.append(e0.elapsed_time(e1))
            s_lk.append(stt.Lk)
    drv.close()
    stream_ms = float(np.median(s_ms))
    stream_flops = 4.0 * Ts * float(np.median(s_lk)) * sst.D * sst.H * sst.L
    log(f"streaming driver: {stream_ms:.2f} ms per chunk (median of chunks {STREAM_TIMED_FROM}..{STREAM_CHUNKS - 1}), "
        f"Lk {int(np.median(s_lk))}, attention {stream_flops / (stream_ms * 1e-3) / 1e12:.1f} TFLOP/s over the chunk")
    del sq, sk, sv, so, slse, s_in

    configs = None
    if not args.no_configs:
        log("sweep over the five workload configurations")
        configs = config_sweep(dev, stream, ws, q, k, v, slot, cuv, cidx, o, lse, wl, attn_ms, a8_ms, a8_dev,
                               retr_ms, repr_ms, not args.no_cpu_baseline)

    counters = profiled_counters()
    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "wan1.3b-history-bank: top-4 retrieval over 200 chunks -> reprojection into 12 frames "
                        "-> biased attention H12 D128 Lq4680 Lk37440 bf16",
            "heads": wl.H, "head_dim": wl.D, "Lq": wl.Lq, "Lk": wl.Lk, "token_grid": [wl.h, wl.w],
            "retrieved_frames": wl.S, "bank_chunks": int(r.bank_c2w.shape[0]), "top_k": r.k,
        },
        "roofline": {
            "bound": "mfma",
            "kernel": "attn_bf16_kernel (+ attn_merge_kernel when the keys are split)",
            "achieved": round(attn_tflops, 2),
            "peak": BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(attn_tflops / BF16_PEAK_TFLOPS, 4),
            "traffic": counters.get("attention"),
            "mfma_busy_profiled": counters.get("mfma_busy_fraction"),
            "valu_busy_profiled": counters.get("valu_busy_fraction"),
            "flops_per_launch": flops,
            "avg_launch_ms": round(attn_ms, 4),
            # the power limit, not the 2.4 GHz peak clock, sets the clock this kernel runs at
            "sustained_power_state": None if power is None else {
                **power, "peak_at_that_clock": round(BF16_PEAK_TFLOPS * power["gfx_clock_mhz"] / PEAK_CLOCK_MHZ, 1),
                "frac_at_that_clock": round(attn_tflops * PEAK_CLOCK_MHZ / (BF16_PEAK_TFLOPS * power["gfx_clock_mhz"]), 4),
            },
        },
        "stages": {
            "retrieval_us": round(retr_ms * 1e3, 2),
            "reprojection_us": round(repr_ms * 1e3, 2),
            "reprojection_tokens_per_s_single_chunk": round(wl.Lq / (repr_ms * 1e-3), 0),
            "reprojection_c3_single_call_us": round(r1_us, 2),
            "attention_ms": round(attn_ms, 4),
            "attention_tflops": round(attn_tflops, 2),
            "reprojection_batched": {
                "problems": B, "tokens": tokens, "ms": round(rb_ms, 4),
                "tokens_per_s": round(tokens / (rb_ms * 1e-3), 0),
                "bytes_per_token": bytes_per_token,
                "achieved_GBs": round(rb_gbs, 1), "peak_GBs": HBM_PEAK_GBS,
                "frac": round(rb_gbs / HBM_PEAK_GBS, 4), "bound": "hbm",
                "traffic": counters.get("reproject"),
            },
            "attention_fp8_logits": {
                "note": "the bench chunk with q, k in fp8 e4m3 (v, o bf16): Q K^T on the fp8 matrix cores",
                "ms": round(a8_ms, 4), "achieved": round(a8_tflops, 2), "unit": "TFLOP/s",
                "peak": FP8_BF16_PEAK_TFLOPS, "frac": round(a8_tflops / FP8_BF16_PEAK_TFLOPS, 4),
                "max_abs_dev_from_bf16_output": a8_dev,
            },
            "reprojection_batched_pooled": {
                "note": "the batched problems on token depth pooled once per stored frame (pool_token_depth), p = 1",
                "ms": round(rp_ms, 4), "tokens_per_s": round(tokens / (rp_ms * 1e-3), 0),
                "bytes_per_token": pooled_bytes_per_token, "achieved_GBs": round(rp_gbs, 1),
                "peak_GBs": HBM_PEAK_GBS, "frac": round(rp_gbs / HBM_PEAK_GBS, 4), "bound": "hbm",
            },
            "reprojection_rotation_batched": {
                "note": "rotation-only correspondence (shared camera centre, homography, no depth) on the same "
                        "number of panorama-clip problems",
                "ms": round(rr_ms, 4), "tokens_per_s": round(tokens / (rr_ms * 1e-3), 0),
                "bytes_per_token": rot_bytes_per_token, "achieved_GBs": round(rr_gbs, 1),
                "peak_GBs": HBM_PEAK_GBS, "frac": round(rr_gbs / HBM_PEAK_GBS, 4), "bound": "hbm",
                "traffic": counters.get("rotation"),
            },
            "kv_pack": {
                "layers": pack_layers, "chunks": r.k, "tokens_per_chunk": T_pack, "store_chunks": n_bank,
                "rope_t_pairs": ROPE_T_PAIRS, "ms": round(pk_ms, 4), "bytes": pk_bytes,
                "achieved_GBs": round(pk_gbs, 1), "peak_GBs": HBM_PEAK_GBS, "frac": round(pk_gbs / HBM_PEAK_GBS, 4),
                "bound": "hbm", "traffic": counters.get("kvpack"),
            },
            "stream": {
                "note": "paper cache layout per chunk: commit, retrieval (k = 1), slot tables, correspondence, "
                        "packing and biased attention for every layer, one rc_stream_step",
                "layers": PACK_LAYERS, "capacity": STREAM_CAPACITY, "chunks_timed": len(s_ms),
                "Lk": int(np.median(s_lk)), "chunk_ms": round(stream_ms, 3),
                "tokens_per_s": round(Ts / (stream_ms * 1e-3), 0),
                "attention_tflops_per_chunk": round(stream_flops / (stream_ms * 1e-3) / 1e12, 2),
            },
            "retrieval_stress": {
                "note": "stress bank outside the configs", "bank_poses": n_stress, "queries": 1, "top_k": 4,
                "us": round(rs_ms * 1e3, 2), "bytes": n_stress * 64, "achieved_GBs": round(rs_gbs, 1),
                "peak_GBs": HBM_PEAK_GBS, "frac": round(rs_gbs / HBM_PEAK_GBS, 4), "bound": "hbm",
            },
        },
    }

    if configs is not None:
        out["configs"] = configs

    if args.copy_calibration_mib:
        n = args.copy_calibration_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        out["copy_calibration_bytes"] = n * 4
        del src, dst

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def _power_state(fn, secs=3.0, settle_s=0.6):
    """Median socket power (W), GFX clock (MHz, mean over the XCDs) and
    hotspot and HBM temperatures (°C) that amd-smi reports while fn runs back
    to back for `secs` seconds, the first `settle_s` of them unsampled; None
    where amd-smi is not available."""
    import re
    import subprocess
    import threading
    import torch
    samples, stop = [], threading.Event()

    def sampler():
        t_start = time.perf_counter()
        while not stop.is_set():
            if time.perf_counter() - t_start < settle_s:
                time.sleep(0.05)
                continue
            try:
                txt = subprocess.run(["amd-smi", "metric", "-p", "-c", "-t", "-g", "0"], capture_output=True,
                                     text=True, timeout=10).stdout
            except (OSError, subprocess.SubprocessError):
                return
            pw = re.search(r"SOCKET_POWER:\s+([0-9.]+)\s*W", txt)
            clk = [float(c) for c in re.findall(r"GFX_\d+:\s+CLK:\s+([0-9.]+)\s*MHz", txt)]
            hot = re.search(r"HOTSPOT:\s+([0-9.]+)", txt)
            mem = re.search(r"\bMEM:\s+([0-9.]+)", txt)
            if pw and clk:
                samples.append((float(pw.group(1)), sum(clk) / len(clk), float(hot.group(1)) if hot else float("nan"),
                                float(mem.group(1)) if mem else float("nan")))
            time.sleep(0.4)

    th = threading.Thread(target=sampler, daemon=True)
    th.start()
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < secs:
        for _ in range(10):
            fn()
        torch.cuda.synchronize()
    stop.set()
    th.join(timeout=15)
    if not samples:
        return None
    med = lambda i: float(np.median([s[i] for s in samples]))
    out = {"socket_power_w": med(0), "gfx_clock_mhz": round(med(1), 1), "samples": len(samples)}
    if not math.isnan(med(2)):
        out["hotspot_c"] = med(2)
    if not math.isnan(med(3)):
        out["hbm_c"] = med(3)
    return out


def _timed(fn, reps, stream):
    """Mean milliseconds per call of fn over `reps` back-to-back calls (after two
    warm-up calls), from HIP events recorded on the launch stream."""
    import torch
    for _ in range(2):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def _timed_rounds(fns, reps, stream, rounds=5, warm_s=0.1):
    """Median over `rounds` rounds of the mean milliseconds per call over `reps`
    back-to-back calls, for each function of the dict `fns`, after `warm_s`
    seconds of untimed calls of each. The functions take turns round by round,
    so that they see the same clock and thermal state. The GPU's clock settles
    to a new load within tens of milliseconds: a short burst right after other
    work (or after idling) measures the transition, not the kernel."""
    import torch
    res = {name: [] for name in fns}
    for fn in fns.values():
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < warm_s:
            for _ in range(5):
                fn()
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    for _ in range(rounds):
        for name, fn in fns.items():
            res[name].append(_timed(fn, reps, stream))
    return {name: float(np.median(v)) for name, v in res.items()}


def _attn_entry(flops, ms_on, ms_off, peak, dtype):
    e = {"dtype": dtype, "flops_per_call": flops, "peak_tflops": peak}
    for tag, ms in (("bias_on", ms_on), ("bias_off", ms_off)):
        if ms is not None:
            e[f"ms_{tag}"] = round(ms, 4)
            e[f"tflops_{tag}"] = round(flops / (ms * 1e-3) / 1e12, 2)
            e[f"frac_{tag}"] = round(flops / (ms * 1e-3) / 1e12 / peak, 4)
    return e


def _oracle_attention_sample(qv, kv, vv, slot, uv, idx, wl, n_rows):
    """Seconds the fp64 oracle takes for n_rows sampled query rows (all heads),
    and the attention flops that covers."""
    from oracle import attention as OA
    rows = np.linspace(0, wl.Lq - 1, n_rows).astype(np.int64)
    t0 = time.perf_counter()
    OA.biased_attention(qv, kv, vv, slot, uv, idx, wl.h, wl.w, wl.softmax_scale, wl.lam, wl.sigma, rows=rows,
                        block=n_rows)
    dt = time.perf_counter() - t0
    return dt, 4.0 * n_rows * wl.Lk * wl.D * wl.H


def config_sweep(dev, stream, ws, q4, k4, v4, slot4, cuv4, cidx4, o4, lse4, wl4, attn4_ms, a8_4_ms, a8_4_dev,
                 retr4_ms, repr4_ms, with_oracle):
    """Every workload configuration at its own shape: attention with the bias on
    and off (fp32 for the tiny reference, bf16 otherwise, plus fp8 logits where
    the configuration has retrieved frames), and the configuration's
    correspondence and retrieval, each timed with HIP events; where asked, the
    fp64 oracle timed on a sample of the same inputs. Q, K and V of the
    Wan-shaped configurations are drawn N(0, 1) on the device (seeded)."""
    import torch

    import paper_2607_21848_amd as rv
    import workloads as W
    from oracle import reprojection as OR, retrieval as ORT

    def t(a):
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    gen = torch.Generator(device=dev)
    threads = blas_threads()
    res = {}

    def randn_bf16(shape, seed):
        gen.manual_seed(seed)
        return torch.randn(shape, generator=gen, device=dev).to(torch.bfloat16)

    def host64(x):
        return x.float().cpu().numpy()

    def attn_call(wl, q, k, v, slot, uv, idx, lam, o, lse):
        return lambda: rv.biased_chunk_attention(q, k, v, slot, uv, idx, h=wl.h, w=wl.w,
                                                 softmax_scale=wl.softmax_scale, lam=lam, sigma=wl.sigma,
                                                 out=(o, lse), workspace=ws)

    def fp8_entry(wl, q, k, v, slot, uv, idx, o_ref, reps):
        q8, k8 = q.float().to(torch.float8_e4m3fn), k.float().to(torch.float8_e4m3fn)
        o8, l8 = torch.empty_like(o_ref), torch.empty((wl.H, wl.Lq), dtype=torch.float32, device=dev)
        ms = _timed_rounds({"fp8": attn_call(wl, q8, k8, v, slot, uv, idx, wl.lam, o8, l8)}, reps, stream,
                           rounds=4)["fp8"]
        d = (o8.float() - o_ref.float()).abs()
        e = _attn_entry(wl.flops, ms, None, FP8_BF16_PEAK_TFLOPS, "fp8 q, k; bf16 v, o")
        e["max_abs_dev_from_bf16_output"] = float(d.max().item())
        e["mean_abs_dev_from_bf16_output"] = float(d.mean().item())
        return e

    # C1: tiny fp32 reference, full oracle
    wl = W.make_c1()
    log("config C1 (tiny fp32 reference)")
    tgt = [t(a) for a in (wl.tgt_depth, wl.tgt_c2w, wl.tgt_K)]
    src = [t(a) for a in (wl.src_depth, wl.src_c2w, wl.src_K)]
    uv = torch.empty((1, wl.S, wl.Lq, 2), dtype=torch.float32, device=dev)
    idx = torch.empty((1, wl.S, wl.Lq), dtype=torch.int32, device=dev)
    r_ms = _timed(lambda: rv.reproject_correspondence(*tgt, *src, p=wl.p, eps=wl.eps, out=(uv, idx)), 50, stream)
    q, k, v, slot = t(wl.q), t(wl.k), t(wl.v), t(wl.slot)
    o = torch.empty_like(q)
    lse = torch.empty((wl.H, wl.Lq), dtype=torch.float32, device=dev)
    tm = _timed_rounds({"on": attn_call(wl, q, k, v, slot, uv[0], idx[0], wl.lam, o, lse),
                        "off": attn_call(wl, q, k, v, slot, None, None, 0.0, o, lse)}, 50, stream, rounds=3)
    on, off = tm["on"], tm["off"]
    e = {"workload": W.CONFIG_NAMES[1], "attention": _attn_entry(wl.flops, on, off, FP32_PEAK_TFLOPS, "f32"),
         "reprojection": {"us": round(r_ms * 1e3, 2), "tokens": wl.Lq, "sources": wl.S,
                          "tokens_per_s": round(wl.Lq / (r_ms * 1e-3), 0)}}
    if with_oracle:
        from oracle import attention as OA
        t0 = time.perf_counter()
        ouv, oidx = OR.reproject(wl.tgt_depth, wl.tgt_c2w, wl.tgt_K, wl.src_depth, wl.src_c2w, wl.src_K, wl.p, wl.eps)
        t1 = time.perf_counter()
        OA.biased_attention(wl.q, wl.k, wl.v, wl.slot, ouv, oidx, wl.h, wl.w, wl.softmax_scale, wl.lam, wl.sigma)
        t2 = time.perf_counter()
        e["oracle"] = {"kind": "oracle", "cores": threads, "sample": "the whole configuration",
                       "reprojection_s": round(t1 - t0, 4), "attention_s": round(t2 - t1, 4),
                       "attention_tflops": round(wl.flops / (t2 - t1) / 1e12, 6)}
    res["C1"] = e

    # C2: plain window, no retrieved frames (bias off)
    wl = W.make_c2("bf16", qkv=False)
    log("config C2 (Wan-1.3B plain window, bias off)")
    q = randn_bf16((wl.Lq, wl.H, wl.D), 201)
    k = randn_bf16((wl.Lk, wl.H, wl.D), 202)
    v = randn_bf16((wl.Lk, wl.H, wl.D), 203)
    slot = t(wl.slot)
    o = torch.empty_like(q)
    lse = torch.empty((wl.H, wl.Lq), dtype=torch.float32, device=dev)
    off = _timed_rounds({"off": attn_call(wl, q, k, v, slot, None, None, 0.0, o, lse)}, 10, stream, rounds=4)["off"]
    e = {"workload": W.CONFIG_NAMES[2], "attention": _attn_entry(wl.flops, None, off, BF16_PEAK_TFLOPS, "bf16")}
    if with_oracle:
        dt, fl = _oracle_attention_sample(host64(q), host64(k), host64(v), wl.slot, None, None, wl, 8)
        e["oracle"] = {"kind": "oracle", "cores": threads, "sample": "8 query rows, all heads and keys",
                       "attention_s": round(dt, 3), "attention_tflops": round(fl / dt / 1e12, 6)}
    res["C2"] = e
    del q, k, v, o

    # C3: loop closure with fixed retrieved frames
    wl = W.make_c3("bf16", qkv=False)
    log("config C3 (Wan-1.3B loop closure)")
    tgt = [t(a[None]) for a in (wl.tgt_depth, wl.tgt_c2w, wl.tgt_K)]
    src = [t(a[None]) for a in (wl.src_depth, wl.src_c2w, wl.src_K)]
    uv = torch.empty((1, wl.S, wl.Lq, 2), dtype=torch.float32, device=dev)
    idx = torch.empty((1, wl.S, wl.Lq), dtype=torch.int32, device=dev)
    r_ms = _timed(lambda: rv.reproject_correspondence(*tgt, *src, p=wl.p, eps=wl.eps, out=(uv, idx)), 50, stream)
    q = randn_bf16((wl.Lq, wl.H, wl.D), 301)
    k = randn_bf16((wl.Lk, wl.H, wl.D), 302)
    v = randn_bf16((wl.Lk, wl.H, wl.D), 303)
    slot = t(wl.slot)
    o = torch.empty_like(q)
    lse = torch.empty((wl.H, wl.Lq), dtype=torch.float32, device=dev)
    tm = _timed_rounds({"on": attn_call(wl, q, k, v, slot, uv[0], idx[0], wl.lam, o, lse),
                        "off": attn_call(wl, q, k, v, slot, None, None, 0.0, o, lse)}, 10, stream, rounds=4)
    on, off = tm["on"], tm["off"]
    attn_call(wl, q, k, v, slot, uv[0], idx[0], wl.lam, o, lse)()  # o: the bias-on output, the fp8 reference
    in_bounds = float((idx[0] >= 0).float().mean().item())
    e = {"workload": W.CONFIG_NAMES[3], "attention": _attn_entry(wl.flops, on, off, BF16_PEAK_TFLOPS, "bf16"),
         "attention_fp8_logits": fp8_entry(wl, q, k, v, slot, uv[0], idx[0], o, 10),
         "reprojection": {"us": round(r_ms * 1e3, 2), "tokens": wl.Lq, "sources": wl.S,
                          "tokens_per_s": round(wl.Lq / (r_ms * 1e-3), 0), "accepted_fraction": round(in_bounds, 4)}}
    if with_oracle:
        t0 = time.perf_counter()
        ouv, oidx = OR.reproject(wl.tgt_depth, wl.tgt_c2w, wl.tgt_K, wl.src_depth, wl.src_c2w, wl.src_K, wl.p, wl.eps)
        t1 = time.perf_counter()
        dt, fl = _oracle_attention_sample(host64(q), host64(k), host64(v), wl.slot, ouv, oidx, wl, 8)
        e["oracle"] = {"kind": "oracle", "cores": threads, "sample": "reprojection of the chunk; attention for 8 "
                       "query rows, all heads and keys", "reprojection_s": round(t1 - t0, 3),
                       "attention_s": round(dt, 3), "attention_tflops": round(fl / dt / 1e12, 6)}
    res["C3"] = e
    del q, k, v, o

    # C4: the headline step's shape; bias on and off timed here in interleaved rounds
    log("config C4 (Wan-1.3B history bank, the headline step)")
    tm = _timed_rounds({"on": attn_call(wl4, q4, k4, v4, slot4, cuv4[0], cidx4[0], wl4.lam, o4, lse4),
                        "off": attn_call(wl4, q4, k4, v4, slot4, None, None, 0.0, o4, lse4)}, 10, stream, rounds=4)
    e8 = _attn_entry(wl4.flops, a8_4_ms, None, FP8_BF16_PEAK_TFLOPS, "fp8 q, k; bf16 v, o")
    e8["max_abs_dev_from_bf16_output"] = a8_4_dev
    res["C4"] = {"workload": W.CONFIG_NAMES[4],
                 "attention": _attn_entry(wl4.flops, tm["on"], tm["off"], BF16_PEAK_TFLOPS, "bf16"),
                 "attention_in_the_headline_steps_ms": round(attn4_ms, 4),
                 "attention_fp8_logits": e8,
                 "retrieval_us": round(retr4_ms * 1e3, 2), "reprojection_us": round(repr4_ms * 1e3, 2),
                 "note": "fp8, retrieval and reprojection times are the headline step's"}

    # C5: Wan-14B 720p with top-2 retrieval from a 300-chunk bank
    wl = W.make_c5("bf16", qkv=False)
    r = wl.retrieval
    log("config C5 (Wan-14B 720p)")
    bank_c2w, q_c2w, q_chunk = t(r.bank_c2w), t(r.query_c2w[:1]), t(r.query_chunk[:1])
    bank = [t(a) for a in (r.bank_frame_depth, r.bank_frame_c2w, r.bank_frame_K)]
    tgt = [t(a[:1]) for a in (r.query_frame_depth, r.query_frame_c2w, r.query_frame_K)]
    ridx = torch.empty((1, r.k), dtype=torch.int32, device=dev)
    rscore = torch.empty((1, r.k), dtype=torch.float32, device=dev)
    rcount = torch.empty((1,), dtype=torch.int32, device=dev)
    rsel = torch.empty((1, r.k * 3), dtype=torch.int32, device=dev)
    uv = torch.empty((1, wl.S, wl.Lq, 2), dtype=torch.float32, device=dev)
    idx = torch.empty((1, wl.S, wl.Lq), dtype=torch.int32, device=dev)
    rt_ms = _timed(lambda: rv.retrieve_chunks(bank_c2w, q_c2w, q_chunk, E=r.E, w_v=r.w_v, tau_c=r.tau_c,
                                              tau_v=r.tau_v, delta=r.delta, first_candidate=r.first_candidate,
                                              k=r.k, frames_per_chunk=3, out=(ridx, rscore, rcount, rsel)),
                   50, stream)
    r_ms = _timed(lambda: rv.reproject_correspondence(*tgt, *bank, p=wl.p, eps=wl.eps, src_sel=rsel,
                                                      out=(uv, idx)), 50, stream)
    q = randn_bf16((wl.Lq, wl.H, wl.D), 501)
    k = randn_bf16((wl.Lk, wl.H, wl.D), 502)
    v = randn_bf16((wl.Lk, wl.H, wl.D), 503)
    slot = t(wl.slot)
    o = torch.empty_like(q)
    lse = torch.empty((wl.H, wl.Lq), dtype=torch.float32, device=dev)
    ws5 = torch.empty(max(rv.attention_workspace_size(torch.bfloat16, wl.Lq, wl.Lk, wl.H, wl.D),
                          rv.attention_workspace_size(torch.float8_e4m3fn, wl.Lq, wl.Lk, wl.H, wl.D), 16),
                      dtype=torch.uint8, device=dev)

    def attn5(lam, uv_, idx_, qq=q, kk=k, oo=o, ll=lse):
        return lambda: rv.biased_chunk_attention(qq, kk, v, slot, uv_, idx_, h=wl.h, w=wl.w,
                                                 softmax_scale=wl.softmax_scale, lam=lam, sigma=wl.sigma,
                                                 out=(oo, ll), workspace=ws5)
    q8, k8 = q.float().to(torch.float8_e4m3fn), k.float().to(torch.float8_e4m3fn)
    o8, l8 = torch.empty_like(o), torch.empty_like(lse)
    tm = _timed_rounds({"on": attn5(wl.lam, uv[0], idx[0]), "off": attn5(0.0, None, None),
                        "fp8": attn5(wl.lam, uv[0], idx[0], q8, k8, o8, l8)}, 5, stream, rounds=3)
    on, off, on8 = tm["on"], tm["off"], tm["fp8"]
    attn5(wl.lam, uv[0], idx[0])()  # o: the bias-on output (the rounds end on other calls)
    d8 = (o8.float() - o.float()).abs()
    e8 = _attn_entry(wl.flops, on8, None, FP8_BF16_PEAK_TFLOPS, "fp8 q, k; bf16 v, o")
    e8["max_abs_dev_from_bf16_output"] = float(d8.max().item())
    e8["mean_abs_dev_from_bf16_output"] = float(d8.mean().item())
    del q8, k8, o8
    e = {"workload": W.CONFIG_NAMES[5], "attention": _attn_entry(wl.flops, on, off, BF16_PEAK_TFLOPS, "bf16"),
         "attention_fp8_logits": e8, "retrieval_us": round(rt_ms * 1e3, 2),
         "retrieved": ridx[0].tolist(),
         "reprojection": {"us": round(r_ms * 1e3, 2), "tokens": wl.Lq, "sources": wl.S,
                          "tokens_per_s": round(wl.Lq / (r_ms * 1e-3), 0),
                          "accepted_fraction": round(float((idx[0] >= 0).float().mean().item()), 4)}}
    if with_oracle:
        t0 = time.perf_counter()
        oi, _, oc = ORT.retrieve(r.bank_c2w, r.query_c2w[:1], r.query_chunk[:1], r.E, r.w_v, r.tau_c, r.tau_v,
                                 r.delta, r.first_candidate, r.k)
        sel = ORT.frame_selection(oi, oc, 3)[0]
        t1 = time.perf_counter()
        ouv, oidx = OR.reproject(r.query_frame_depth[0], r.query_frame_c2w[0], r.query_frame_K[0],
                                 r.bank_frame_depth, r.bank_frame_c2w, r.bank_frame_K, wl.p, wl.eps, src_sel=sel)
        t2 = time.perf_counter()
        dt, fl = _oracle_attention_sample(host64(q), host64(k), host64(v), wl.slot, ouv, oidx, wl, 4)
        e["oracle"] = {"kind": "oracle", "cores": threads, "sample": "retrieval and reprojection of the chunk; "
                       "attention for 4 query rows, all heads and keys", "retrieval_s": round(t1 - t0, 4),
                       "reprojection_s": round(t2 - t1, 3), "attention_s": round(dt, 3),
                       "attention_tflops": round(fl / dt / 1e12, 6)}
    res["C5"] = e
    del q, k, v, o, ws5
    torch.cuda.empty_cache()
    return res


def cpu_baseline(wl, target_s):
    """The fp64 oracle on this host: retrieval + reprojection of the same
    query chunk, then attention for blocks of 64 query rows (all heads,
    all Lk keys) until about ``target_s`` seconds have passed. Reported in the
    metric's unit: attention flops processed per second."""
    from oracle import attention as OA, reprojection as OR, retrieval as ORT

    r = wl.retrieval
    qs = slice(BENCH_QUERY, BENCH_QUERY + 1)
    log("cpu baseline: oracle retrieval + reprojection")
    t0 = time.perf_counter()
    oi, _, oc = ORT.retrieve(r.bank_c2w, r.query_c2w[qs], r.query_chunk[qs], r.E, r.w_v, r.tau_c, r.tau_v, r.delta,
                             r.first_candidate, r.k)
    sel = ORT.frame_selection(oi, oc, 3)[0]
    t1 = time.perf_counter()
    uv, idx = OR.reproject(r.query_frame_depth[BENCH_QUERY], r.query_frame_c2w[BENCH_QUERY],
                           r.query_frame_K[BENCH_QUERY], r.bank_frame_depth, r.bank_frame_c2w, r.bank_frame_K,
                           wl.p, wl.eps, src_sel=sel)
    t2 = time.perf_counter()
    qv, kv, vv = wl.values("q"), wl.values("k"), wl.values("v")
    rows_done = 0
    block = 64
    t3 = time.perf_counter()
    while rows_done < wl.Lq and time.perf_counter() - t3 < target_s:
        rows = np.arange(rows_done, min(rows_done + block, wl.Lq))
        OA.biased_attention(qv, kv, vv, wl.slot, uv, idx, wl.h, wl.w, wl.softmax_scale, wl.lam, wl.sigma,
                            rows=rows, block=block)
        rows_done += len(rows)
        log(f"cpu baseline: {rows_done} query rows, {time.perf_counter() - t3:.1f} s")
    t4 = time.perf_counter()
    attn_flops = 4.0 * rows_done * wl.Lk * wl.D * wl.H
    attn_s = t4 - t3
    # whole-chunk estimate: attention scaled to all Lq rows plus the measured retrieval + reprojection
    chunk_s = attn_s * wl.Lq / rows_done + (t2 - t0)
    return {
        "value": round(attn_flops / attn_s / 1e12, 6),
        "unit": "TFLOP/s",
        "cores": blas_threads(),
        "kind": "oracle",
        "sample": f"fp64 NumPy oracle on the bench chunk: retrieval ({1e3 * (t1 - t0):.1f} ms) + reprojection "
                  f"({1e3 * (t2 - t1):.1f} ms, 1 core) + biased attention for {rows_done} of {wl.Lq} query rows, "
                  f"all {wl.H} heads and {wl.Lk} keys ({attn_s:.1f} s, BLAS threads); value = attention flops / "
                  f"attention time; whole chunk extrapolates to {chunk_s:.1f} s",
        "host_cpu": host_info(),
        "chunk_seconds_extrapolated": round(chunk_s, 2),
    }


if __name__ == "__main__":
    main()
