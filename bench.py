#!/usr/bin/env python3
"""Benchmark of the RAG-synthesis attention path on one MI355X.

One step = one pass of the hot path over the 7B-class stuff batch
(16 queries, 64 query tokens + U{5..20} chunks of 512 tokens each):
  1. prompt planning (rag_plan_prompts, host),
  2. packed varlen causal prefill of all 16 prompts (rag_attn_prefill_varlen),
  3. 128 decode steps of paged attention (rag_attn_decode_paged), kv_len
     growing by one per step.
Inputs (Q/K/V, paged KV pools, per-step queries and kv lengths) are resident
in HBM before the timed region.  Two KV pools alternate between decode steps
so that a step does not find the previous step's pages in the 256 MB
Infinity Cache.

Printed: one JSON line with the prefill TFLOP/s (value; median over the timed
steps), the decode KV GB/s, roofline objects, extra phases (map_reduce mappers,
70B long stuff, mixed decode + chunked prefill, KV-cache write, int4 GEMMs,
query streams), the clocks (idle, and under a prefill load, with the MFMA
fractions at that shader clock) and the oracle's CPU baseline: for every
workload a bounded sample (measured seconds) and the full work's time
extrapolated from it.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-extra] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "prefill attn TFLOP/s (% MFMA peak); decode attn KV GB/s (% HBM peak)"
PEAK_BF16_TFLOPS = 2516.6     # 256 CU x 4096 FLOP/clk x 2.4 GHz, dense
PEAK_HBM_GBS = 8000.0
WARMUP_REPS = 5               # untimed repetitions before each extra phase
CPU_BUDGET_S = 2.0            # oracle seconds per sampled part of each workload
PROFILES = os.path.join(ROOT, "profiles")


# ---------------------------------------------------------------------------
# algorithmic work (what the method must do; no masked or padded work)
# ---------------------------------------------------------------------------
def prefill_flops(lens_q, lens_k, hq, d):
    pairs = 0
    for nq, nk in zip(lens_q, lens_k):
        pairs += nq * (nk - nq) + nq * (nq + 1) // 2
    return 4.0 * d * hq * pairs


def prefill_bytes(lens_q, lens_k, hq, hkv, d):
    return float(sum(2 * nq * hq * d * 2 + 2 * nk * hkv * d * 2
                     for nq, nk in zip(lens_q, lens_k)))


def decode_bytes(kv_lens, hq, hkv, d, q_rows=None):
    g = hq // hkv
    rows = q_rows or [1] * len(kv_lens)
    return float(sum(n * hkv * d * 2 * 2 + 2 * r * g * hkv * d * 2 + 4 * ((n + 15) // 16) + 4
                     for n, r in zip(kv_lens, rows)))


# The sources of the attention kernels the stored traffic counters measure:
# their translation unit and the headers it includes.
ATTN_SOURCES = ("kernels.hip", "common.h", "prefill_tile.h", "decode_unit.h", "launch.h")


def kernel_source_hash():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2412_10543_amd", "csrc")
    for name in ATTN_SOURCES:
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def decode_kernel_name(num_decode, hkv):
    """The decode kernel a default-policy launch of `num_decode` rows runs:
    balanced units when rows x kv heads leave CUs idle (fewer than 256
    pairs), one workgroup per (row, kv head, split) otherwise."""
    if num_decode * hkv < 256:
        return "paged_decode_balanced_kernel<128, false>"
    return "paged_decode_kernel<128, false>"


def stored_traffic(kernel_key):
    """HBM traffic per launch from the committed counter summary, if it was
    taken on the current kernel sources."""
    path = os.path.join(PROFILES, "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_hash") != kernel_source_hash():
        return None
    k = t.get("kernels", {}).get(kernel_key)
    return None if k is None else k.get("bytes_per_launch")


class Timer:
    """HIP events on the current stream (the stream every call is enqueued on)."""

    def __init__(self, torch):
        self.torch = torch
        self.pairs = {}

    def start(self, name):
        e = self.torch.cuda.Event(enable_timing=True)
        e.record()
        self.pairs.setdefault(name, []).append([e, None])

    def stop(self, name):
        e = self.torch.cuda.Event(enable_timing=True)
        e.record()
        self.pairs[name][-1][1] = e

    def ms(self, name):
        return [a.elapsed_time(b) for a, b in self.pairs.get(name, [])]


def read_clocks():
    """Current and maximum shader clock and memory clock of GPU 0 from
    `amd-smi metric --clock --json` (a child process; read-only).  None-valued
    or an error note when the tool or a field is missing."""
    import signal
    import subprocess
    try:
        # own session: whatever the tool leaves behind is ended with its group
        p = subprocess.Popen(["amd-smi", "metric", "--clock", "--json"], stdout=subprocess.PIPE,
                             stderr=subprocess.DEVNULL, text=True, start_new_session=True)
        try:
            out, _ = p.communicate(timeout=30)
        finally:
            try:
                os.killpg(p.pid, signal.SIGKILL)
            except ProcessLookupError:
                pass
            p.wait()
        d = json.loads(out[out.index("{"):] if "{" in out else "{}")
        gpus = d.get("gpu_data", d) if isinstance(d, dict) else d
        c = gpus[0]["clock"]

        def vals(prefix, field):
            out = []
            for k, v in c.items():
                f = v.get(field) if k.startswith(prefix) and isinstance(v, dict) else None
                if isinstance(f, dict) and isinstance(f.get("value"), (int, float)):
                    out.append(f["value"])
            return max(out) if out else None
        return {"sclk_mhz": vals("gfx", "clk"), "sclk_max_mhz": vals("gfx", "max_clk"),
                "mclk_mhz": vals("mem", "clk")}
    except Exception as e:   # a missing tool must not stop the bench
        return {"error": f"{type(e).__name__}: {str(e)[:60]}"}


class ClockSampler:
    """One clock reading taken `delay` seconds after start(), from a thread,
    while the GPU is busy with the work that follows."""

    def __init__(self, delay=2.0):
        import threading
        self.result = None
        self.thread = threading.Thread(target=self._run, args=(delay,), daemon=True)

    def _run(self, delay):
        time.sleep(delay)
        self.result = read_clocks()

    def start(self):
        self.thread.start()

    def join(self):
        self.thread.join(timeout=60)
        return self.result


def clock_under_load(torch, st, seconds=2.5):
    """Clocks read (from a thread) while the GPU runs the step's prefill back
    to back for `seconds`: the shader clock the MFMA-bound work runs at."""
    sampler = ClockSampler(delay=0.6 * seconds)
    sampler.start()
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(10):
            run_stuff_step(st, None, plan=False, decode=False)
        torch.cuda.synchronize()
    return sampler.join()


# ---------------------------------------------------------------------------
# workload set-up
# ---------------------------------------------------------------------------
def setup_stuff(torch, w, dev, n_pools=2):
    from paper_2412_10543_amd import binding
    from paper_2412_10543_amd.workloads import normal_bf16, paged_pool
    cu, dec = binding.rag_plan_prompts(w.method, w.query_lens, w.num_chunks, w.chunk_len,
                                       w.intermediate_length, w.answer_len)
    lens = [b - a for a, b in zip(cu[:-1], cu[1:])]
    T = cu[-1]
    st = {"w": w, "lens": lens, "cu": cu, "decode_steps": max(dec) if dec else 0}
    st["q"] = normal_bf16((T, w.hq, w.d), w.seed, dev)
    st["k"] = normal_bf16((T, w.hkv, w.d), w.seed + 1, dev)
    st["v"] = normal_bf16((T, w.hkv, w.d), w.seed + 2, dev)
    st["o"] = torch.empty_like(st["q"])
    st["cu_t"] = torch.tensor(cu, dtype=torch.int32, device=dev)
    nsteps = st["decode_steps"]
    S = len(lens)
    if nsteps > 0:
        full = [n + nsteps for n in lens]
        st["pools"] = [paged_pool(full, w.hkv, w.d, w.seed + 100 + i, device=dev)
                       for i in range(n_pools)]
        st["dq"] = normal_bf16((nsteps, S, w.hq, w.d), w.seed + 7, dev)
        st["do"] = torch.empty((S, w.hq, w.d), dtype=torch.bfloat16, device=dev)
        kv = torch.tensor([[n + t + 1 for n in lens] for t in range(nsteps)], dtype=torch.int32,
                          device=dev)
        st["kv_steps"] = kv
        mb = st["pools"][0].block_tables.shape[1]
        n = binding.rag_attn_decode_workspace_size(S, w.hq, w.hkv, w.d, mb)
        st["ws"] = torch.zeros(max(n, 256), dtype=torch.uint8, device=dev)
        st["splits"] = binding.rag_attn_decode_num_splits(S, w.hkv, mb)
    return st


def run_stuff_step(st, timer=None, plan=True, decode=True):
    from paper_2412_10543_amd import binding
    w = st["w"]
    if plan:
        binding.rag_plan_prompts(w.method, w.query_lens, w.num_chunks, w.chunk_len,
                                 w.intermediate_length, w.answer_len)
    L = max(st["lens"])
    if timer:
        timer.start("prefill")
    binding.rag_attn_prefill_varlen(st["q"], st["k"], st["v"], st["o"], None, st["cu_t"],
                                    st["cu_t"], L, L, w.scale, True)
    if timer:
        timer.stop("prefill")
    # The decode launches go back to back between one pair of events: an
    # event pair around every launch would add the events' own cost to each
    # (about 2.5 us of 81).  The average launch duration is the pair's time
    # over the number of launches (inter-launch gaps included).  With a
    # captured graph (capture_decode) the launches are one graph replay, as a
    # serving loop runs its per-token steps.
    if not decode:
        return
    if timer and st["decode_steps"]:
        timer.start("decode")
    if st.get("graph") is not None:
        st["graph"].replay()
    else:
        run_decode_launches(st)
    if timer and st["decode_steps"]:
        timer.stop("decode")


def run_decode_launches(st):
    """The workload's decode steps, one paged-decode launch each; KV pools
    alternate between steps (no step finds the previous one's pages in the
    256 MB Infinity Cache)."""
    from paper_2412_10543_amd import binding
    w = st["w"]
    pools = st.get("pools", [])
    for t in range(st["decode_steps"]):
        pool = pools[t % len(pools)]
        binding.rag_attn_decode_paged(st["dq"][t], pool.k_cache, pool.v_cache, st["do"],
                                      pool.block_tables, st["kv_steps"][t], w.scale,
                                      workspace=st["ws"])


def capture_decode(torch, st):
    """Captures the decode steps (the launches of run_decode_launches) in a
    HIP graph and keeps the eager result of the last step to check every
    replay against (check_decode_replay).  No memset or allocation is
    recorded: the kernels leave the workspace's counters zero themselves."""
    if not st["decode_steps"]:
        return
    run_decode_launches(st)
    torch.cuda.synchronize()
    st["do_eager"] = st["do"].clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            run_decode_launches(st)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    st["graph"] = g
    check_decode_replay(torch, st)


def check_decode_replay(torch, st):
    """The last decode step's output after a replay equals the eager one, bit
    for bit (run after the replay's events, outside the timed pair)."""
    if st.get("graph") is None:
        return
    st["do"].zero_()
    st["graph"].replay()
    torch.cuda.synchronize()
    if not torch.equal(st["do"].view(torch.int16), st["do_eager"].view(torch.int16)):
        raise RuntimeError("decode graph replay differs from the eager launches")


def eager_decode_ms(torch, st, reps=5):
    """Median time of the decode steps launched one by one from the host."""
    ts = []
    for _ in range(reps):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        run_decode_launches(st)
        b.record()
        torch.cuda.synchronize()
        ts.append(a.elapsed_time(b))
    return median(ts)


def stuff_work(st):
    w = st["w"]
    lens = st["lens"]
    fl = prefill_flops(lens, lens, w.hq, w.d)
    pb = prefill_bytes(lens, lens, w.hq, w.hkv, w.d)
    db = [decode_bytes([n + t + 1 for n in lens], w.hq, w.hkv, w.d)
          for t in range(st["decode_steps"])]
    return fl, pb, db


def roofline(bound, achieved, peak, unit, traffic=None, kernel=None):
    r = {"bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
         "frac": round(achieved / peak, 4), "traffic": traffic}
    if kernel:
        r["kernel"] = kernel
    return r


def median(x):
    s = sorted(x)
    if not s:
        return float("nan")
    n = len(s)
    return s[n // 2] if n % 2 else 0.5 * (s[n // 2 - 1] + s[n // 2])


# ---------------------------------------------------------------------------
# extra phases (other workloads; measured, not part of the step)
# ---------------------------------------------------------------------------
def bench_phase_stuff(torch, w, dev, reps, cpu=None):
    """`cpu` (seconds) also samples the oracle on this workload (returned under
    "_cpu", moved to cpu_baseline by the caller)."""
    st = setup_stuff(torch, w, dev)
    fl, pb, db = stuff_work(st)
    for _ in range(WARMUP_REPS):
        run_stuff_step(st, None, plan=False)
    torch.cuda.synchronize()
    eager_ms = eager_decode_ms(torch, st) if st["decode_steps"] else None
    capture_decode(torch, st)
    timer = Timer(torch)
    for _ in range(reps):
        run_stuff_step(st, timer, plan=False)
        check_decode_replay(torch, st)
    torch.cuda.synchronize()
    pf_ms = median(timer.ms("prefill"))
    dec_ms = timer.ms("decode")
    out = {"tokens": st["cu"][-1], "seqs": len(st["lens"]), "hq": w.hq, "hkv": w.hkv, "d": w.d,
           "prefill_ms": round(pf_ms, 4), "prefill_tflops": round(fl / pf_ms / 1e9, 1),
           "prefill_frac_mfma": round(fl / pf_ms / 1e9 / PEAK_BF16_TFLOPS, 4),
           "prefill_hbm_gbs": round(pb / pf_ms / 1e6, 1)}
    if dec_ms:
        per = st["decode_steps"]
        tot = median(dec_ms)
        gbs = sum(db) / tot / 1e6
        out.update({"decode_steps": per, "decode_us_per_step": round(tot / per * 1e3, 2),
                    "decode_gbs": round(gbs, 1), "decode_frac_hbm": round(gbs / PEAK_HBM_GBS, 4),
                    "decode_us_per_step_eager": round(eager_ms / per * 1e3, 2),
                    "decode_splits": st["splits"]})
    if cpu:
        if w.name == "mapred7b":
            out["_cpu"] = cpu_baseline_mapred(torch, st, cpu, seed=w.seed)
        else:
            out["_cpu"] = cpu_baseline_stuff(torch, st, cpu, seed=w.seed)
    del st
    torch.cuda.empty_cache()
    return out


def setup_mixed(torch, dev, n_pools=2):
    """The mixed workload: 256 decode rows followed by 4 chunked-prefill
    pieces, in one paged batch."""
    from paper_2412_10543_amd import binding
    from paper_2412_10543_amd.workloads import mixed, normal_bf16, paged_pool
    w = mixed()
    kv = w.decode_kv_lens + [p + w.piece_len for p in w.piece_prior]
    q_lens = [1] * len(w.decode_kv_lens) + [w.piece_len] * len(w.piece_prior)
    cu = [0]
    for n in q_lens:
        cu.append(cu[-1] + n)
    st = {"w": w, "kv": kv, "q_lens": q_lens, "cu": cu, "nd": len(w.decode_kv_lens)}
    st["pools"] = [paged_pool(kv, w.hkv, w.d, w.seed + i, device=dev) for i in range(n_pools)]
    st["q"] = normal_bf16((cu[-1], w.hq, w.d), w.seed + 9, dev)
    st["o"] = torch.empty_like(st["q"])
    mb = st["pools"][0].block_tables.shape[1]
    n = binding.rag_attn_decode_workspace_size(st["nd"], w.hq, w.hkv, w.d, mb)
    st["ws"] = torch.zeros(max(n, 256), dtype=torch.uint8, device=dev)
    st["cu_t"] = torch.tensor(cu, dtype=torch.int32, device=dev)
    st["kv_t"] = torch.tensor(kv, dtype=torch.int32, device=dev)
    st["splits"] = binding.rag_attn_decode_num_splits(st["nd"], w.hkv, mb)
    return st


def run_mixed(st, pool_index=0):
    from paper_2412_10543_amd import binding
    w = st["w"]
    pool = st["pools"][pool_index]
    binding.rag_attn_decode_paged(st["q"], pool.k_cache, pool.v_cache, st["o"], pool.block_tables,
                                  st["kv_t"], w.scale, cu_seqlens_q=st["cu_t"],
                                  num_decode_seqs=st["nd"], max_seqlen_q=w.piece_len,
                                  workspace=st["ws"])


def bench_phase_mixed(torch, dev, reps, cpu=None):
    st = setup_mixed(torch, dev)
    w = st["w"]
    for i in range(max(WARMUP_REPS, len(st["pools"]))):   # includes first touch of each pool
        run_mixed(st, i % len(st["pools"]))
    torch.cuda.synchronize()
    timer = Timer(torch)
    for r in range(reps):
        timer.start("mixed")
        run_mixed(st, r % 2)
        timer.stop("mixed")
    torch.cuda.synchronize()
    ms = median(timer.ms("mixed"))
    dbytes = decode_bytes(w.decode_kv_lens, w.hq, w.hkv, w.d)
    pl_q = [w.piece_len] * len(w.piece_prior)
    pl_k = [p + w.piece_len for p in w.piece_prior]
    pfl = prefill_flops(pl_q, pl_k, w.hq, w.d)
    pbytes = decode_bytes(pl_k, w.hq, w.hkv, w.d, q_rows=pl_q)
    t_hbm = (dbytes + pbytes) / (PEAK_HBM_GBS * 1e6)
    t_mfma = pfl / (PEAK_BF16_TFLOPS * 1e9)
    out = {"decode_seqs": st["nd"], "pieces": len(w.piece_prior), "piece_len": w.piece_len,
           "ms": round(ms, 4), "kv_gbs": round((dbytes + pbytes) / ms / 1e6, 1),
           "piece_tflops": round(pfl / ms / 1e9, 1),
           "roofline_ms_overlapped": round(max(t_hbm, t_mfma), 4),
           "roofline_ms_serial": round(t_hbm + t_mfma, 4),
           "frac_of_overlapped_roofline": round(max(t_hbm, t_mfma) / ms, 4),
           "splits": st["splits"]}
    if cpu:
        out["_cpu"] = cpu_baseline_mixed(torch, st, cpu, seed=w.seed)
    del st
    torch.cuda.empty_cache()
    return out


def bench_phase_kv_write(torch, dev, reps):
    """Paged KV-cache write of the stuff7b prompt tokens (what a prefill hands
    to decode) and of one decode step (one token per sequence), into a pool of
    randomly permuted pages.  HBM-bound copy: bytes = K and V read once and
    written once, plus the slot mapping.

    `us` is one call timed with HIP events around it, host launch included;
    for the decode step (a few microseconds of GPU work) that is mostly the
    launch path, so `us_gpu` times the same call captured in a HIP graph (10
    per replay, each replay's cache checked bit for bit against the eager
    result) and the rates use `us_gpu`."""
    import numpy as np

    from paper_2412_10543_amd import binding
    from paper_2412_10543_amd.workloads import normal_bf16, stuff7b
    w = stuff7b()
    cu, _ = binding.rag_plan_prompts(w.method, w.query_lens, w.num_chunks, w.chunk_len,
                                     w.intermediate_length, w.answer_len)
    T = cu[-1]
    nblocks = int(math.ceil(T / 16 * 1.25))
    out = {}
    for name, ntok in (("prompt_tokens", T), ("decode_step", len(cu) - 1)):
        rng = np.random.Generator(np.random.PCG64(17))
        slots = torch.tensor(rng.permutation(nblocks * 16)[:ntok].astype(np.int32), device=dev)
        k = normal_bf16((ntok, w.hkv, w.d), 31, dev)
        v = normal_bf16((ntok, w.hkv, w.d), 32, dev)
        kc = torch.empty((nblocks, w.hkv, 16, w.d), dtype=torch.bfloat16, device=dev)
        vc = torch.empty_like(kc)
        for _ in range(WARMUP_REPS):
            binding.rag_kv_cache_write(k, v, kc, vc, slots)
        torch.cuda.synchronize()
        timer = Timer(torch)
        for _ in range(reps):
            timer.start("w")
            binding.rag_kv_cache_write(k, v, kc, vc, slots)
            timer.stop("w")
        torch.cuda.synchronize()
        ms = median(timer.ms("w"))
        ms_gpu = ms
        if ntok < 4096:
            kc.zero_()
            vc.zero_()
            binding.rag_kv_cache_write(k, v, kc, vc, slots)
            torch.cuda.synchronize()
            want_k, want_v = kc.clone(), vc.clone()
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            cg = torch.cuda.CUDAGraph()
            with torch.cuda.stream(side):
                with torch.cuda.graph(cg, stream=side):
                    for _ in range(10):
                        binding.rag_kv_cache_write(k, v, kc, vc, slots)
            torch.cuda.current_stream().wait_stream(side)
            torch.cuda.synchronize()
            gms = []
            for _ in range(5):
                kc.zero_()
                vc.zero_()
                torch.cuda.synchronize()
                timer = Timer(torch)
                timer.start("r")
                cg.replay()
                timer.stop("r")
                torch.cuda.synchronize()
                if not (torch.equal(kc.view(torch.int16), want_k.view(torch.int16))
                        and torch.equal(vc.view(torch.int16), want_v.view(torch.int16))):
                    raise RuntimeError("kv write: graph replay differs from the eager call")
                gms.append(timer.ms("r")[0] / 10)
            ms_gpu = median(gms)
            del cg, want_k, want_v
        nbytes = 2.0 * 2 * ntok * w.hkv * w.d * 2 + 4 * ntok
        gbs = nbytes / ms_gpu / 1e6
        out[name] = {"tokens": ntok, "us": round(ms * 1e3, 2), "us_gpu": round(ms_gpu * 1e3, 2),
                     "gbs": round(gbs, 1), "frac_hbm": round(gbs / PEAK_HBM_GBS, 4)}
        del k, v, kc, vc
    torch.cuda.empty_cache()
    return out


def bench_phase_fused_kv(torch, dev, reps):
    """The KV-cache writes on either side of the hot path, separate and fused:
    prompt prefill then rag_kv_cache_write vs rag_attn_prefill_varlen_kvcache
    (stuff7b and the map_reduce mappers; each sequence's tokens in consecutive
    slots of randomly permuted pages), and a stuff7b decode step as
    rag_kv_cache_write + rag_attn_decode_paged vs rag_attn_decode_paged_append."""
    import numpy as np

    from paper_2412_10543_amd import binding, workloads
    from paper_2412_10543_amd.workloads import normal_bf16, paged_pool
    out = {}

    def timed(fn, name):
        for _ in range(WARMUP_REPS):
            fn()
        torch.cuda.synchronize()
        timer = Timer(torch)
        for _ in range(reps):
            timer.start(name)
            fn()
            timer.stop(name)
        torch.cuda.synchronize()
        return median(timer.ms(name))

    for wname in ("mapred7b", "stuff7b"):
        w = getattr(workloads, wname)()
        cu, dec = binding.rag_plan_prompts(w.method, w.query_lens, w.num_chunks, w.chunk_len,
                                           w.intermediate_length, w.answer_len)
        lens = [b - a for a, b in zip(cu[:-1], cu[1:])]
        T, L = cu[-1], max(lens)
        q = normal_bf16((T, w.hq, w.d), w.seed, dev)
        k = normal_bf16((T, w.hkv, w.d), w.seed + 1, dev)
        v = normal_bf16((T, w.hkv, w.d), w.seed + 2, dev)
        o = torch.empty_like(q)
        cu_t = torch.tensor(cu, dtype=torch.int32, device=dev)
        nblk = [(n + 15) // 16 for n in lens]
        num_blocks = int(sum(nblk) * 1.25) + 1
        perm = np.random.Generator(np.random.PCG64(23)).permutation(num_blocks)
        slots, pos = [], 0
        for n, nb in zip(lens, nblk):
            pages = perm[pos:pos + nb]
            pos += nb
            j = np.arange(n)
            slots.append(pages[j // 16] * 16 + j % 16)
        slots_t = torch.tensor(np.concatenate(slots).astype(np.int32), device=dev)
        kc = torch.empty((num_blocks, w.hkv, 16, w.d), dtype=torch.bfloat16, device=dev)
        vc = torch.empty_like(kc)

        def prefill():
            binding.rag_attn_prefill_varlen(q, k, v, o, None, cu_t, cu_t, L, L, w.scale, True)

        def separate():
            prefill()
            binding.rag_kv_cache_write(k, v, kc, vc, slots_t)

        def fused():
            binding.rag_attn_prefill_varlen_kvcache(q, k, v, o, None, cu_t, L, w.scale, kc, vc,
                                                    slots_t)
        ms = {n: timed(f, n) for n, f in (("prefill", prefill), ("separate", separate),
                                          ("fused", fused))}
        out[f"{wname}_prefill"] = {
            "tokens": T, "prefill_only_ms": round(ms["prefill"], 4),
            "prefill_then_write_ms": round(ms["separate"], 4),
            "fused_ms": round(ms["fused"], 4),
            "write_cost_fused_ms": round(ms["fused"] - ms["prefill"], 4),
            "write_cost_separate_ms": round(ms["separate"] - ms["prefill"], 4)}
        del q, k, v, o, kc, vc
        torch.cuda.empty_cache()

    # decode step 0 of stuff7b with its new token appended
    w = workloads.stuff7b()
    cu, _ = binding.rag_plan_prompts(w.method, w.query_lens, w.num_chunks, w.chunk_len,
                                     w.intermediate_length, w.answer_len)
    lens = [b - a for a, b in zip(cu[:-1], cu[1:])]
    S = len(lens)
    kvl = [n + 1 for n in lens]
    pools = [paged_pool(kvl, w.hkv, w.d, w.seed + 300 + i, device=dev, poison=False)
             for i in range(2)]
    kvl_t = torch.tensor(kvl, dtype=torch.int32, device=dev)
    qd = normal_bf16((S, w.hq, w.d), 61, dev)
    kn = normal_bf16((S, w.hkv, w.d), 62, dev)
    vn = normal_bf16((S, w.hkv, w.d), 63, dev)
    od = torch.empty_like(qd)
    mb = pools[0].block_tables.shape[1]
    nws = binding.rag_attn_decode_workspace_size(S, w.hq, w.hkv, w.d, mb)
    ws = torch.zeros(max(nws, 256), dtype=torch.uint8, device=dev)
    new_slots = []
    for pool in pools:
        tb = pool.block_tables.cpu().numpy()
        new_slots.append(torch.tensor([int(tb[s, (n - 1) // 16]) * 16 + (n - 1) % 16
                                       for s, n in enumerate(kvl)], dtype=torch.int32,
                                      device=dev))
    it = [0]

    def separate_step():
        i = it[0] = it[0] ^ 1
        p = pools[i]
        binding.rag_kv_cache_write(kn, vn, p.k_cache, p.v_cache, new_slots[i])
        binding.rag_attn_decode_paged(qd, p.k_cache, p.v_cache, od, p.block_tables, kvl_t,
                                      w.scale, workspace=ws)

    def append_step():
        i = it[0] = it[0] ^ 1
        p = pools[i]
        binding.rag_attn_decode_paged_append(qd, kn, vn, p.k_cache, p.v_cache, od,
                                             p.block_tables, kvl_t, w.scale, workspace=ws)

    def loop(fn):
        def run():
            for _ in range(16):
                fn()
        return run
    sep = timed(loop(separate_step), "dsep") / 16
    app = timed(loop(append_step), "dapp") / 16
    out["stuff7b_decode_step"] = {"write_then_decode_us": round(sep * 1e3, 2),
                                  "append_us": round(app * 1e3, 2),
                                  "note": "16 launches (pairs) back to back between one event "
                                          "pair, two pools alternating"}
    del pools
    torch.cuda.empty_cache()
    return out


def bench_phase_awq(torch, dev, reps, batches=(16, 8192), graph=True, dense=True):
    """Group-quantized int4-weight GEMMs of the 7B model's linear layers
    (qkv, o, gate_up, down) at a decode batch of 16 rows (HBM-bound: the packed
    weights dominate) and a chunked-prefill batch of 8192 rows (MFMA-bound).
    Algorithmic bytes: x and y in bf16, codes at 4 bits, one bf16 scale and one
    uint8 zero point per group of 128 k; flops 2 M N K.

    `us` is one call timed with HIP events around it, host launch included; at
    16 rows that is mostly the launch path, so `us_gpu` times the same calls
    captured in a HIP graph (10 per replay; every replay's output is checked
    bit for bit against the eager result) and the rates use `us_gpu`.

    For context, `dense_bf16_library_us` times torch's bf16 matmul (the
    vendor GEMM library) of x with a dense bf16 weight of the same shape,
    i.e. the same product without the quantisation (ten back-to-back calls
    between two events); `vs_dense_library` is that time over `us_gpu`."""
    from paper_2412_10543_amd import binding
    from paper_2412_10543_amd.workloads import AWQ_LAYERS_7B, awq_problem
    out = {}
    for name, K, N in AWQ_LAYERS_7B:
        p = awq_problem(max(batches), N, K, seed=K + N, device=dev)
        qw = torch.from_numpy(binding.rag_awq_pack_weights(p.codes)).to(dev)
        sc, z = p.scales.to(dev), torch.from_numpy(p.zeros).to(dev)
        for M in batches:
            x = p.x[:M]
            y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
            ws = torch.zeros(max(binding.rag_awq_workspace_size(M, N, K), 1), dtype=torch.uint8,
                             device=dev)
            for _ in range(WARMUP_REPS):
                binding.rag_awq_gemm(x, qw, sc, z, y, ws)
            torch.cuda.synchronize()
            want = y.clone()
            timer = Timer(torch)
            for _ in range(reps):
                timer.start("g")
                binding.rag_awq_gemm(x, qw, sc, z, y, ws)
                timer.stop("g")
            torch.cuda.synchronize()
            ms = median(timer.ms("g"))
            ms_gpu = ms
            if graph and M <= 64:
                side = torch.cuda.Stream()
                side.wait_stream(torch.cuda.current_stream())
                cg = torch.cuda.CUDAGraph()
                with torch.cuda.stream(side):
                    with torch.cuda.graph(cg, stream=side):
                        for _ in range(10):
                            binding.rag_awq_gemm(x, qw, sc, z, y, ws)
                torch.cuda.current_stream().wait_stream(side)
                torch.cuda.synchronize()
                gms = []
                for _ in range(5):
                    y.zero_()
                    torch.cuda.synchronize()
                    timer = Timer(torch)
                    timer.start("r")
                    cg.replay()
                    timer.stop("r")
                    torch.cuda.synchronize()
                    if not torch.equal(y.view(torch.int16), want.view(torch.int16)):
                        raise RuntimeError(f"awq {name} M={M}: graph replay differs from eager")
                    gms.append(timer.ms("r")[0] / 10)
                ms_gpu = median(gms)
                del cg
            ms_dense = None
            if dense:
                wd = torch.empty((K, N), dtype=torch.bfloat16, device=dev).normal_(0, K ** -0.5)
                for _ in range(WARMUP_REPS):
                    yd = x @ wd
                torch.cuda.synchronize()
                dms = []
                for _ in range(5):
                    timer = Timer(torch)
                    timer.start("d")
                    for _ in range(10):
                        yd = x @ wd
                    timer.stop("d")
                    torch.cuda.synchronize()
                    dms.append(timer.ms("d")[0] / 10)
                ms_dense = median(dms)
                del wd, yd
            nbytes = 2.0 * M * K + K * N / 2 + (K // 128) * N * 3 + 2.0 * M * N
            tflops = 2.0 * M * N * K / ms_gpu / 1e9
            gbs = nbytes / ms_gpu / 1e6
            out[f"{name}_m{M}"] = {"M": M, "N": N, "K": K, "us": round(ms * 1e3, 2),
                                   "us_gpu": round(ms_gpu * 1e3, 2),
                                   "tflops": round(tflops, 1), "gbs": round(gbs, 1),
                                   "frac_mfma": round(tflops / PEAK_BF16_TFLOPS, 4),
                                   "frac_hbm": round(gbs / PEAK_HBM_GBS, 4),
                                   "dense_bf16_library_us":
                                       None if ms_dense is None else round(ms_dense * 1e3, 2),
                                   "vs_dense_library":
                                       None if ms_dense is None else round(ms_dense / ms_gpu, 3)}
            del x, y, ws
        del p, qw, sc, z
    torch.cuda.empty_cache()
    return out


def bench_phase_library_attention(torch, dev, reps=5):
    """For context: torch's own fused attention (scaled_dot_product_attention
    restricted to its flash backend, the framework's library kernel; no other
    backend is allowed to run) on the prompts of stuff7b, mapred7b and
    long70b, causal, bf16.  Prompts of different lengths are one call each;
    equal lengths (the mappers) one batched call.  K and V are expanded to
    the q heads (repeat_interleave) for the call; the FLOP count is the same
    as the prefill phases'.  Not part of the product path."""
    import torch.nn.functional as F
    from torch.nn.attention import SDPBackend, sdpa_kernel

    from paper_2412_10543_amd import binding, workloads
    from paper_2412_10543_amd.workloads import normal_bf16
    out = {}
    for name in ("stuff7b", "mapred7b", "long70b"):
        w = getattr(workloads, name)()
        cu, _ = binding.rag_plan_prompts(w.method, w.query_lens, w.num_chunks, w.chunk_len,
                                         w.intermediate_length, w.answer_len)
        lens = [b - a for a, b in zip(cu[:-1], cu[1:])]
        g = w.hq // w.hkv
        groups = [(len(lens), lens[0])] if len(set(lens)) == 1 else [(1, n) for n in lens]
        calls = []
        for i, (batch, n) in enumerate(groups):
            q = normal_bf16((batch, w.hq, n, w.d), w.seed + 10 * i, dev)
            k = normal_bf16((batch, w.hkv, n, w.d), w.seed + 10 * i + 1, dev)
            v = normal_bf16((batch, w.hkv, n, w.d), w.seed + 10 * i + 2, dev)
            calls.append((q, k.repeat_interleave(g, dim=1).contiguous(),
                          v.repeat_interleave(g, dim=1).contiguous()))
            del k, v

        def run():
            with sdpa_kernel([SDPBackend.FLASH_ATTENTION]):
                for q, k, v in calls:
                    F.scaled_dot_product_attention(q, k, v, is_causal=True)
        try:
            run()
            torch.cuda.synchronize()
        except RuntimeError as e:
            out[name] = {"error": str(e)[:200]}
            continue
        timer = Timer(torch)
        for _ in range(reps):
            timer.start("a")
            run()
            timer.stop("a")
        torch.cuda.synchronize()
        ms = median(timer.ms("a"))
        out[name] = {"ms": round(ms, 4),
                     "tflops": round(prefill_flops(lens, lens, w.hq, w.d) / ms / 1e9, 1),
                     "calls": len(calls)}
        del calls
    torch.cuda.empty_cache()
    return out


def bench_phase_stream(torch, n=32, rate=100.0, budget_gb=16):
    """A synthetic query stream (Poisson arrivals, random profiles) through the
    configuration planner and the kernels: 7B-class shape (Hq 32, Hkv 8, d 128,
    32 layers for the KV budget), 512-token chunks, `budget_gb` GB of KV."""
    from paper_2412_10543_amd import stream
    eng = stream.Engine(kv_budget_bytes=int(budget_gb * (1 << 30)), chunk_len=512, answer_len=32,
                        layers=32, seed=5)
    res = stream.run_stream(stream.synthetic_queries(n, rate, seed=2024), eng)
    res["rate_per_s"] = rate
    res["kv_budget_gb"] = budget_gb
    del eng
    torch.cuda.empty_cache()
    return res


# ---------------------------------------------------------------------------
# CPU baseline: the oracle on a bounded sample of each workload
# ---------------------------------------------------------------------------
def _cores():
    return len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def _f64_of(t):
    """GPU bf16 tensor -> fp64 numpy (exact widening), outside the timed calls."""
    import oracle
    from paper_2412_10543_amd.workloads import bf16_bits
    return oracle.bf16_bits_to_f64(bf16_bits(t))


def oracle_prefill_sample(torch, q, k, v, cu_q, cu_k, hq, scale, budget_s, seed):
    """The oracle on seeded random (row, head) pairs of packed prompts, drawn
    sequence by sequence (sequences in proportion to their work) until
    `budget_s` seconds of oracle time; the full launch's time is extrapolated
    from the sampled pairs' share of the algorithmic FLOPs."""
    import numpy as np

    import oracle
    orc = oracle.default()
    d = q.shape[2]
    lq = [b - a for a, b in zip(cu_q[:-1], cu_q[1:])]
    lk = [b - a for a, b in zip(cu_k[:-1], cu_k[1:])]
    full = prefill_flops(lq, lk, hq, d)
    per_seq = np.array([prefill_flops([a], [b], hq, d) for a, b in zip(lq, lk)])
    rng = np.random.Generator(np.random.PCG64(seed))
    flops, secs, pairs, seqs = 0.0, 0.0, 0, set()
    while secs < budget_s:
        s = int(rng.choice(len(lq), p=per_seq / per_seq.sum()))
        nq, nk = lq[s], lk[s]
        kk, vv = _f64_of(k[cu_k[s]:cu_k[s + 1]]), _f64_of(v[cu_k[s]:cu_k[s + 1]])
        for _ in range(4):
            rows = np.sort(rng.integers(0, nq, size=128)).astype(np.int32)
            heads = rng.integers(0, hq, size=128).astype(np.int32)
            qr = _f64_of(q[cu_q[s]:cu_q[s + 1]][torch.as_tensor(rows, device=q.device).long(),
                                                 torch.as_tensor(heads, device=q.device).long()])
            t0 = time.perf_counter()
            orc.seq_rows(qr, kk, vv, nq, rows, heads, hq, scale, True)
            secs += time.perf_counter() - t0
            flops += float(sum(4 * d * (nk - nq + int(r) + 1) for r in rows))
            pairs += len(rows)
            if secs >= budget_s:
                break
        seqs.add(s)
    return {"sample": f"{pairs} random (row, head) pairs of {len(seqs)} of {len(lq)} prompts",
            "sample_s": round(secs, 3), "sample_gflop": round(flops / 1e9, 3),
            "tflops": round(flops / secs / 1e12, 6),
            "full_tflop": round(full / 1e12, 4),
            "extrapolated_full_s": round(secs * full / flops, 1)}


def oracle_decode_sample(torch, q_rows, pool, kv_lens, seqs, hq, scale, full_bytes, budget_s):
    """The oracle on one decode row per listed sequence (all heads), pages
    gathered from the pool, until `budget_s` seconds; the full phase's time is
    extrapolated from the sampled rows' share of the algorithmic bytes."""
    import numpy as np

    import oracle
    orc = oracle.default()
    hkv, d = pool.k_cache.shape[1], pool.k_cache.shape[3]
    tables = pool.block_tables.cpu().numpy()
    nbytes, secs, n = 0.0, 0.0, 0
    for s in seqs:
        nb = (kv_lens[s] + 15) // 16
        blocks = torch.as_tensor(tables[s, :nb], device=pool.k_cache.device).long()
        kc, vc = _f64_of(pool.k_cache[blocks]), _f64_of(pool.v_cache[blocks])
        qd = _f64_of(q_rows[s:s + 1])
        t0 = time.perf_counter()
        orc.paged(qd, kc, vc, np.arange(nb, dtype=np.int32)[None, :], [kv_lens[s]], scale,
                  want_lse=False)
        secs += time.perf_counter() - t0
        nbytes += decode_bytes([kv_lens[s]], hq, hkv, d)
        n += 1
        if secs >= budget_s:
            break
    return {"sample": f"one decode row (all {hq} heads) of {n} sequences",
            "sample_s": round(secs, 3), "sample_gb": round(nbytes / 1e9, 4),
            "gbs": round(nbytes / secs / 1e9, 4), "full_gb": round(full_bytes / 1e9, 3),
            "extrapolated_full_s": round(secs * full_bytes / nbytes, 1)}


def cpu_baseline_tiny(torch, dev):
    """The tiny stuff query in full: prefill of its 288 tokens and its 16
    decode steps (measured, nothing extrapolated)."""
    import oracle
    from paper_2412_10543_amd import binding
    from paper_2412_10543_amd.workloads import normal_bf16, paged_pool, tiny
    w = tiny()
    cu, dec = binding.rag_plan_prompts(w.method, w.query_lens, w.num_chunks, w.chunk_len,
                                       w.intermediate_length, w.answer_len)
    T = cu[-1]
    q = _f64_of(normal_bf16((T, w.hq, w.d), w.seed, dev))
    k = _f64_of(normal_bf16((T, w.hkv, w.d), w.seed + 1, dev))
    v = _f64_of(normal_bf16((T, w.hkv, w.d), w.seed + 2, dev))
    orc = oracle.default()
    t0 = time.perf_counter()
    orc.varlen(q, k, v, cu, cu, w.scale, True)
    pf_s = time.perf_counter() - t0
    steps = dec[0]
    pool = paged_pool([T + steps], w.hkv, w.d, w.seed + 100, device=dev)
    kc, vc = _f64_of(pool.k_cache), _f64_of(pool.v_cache)
    table = pool.block_tables.cpu().numpy()
    qd = _f64_of(normal_bf16((steps, 1, w.hq, w.d), w.seed + 7, dev))
    t0 = time.perf_counter()
    for t in range(steps):
        orc.paged(qd[t], kc, vc, table, [T + t + 1], w.scale, want_lse=False)
    dec_s = time.perf_counter() - t0
    fl = prefill_flops([T], [T], w.hq, w.d)
    db = sum(decode_bytes([T + t + 1], w.hq, w.hkv, w.d) for t in range(steps))
    return {"prefill": {"sample": "full", "sample_s": round(pf_s, 4),
                        "tflops": round(fl / pf_s / 1e12, 6)},
            "decode": {"sample": f"all {steps} steps", "sample_s": round(dec_s, 4),
                       "gbs": round(db / dec_s / 1e9, 4)}}


def cpu_baseline_stuff(torch, st, budget_s, seed):
    """Sampled prefill rows and decode rows of a stuff-shaped workload (the
    step's stuff7b or the long70b phase)."""
    w = st["w"]
    out = {"prefill": oracle_prefill_sample(torch, st["q"], st["k"], st["v"], st["cu"], st["cu"],
                                            w.hq, w.scale, budget_s, seed)}
    if st["decode_steps"]:
        lens = st["lens"]
        full = sum(decode_bytes([n + t + 1 for n in lens], w.hq, w.hkv, w.d)
                   for t in range(st["decode_steps"]))
        order = sorted(range(len(lens)), key=lambda s: -lens[s])
        out["decode"] = oracle_decode_sample(torch, st["dq"][0], st["pools"][0],
                                             [n + 1 for n in lens], order, w.hq, w.scale,
                                             full, budget_s)
        out["decode"]["sample"] += " (step 0, longest first)"
    return out


def cpu_baseline_mapred(torch, st, budget_s, seed):
    """Whole mapper prompts (every row and head) of the map_reduce map phase,
    one after another until the budget, and sampled decode rows."""
    import numpy as np

    import oracle
    w = st["w"]
    orc = oracle.default()
    lens, cu = st["lens"], st["cu"]
    rng = np.random.Generator(np.random.PCG64(seed))
    flops, secs, n = 0.0, 0.0, 0
    for s in rng.permutation(len(lens)):
        s = int(s)
        sl = slice(cu[s], cu[s + 1])
        qq, kk, vv = _f64_of(st["q"][sl]), _f64_of(st["k"][sl]), _f64_of(st["v"][sl])
        t0 = time.perf_counter()
        orc.varlen(qq, kk, vv, [0, lens[s]], [0, lens[s]], w.scale, True, want_lse=False)
        secs += time.perf_counter() - t0
        flops += prefill_flops([lens[s]], [lens[s]], w.hq, w.d)
        n += 1
        if secs >= budget_s:
            break
    full = prefill_flops(lens, lens, w.hq, w.d)
    out = {"prefill": {"sample": f"{n} whole mapper prompts of {len(lens)} (every row and head)",
                       "sample_s": round(secs, 3), "sample_gflop": round(flops / 1e9, 3),
                       "tflops": round(flops / secs / 1e12, 6), "full_tflop": round(full / 1e12, 4),
                       "extrapolated_full_s": round(secs * full / flops, 1)}}
    fullb = sum(decode_bytes([x + t + 1 for x in lens], w.hq, w.hkv, w.d)
                for t in range(st["decode_steps"]))
    out["decode"] = oracle_decode_sample(torch, st["dq"][0], st["pools"][0],
                                         [x + 1 for x in lens],
                                         [int(x) for x in rng.permutation(len(lens))], w.hq,
                                         w.scale, fullb, budget_s)
    out["decode"]["sample"] += " (step 0)"
    return out


def cpu_baseline_mixed(torch, st, budget_s, seed):
    """Sampled decode rows and chunked-prefill rows of the mixed batch."""
    import numpy as np
    w = st["w"]
    nd = st["nd"]
    pool = st["pools"][0]
    out = {}
    full = decode_bytes(w.decode_kv_lens, w.hq, w.hkv, w.d)
    rng = np.random.Generator(np.random.PCG64(seed))
    out["decode"] = oracle_decode_sample(torch, st["q"], pool, st["kv"],
                                         [int(s) for s in rng.permutation(nd)], w.hq, w.scale,
                                         full, budget_s)
    # pieces: rows of each piece against its paged keys (gathered densely)
    cu = st["cu"]
    qs, ks, vs, cq, ck = [], [], [], [0], [0]
    tables = pool.block_tables.cpu().numpy()
    for s in range(nd, len(st["kv"])):
        n = st["kv"][s]
        nb = (n + 15) // 16
        blocks = torch.as_tensor(tables[s, :nb], device=pool.k_cache.device).long()
        ks.append(pool.k_cache[blocks].permute(0, 2, 1, 3).reshape(nb * 16, w.hkv, w.d)[:n])
        vs.append(pool.v_cache[blocks].permute(0, 2, 1, 3).reshape(nb * 16, w.hkv, w.d)[:n])
        qs.append(st["q"][cu[s]:cu[s + 1]])
        cq.append(cq[-1] + cu[s + 1] - cu[s])
        ck.append(ck[-1] + n)
    out["pieces"] = oracle_prefill_sample(torch, torch.cat(qs), torch.cat(ks), torch.cat(vs),
                                          cq, ck, w.hq, w.scale, budget_s, seed + 1)
    return out


def cpu_baseline_summary(per_config):
    """The headline figure (stuff7b prefill, the bench's `value` metric) with
    the per-workload samples beside it."""
    pf = per_config["stuff7b"]["prefill"]
    return {"value": pf["tflops"], "unit": "TFLOP/s", "cores": _cores(), "kind": "oracle",
            "sample": f"stuff7b prefill: {pf['sample']}, {pf['sample_s']} s of oracle time "
                      f"(full launch extrapolated: {pf['extrapolated_full_s']} s)",
            "cpu_model": _cpu_model(), "omp_threads": os.environ.get("OMP_NUM_THREADS", "default"),
            "note": "oracle = plain fp64 C (OpenMP over sequence x head); sample_s measured, "
                    "extrapolated_full_s = sample_s x (full work / sampled work)",
            "per_config": per_config}


# ---------------------------------------------------------------------------
def prefill_only(torch, name, dev, reps):
    """The packed prefill of one workload, `reps` launches back to back (the
    first warms up), for counter runs that should see nothing else."""
    from paper_2412_10543_amd import binding, workloads
    w = getattr(workloads, name)()
    cu, _ = binding.rag_plan_prompts(w.method, w.query_lens, w.num_chunks, w.chunk_len,
                                     w.intermediate_length, w.answer_len)
    lens = [b - a for a, b in zip(cu[:-1], cu[1:])]
    T = cu[-1]
    q = workloads.normal_bf16((T, w.hq, w.d), w.seed, dev)
    k = workloads.normal_bf16((T, w.hkv, w.d), w.seed + 1, dev)
    v = workloads.normal_bf16((T, w.hkv, w.d), w.seed + 2, dev)
    o = torch.empty_like(q)
    cu_t = torch.tensor(cu, dtype=torch.int32, device=dev)
    timer = Timer(torch)
    for _ in range(reps):
        timer.start("p")
        binding.rag_attn_prefill_varlen(q, k, v, o, None, cu_t, cu_t, max(lens), max(lens),
                                        w.scale, True)
        timer.stop("p")
    torch.cuda.synchronize()
    return {"workload": name, "launches": reps, "ms": [round(x, 4) for x in timer.ms("p")],
            "algorithmic_flops": prefill_flops(lens, lens, w.hq, w.d),
            "algorithmic_bytes": prefill_bytes(lens, lens, w.hq, w.hkv, w.d)}


def ceilings(torch, dev, reps=5, clocks=True):
    """Hardware ceilings the roofline fractions are read against, measured
    with the probes of libceiling_probes.so (HIP events around one launch,
    median of `reps`): random 4 KB page reads (two disjoint 512 MB page sets
    of an 8 GB pool alternate, so neither is found in the 256 MB Infinity
    Cache), K and V pages loaded as the paged decode kernel loads them (and
    as whole rows), a contiguous 4 GB read -- the reads under the default and
    the non-temporal load policy -- a dependency-free bf16 MFMA loop, the prefill kernel's steady 32-key slot
    on LDS-resident tiles, that slot's MFMA + softmax instruction mix with
    register operands, and the slot's work split between specialised wave
    pairs.  Slot rates count 4 * d FLOP per query-key pair, as the prefill's
    algorithmic FLOPs do."""
    import ctypes

    import numpy as np

    from paper_2412_10543_amd import build as pb
    L = ctypes.CDLL(pb.PROBES)
    vp = ctypes.c_void_p
    L.rag_probe_page_read.argtypes = [vp, vp, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, vp, vp]
    L.rag_probe_stream_read.argtypes = [vp, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, vp,
                                        vp]
    L.rag_probe_kv_page_read.argtypes = [vp, vp, vp, ctypes.c_int64, ctypes.c_int32,
                                         ctypes.c_int32, vp, vp]
    L.rag_probe_mfma_loop.argtypes = [ctypes.c_int32, ctypes.c_int32, vp, vp]
    L.rag_probe_attn_slot.argtypes = [ctypes.c_int32, ctypes.c_int32, vp, vp]
    L.rag_probe_softmax_mfma.argtypes = [ctypes.c_int32, ctypes.c_int32, vp, vp]
    L.rag_probe_attn_pair.argtypes = [ctypes.c_int32, ctypes.c_int32, vp, vp]
    stream = torch.cuda.current_stream().cuda_stream
    sink = torch.zeros(1 << 16, dtype=torch.int32, device=dev)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        return median(ts)

    out = {}
    pool_pages = 2 << 20                      # 8 GiB of 4 KB pages
    pool = torch.empty(pool_pages * 1024, dtype=torch.int32, device=dev)
    pool.fill_(7)
    n = 128 << 10                             # 512 MiB per launch
    perm = np.random.Generator(np.random.PCG64(5)).permutation(pool_pages).astype(np.int32)
    sets = [torch.from_numpy(perm[i * n:(i + 1) * n].copy()).to(dev) for i in range(2)]
    pages = {}
    for hint in (0, 1):
        for wg in (256, 512, 1024, 2048):
            it = [0]

            def run(wg=wg, hint=hint):
                ids = sets[it[0] % 2]
                it[0] += 1
                assert L.rag_probe_page_read(pool.data_ptr(), ids.data_ptr(), n, wg, hint,
                                             sink.data_ptr(), stream) == 0
            ms = timed(run)
            pages[f"{'nt' if hint else 'default'}_wg{wg}"] = round(n * 4096 / ms / 1e6, 1)
    out["random_4k_page_read_gbs"] = pages
    out["random_4k_page_read_best_gbs"] = max(pages.values())
    del pool
    # K and V pages per id from two 4 GiB pools, two disjoint sets of 2^16
    # random ids (256 MiB of K and of V per launch) alternating: the decode
    # kernel's loads, and both pools as whole rows under either policy
    kpool = torch.empty(pool_pages * 512, dtype=torch.int32, device=dev)
    kpool.fill_(5)
    vpool = torch.empty_like(kpool)
    vpool.fill_(9)
    nkv = 64 << 10
    perm_kv = np.random.Generator(np.random.PCG64(6)).permutation(pool_pages // 2)
    kv_sets = [torch.from_numpy(perm_kv[i * nkv:(i + 1) * nkv].astype(np.int32)).to(dev)
               for i in range(2)]
    kv = {}
    for pattern, key in ((0, "decode_loads"), (1, "rows_default"), (2, "rows_nt")):
        for wg in (512, 1024, 2048):
            it = [0]

            def run_kv(wg=wg, pattern=pattern):
                ids = kv_sets[it[0] % 2]
                it[0] += 1
                assert L.rag_probe_kv_page_read(kpool.data_ptr(), vpool.data_ptr(), ids.data_ptr(),
                                                nkv, wg, pattern, sink.data_ptr(), stream) == 0
            ms = timed(run_kv)
            kv[f"{key}_wg{wg}"] = round(nkv * 8192 / ms / 1e6, 1)
    out["kv_page_read_gbs"] = kv
    out["kv_page_read_decode_loads_best_gbs"] = max(v for k, v in kv.items()
                                                    if k.startswith("decode_loads"))
    del kpool, vpool, sets, kv_sets
    torch.cuda.empty_cache()
    buf = torch.empty(1 << 30, dtype=torch.int32, device=dev)   # 4 GiB
    buf.fill_(3)
    stream_gbs = {}
    for hint in (0, 1):
        for wg in (1024, 2048, 4096):
            ms = timed(lambda wg=wg, hint=hint: L.rag_probe_stream_read(
                buf.data_ptr(), buf.numel() * 4, wg, hint, sink.data_ptr(), stream))
            stream_gbs[f"{'nt' if hint else 'default'}_wg{wg}"] = \
                round(buf.numel() * 4 / ms / 1e6, 1)
    out["stream_read_gbs"] = stream_gbs
    out["stream_read_best_gbs"] = max(stream_gbs.values())
    del buf
    torch.cuda.empty_cache()
    mfma = {}
    iters = 20000
    for wg in (256, 512):
        ms = timed(lambda wg=wg: L.rag_probe_mfma_loop(iters, wg, sink.data_ptr(), stream))
        flops = wg * 8 * 4 * iters * 32768.0
        mfma[f"wg{wg}_waves_per_simd{wg // 128}"] = round(flops / ms / 1e9, 1)
    out["mfma_bf16_loop_tflops"] = mfma
    out["mfma_bf16_loop_best_tflops"] = max(mfma.values())
    # 32 rows x 32 keys x 4 x 128 FLOP per slot and wave, two slots per iteration
    slot_flops = 32 * 32 * 4 * 128
    for key, fn in (("attn_slot_lds_tflops", L.rag_probe_attn_slot),
                    ("softmax_mfma_mix_tflops", L.rag_probe_softmax_mfma)):
        iters = 4000
        ms = timed(lambda fn=fn: fn(iters, 256, sink.data_ptr(), stream))
        out[key] = round(256 * 8 * 2 * iters * slot_flops / ms / 1e9, 1)
    # the same work split between the two waves of a SIMD: per 32-key block
    # and pair, 64 rows x 32 keys x 4 x 128 FLOP
    blocks = 8000
    ms = timed(lambda: L.rag_probe_attn_pair(blocks, 256, sink.data_ptr(), stream))
    out["attn_pair_lds_tflops"] = round(256 * 4 * blocks * 2 * slot_flops / ms / 1e9, 1)
    if clocks:
        # the shader clock while the MFMA loop runs (about 2 s of launches)
        sampler = ClockSampler(delay=1.0)
        sampler.start()
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < 2.0:
            L.rag_probe_mfma_loop(iters, 256, sink.data_ptr(), stream)
            torch.cuda.synchronize()
        out["clocks_during_mfma_loop"] = sampler.join()
        out["clocks_idle"] = read_clocks()
    out["peaks"] = {"hbm_gbs": PEAK_HBM_GBS, "bf16_tflops": PEAK_BF16_TFLOPS}
    return out


def copy_calibration(torch, gib=1.0):
    """A plain device copy of known size, for scaling the HBM traffic counters."""
    n = int(gib * (1 << 30))
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": n, "launches": 3}))


TRAFFIC_COMMANDS = [
    "rocprofv3 --pmc FETCH_SIZE --output-format csv -d {d}/pmc_FETCH_SIZE -o p -- "
    "python3 -u bench.py --steps 1 --warmup 0 --no-extra --no-cpu-baseline",
    "rocprofv3 --pmc WRITE_SIZE --output-format csv -d {d}/pmc_WRITE_SIZE -o p -- "
    "python3 -u bench.py --steps 1 --warmup 0 --no-extra --no-cpu-baseline",
    "rocprofv3 --pmc FETCH_SIZE --output-format csv -d {d}/cal_FETCH_SIZE -o p -- "
    "python3 -u bench.py --copy-calibration",
    "rocprofv3 --pmc WRITE_SIZE --output-format csv -d {d}/cal_WRITE_SIZE -o p -- "
    "python3 -u bench.py --copy-calibration",
]


def traffic_summary(prof_dir, out_path):
    """HBM traffic per launch of the attention kernels of the default command,
    from the four counter runs of TRAFFIC_COMMANDS with {d} = `prof_dir`:
    FETCH_SIZE and WRITE_SIZE (KiB per dispatch) of each kernel, scaled by
    what the same counters read for the calibration copy of 1 GiB."""
    import collections
    import csv

    def load(sub):
        out = collections.defaultdict(list)
        with open(os.path.join(prof_dir, sub, "p_counter_collection.csv")) as f:
            for r in csv.DictReader(f):
                out[r["Kernel_Name"]].append(float(r["Counter_Value"]))
        return out

    def short(name):   # "void rag::(anon)::k<128, false>(args)" -> "k<128, false>"
        return name.split("(")[0].replace("void ", "").split("::")[-1]

    cal_f, cal_w = load("cal_FETCH_SIZE"), load("cal_WRITE_SIZE")
    copy = [k for k in cal_f if "copyBuffer" in k][0]
    cf = sorted(cal_f[copy])[len(cal_f[copy]) // 2]       # median of the 3 copies
    cw = sorted(cal_w[copy])[len(cal_w[copy]) // 2]
    copy_kib = (1 << 30) / 1024
    ff, wf = copy_kib / cf, copy_kib / cw
    pf, pw = load("pmc_FETCH_SIZE"), load("pmc_WRITE_SIZE")
    kern = {}
    for name in pf:
        key = short(name)
        if not (key.startswith("prefill_varlen_kernel") or key.startswith("paged_decode")):
            continue
        f = sum(pf[name]) / len(pf[name])
        wr = sum(pw[name]) / len(pw[name])
        kern[key] = {"kernel": name.split("(")[0].replace("void ", ""),
                     "dispatches": len(pf[name]),
                     "fetch_kib_per_dispatch": round(f, 1), "write_kib_per_dispatch": round(wr, 1),
                     "fetch_bytes_per_launch": round(f * 1024 * ff),
                     "write_bytes_per_launch": round(wr * 1024 * wf),
                     "bytes_per_launch": round(f * 1024 * ff + wr * 1024 * wf)}
    t = {"source_hash": kernel_source_hash(),
         "workload": "stuff7b (16 prompts, 102,400 tokens, Hq=32, Hkv=8, d=128; 128 decode steps)",
         "calibration": {"copy_bytes": 1 << 30, "copy_fetch_kib": cf, "copy_write_kib": cw,
                         "fetch_factor": round(ff, 4), "write_factor": round(wf, 4)},
         "commands": [c.format(d=prof_dir.rstrip("/")) for c in TRAFFIC_COMMANDS]
                     + [f"python3 bench.py --traffic-summary {prof_dir}"],
         "kernels": kern}
    with open(out_path, "w") as f:
        json.dump(t, f, indent=1)
    return t


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-extra", action="store_true", help="skip the other workloads")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--extra-reps", type=int, default=20)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 1 GiB device copy (counter calibration)")
    ap.add_argument("--awq-only", action="store_true",
                    help="only the int4-weight GEMM phase, eager calls (for profiling)")
    ap.add_argument("--prefill-only", metavar="WORKLOAD",
                    help="only run this workload's packed prefill --reps times (for counter runs)")
    ap.add_argument("--reps", type=int, default=2)
    ap.add_argument("--ceilings", action="store_true",
                    help="only the hardware ceiling probes (page reads, stream read, MFMA loop, "
                         "attention slot, softmax-MFMA mix)")
    ap.add_argument("--no-clocks", action="store_true",
                    help="do not query amd-smi for the clocks (skipped under rocprofv3 anyway)")
    ap.add_argument("--traffic-summary", metavar="PROF_DIR",
                    help="no GPU: write profiles/traffic.json from the csv of the counter runs")
    args = ap.parse_args()
    if args.traffic_summary:
        t = traffic_summary(args.traffic_summary, os.path.join(PROFILES, "traffic.json"))
        print(json.dumps(t, indent=1))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the library has no multi-GPU path "
              "(sequences would shard across GPUs with no exchange between them). "
              "Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    # Clock readings come from an amd-smi child process; not under a profiler,
    # whose preloaded library the child would inherit.
    under_profiler = any(k.startswith("ROCPROF") for k in os.environ) or \
        "rocprof" in os.environ.get("LD_PRELOAD", "")
    want_clocks = not (args.no_clocks or under_profiler or args.copy_calibration or args.awq_only
                       or args.prefill_only or args.ceilings)
    clocks = {"idle_before": read_clocks()} if want_clocks else None

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.copy_calibration:
        copy_calibration(torch)
        return
    if args.ceilings:
        res = ceilings(torch, torch.device("cuda:0"), clocks=not under_profiler)
        print(json.dumps({"ceilings": res}))
        return
    if args.awq_only:
        print(json.dumps({"awq_gemm_7b": bench_phase_awq(torch, torch.device("cuda:0"),
                                                         max(args.extra_reps, 10), graph=False,
                                                         dense=False)}))
        return
    from paper_2412_10543_amd import binding
    from paper_2412_10543_amd.workloads import long70b, mapred7b, stuff7b
    binding.lib()
    dev = torch.device("cuda:0")
    if args.prefill_only:
        print(json.dumps(prefill_only(torch, args.prefill_only, dev, args.reps)))
        return

    w = stuff7b()
    st = setup_stuff(torch, w, dev)
    fl, pb, db = stuff_work(st)
    for _ in range(args.warmup):
        run_stuff_step(st)
    torch.cuda.synchronize()
    dec_eager = eager_decode_ms(torch, st) if st["decode_steps"] else None
    capture_decode(torch, st)

    timer = Timer(torch)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        if st.get("graph") is not None:
            st["do"].zero_()
        run_stuff_step(st, timer)
        if st.get("graph") is not None and not torch.equal(st["do"].view(torch.int16),
                                                           st["do_eager"].view(torch.int16)):
            raise RuntimeError("decode graph replay differs from the eager launches")
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    pf_ms = timer.ms("prefill")
    dec_ms = timer.ms("decode")
    pf_med = median(pf_ms)                                 # headline: median over steps
    pf_mean = sum(pf_ms) / len(pf_ms)
    dec_total = median(dec_ms)                             # ms of decode per step (median)
    nsteps = st["decode_steps"]
    dec_avg = dec_total / nsteps                           # ms per decode launch
    tflops = fl / pf_med / 1e9
    dec_gbs = sum(db) / dec_total / 1e6
    dec_bytes_avg = sum(db) / nsteps

    rl_pf = roofline("mfma", tflops, PEAK_BF16_TFLOPS, "TFLOP/s",
                     traffic=stored_traffic("prefill_varlen_kernel<128>"),
                     kernel="prefill_varlen_kernel<128>")
    dec_kernel = decode_kernel_name(len(st["lens"]), w.hkv)
    rl_dec = roofline("hbm", dec_gbs, PEAK_HBM_GBS, "GB/s",
                      traffic=stored_traffic(dec_kernel),
                      kernel=f"{dec_kernel} (rag_attn_decode_paged)")
    dominant = rl_dec if dec_total > pf_med else rl_pf

    res = {
        "metric": METRIC, "value": round(tflops, 2), "unit": "TFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic: seeded N(0,1) fp32 rounded to bf16; RAG prompt shapes",
        "config": {"workload": "stuff7b", "queries": 16, "query_tokens": 64, "chunk_len": 512,
                   "num_chunks": w.num_chunks, "tokens": st["cu"][-1], "hq": w.hq,
                   "hkv": w.hkv, "d": w.d, "decode_steps": nsteps, "block_size": 16,
                   "decode_splits": st["splits"]},
        "prefill": {"ms": round(pf_med, 4), "ms_mean": round(pf_mean, 4),
                    "ms_min": round(min(pf_ms), 4), "ms_max": round(max(pf_ms), 4),
                    "tflops": round(tflops, 2),
                    "frac_mfma": round(tflops / PEAK_BF16_TFLOPS, 4),
                    "algorithmic_flops": fl, "algorithmic_bytes": pb},
        "decode": {"value": round(dec_gbs, 1), "unit": "GB/s",
                   "frac_hbm": round(dec_gbs / PEAK_HBM_GBS, 4),
                   "us_per_step": round(dec_avg * 1e3, 3),
                   "us_per_step_mean": round(sum(dec_ms) / len(dec_ms) / nsteps * 1e3, 3),
                   "us_per_step_eager": round(dec_eager / nsteps * 1e3, 3) if dec_eager else None,
                   "algorithmic_bytes_per_launch": round(dec_bytes_avg)},
        "timing": "median over the timed steps: prefill = one event pair per launch; decode = "
                  "one event pair around a replay of the step's launches captured in a HIP graph "
                  "(every replay checked bit for bit against the eager launches), divided by their "
                  "number; us_per_step_eager = the same launches issued one by one from the host",
        "roofline": dominant,
        "rooflines": {"prefill": rl_pf, "decode": rl_dec},
    }
    if want_clocks:
        clocks["under_load"] = clock_under_load(torch, st)
    if not args.no_extra:
        phases = {}
        cpu = None if args.no_cpu_baseline else CPU_BUDGET_S
        for fn in (mapred7b, long70b):
            phases[fn.__name__] = bench_phase_stuff(torch, fn(), dev, args.extra_reps, cpu=cpu)
        phases["mixed"] = bench_phase_mixed(torch, dev, args.extra_reps, cpu=cpu)
        phases["kv_write"] = bench_phase_kv_write(torch, dev, max(args.extra_reps, 10))
        phases["fused_kv"] = bench_phase_fused_kv(torch, dev, max(args.extra_reps, 10))
        phases["awq_gemm_7b"] = bench_phase_awq(torch, dev, max(args.extra_reps, 10),
                                                dense=not under_profiler)
        if not under_profiler:
            lib_attn = bench_phase_library_attention(torch, dev)
            ours = {"stuff7b": res["prefill"]["ms"],
                    "mapred7b": phases["mapred7b"]["prefill_ms"],
                    "long70b": phases["long70b"]["prefill_ms"]}
            for name, r in lib_attn.items():
                if "ms" in r:
                    r["ours_speedup"] = round(r["ms"] / ours[name], 2)
            phases["torch_sdpa_flash"] = lib_attn
        phases["query_stream"] = bench_phase_stream(torch)
        phases["query_stream_tight"] = bench_phase_stream(torch, n=32, rate=2000.0, budget_gb=1)
        res["phases"] = phases
    if not args.no_cpu_baseline:
        per = {"tiny": cpu_baseline_tiny(torch, dev),
               "stuff7b": cpu_baseline_stuff(torch, st, CPU_BUDGET_S, seed=w.seed)}
        for name, ph in res.get("phases", {}).items():
            if isinstance(ph, dict) and "_cpu" in ph:
                per[name] = ph.pop("_cpu")
        res["cpu_baseline"] = cpu_baseline_summary(per)
    if want_clocks:
        clocks["idle_after"] = read_clocks()
        res["clocks"] = clocks
        sclk = (clocks.get("under_load") or {}).get("sclk_mhz")
        if isinstance(sclk, (int, float)) and sclk > 0:
            # the same work against the MFMA peak at the shader clock read under load
            peak = PEAK_BF16_TFLOPS * sclk / 2400.0
            res["at_measured_sclk"] = {
                "sclk_mhz": sclk, "bf16_peak_tflops": round(peak, 1),
                "prefill_frac_mfma": round(tflops / peak, 4),
                "phases_prefill_frac_mfma": {
                    k: round(v["prefill_tflops"] / peak, 4)
                    for k, v in res.get("phases", {}).items()
                    if isinstance(v, dict) and "prefill_tflops" in v}}
    print(json.dumps(res))


if __name__ == "__main__":
    main()
