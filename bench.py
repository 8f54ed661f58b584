#!/usr/bin/env python3
"""Prefix-extend attention benchmark on one MI355X.

One step = one pass of the whole hot path over one batch: the host work plan,
store_kv of the uncached suffix's K/V into the paged pool, and extend_attention
of the suffix over its cached prefix and itself.  Inputs are synthetic, seeded,
and resident in HBM before the timed region; the cached prefixes were written
into the pool by an earlier (untimed) turn.

Prints one JSON line: algorithmic TFLOP/s of the step (4*d*Hq per visible causal
(query, key) pair), its fraction of the bf16 dense MFMA peak, uncached tokens/s,
the attention kernel's roofline entry, and the CPU oracle timed on a bounded
sample of the same workload.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--config wide70b]

The default workload is the largest single-GPU one, the 70B-shaped layer
(48 requests, 64 query / 8 KV heads, 6.3e14 FLOP per step).
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6  # 256 CUs x 2.4 GHz x 4096 dense bf16 flop/clk/CU
PEAK_HBM_GBPS = 8000.0
CPU_SAMPLE_TRIPLES = 330_000_000  # oracle sample size in (row, query head, key) triples

DESCRIPTIONS = {
    "tiny": "4 requests, P {0,64,208,512}, E {32,16,100,8}, Hq 4 / Hkv 2, d 64, page 16, bf16 K/V",
    "llama8b": "Llama-3-8B-shaped layer: 16 returning agents, P~U[4096,32768] (page-rounded), "
               "E~U[64,2048], Hq 32 / Hkv 8, d 128, page 16, bf16 K/V, values N(0,0.25)",
    "tail_outlier": "1 fully evicted agent (P 0, E 131072) + 31 agents P~U[32768,98304], E~U[256,1024], "
                    "Hq 32 / Hkv 8, d 128, page 16, bf16 K/V",
    "rr_partial": "64 agents, context~logU[8192,196608], k~U{1..4} lost 2048-token tail chunks, "
                  "E = 2048k + U[128,4096], Hq 32 / Hkv 8, d 128, page 16, bf16 K/V",
    "wide70b": "70B-shaped layer: 48 requests, P~logU[16384,262144], E~U[512,8192], Hq 64 / Hkv 8, d 128, "
               "page 16, bf16 K/V",
    "wide70b_fp8": "70B-shaped layer: 48 requests, P~logU[16384,262144], E~U[512,8192], Hq 64 / Hkv 8, d 128, "
                   "page 16, fp8 e4m3 K/V with per-head scales U[0.01,0.1]",
    "decode_llama8b": "decode step (E = 1): 128 agents, P~U[4096,32768] (page-rounded), Hq 32 / Hkv 8, d 128, "
                      "page 16, bf16 K/V, values N(0,0.25)",
    "decode_long": "decode step (E = 1): 32 agents, P~U[65536,131072] (page-rounded), Hq 32 / Hkv 8, d 128, "
                   "page 16, bf16 K/V",
}


def is_decode(config: str) -> bool:
    """Decode steps (one suffix token per request) run the decode kernel."""
    return config.startswith("decode")


def code_only(text: str) -> str:
    """C/C++ source text without its comments and blank lines, each line stripped:
    an edit of comments or layout alone leaves it unchanged."""
    out, i, n, quote = [], 0, len(text), None
    while i < n:
        c = text[i]
        if quote:
            out.append(c)
            if c == "\\" and i + 1 < n:
                out.append(text[i + 1])
                i += 2
                continue
            if c == quote:
                quote = None
            i += 1
        elif c in "\"'":
            quote = c
            out.append(c)
            i += 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(c)
            i += 1
    lines = (ln.strip() for ln in "".join(out).splitlines())
    return "\n".join(ln for ln in lines if ln)


def code_hash(path: str) -> str:
    """sha256[:16] of a source file's code (comments and blank lines removed)."""
    return hashlib.sha256(code_only(open(path, encoding="utf-8").read()).encode()).hexdigest()[:16]


def attn_source_hash(config: str = "llama8b") -> str:
    """Code hash of the attention (or decode) kernel source: committed counter
    summaries carry it, and their traffic is used only while it matches."""
    name = "kvx_decode.hip" if is_decode(config) else "kvx_attn.hip"
    return code_hash(os.path.join(ROOT, "paper_2609_32278_amd", "csrc", name))


def traffic_from_profiles(config: str):
    """HBM bytes per attention launch from the committed rocprofv3 counter summary,
    only if it was taken on the current kernel source; else None."""
    kernel = "decode_kernel" if is_decode(config) else "extend_attn"
    path = os.path.join(ROOT, "profiles", f"{kernel}_{config}_hbm_counters.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_hash = re.search(r"kernel code sha256\[:16\][^:`]*:\s*`?([0-9a-f]{16})", text)
    m_bytes = re.search(r"HBM bytes per launch \(scaled\):\s*`?([0-9.eE+]+)", text)
    if not (m_hash and m_bytes) or m_hash.group(1) != attn_source_hash(config):
        return None
    return float(m_bytes.group(1))


def rope_args(w, dev="cuda"):
    """Keyword arguments of store_kv_rope for the Qwen3-shaped setting: half-layout
    rotation of the whole head, base 10^6, RMS norm of every Q and K head."""
    from paper_2609_32278_amd import workloads as wl
    spec = wl.RopeSpec(rotary_dim=w.head_dim)
    qn, kn = wl.norm_weights(w, dev)
    return dict(theta=spec.theta, rotary_dim=spec.rotary_dim, style=spec.style, q_norm=qn, k_norm=kn,
                norm_eps=spec.eps)


def setup(config: str, seed: int = 0, rope: bool = False):
    import torch
    from paper_2609_32278_amd import kvx
    from paper_2609_32278_amd import workloads as wl

    w = wl.make_workload(config, seed)
    dev = "cuda"
    pool = kvx.kv_pool_create(w.num_pages, w.page_size, w.num_kv_heads, w.head_dim, w.kv_dtype, w.k_scale, w.v_scale)
    rk = rope_args(w, dev) if rope else None
    qs, ke, ve = [], [], []
    for r in range(w.num_reqs):
        k, v = wl.request_kv(w, r, dev)
        p = int(w.prefix_lens[r])
        if p > 0:  # the earlier turn that cached this prefix
            n = (p + w.page_size - 1) // w.page_size
            ids = torch.from_numpy(np.ascontiguousarray(w.pages_of(r)[:n])).to(dev)
            hb = kvx.Batch([0], [p], [0, n], ids)
            if rope:
                kvx.store_kv_rope(pool, hb, k[:p].contiguous(), v[:p].contiguous(), **rk)
            else:
                kvx.store_kv(pool, hb, k[:p].contiguous(), v[:p].contiguous())
            torch.cuda.synchronize()
        qs.append(wl.request_q(w, r, dev))
        ke.append(k[p:].clone())
        ve.append(v[p:].clone())
        del k, v
    q = torch.cat(qs).contiguous()
    k_ext = torch.cat(ke).contiguous()
    v_ext = torch.cat(ve).contiguous()
    del qs, ke, ve
    ids = torch.from_numpy(w.page_ids).to(dev)
    batch = kvx.Batch(w.prefix_lens, w.extend_lens, w.page_indptr, ids)
    out = torch.empty_like(q)
    torch.cuda.synchronize()
    return dict(w=w, pool=pool, batch=batch, ids=ids, q=q, k_ext=k_ext, v_ext=v_ext, out=out, rope=rk)


def run_gpu(config: str, steps: int, warmup: int, rope: bool = False, scaled_q_steps: int = 0):
    import torch
    from paper_2609_32278_amd import kvx

    print(f"[bench] setup {config}", file=sys.stderr, flush=True)
    s = setup(config, rope=rope)
    w, pool, batch = s["w"], s["pool"], s["batch"]
    print(f"[bench] timing {warmup} + {steps} steps", file=sys.stderr, flush=True)
    q, k_ext, v_ext, out = s["q"], s["k_ext"], s["v_ext"], s["out"]
    q_rot = torch.empty_like(q) if rope else q

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        if rope:  # norm + rotate Q and K, store K and V: one fused kernel
            kvx.store_kv_rope(pool, batch, k_ext, v_ext, q=q, num_q_heads=w.num_q_heads, q_out=q_rot, **s["rope"])
        else:
            kvx.store_kv(pool, batch, k_ext, v_ext)
        if ev is not None:
            ev[1].record()
        kvx.extend_attention(pool, batch, q_rot, w.num_q_heads, w.sm_scale, out)
        if ev is not None:
            ev[2].record()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        step(evs[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    store_t = np.array([e[0].elapsed_time(e[1]) for e in evs])
    attn_t = np.array([e[1].elapsed_time(e[2]) for e in evs])
    ms_step = (t1 - t0) * 1e3 / steps
    assert torch.isfinite(out.float()).all(), "non-finite attention output"
    scaled = None
    if scaled_q_steps > 0 and w.kv_dtype == 0:
        # the pool's scaled-Q setting (folded softmax) on the same pool and inputs: the
        # attention kernel alone, after the exact steps
        print(f"[bench] scaled-Q mode: {warmup} + {scaled_q_steps} attention launches", file=sys.stderr, flush=True)
        kvx.kv_pool_set_scaled_q(pool, True)
        out_sq = torch.empty_like(out)
        for _ in range(warmup):
            kvx.extend_attention(pool, batch, q_rot, w.num_q_heads, w.sm_scale, out_sq)
        ev2 = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(scaled_q_steps)]
        torch.cuda.synchronize()
        for e in ev2:
            e[0].record()
            kvx.extend_attention(pool, batch, q_rot, w.num_q_heads, w.sm_scale, out_sq)
            e[1].record()
        torch.cuda.synchronize()
        kvx.kv_pool_set_scaled_q(pool, False)
        assert torch.isfinite(out_sq.float()).all(), "non-finite attention output (scaled-Q mode)"
        scaled = (np.array([e[0].elapsed_time(e[1]) for e in ev2]), out_sq)
    kvx.kv_pool_destroy(pool)
    return w, ms_step, store_t, attn_t, out, scaled


def _parity(gpu_out, qo, rows, ref):
    """Errors of the GPU output's sampled rows against the oracle's."""
    import torch
    gidx = torch.from_numpy(np.array([qo[r] + i for r, i in rows], dtype=np.int64))
    got = gpu_out[gidx.to(gpu_out.device)].float().cpu().numpy().astype(np.float64)
    err = np.abs(got - ref)
    return {"rows": int(len(rows)), "max_abs_err": float(err.max()), "mean_abs_err": float(err.mean()),
            "rel_rms_err": float(np.sqrt((err ** 2).mean()) / max(np.sqrt((ref ** 2).mean()), 1e-300)),
            "gate": "max <= 2e-2, mean <= 2e-3 (fp64 oracle)",
            "pass": bool(err.max() <= 2e-2 and err.mean() <= 2e-3)}


def run_cpu_baseline(config: str, rows_per_req: int, max_reqs: int, gpu_out=None, gpu_out_scaled=None):
    """The oracle as it stands, on a bounded sample of the same workload.  With the
    GPU's output of the timed steps, also the parity of the sampled rows (and of the
    scaled-Q mode's output against the oracle's definition of that mode)."""
    import torch
    import oracle
    from paper_2609_32278_amd import workloads as wl

    w = wl.make_workload(config)
    reqs = list(range(min(w.num_reqs, max_reqs)))
    if rows_per_req <= 0:
        # about CPU_SAMPLE_TRIPLES (row, query head, key) triples, ~15 s of the oracle on 16 cores; an fp8
        # pool's keys cost the oracle 2.3x (it decodes every code).  Each request contributes at least its
        # first, last and page-boundary rows, so the largest configs also sample fewer requests.
        weight = 2.3 if w.kv_dtype != 0 else 1.0
        cost = [weight * w.num_q_heads * (int(w.prefix_lens[r]) + int(w.extend_lens[r]) / 2) for r in reqs]
        rows_per_req = int(min(32, max(4, CPU_SAMPLE_TRIPLES // max(sum(cost), 1))))
        if rows_per_req == 4:
            keep, total = 0, 0.0
            while keep < len(reqs) and (keep < 2 or total + 4 * cost[keep] <= CPU_SAMPLE_TRIPLES):
                total += 4 * cost[keep]
                keep += 1
            reqs = reqs[:keep]
    print(f"[bench] cpu baseline: {rows_per_req} rows per request of {len(reqs)} requests", file=sys.stderr,
          flush=True)
    sub = w.subset(reqs)
    t = wl.batch_tensors(sub, device="cuda")
    t = {k: v.cpu() for k, v in t.items()}
    # the oracle's own pool: cached prefixes (the earlier turn), then this turn's suffix
    pool = oracle.OraclePool(sub.num_pages, sub.num_kv_heads, sub.head_dim, sub.kv_dtype, sub.page_size,
                             sub.k_scale, sub.v_scale)
    h = wl.history_batch(sub)
    oracle.store_kv(pool, h.prefix_lens, h.extend_lens, h.page_indptr, h.page_ids, t["k_hist"], t["v_hist"])
    oracle.store_kv(pool, sub.prefix_lens, sub.extend_lens, sub.page_indptr, sub.page_ids, t["k_ext"], t["v_ext"])
    rows = wl.sample_rows(sub, rows_per_req)
    qo = sub.qo_indptr.astype(np.int64)
    q_rows = t["q"][torch.from_numpy(np.array([qo[r] + i for r, i in rows], dtype=np.int64))]
    # the host's share of cores: the affinity mask, capped by OMP_NUM_THREADS when set
    cores = len(os.sched_getaffinity(0))
    if os.environ.get("OMP_NUM_THREADS", "").isdigit():
        cores = min(cores, int(os.environ["OMP_NUM_THREADS"]))
    t0 = time.perf_counter()
    ref = oracle.extend_attention(pool, sub.prefix_lens, sub.extend_lens, sub.page_indptr, sub.page_ids, q_rows,
                                  rows[:, 0], rows[:, 1], w.num_q_heads, w.sm_scale, num_threads=cores)
    dt = time.perf_counter() - t0
    used = oracle.max_threads()
    visible = int(sum(int(sub.prefix_lens[r]) + int(i) + 1 for r, i in rows))
    flops = 4.0 * w.head_dim * w.num_q_heads * visible
    parity = parity_sq = None
    # the sampled requests are the batch's first ones, so their rows sit at the same offsets
    if gpu_out is not None:
        parity = _parity(gpu_out, qo, rows, ref)
    if gpu_out_scaled is not None:
        ref_sq = oracle.extend_attention(pool, sub.prefix_lens, sub.extend_lens, sub.page_indptr, sub.page_ids,
                                         q_rows, rows[:, 0], rows[:, 1], w.num_q_heads, w.sm_scale,
                                         num_threads=cores, scaled_q=True)
        parity_sq = _parity(gpu_out_scaled, qo, rows, ref_sq)
    return parity, parity_sq, {
        "value": flops / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": used,
        "kind": "oracle",
        "sample": f"{len(rows)} suffix rows x {w.num_q_heads} heads ({rows_per_req} per request: first, last, "
                  f"page-boundary and seeded random rows) of the first {len(reqs)} requests; "
                  f"{visible} visible (row, key) pairs per head, fp64, {dt:.1f} s",
        "row_heads_per_s": len(rows) * w.num_q_heads / dt,
        "seconds": dt,
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="wide70b", choices=sorted(DESCRIPTIONS))
    ap.add_argument("--rope", action="store_true",
                    help="the step's store also RMS-normalises and rotates Q and K (store_kv_rope)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=0,
                    help="oracle sample rows per request (0: sized to about 15 s of oracle work, at most 32)")
    ap.add_argument("--cpu-reqs", type=int, default=16)
    ap.add_argument("--scaled-q-steps", type=int, default=-1,
                    help="attention launches timed in the pool's scaled-Q mode after the exact steps "
                         "(bf16 pools; -1: as many as --steps, 0: skip)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="run only a plain 1 GiB device copy kernel (HBM counter calibration)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}): kvx has no "
              f"multi-GPU path", file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    torch.cuda.set_device(0)

    if args.calib_copy:
        # a plain elementwise kernel that reads 1 GiB and writes 1 GiB, three launches
        n = (1 << 30) // 4
        x = torch.ones(n, dtype=torch.float32, device="cuda")
        y = torch.empty_like(x)
        for _ in range(3):
            torch.mul(x, 1.0, out=y)
        torch.cuda.synchronize()
        print(json.dumps({"calib_copy_bytes_read": 4 * n, "calib_copy_bytes_written": 4 * n, "launches": 3}))
        return

    sq_steps = args.steps if args.scaled_q_steps < 0 else args.scaled_q_steps
    if is_decode(args.config):
        sq_steps = 0  # decode steps are always exact
    w, ms_step, store_t, attn_t, gpu_out, scaled = run_gpu(args.config, args.steps, args.warmup, args.rope,
                                                           sq_steps)
    # the roofline entry takes the kernel's average launch time; medians are reported beside it
    store_ms, attn_ms = float(store_t.mean()), float(attn_t.mean())
    store_med, attn_med = float(np.median(store_t)), float(np.median(attn_t))
    flops = w.flops()
    T = w.total_extend
    tflops_step = flops / (ms_step * 1e-3) / 1e12
    tflops_attn = flops / (attn_ms * 1e-3) / 1e12
    eb = 2 if w.kv_dtype == 0 else 1
    store_bytes = T * w.num_kv_heads * w.head_dim * 2 * (2 + eb)
    if args.rope:  # plus Q read and written back rotated
        store_bytes += T * w.num_q_heads * w.head_dim * 2 * 2
    ctx = int(w.seq_lens.sum())
    attn_alg_bytes = (2 * T * w.num_q_heads * w.head_dim * 2 + 2 * eb * ctx * w.num_kv_heads * w.head_dim
                      + 4 * int(np.ceil(w.seq_lens / 16).sum()))
    traffic = traffic_from_profiles(args.config)
    result = {
        "metric": "prefix-extend attention TFLOP/s (% bf16 MFMA peak) + uncached tokens/s",
        "value": round(tflops_step, 2),
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
            "workload": f"{args.config}: {DESCRIPTIONS[args.config]}"
                        + ("; store fused with Q/K RMS norm + RoPE (half layout, base 1e6)" if args.rope else ""),
            "requests": w.num_reqs,
            "uncached_tokens": T,
            "context_tokens": ctx,
            "algorithmic_flop": flops,
            "kv_pool": "fp8_e4m3" if w.kv_dtype else "bf16",
        },
        "pct_bf16_peak": round(100.0 * tflops_step / PEAK_BF16_TFLOPS, 2),
        "uncached_tokens_per_s": round(T / (ms_step * 1e-3), 1),
        "attn_ms": round(attn_ms, 4),
        "attn_ms_median": round(attn_med, 4),
        "attn_ms_min_max": [round(float(attn_t.min()), 4), round(float(attn_t.max()), 4)],
        "attn_tflops": round(tflops_attn, 2),
        "attn_tflops_median": round(flops / (attn_med * 1e-3) / 1e12, 2),
        "pct_bf16_peak_attn_median": round(100.0 * flops / (attn_med * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 2),
        "uncached_tokens_per_s_attn_only": round(T / (attn_med * 1e-3), 1),
        "store_kernel": "store_kv_rope_kernel" if args.rope else "store_kv_kernel",
        "store_ms": round(store_ms, 4),
        "store_ms_median": round(store_med, 4),
        "store_GBps": round(store_bytes / (store_med * 1e-3) / 1e9, 1),
        "store_roofline_frac": round(store_bytes / (store_med * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
        "roofline": {
            "kernel": "extend_attn_fp8_kernel" if w.kv_dtype else "extend_attn_kernel",
            "bound": "mfma",
            "achieved": round(tflops_attn, 2),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(tflops_attn / PEAK_BF16_TFLOPS, 4),
            "traffic": traffic,
            "algorithmic_bytes": attn_alg_bytes,
            "kernel_source": attn_source_hash(args.config),
        },
    }
    if is_decode(args.config):
        # one query per request: intensity ~ 2 Hq/Hkv / b_kv flop/B, far below the ridge -> HBM-bound
        gbps = attn_alg_bytes / (attn_ms * 1e-3) / 1e9
        result["roofline"].update({"kernel": "decode_kernel", "bound": "hbm", "achieved": round(gbps, 1),
                                   "peak": PEAK_HBM_GBPS, "unit": "GB/s", "frac": round(gbps / PEAK_HBM_GBPS, 4)})
    if traffic is not None:
        result["roofline"]["traffic_GBps"] = round(traffic / (attn_ms * 1e-3) / 1e9, 1)
        result["roofline"]["traffic_over_algorithmic"] = round(traffic / attn_alg_bytes, 2)
    if scaled is not None:
        sq_t, _ = scaled
        sq_med = float(np.median(sq_t))
        result["scaled_q_mode"] = {
            "what": "kv_pool_set_scaled_q: Q times the softmax scale rounded to bf16, no FMA per score "
                    "(a precision option, not the headline)",
            "attn_ms_median": round(sq_med, 4),
            "attn_ms_min_max": [round(float(sq_t.min()), 4), round(float(sq_t.max()), 4)],
            "attn_tflops_median": round(flops / (sq_med * 1e-3) / 1e12, 2),
            "pct_bf16_peak_attn_median": round(100.0 * flops / (sq_med * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 2),
        }
    if not args.no_cpu_baseline:
        parity, parity_sq, cb = run_cpu_baseline(args.config, args.cpu_rows, args.cpu_reqs, gpu_out,
                                                 scaled[1] if scaled is not None else None)
        result["cpu_baseline"] = {k: (round(v, 6) if isinstance(v, float) else v) for k, v in cb.items()}
        result["parity"] = parity
        if parity_sq is not None:
            result["scaled_q_mode"]["parity"] = parity_sq
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
