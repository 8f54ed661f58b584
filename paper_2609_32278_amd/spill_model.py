"""Reload instead of recompute: measured rates and the per-token timing model.

An agent whose tail chunk was evicted either recomputes it on its next turn
(prefill of those tokens over the rest of its prefix) or, with a host tier,
reloads the spilled KV pages (the paper's future work, Section 6).  Per token
and attention layer:

    reload    = 2 * Hkv * d * b_kv bytes / (host link rate of kv_pool_reload)
    recompute = 2 * W_layer flop / (GEMM rate)                      projections + MLP
              + 4 * d * Hq * (P + 1/2 ...) flop / (extend_attention rate)   attention over the prefix

This tool measures every rate on the GPU it runs on: kv_pool_spill and
kv_pool_reload over pinned host memory (and a plain device-to-host copy for
reference), extend_attention on chunk recomputes at several prefix lengths, and
torch's bf16 GEMM of a layer's MLP shape.  It prints one JSON object.

    python -m paper_2609_32278_amd.spill_model [--heads 32,8,128] [--pages 16384]
"""

from __future__ import annotations

import argparse
import json
import sys

import numpy as np

from . import kvx
from . import workloads as wl


def _time(fn, reps=5):
    import torch
    fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        fn()
    e1.record()
    e1.synchronize()
    return e0.elapsed_time(e1) / reps * 1e-3  # seconds per call


def link_rates(hkv: int, d: int, pages: int):
    import torch
    pool = kvx.kv_pool_create(pages, wl.PAGE_SIZE, hkv, d)  # zero-filled bf16 pool
    try:
        rb = kvx.kv_pool_record_bytes(pool)
        host = torch.empty(pages * rb, dtype=torch.uint8, pin_memory=True)
        rng = np.random.default_rng(0)
        ids = rng.permutation(pages).astype(np.int32)
        slots = np.arange(pages, dtype=np.int32)
        t_spill = _time(lambda: kvx.kv_pool_spill(pool, ids, slots, host, pages))
        t_reload = _time(lambda: kvx.kv_pool_reload(pool, ids, slots, host, pages))
        dev = torch.empty(pages * rb, dtype=torch.uint8, device="cuda")
        t_d2h = _time(lambda: host.copy_(dev, non_blocking=True))
        t_h2d = _time(lambda: dev.copy_(host, non_blocking=True))
        n = pages * rb
        return {"record_bytes": rb, "bytes": n, "spill_GBps": n / t_spill / 1e9, "reload_GBps": n / t_reload / 1e9,
                "copy_d2h_GBps": n / t_d2h / 1e9, "copy_h2d_GBps": n / t_h2d / 1e9}
    finally:
        kvx.kv_pool_destroy(pool)


def recompute_attention_rate(hq: int, hkv: int, d: int, prefix: int, chunk: int, reqs: int):
    """Seconds per recomputed token of one attention layer: `reqs` agents each
    recomputing a `chunk`-token tail over a `prefix`-token cached prefix."""
    import torch
    w = wl.make_custom([prefix] * reqs, [chunk] * reqs, hq, hkv, d, seed=1, pool_factor=1.05, placement="linear",
                       name="recompute")
    pool = kvx.kv_pool_create(w.num_pages, w.page_size, hkv, d)
    try:
        ids = torch.from_numpy(w.page_ids).to("cuda")
        b = kvx.Batch(w.prefix_lens, w.extend_lens, w.page_indptr, ids)
        g = torch.Generator(device="cuda").manual_seed(3)
        # the cached prefixes hold N(0, 1) values like every other workload (MFMA
        # clocks depend on the data: an all-zero prefix would run faster)
        for p0 in range(0, w.num_pages, 4096):
            n = min(4096, w.num_pages - p0)
            kv = torch.randn((n, hkv, wl.PAGE_SIZE, d), generator=g, device="cuda").to(torch.bfloat16)
            kvx.kv_pool_write_pages(pool, np.arange(p0, p0 + n, dtype=np.int32), kv, kv)
        T = w.total_extend
        q = torch.randn((T, hq, d), generator=g, device="cuda").to(torch.bfloat16)
        k = torch.randn((T, hkv, d), generator=g, device="cuda").to(torch.bfloat16)
        out = torch.empty_like(q)

        def step():
            kvx.store_kv(pool, b, k, k)
            kvx.extend_attention(pool, b, q, hq, d ** -0.5, out)

        t = _time(step, reps=3)
        return {"prefix": prefix, "chunk": chunk, "requests": reqs, "s_per_token": t / T,
                "tflops": w.flops() / t / 1e12}
    finally:
        kvx.kv_pool_destroy(pool)


def gemm_rate(m: int, k: int, n: int):
    import torch
    a = torch.randn((m, k), device="cuda").to(torch.bfloat16)
    b = torch.randn((k, n), device="cuda").to(torch.bfloat16)
    t = _time(lambda: torch.matmul(a, b))
    return 2.0 * m * k * n / t / 1e12


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--heads", default="32,8,128", help="Hq,Hkv,head_dim of the layer")
    ap.add_argument("--hidden", type=int, default=4096, help="model width (Llama-3-8B: 4096)")
    ap.add_argument("--ffn", type=int, default=14336, help="MLP width (Llama-3-8B: 14336)")
    ap.add_argument("--pages", type=int, default=16384, help="pages moved per spill / reload call")
    ap.add_argument("--chunk", type=int, default=2048, help="tokens per recomputed tail chunk")
    ap.add_argument("--prefixes", default="0,8192,32768,131072")
    args = ap.parse_args(argv)
    import torch
    torch.cuda.set_device(0)
    hq, hkv, d = (int(x) for x in args.heads.split(","))
    H, F = args.hidden, args.ffn
    w_layer = H * (hq * d + 2 * hkv * d) + hq * d * H + 3 * H * F  # QKV, O, gate/up/down
    link = link_rates(hkv, d, args.pages)
    gemm_tflops = gemm_rate(args.chunk * 4, H, F)
    bytes_tok = link["record_bytes"] / wl.PAGE_SIZE
    t_reload = bytes_tok / (link["reload_GBps"] * 1e9)
    t_gemm = 2.0 * w_layer / (gemm_tflops * 1e12)
    rows = []
    for p in (int(x) for x in args.prefixes.split(",")):
        reqs = max(1, min(64, (1 << 22) // max(args.chunk * max(p, args.chunk) // 1024, 1)))
        a = recompute_attention_rate(hq, hkv, d, p, args.chunk, reqs)
        t_re = t_gemm + a["s_per_token"]
        rows.append({**a, "recompute_ns_per_token": 1e9 * t_re, "reload_ns_per_token": 1e9 * t_reload,
                     "recompute_over_reload": t_re / t_reload})
    print(json.dumps({"heads": [hq, hkv, d], "hidden": H, "ffn": F, "layer_params": w_layer, "link": link,
                      "kv_bytes_per_token_per_layer": bytes_tok, "gemm_tflops": gemm_tflops,
                      "gemm_ns_per_token": 1e9 * t_gemm, "chunks": rows}), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
