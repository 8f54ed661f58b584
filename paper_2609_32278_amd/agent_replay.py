"""Replay a synthetic multi-agent workload through the prefix cache and the hot path.

Every scheduler tick, the agents whose idle time has run out start their next
turn: the cache (include/kvx_cache.h) reuses what is left of each agent's history,
evicts idle agents' pages by the chosen policy when the pool runs short, and
returns the turn's page table.  The tick's starting turns form one prefix-extend
batch: store_kv writes their uncached suffix K/V into the pool and
extend_attention computes the suffix rows (paper Sections 1 and 2).  A turn then
decodes for a few ticks (its pages pinned), ends, and the agent idles for its
tool / user latency; an agent that finishes its last turn sends the completion
signal (Section 3.2).

The figures this produces are the paper's: uncached prompt tokens per returning
turn (Section 4) and, with the GPU, the time of each batch's KV store + attention.

With a host tier (``--host-pages``, the paper's future work in Section 6), pages
the policy evicts are spilled to pinned host memory and a returning agent's
spilled pages are reloaded instead of recomputed: each turn start's spills and
reloads run on the pool (kv_pool_spill / kv_pool_reload, in call order) before the
batch's store, inside the batch's timed region.

    python -m paper_2609_32278_amd.agent_replay --policy both --agents 48 --turns 8
"""

from __future__ import annotations

import argparse
import json
import sys
import time
from dataclasses import dataclass, field

import numpy as np

from . import kvx
from . import workloads as wl

POLICIES = {"lru": kvx.KVX_EVICT_LRU, "rr": kvx.KVX_EVICT_RR}


@dataclass
class TurnRecord:
    agent: int
    turn: int
    tick: int
    prompt: int        # tokens of the turn's prompt
    prefix: int        # tokens reused from the cache (device pages and reloaded host pages)
    history: int       # tokens of context the agent had before this turn
    reloaded: int = 0  # tokens of the prefix reloaded from the host tier

    @property
    def uncached(self) -> int:
        return self.prompt - self.prefix

    @property
    def recomputed_history(self) -> int:
        """Old-prefix recomputation (the X of Section 3.3, in tokens)."""
        return self.history - min(self.prefix, self.history)


@dataclass
class ReplayResult:
    policy: str
    turns: list = field(default_factory=list)
    events: list = field(default_factory=list)   # ("begin", agent, prompt, prefix | None), ("end", a), ("complete", a)
    moves: list = field(default_factory=list)    # per tiered turn start: (spills, reloads) page counts
    batch_ms: list = field(default_factory=list)
    stats: dict = field(default_factory=dict)
    cache_calls: int = 0
    cache_seconds: float = 0.0  # host time inside the cache's calls

    def summary(self) -> dict:
        back = [t for t in self.turns if t.turn > 0]
        u = np.array([t.uncached for t in back], dtype=np.float64)
        x = np.array([t.recomputed_history / max(t.history, 1) for t in back], dtype=np.float64)
        out = {
            "policy": self.policy,
            "turns": len(self.turns),
            "returning_turns": len(back),
            "uncached_tokens_total": int(sum(t.uncached for t in self.turns)),
        }
        if len(back):
            out.update({
                "uncached_p50": float(np.percentile(u, 50)),
                "uncached_p90": float(np.percentile(u, 90)),
                "uncached_p99": float(np.percentile(u, 99)),
                "uncached_max": float(u.max()),
                "uncached_mean": float(u.mean()),
                "history_recomputed_mean": float(x.mean()),
                "history_recomputed_p99": float(np.percentile(x, 99)),
                "full_misses": int(sum(1 for t in back if t.prefix == 0)),
                "reloaded_tokens_total": int(sum(t.reloaded for t in back)),
            })
        if self.batch_ms:
            b = np.array(self.batch_ms)
            out.update({"batches": len(b), "prefill_ms_total": float(b.sum()),
                        "prefill_ms_p50": float(np.percentile(b, 50)), "prefill_ms_p99": float(np.percentile(b, 99))})
        out["cache"] = self.stats
        out["cache_us_per_call"] = 1e6 * self.cache_seconds / max(self.cache_calls, 1)
        return out


def replay(tr: wl.AgentTrace, policy: str, num_pages: int, *, chunk_tokens: int = 1024, decode_ticks: int = 2,
           completion_signals: bool = True, gpu: bool = True, on_batch=None, max_ticks: int = 1_000_000,
           host_pages: int = 0, layer_gemms: tuple | None = None, tier_width: int = 0) -> ReplayResult:
    """Run the trace; `on_batch(requests, q, out)` sees each GPU batch (requests:
    list of TurnRecord, q / out: the batch's [rows, Hq, d] tensors).  With
    `layer_gemms` = (hidden, ffn), each batch's timed region also runs the
    projection and MLP GEMMs of one transformer layer (torch bf16 matmuls with
    random weights) for its uncached tokens, so that the batch time is the
    recompute cost of a whole layer rather than of its attention alone."""
    res = ReplayResult(policy)
    tiered = host_pages > 0
    cache = kvx.kvx_cache_create_tiered(num_pages, host_pages, wl.PAGE_SIZE, chunk_tokens, POLICIES[policy])
    if tier_width:
        kvx.kvx_cache_set_recency_tiers(cache, tier_width)
    if tr.shared >= wl.PAGE_SIZE:  # every agent shares the common system prompt's pages
        for a in range(tr.num_agents):
            kvx.kvx_cache_join(cache, a, 0, tr.shared)
    pool = None
    torch = None
    host = None
    if gpu:
        import torch  # noqa: F811  (device memory and streams only)
        pool = kvx.kv_pool_create(num_pages, wl.PAGE_SIZE, tr.num_kv_heads, tr.head_dim)
        if tiered:
            host = torch.empty(host_pages * kvx.kv_pool_record_bytes(pool), dtype=torch.uint8, pin_memory=True)
    tier = (host, host_pages)
    if gpu:
        _warmup(tr, pool, torch, tier)
    gemm = None
    if gpu and layer_gemms is not None:
        H, F = layer_gemms
        g = torch.Generator(device="cuda").manual_seed(11)
        qkv = (tr.num_q_heads + 2 * tr.num_kv_heads) * tr.head_dim

        def wgt(a, b):
            return (torch.randn((a, b), generator=g, device="cuda") * a ** -0.5).to(torch.bfloat16)

        gemm = {"x": H, "w_qkv": wgt(H, qkv), "w_o": wgt(tr.num_q_heads * tr.head_dim, H),
                "w_gu": wgt(H, 2 * F), "w_d": wgt(F, H)}
    n = tr.num_agents
    turns = len(tr.new[0])
    ctx = [0] * n
    turn = [0] * n
    due = list(tr.start)          # tick at which the next turn may start
    running_until = [-1] * n      # tick at which the running turn ends, -1 = idle
    done = [False] * n
    try:
        tick = 0
        while not all(done):
            if tick > max_ticks:
                raise RuntimeError("replay did not finish (capacity below the active demand?)")
            for a in range(n):
                if running_until[a] == tick:
                    t0 = time.perf_counter()
                    kvx.kvx_cache_end_turn(cache, a)
                    res.cache_seconds += time.perf_counter() - t0
                    res.cache_calls += 1
                    res.events.append(("end", a))
                    running_until[a] = -1
                    ctx[a] += tr.reply[a][turn[a]]
                    due[a] = tick + tr.idle[a][turn[a]]
                    turn[a] += 1
                    if turn[a] == turns:
                        done[a] = True
                        if completion_signals:
                            kvx.kvx_cache_complete(cache, a)
                            res.events.append(("complete", a))
            batch = []
            moves = []  # page moves of this tick's turn starts, in call order
            for a in range(n):
                if done[a] or running_until[a] >= 0 or due[a] > tick:
                    continue
                prompt = ctx[a] + tr.new[a][turn[a]]
                t0 = time.perf_counter()
                mv = None
                try:
                    if tiered:
                        prefix, table, mv = kvx.kvx_cache_begin_turn_tiered(cache, a, prompt)
                    else:
                        prefix, table = kvx.kvx_cache_begin_turn(cache, a, prompt)
                except kvx.KvxError as e:
                    res.cache_seconds += time.perf_counter() - t0
                    res.cache_calls += 1
                    if e.status != kvx.KVX_ENOMEM:
                        raise
                    if isinstance(e, kvx.KvxNoMemory):  # its spills still run
                        moves.append(e.moves)
                        res.moves.append((len(e.moves["spill_pages"]), 0))
                    res.events.append(("begin", a, prompt, None))
                    continue  # waits for pages to free up
                res.cache_seconds += time.perf_counter() - t0
                res.cache_calls += 1
                res.events.append(("begin", a, prompt, prefix))
                reloaded = 0
                if mv is not None:
                    moves.append(mv)
                    res.moves.append((len(mv["spill_pages"]), len(mv["reload_pages"])))
                    reloaded = len(mv["reload_pages"]) * wl.PAGE_SIZE
                rec = TurnRecord(a, turn[a], tick, prompt, prefix, ctx[a], reloaded)
                res.turns.append(rec)
                batch.append((rec, table))
                running_until[a] = tick + decode_ticks
                ctx[a] = prompt
            if (batch or moves) and gpu:
                ms = _run_batch(tr, pool, batch, on_batch, torch, moves, tier, gemm)
                if batch:
                    res.batch_ms.append(ms)
            tick += 1
        res.stats = kvx.kvx_cache_stats(cache)
    finally:
        kvx.kvx_cache_destroy(cache)
        if pool is not None:
            kvx.kv_pool_destroy(pool)
    return res


def _warmup(tr, pool, torch, tier):
    """Run every kernel a batch may use once, untimed, so that no batch pays for
    loading code: store_kv, a short and a split extend_attention, the page moves."""
    n = min(int(kvx.kv_pool_layout(pool)["num_pages"]), 4096 // wl.PAGE_SIZE + 2)
    ids = torch.arange(n, dtype=torch.int32, device="cuda")
    for P, E in ((0, 64), ((n - 2) * wl.PAGE_SIZE, 16)):
        b = kvx.Batch([P], [E], [0, n], ids)
        k = torch.zeros((E, tr.num_kv_heads, tr.head_dim), dtype=torch.bfloat16, device="cuda")
        q = torch.zeros((E, tr.num_q_heads, tr.head_dim), dtype=torch.bfloat16, device="cuda")
        kvx.store_kv(pool, b, k, k)
        kvx.extend_attention(pool, b, q, tr.num_q_heads, tr.sm_scale, torch.empty_like(q))
    host, host_pages = tier
    if host is not None:
        kvx.kv_pool_spill(pool, [0], [0], host, host_pages)
        kvx.kv_pool_reload(pool, [0], [0], host, host_pages)
    torch.cuda.synchronize()


def _run_moves(pool, moves, tier, kvx_mod=kvx):
    host, host_pages = tier
    for mv in moves:  # in call order: a later call may reuse records an earlier one reloaded from
        if len(mv["spill_pages"]):
            kvx_mod.kv_pool_spill(pool, mv["spill_pages"], mv["spill_slots"], host, host_pages)
        if len(mv["reload_pages"]):
            kvx_mod.kv_pool_reload(pool, mv["reload_pages"], mv["reload_slots"], host, host_pages)


GEMM_BUCKET = 512  # GEMM rows are padded to a multiple of this (one library kernel choice per bucket)


def _layer_inputs(gemm, T, torch):
    """N(0, 1) activations for T tokens, grown outside the timed region, and one
    untimed run of the bucket's GEMMs the first time it is used (the library
    picks and loads its kernels per shape)."""
    m = -(-T // GEMM_BUCKET) * GEMM_BUCKET
    if gemm.get("x_buf") is None or gemm["x_buf"].shape[0] < m:
        n = max(m, 2 * (0 if gemm.get("x_buf") is None else gemm["x_buf"].shape[0]))
        gemm["x_buf"] = torch.randn((n, gemm["x"]), device="cuda").to(torch.bfloat16)
        gemm["o_buf"] = torch.randn((n, gemm["w_o"].shape[0]), device="cuda").to(torch.bfloat16)
    seen = gemm.setdefault("seen", set())
    if m not in seen:
        seen.add(m)
        _layer_gemms(gemm, T, torch)


def _layer_gemms(gemm, T, torch):
    """Projection and MLP GEMMs of one layer for T tokens (padded to the bucket;
    values unused)."""
    m = -(-T // GEMM_BUCKET) * GEMM_BUCKET
    x = gemm["x_buf"][:m]
    torch.matmul(x, gemm["w_qkv"])
    o = torch.matmul(gemm["o_buf"][:m], gemm["w_o"])
    gu = torch.matmul(o, gemm["w_gu"])
    f = gemm["w_d"].shape[0]
    torch.matmul(torch.nn.functional.silu(gu[:, :f]) * gu[:, f:], gemm["w_d"])


def _run_batch(tr, pool, batch, on_batch, torch, moves=(), tier=(None, 0), gemm=None) -> float:
    dev = "cuda"
    if not batch:  # only spills of failed turn starts
        _run_moves(pool, moves, tier)
        return 0.0
    P = np.array([r.prefix for r, _ in batch], np.int32)
    E = np.array([r.uncached for r, _ in batch], np.int32)
    indptr = np.zeros(len(batch) + 1, np.int32)
    indptr[1:] = np.cumsum([len(t) for _, t in batch])
    ids = torch.from_numpy(np.concatenate([t for _, t in batch]).astype(np.int32)).to(dev)
    b = kvx.Batch(P, E, indptr, ids.data_ptr())
    k_ext, v_ext, q = [], [], []
    for r, _ in batch:
        k, v = wl.agent_kv(tr, r.agent, r.prompt, dev)
        k_ext.append(k[r.prefix:])
        v_ext.append(v[r.prefix:])
        q.append(wl.agent_q(tr, r.agent, r.turn, r.uncached, dev))
    k_ext = torch.cat(k_ext).contiguous()
    v_ext = torch.cat(v_ext).contiguous()
    q = torch.cat(q).contiguous()
    out = torch.empty_like(q)
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    if gemm is not None:
        _layer_inputs(gemm, int(E.sum()), torch)
    e0.record(stream)
    _run_moves(pool, moves, tier)
    kvx.store_kv(pool, b, k_ext, v_ext)
    kvx.extend_attention(pool, b, q, tr.num_q_heads, tr.sm_scale, out)
    if gemm is not None:
        _layer_gemms(gemm, int(E.sum()), torch)
    e1.record(stream)
    e1.synchronize()
    if on_batch is not None:
        on_batch([r for r, _ in batch], q, out)
    return e0.elapsed_time(e1)


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--policy", choices=["lru", "rr", "both"], default="both")
    ap.add_argument("--agents", type=int, default=48)
    ap.add_argument("--turns", type=int, default=8)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--capacity", type=float, default=0.5,
                    help="pool size as a fraction of the summed final contexts of all agents")
    ap.add_argument("--pool-tokens", type=int, default=0,
                    help="pool size in tokens (overrides --capacity; a fixed pool for concurrency sweeps)")
    ap.add_argument("--chunk-tokens", type=int, default=1024)
    ap.add_argument("--decode-ticks", type=int, default=2)
    ap.add_argument("--heads", default="32,8,128", help="Hq,Hkv,head_dim")
    ap.add_argument("--host-pages", type=float, default=0.0,
                    help="host tier size as a multiple of the device pool (0: no host tier)")
    ap.add_argument("--layer-gemms", default="",
                    help="hidden,ffn: time each batch with one layer's projection + MLP GEMMs (e.g. 4096,14336)")
    ap.add_argument("--no-completion", action="store_true", help="agents send no completion signal")
    ap.add_argument("--shared", type=int, default=0, help="tokens of a system prompt every agent shares")
    ap.add_argument("--tiers", type=int, default=0, help="recency tier width for rr (logical clock ticks; 0: off)")
    ap.add_argument("--no-gpu", action="store_true")
    args = ap.parse_args(argv)
    lg = tuple(int(x) for x in args.layer_gemms.split(",")) if args.layer_gemms else None
    hq, hkv, d = (int(x) for x in args.heads.split(","))
    tr = wl.make_agent_trace(args.agents, args.turns, seed=args.seed, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                             shared=args.shared)
    total = sum(tr.max_context(i) for i in range(tr.num_agents))
    num_pages = (args.pool_tokens if args.pool_tokens > 0 else int(args.capacity * total)) // wl.PAGE_SIZE
    for pol in (["lru", "rr"] if args.policy == "both" else [args.policy]):
        host_pages = int(args.host_pages * num_pages)
        r = replay(tr, pol, num_pages, chunk_tokens=args.chunk_tokens, decode_ticks=args.decode_ticks,
                   gpu=not args.no_gpu, host_pages=host_pages, layer_gemms=lg,
                   completion_signals=not args.no_completion, tier_width=args.tiers if pol == "rr" else 0)
        s = r.summary()
        s.update({"agents": args.agents, "turns_per_agent": args.turns, "num_pages": num_pages, "host_pages": host_pages,
                  "layer_gemms": list(lg) if lg else None,
                  "completion_signals": not args.no_completion, "shared": args.shared, "tiers": args.tiers if pol == "rr" else 0,
                  "context_tokens_total": total, "heads": [hq, hkv, d], "chunk_tokens": args.chunk_tokens})
        print(json.dumps(s), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
