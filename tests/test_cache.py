"""The library's prefix cache (include/kvx_cache.h) against the eviction oracle on
random multi-agent traces: identical reuse decisions, cached histories and
counters after every call; page tables that are valid, disjoint and stable."""

import os

import numpy as np
import pytest

from oracle.evict import NoMemory, OracleCache
from paper_2609_32278_amd import kvx

PAGE = 16


@pytest.fixture(scope="module", autouse=True)
def _built():
    if not os.path.exists(kvx.LIB_PATH):
        from paper_2609_32278_amd import build
        build.build()


def _err(fn, *a):
    with pytest.raises(kvx.KvxError) as e:
        fn(*a)
    return e.value.status


def test_argument_errors():
    assert _err(kvx.kvx_cache_create, 0, 16, 1024, kvx.KVX_EVICT_RR) == kvx.KVX_EINVAL
    assert _err(kvx.kvx_cache_create, 64, 8, 1024, kvx.KVX_EVICT_RR) == kvx.KVX_EUNSUPPORTED
    assert _err(kvx.kvx_cache_create, 64, 16, 24, kvx.KVX_EVICT_RR) == kvx.KVX_EINVAL
    assert _err(kvx.kvx_cache_create, 64, 16, 1024, 5) == kvx.KVX_EINVAL
    c = kvx.kvx_cache_create(64, 16, 64, kvx.KVX_EVICT_RR)
    try:
        assert _err(kvx.kvx_cache_begin_turn, c, 1, 0) == kvx.KVX_EINVAL
        assert _err(kvx.kvx_cache_end_turn, c, 1) == kvx.KVX_EINVAL      # not inside a turn
        assert _err(kvx.kvx_cache_complete, c, 1) == kvx.KVX_EINVAL      # unknown
        kvx.kvx_cache_begin_turn(c, 1, 40)
        assert _err(kvx.kvx_cache_begin_turn, c, 1, 50) == kvx.KVX_EINVAL  # already active
        assert _err(kvx.kvx_cache_complete, c, 1) == kvx.KVX_EINVAL      # active
        ids = np.zeros(2, np.int32)
        prefix = kvx.ctypes.c_int32()
        st = kvx.lib().kvx_cache_begin_turn(c, 2, 100, kvx.ctypes.byref(prefix), ids.ctypes.data, 2)
        assert st == kvx.KVX_EINVAL                                       # page_ids too short
        assert kvx.kvx_cache_stats(c)["agents"] == 1                      # checked before any change
        assert _err(kvx.kvx_cache_begin_turn, c, 3, 65 * PAGE) == kvx.KVX_ENOMEM
    finally:
        kvx.kvx_cache_destroy(c)


class _Pair:
    """The library cache and the oracle, driven in lockstep."""

    def __init__(self, num_pages, chunk_tokens, policy, tier_width=0):
        self.c = kvx.kvx_cache_create(num_pages, PAGE, chunk_tokens, policy)
        if tier_width:
            kvx.kvx_cache_set_recency_tiers(self.c, tier_width)
        self.o = OracleCache(num_pages, PAGE, chunk_tokens, OracleCache.RR if policy == kvx.KVX_EVICT_RR
                             else OracleCache.LRU, tier_width=tier_width)
        self.num_pages = num_pages
        self.tables = {}  # active agent -> page table of its running turn

    def close(self):
        kvx.kvx_cache_destroy(self.c)

    def begin(self, agent, prompt):
        cached_before, pages_before = kvx.kvx_cache_agent(self.c, agent)
        try:
            want = self.o.begin_turn(agent, prompt)
        except NoMemory:
            want = None
        if want is None:
            with pytest.raises(kvx.KvxError) as e:
                kvx.kvx_cache_begin_turn(self.c, agent, prompt)
            assert e.value.status == kvx.KVX_ENOMEM
            return None
        prefix, table = kvx.kvx_cache_begin_turn(self.c, agent, prompt)
        assert prefix == want
        assert len(table) == -(-prompt // PAGE)
        # the reused prefix keeps its physical pages
        assert (table[: prefix // PAGE] == pages_before[: prefix // PAGE]).all()
        self.tables[agent] = table
        return prefix

    def end(self, agent):
        self.o.end_turn(agent)
        kvx.kvx_cache_end_turn(self.c, agent)
        table = self.tables.pop(agent)
        cached, pages = kvx.kvx_cache_agent(self.c, agent)
        assert (pages == table[: cached // PAGE]).all()  # the turn's whole pages stay, in order

    def complete(self, agent):
        self.o.complete(agent)
        kvx.kvx_cache_complete(self.c, agent)

    def check(self):
        st = kvx.kvx_cache_stats(self.c)
        assert st["free_pages"] == self.o.free
        assert st["evicted_pages"] == self.o.evicted_pages
        assert st["evictions"] == self.o.evictions
        assert st["agents"] == len(self.o.agents)
        owned = []
        for a in self.o.agents:
            cached, pages = kvx.kvx_cache_agent(self.c, a)
            assert cached == self.o.cached_tokens(a)
            owned.extend(pages.tolist())
        for a, t in self.tables.items():
            cached, _ = kvx.kvx_cache_agent(self.c, a)
            owned.extend(t[cached // PAGE:].tolist())  # the running turn's fresh pages
        assert len(owned) == len(set(owned)), "a page is owned twice"
        assert all(0 <= p < self.num_pages for p in owned)
        assert len(owned) + st["free_pages"] == self.num_pages


def _trace(seed, policy, n_agents, num_pages, chunk_tokens, steps, tier_width=0, complete_prob=0.05):
    rng = np.random.default_rng(seed)
    pair = _Pair(num_pages, chunk_tokens, policy, tier_width)
    ctx = {}
    active = set()
    try:
        for _ in range(steps):
            a = int(rng.integers(n_agents))
            r = rng.random()
            if a in active:
                if r < 0.85:
                    pair.end(a)
                    active.discard(a)
                    ctx[a] += int(rng.integers(0, 300))  # the model's reply joins the context
            elif a in ctx and r < complete_prob:
                pair.complete(a)
                del ctx[a]
            else:
                prompt = ctx.get(a, int(rng.integers(1, 400))) + int(rng.integers(1, 600))
                if pair.begin(a, prompt) is not None:
                    active.add(a)
                    ctx[a] = prompt
            pair.check()
    finally:
        pair.close()


@pytest.mark.parametrize("seed", range(3))
@pytest.mark.parametrize("tier_width", [1, 7, 60])
def test_recency_tiers_match_the_oracle(seed, tier_width):
    """Round robin with recency tiers and no completion signals (the case tiers exist for)."""
    _trace(seed, kvx.KVX_EVICT_RR, n_agents=16, num_pages=400, chunk_tokens=32, steps=800,
           tier_width=tier_width, complete_prob=0.0)


def test_recency_tier_errors():
    c = kvx.kvx_cache_create(64, 16, 64, kvx.KVX_EVICT_LRU)
    try:
        assert _err(kvx.kvx_cache_set_recency_tiers, c, 4) == kvx.KVX_EINVAL  # LRU
    finally:
        kvx.kvx_cache_destroy(c)
    c = kvx.kvx_cache_create(64, 16, 64, kvx.KVX_EVICT_RR)
    try:
        assert _err(kvx.kvx_cache_set_recency_tiers, c, -1) == kvx.KVX_EINVAL
        kvx.kvx_cache_set_recency_tiers(c, 0)
    finally:
        kvx.kvx_cache_destroy(c)


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("policy", [kvx.KVX_EVICT_RR, kvx.KVX_EVICT_LRU])
def test_random_traces_match_the_oracle(seed, policy):
    _trace(seed, policy, n_agents=12, num_pages=700, chunk_tokens=64 * (1 + seed % 3), steps=600)


@pytest.mark.parametrize("policy", [kvx.KVX_EVICT_RR, kvx.KVX_EVICT_LRU])
def test_random_traces_under_heavy_pressure(policy):
    """Capacity near the active demand: frequent evictions and failed turn starts."""
    _trace(99, policy, n_agents=30, num_pages=260, chunk_tokens=16, steps=1500)


@pytest.mark.parametrize("policy,expect", [(kvx.KVX_EVICT_RR, "even"), (kvx.KVX_EVICT_LRU, "whole")])
def test_homogeneous_regime_closed_forms(policy, expect):
    """Equations 2 and 3 on the library: n = 10, n a = 4, m = 7 prefixes of u pages."""
    n, na, m = 10, 4, 7
    ns = n - na
    u = 8 * ns
    c = kvx.kvx_cache_create(m * u, PAGE, PAGE, policy)
    try:
        for i in range(ns):
            kvx.kvx_cache_begin_turn(c, i, u * PAGE + 1)
            kvx.kvx_cache_end_turn(c, i)
        for j in range(na):
            kvx.kvx_cache_begin_turn(c, 1000 + j, u * PAGE)
        kept = [kvx.kvx_cache_agent(c, i)[0] / (u * PAGE) for i in range(ns)]
    finally:
        kvx.kvx_cache_destroy(c)
    h = (m - na) / ns
    if expect == "even":
        assert all(abs(k - h) < 1e-12 for k in kept)
    else:
        assert kept == [0.0] * (n - m) + [1.0] * (m - na)


@pytest.mark.parametrize("policy", ["lru", "rr"])
def test_replay_decisions_match_the_oracle(policy):
    """The replay tool's cache calls, re-run through the oracle, give the same reuse."""
    from paper_2609_32278_amd import agent_replay
    from paper_2609_32278_amd import workloads as wl
    tr = wl.make_agent_trace(24, 6, seed=5)
    total = sum(tr.max_context(i) for i in range(tr.num_agents))
    num_pages = int(0.5 * total) // PAGE
    res = agent_replay.replay(tr, policy, num_pages, chunk_tokens=1024, gpu=False)
    o = OracleCache(num_pages, PAGE, 1024, OracleCache.RR if policy == "rr" else OracleCache.LRU)
    for ev in res.events:
        if ev[0] == "begin":
            try:
                got = o.begin_turn(ev[1], ev[2])
            except NoMemory:
                got = None
            assert got == ev[3], ev
        elif ev[0] == "end":
            o.end_turn(ev[1])
        else:
            o.complete(ev[1])
    assert o.evictions == res.stats["evictions"] > 0
    assert len(res.turns) == tr.num_agents * 6


def test_round_robin_spreads_the_loss_on_a_replay():
    """The paper's claim on a synthetic agent workload: round-robin tail eviction
    leaves fewer full misses and a smaller tail of uncached tokens than LRU."""
    from paper_2609_32278_amd import agent_replay
    from paper_2609_32278_amd import workloads as wl
    tr = wl.make_agent_trace(48, 8, seed=0)
    total = sum(tr.max_context(i) for i in range(tr.num_agents))
    num_pages = int(0.6 * total) // PAGE
    s = {p: agent_replay.replay(tr, p, num_pages, gpu=False).summary() for p in ("lru", "rr")}
    assert s["rr"]["full_misses"] < s["lru"]["full_misses"]
    assert s["rr"]["uncached_p99"] < s["lru"]["uncached_p99"]


def test_replay_cli_fixed_pool(capsys):
    """--pool-tokens fixes the pool across a concurrency sweep: the CLI reports that
    pool, and once 28 agents overflow 200k tokens round robin keeps the P99 tail
    below LRU's (seed 0: 7454 vs 12399 uncached tokens)."""
    import json
    from paper_2609_32278_amd import agent_replay
    assert agent_replay.main(["--no-gpu", "--agents", "28", "--turns", "8", "--pool-tokens", "200000"]) == 0
    rows = [json.loads(x) for x in capsys.readouterr().out.splitlines() if x.startswith("{")]
    by = {r["policy"]: r for r in rows}
    assert by["lru"]["num_pages"] == by["rr"]["num_pages"] == 200000 // PAGE
    assert by["rr"]["uncached_p99"] < 0.7 * by["lru"]["uncached_p99"]
    assert by["rr"]["full_misses"] < by["lru"]["full_misses"]


# ------------------------------------------------------------------ host tier

class _TieredPair(_Pair):
    """The library's tiered cache and the oracle in lockstep, plus a model of the
    data: what (agent, logical page) each device page and host record holds, moved
    by the cache's spills and reloads exactly as kv_pool_spill / kv_pool_reload
    would move it, so every reused prefix can be checked to hold the agent's own
    pages in logical order."""

    def __init__(self, num_pages, host_pages, chunk_tokens, policy):
        self.c = kvx.kvx_cache_create_tiered(num_pages, host_pages, PAGE, chunk_tokens, policy)
        self.o = OracleCache(num_pages, PAGE, chunk_tokens, OracleCache.RR if policy == kvx.KVX_EVICT_RR
                             else OracleCache.LRU, host_pages=host_pages)
        self.num_pages = num_pages
        self.host_pages = host_pages
        self.tables = {}
        self.dev = {}   # page -> (agent, logical page)
        self.host = {}  # record -> (agent, logical page)

    def begin(self, agent, prompt):
        try:
            want = self.o.begin_turn(agent, prompt)
        except NoMemory:
            want = None
        try:
            prefix, table, mv = kvx.kvx_cache_begin_turn_tiered(self.c, agent, prompt)
        except kvx.KvxNoMemory as e:
            assert want is None
            self._apply(e.moves)
            assert (len(e.moves["spill_pages"]), 0) == self.o.last_moves
            return None
        assert want is not None and prefix == want
        assert (len(mv["spill_pages"]), len(mv["reload_pages"])) == self.o.last_moves
        assert len(set(mv["spill_slots"].tolist())) == len(mv["spill_slots"])
        self._apply(mv)
        n = -(-prompt // PAGE)
        assert len(table) == n and len(set(table.tolist())) == n
        # the reused prefix holds this agent's pages in logical order
        for j in range(prefix // PAGE):
            assert self.dev.get(int(table[j])) == (agent, j), (agent, j)
        # this turn writes its suffix pages (store_kv)
        for j in range(prefix // PAGE, n):
            self.dev[int(table[j])] = (agent, j)
        self.tables[agent] = table
        return prefix

    def _apply(self, mv):
        for pg, rec in zip(mv["spill_pages"], mv["spill_slots"]):
            assert int(pg) in self.dev
            self.host[int(rec)] = self.dev[int(pg)]
        for pg, rec in zip(mv["reload_pages"], mv["reload_slots"]):
            self.dev[int(pg)] = self.host[int(rec)]

    def check(self):
        super().check()
        st = kvx.kvx_cache_stats(self.c)
        for key in ("spilled_pages", "reloaded_pages", "host_dropped_pages", "host_used"):
            assert st[key] == getattr(self.o, key), key
        recs = []
        for a in self.o.agents:
            tok, slots = kvx.kvx_cache_agent_host(self.c, a)
            assert tok == self.o.host_tokens(a)
            cached = kvx.kvx_cache_agent(self.c, a)[0] // PAGE
            for k, r in enumerate(slots.tolist()):
                assert self.host.get(r) == (a, cached + k), "host pages must continue the device prefix"
            recs.extend(slots.tolist())
        assert len(recs) == len(set(recs)) == st["host_used"]
        assert all(0 <= r < self.host_pages for r in recs)


def _tiered_trace(seed, policy, n_agents, num_pages, host_pages, chunk_tokens, steps):
    rng = np.random.default_rng(seed)
    pair = _TieredPair(num_pages, host_pages, chunk_tokens, policy)
    ctx = {}
    active = set()
    try:
        for _ in range(steps):
            a = int(rng.integers(n_agents))
            r = rng.random()
            if a in active:
                if r < 0.85:
                    pair.end(a)
                    active.discard(a)
                    ctx[a] += int(rng.integers(0, 300))
            elif a in ctx and r < 0.05:
                pair.complete(a)
                del ctx[a]
            else:
                grow = int(rng.integers(1, 600)) if r < 0.9 else -int(rng.integers(0, 200))  # sometimes shorter
                prompt = max(1, ctx.get(a, int(rng.integers(1, 400))) + grow)
                if pair.begin(a, prompt) is not None:
                    active.add(a)
                    ctx[a] = prompt
            pair.check()
    finally:
        pair.close()


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("policy", [kvx.KVX_EVICT_RR, kvx.KVX_EVICT_LRU])
@pytest.mark.parametrize("host_pages", [1, 40, 400])
def test_tiered_random_traces_match_the_oracle(seed, policy, host_pages):
    _tiered_trace(seed, policy, n_agents=12, num_pages=500, host_pages=host_pages,
                  chunk_tokens=64 * (1 + seed % 3), steps=500)


@pytest.mark.parametrize("policy", [kvx.KVX_EVICT_RR, kvx.KVX_EVICT_LRU])
def test_tiered_traces_under_heavy_pressure(policy):
    _tiered_trace(98, policy, n_agents=30, num_pages=260, host_pages=120, chunk_tokens=16, steps=1500)


def test_tiered_argument_errors():
    assert _err(kvx.kvx_cache_create_tiered, 64, -1, 16, 64, kvx.KVX_EVICT_RR) == kvx.KVX_EINVAL
    c = kvx.kvx_cache_create_tiered(64, 8, 16, 64, kvx.KVX_EVICT_RR)
    try:
        assert _err(kvx.kvx_cache_begin_turn, c, 1, 40) == kvx.KVX_EINVAL  # spills would be lost
        ids = np.zeros(4, np.int32)
        prefix = kvx.ctypes.c_int32()
        st = kvx.lib().kvx_cache_begin_turn_tiered(c, 1, 40, kvx.ctypes.byref(prefix), ids.ctypes.data, 4, None)
        assert st == kvx.KVX_EINVAL
        assert kvx.kvx_cache_stats(c)["agents"] == 0
    finally:
        kvx.kvx_cache_destroy(c)


# ------------------------------------------------------------------ shared prefixes

class _GroupPair(_TieredPair):
    """_TieredPair with shared-prefix groups: a shared page holds the group's
    content ('G', group, j), the same whichever member computed it."""

    def __init__(self, num_pages, host_pages, chunk_tokens, policy, groups):
        super().__init__(num_pages, host_pages, chunk_tokens, policy)
        self.groups = groups      # group -> shared pages S
        self.member = {}          # agent -> group

    def join(self, agent, group):
        S = self.groups[group]
        self.o.join(agent, group, S * PAGE)
        kvx.kvx_cache_join(self.c, agent, group, S * PAGE + 7)  # rounds down to whole pages
        self.member[agent] = group

    def _content(self, agent, j):
        g = self.member.get(agent)
        return ("G", g, j) if g is not None and j < self.groups[g] else (agent, j)

    def begin(self, agent, prompt):
        try:
            want = self.o.begin_turn(agent, prompt)
        except NoMemory:
            want = None
        try:
            prefix, table, mv = kvx.kvx_cache_begin_turn_tiered(self.c, agent, prompt)
        except kvx.KvxNoMemory as e:
            assert want is None
            self._apply(e.moves)
            return None
        assert want is not None and prefix == want
        assert (len(mv["spill_pages"]), len(mv["reload_pages"])) == self.o.last_moves
        self._apply(mv)
        n = -(-prompt // PAGE)
        assert len(table) == n and len(set(table.tolist())) == n
        for j in range(prefix // PAGE):
            assert self.dev.get(int(table[j])) == self._content(agent, j), (agent, j)
        for j in range(prefix // PAGE, n):
            self.dev[int(table[j])] = self._content(agent, j)
        self.tables[agent] = table
        return prefix

    def end(self, agent):
        self.o.end_turn(agent)
        kvx.kvx_cache_end_turn(self.c, agent)
        self.tables.pop(agent)

    def check(self):
        st = kvx.kvx_cache_stats(self.c)
        assert st["free_pages"] == self.o.free
        assert st["evicted_pages"] == self.o.evicted_pages
        assert st["evictions"] == self.o.evictions
        assert st["group_pages"] == sum(self.o.group_tokens(g) for g in self.groups) // PAGE
        owned = []
        for g in self.groups:
            tok, pages = kvx.kvx_cache_group(self.c, g)
            assert tok == self.o.group_tokens(g)
            for j, pg in enumerate(pages.tolist()):
                assert self.dev.get(pg) == ("G", g, j)
            owned.extend(pages.tolist())
        for a in self.o.agents:
            cached, pages = kvx.kvx_cache_agent(self.c, a)
            assert cached == self.o.cached_tokens(a)
            g = self.member.get(a)
            start = self.groups[g] if g is not None else 0
            for k, pg in enumerate(pages.tolist()):
                assert self.dev.get(pg) == self._content(a, start + k)
            owned.extend(pages.tolist())
        for a, t in self.tables.items():
            # the running turn's own pages: everything past the shared pages and cached ones it reuses
            g = self.member.get(a)
            shared = set(kvx.kvx_cache_group(self.c, g)[1].tolist()) if g is not None else set()
            cached = set(kvx.kvx_cache_agent(self.c, a)[1].tolist())
            owned.extend(p for p in t.tolist() if p not in shared and p not in cached)
        assert len(owned) == len(set(owned)), "a page is owned twice"
        assert len(owned) + st["free_pages"] == self.num_pages


def _group_trace(seed, policy, host_pages, steps=700):
    rng = np.random.default_rng(seed)
    groups = {0: 6, 1: 3}
    pair = _GroupPair(400, host_pages, 32, policy, groups)
    ctx, active, known = {}, set(), set()
    try:
        for _ in range(steps):
            a = int(rng.integers(14))
            r = rng.random()
            if a not in known:
                known.add(a)
                if a % 3 != 2:                       # two agents in three share a prompt
                    pair.join(a, a % 2)
            if a in active:
                if r < 0.85:
                    pair.end(a)
                    active.discard(a)
                    ctx[a] += int(rng.integers(0, 300))
            elif a in ctx and r < 0.04:
                pair.complete(a)
                del ctx[a]
                known.discard(a)
                pair.member.pop(a, None)
            else:
                g = pair.member.get(a)
                base = pair.groups[g] * PAGE + int(rng.integers(0, 40)) if g is not None else int(rng.integers(1, 400))
                prompt = ctx.get(a, base) + int(rng.integers(1, 500))
                if r > 0.97:
                    prompt = int(rng.integers(1, 60))  # now and then a prompt inside the shared span
                if pair.begin(a, prompt) is not None:
                    active.add(a)
                    ctx[a] = prompt
            pair.check()
    finally:
        pair.close()
    return pair


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("policy", [kvx.KVX_EVICT_RR, kvx.KVX_EVICT_LRU])
@pytest.mark.parametrize("host_pages", [0, 60])
def test_shared_prefix_traces_match_the_oracle(seed, policy, host_pages):
    _group_trace(seed, policy, host_pages)


def test_join_errors():
    c = kvx.kvx_cache_create(64, 16, 64, kvx.KVX_EVICT_RR)
    try:
        assert _err(kvx.kvx_cache_join, c, 1, 0, 15) == kvx.KVX_EINVAL     # below one page
        kvx.kvx_cache_join(c, 1, 0, 64)
        assert _err(kvx.kvx_cache_join, c, 1, 0, 64) == kvx.KVX_EINVAL     # already a member
        assert _err(kvx.kvx_cache_join, c, 2, 0, 80) == kvx.KVX_EINVAL     # other span
        kvx.kvx_cache_begin_turn(c, 3, 40)
        assert _err(kvx.kvx_cache_join, c, 3, 0, 64) == kvx.KVX_EINVAL     # inside a turn
        kvx.kvx_cache_end_turn(c, 3)
        assert _err(kvx.kvx_cache_join, c, 3, 0, 64) == kvx.KVX_EINVAL     # holds pages
        assert kvx.kvx_cache_group(c, 0)[0] == 0 and kvx.kvx_cache_group(c, 5)[0] == 0
    finally:
        kvx.kvx_cache_destroy(c)
