"""The library's token-content prefix cache (kvx_radix, include/kvx_radix.h) in
lockstep with the oracle (oracle/radix.py) on seeded branching multi-agent traces
-- no GPU: every request's reused prefix and page table, every counter after every
call, and the longest-prefix probe must agree -- plus its argument errors."""

import numpy as np
import pytest

from oracle import radix as R
from paper_2609_32278_amd import kvx

PAGE = 16


def _branching_trace(seed, agents=6, steps=160):
    """Agents that share a system prompt, extend private histories turn by turn, and
    now and then branch: resume from an earlier point of their own history (a retry)
    or fork another agent's history.  Returns (op, agent, tokens) events."""
    rng = np.random.default_rng([43, seed])
    system = list(rng.integers(0, 50_000, 3 * PAGE + 5))
    hist = {a: list(system) for a in range(agents)}
    running = set()
    events = []
    for _ in range(steps):
        a = int(rng.integers(0, agents))
        if a in running:
            events.append(("end", a, None))
            running.discard(a)
            continue
        u = rng.random()
        if u < 0.1 and len(hist[a]) > len(system) + 8:
            hist[a] = hist[a][: int(rng.integers(len(system), len(hist[a])))]  # retry from earlier
        elif u < 0.15:
            b = int(rng.integers(0, agents))
            hist[a] = list(hist[b][: int(rng.integers(1, len(hist[b]) + 1))])  # fork another history
        elif u < 0.18:
            events.append(("complete", a, None))
            continue
        hist[a] = hist[a] + list(rng.integers(0, 50_000, int(rng.integers(1, 120))))
        events.append(("begin", a, list(hist[a])))
        running.add(a)
    return events


@pytest.mark.parametrize("policy", [kvx.KVX_EVICT_RR, kvx.KVX_EVICT_LRU])
@pytest.mark.parametrize("seed", range(5))
def test_library_matches_the_oracle_step_by_step(policy, seed):
    events = _branching_trace(seed)
    num_pages, chunk = 90, 2 * PAGE
    o = R.OracleRadix(num_pages, PAGE, chunk, R.RR if policy == kvx.KVX_EVICT_RR else R.LRU)
    t = kvx.kvx_radix_create(num_pages, PAGE, chunk, policy)
    fails = begins = reused = 0
    try:
        for op, a, tokens in events:
            if op == "begin":
                begins += 1
                try:
                    want = o.begin(a, tokens)
                except R.NoMemory:
                    want = None
                try:
                    p, table = kvx.kvx_radix_begin(t, a, tokens)
                    got = (p, list(table))
                except kvx.KvxError as e:
                    assert e.status == kvx.KVX_ENOMEM
                    got = None
                assert got == want, (op, a, len(tokens))
                fails += want is None
                reused += bool(want and want[0] > 0)
            elif op == "end":
                if a in o.running:
                    o.end(a)
                    kvx.kvx_radix_end(t, a)
            else:
                if a not in o.running:
                    o.complete(a)
                    kvx.kvx_radix_complete(t, a)
            st = kvx.kvx_radix_stats(t)
            want_st = o.stats()
            assert {k: st[k] for k in want_st} == want_st
            assert st["free_pages"] + st["cached_pages"] + st["temp_pages"] == num_pages
            if tokens is not None:
                for probe in (tokens, tokens[: len(tokens) // 2 + 1]):
                    m_lib, m_or = kvx.kvx_radix_match(t, probe), o.match(probe)
                    assert m_lib[0] == m_or[0] and list(m_lib[1]) == m_or[1]
        assert o.evictions > 0 and reused > 0  # the trace exercises eviction and reuse
    finally:
        kvx.kvx_radix_destroy(t)


def test_argument_errors():
    with pytest.raises(kvx.KvxError) as e:
        kvx.kvx_radix_create(0, PAGE, PAGE, kvx.KVX_EVICT_RR)
    assert e.value.status == kvx.KVX_EINVAL
    with pytest.raises(kvx.KvxError) as e:
        kvx.kvx_radix_create(10, 8, PAGE, kvx.KVX_EVICT_RR)
    assert e.value.status == kvx.KVX_EUNSUPPORTED
    with pytest.raises(kvx.KvxError):
        kvx.kvx_radix_create(10, PAGE, 24, kvx.KVX_EVICT_RR)
    with pytest.raises(kvx.KvxError):
        kvx.kvx_radix_create(10, PAGE, PAGE, 9)
    t = kvx.kvx_radix_create(10, PAGE, PAGE, kvx.KVX_EVICT_RR)
    try:
        with pytest.raises(kvx.KvxError):
            kvx.kvx_radix_begin(t, 1, [])
        kvx.kvx_radix_begin(t, 1, list(range(40)))
        with pytest.raises(kvx.KvxError) as e:
            kvx.kvx_radix_begin(t, 1, list(range(40)))  # already running
        assert e.value.status == kvx.KVX_EINVAL
        with pytest.raises(kvx.KvxError):
            kvx.kvx_radix_complete(t, 1)  # running
        with pytest.raises(kvx.KvxError):
            kvx.kvx_radix_end(t, 2)  # not running
        with pytest.raises(kvx.KvxError) as e:
            kvx.kvx_radix_begin(t, 3, list(range(1000, 1200)))  # 13 pages of 10
        assert e.value.status == kvx.KVX_ENOMEM
        kvx.kvx_radix_end(t, 1)
        assert kvx.kvx_radix_stats(t)["active"] == 0
    finally:
        kvx.kvx_radix_destroy(t)
