"""Pins of the eviction oracle (oracle/evict.py) against the paper: the closed
forms of the homogeneous analysis (Section 3.3, Equations 1-3) and hand-traced
runs of Algorithm 1 and of the LRU baseline on toy histories."""

import pytest

from oracle.evict import NoMemory, OracleCache

PAGE = 16


def _fill(cache, agent, pages):
    """One turn that leaves `pages` whole pages cached for `agent`."""
    cache.begin_turn(agent, pages * PAGE + 1)
    cache.end_turn(agent)


def _homogeneous(policy, n, na, m, u, chunk_pages):
    """n trajectories of u pages each; ns = n - na idle ones cached first, then na
    fresh active ones start turns that need their whole prompt; capacity m * u pages
    (Section 3.3's model, with every idle prefix one unit)."""
    ns = n - na
    c = OracleCache(m * u, PAGE, chunk_pages * PAGE, policy)
    for i in range(ns):
        _fill(c, i, u)
    for j in range(na):
        c.begin_turn(1000 + j, u * PAGE)  # u pages, prefix 0, active
    return c, [c.cached_tokens(i) / (u * PAGE) for i in range(ns)]


# (n, na, m): na < m < n (Equation 1) and ns <= m so every idle prefix fits first
REGIME = [(10, 4, 7), (12, 4, 9), (20, 8, 15), (6, 2, 5)]


@pytest.mark.parametrize("n,na,m", REGIME)
def test_round_robin_keeps_the_same_fraction_of_every_idle_prefix(n, na, m):
    """Equation 2: ideal round-robin retains h = (m - na) / (n s) of every idle prefix."""
    ns = n - na
    u = 8 * ns  # (n - m) * u pages split evenly over ns agents
    c, kept = _homogeneous(OracleCache.RR, n, na, m, u, chunk_pages=1)
    h = (m - na) / ns
    assert all(abs(k - h) < 1e-12 for k in kept), (kept, h)
    q = 1 - h
    assert abs(q - (n - m) / ns) < 1e-12
    # Equation 3: X_RR = q for every returning idle agent
    assert all(abs((1 - k) - q) < 1e-12 for k in kept)


@pytest.mark.parametrize("n,na,m", REGIME)
def test_round_robin_with_coarse_chunks_stays_within_one_chunk(n, na, m):
    ns = n - na
    u = 64
    chunk = 8
    c, kept = _homogeneous(OracleCache.RR, n, na, m, u, chunk_pages=chunk)
    h = (m - na) / ns
    assert all(abs(k - h) <= chunk / u + 1e-12 for k in kept), (kept, h)


@pytest.mark.parametrize("n,na,m", REGIME)
def test_lru_removes_whole_prefixes_of_a_fraction_q(n, na, m):
    """Equation 3: LRU retains m - na idle prefixes whole and loses n - m whole."""
    ns = n - na
    c, kept = _homogeneous(OracleCache.LRU, n, na, m, 16, chunk_pages=1)
    assert sorted(kept) == [0.0] * (n - m) + [1.0] * (m - na)
    # the least recently used ones go first
    assert kept[: n - m] == [0.0] * (n - m)
    q = (n - m) / ns
    x = [1 - k for k in kept]
    assert abs(sum(x) / ns - q) < 1e-12  # E[X_LRU] = q
    assert abs(sum(x) / ns - (1 - sum(_homogeneous(OracleCache.RR, n, na, m, 8 * ns, 1)[1]) / ns)) < 1e-12


@pytest.mark.parametrize("policy", [OracleCache.LRU, OracleCache.RR])
def test_no_eviction_when_everything_fits(policy):
    """m >= n: eviction is unnecessary (Equation 1's upper bound)."""
    n, na, u = 8, 3, 32
    c, kept = _homogeneous(policy, n, na, n, u, 1)
    assert kept == [1.0] * (n - na) and c.evictions == 0


@pytest.mark.parametrize("policy", [OracleCache.LRU, OracleCache.RR])
def test_active_demand_above_capacity_cannot_be_met(policy):
    """m < na: active trajectories alone exceed the capacity (Equation 1's lower bound)."""
    n, na, m, u = 8, 5, 4, 16
    c = OracleCache(m * u, PAGE, PAGE, policy)
    for i in range(n - na):
        _fill(c, i, 1)
    with pytest.raises(NoMemory):
        for j in range(na):
            c.begin_turn(1000 + j, u * PAGE)
    assert all(c.cached_tokens(i) == 0 for i in range(n - na))  # every idle page was given up


def _toy(policy):
    """Agents 1, 2, 3 idle with 5, 1 and 4 cached pages (one node each), 2 pages free."""
    c = OracleCache(12, PAGE, 2 * PAGE, policy)
    _fill(c, 1, 5)
    _fill(c, 2, 1)
    _fill(c, 3, 4)
    assert c.free == 2
    return c


def test_algorithm1_hand_trace():
    """Reclaim 9 pages with 2-page chunks: queue [1, 2, 3];
    1 loses 2 (3 left), 2 loses its last page and leaves the queue, 3 loses 2,
    1 loses 2, 3 loses its last 2 -> 9 freed in 5 steps."""
    c = _toy(OracleCache.RR)
    assert c.begin_turn(9, 11 * PAGE) == 0  # needs 11 pages, 2 free
    assert [c.cached_tokens(i) // PAGE for i in (1, 2, 3)] == [1, 0, 0]
    assert (c.evictions, c.evicted_pages, c.free) == (5, 9, 0)
    assert c.rr_last == 3
    # the next reclamation continues the rotation after agent 3: agent 9 (now idle,
    # 11 pages) comes before agent 1
    c.end_turn(9)
    _fill(c, 4, 1)  # needs 2 pages, none free
    assert (c.cached_tokens(9), c.cached_tokens(1)) == (9 * PAGE, PAGE)


def test_algorithm1_rotation_continues_across_reclamations():
    c = OracleCache(6, PAGE, PAGE, OracleCache.RR)
    for a in (1, 2, 3):
        c.begin_turn(a, 2 * PAGE)  # two whole pages, nothing partial
        c.end_turn(a)
    assert c.free == 0
    order = []
    for k in range(3):  # three one-page reclamations, the new agents stay active
        before = [c.cached_tokens(a) for a in (1, 2, 3)]
        c.begin_turn(10 + k, PAGE)
        after = [c.cached_tokens(a) for a in (1, 2, 3)]
        order.append([a for a, x, y in zip((1, 2, 3), before, after) if y < x])
    assert order == [[1], [2], [3]]


def test_algorithm1_skips_active_trajectories():
    c = _toy(OracleCache.RR)
    c.begin_turn(1, 5 * PAGE + 1)  # agent 1 resumes: active, its 5 pages pinned (needs 1 more)
    assert c.cached_tokens(1) == 5 * PAGE
    c.begin_turn(9, 5 * PAGE)  # needs 5; 1 free -> reclaim 4 from agents 2 and 3 only
    assert c.cached_tokens(1) == 5 * PAGE
    assert [c.cached_tokens(i) // PAGE for i in (2, 3)] == [0, 1]


def test_lru_hand_trace():
    """Same toy history: LRU drops whole leaves oldest first -- agent 1 (5 pages),
    agent 2 (1), agent 3 (4) -- and over-reclaims the last node."""
    c = _toy(OracleCache.LRU)
    c.begin_turn(9, 11 * PAGE)
    assert [c.cached_tokens(i) for i in (1, 2, 3)] == [0, 0, 0]
    assert (c.evictions, c.evicted_pages, c.free) == (3, 10, 1)


def test_lru_takes_a_whole_synchronized_path_before_the_next_agent():
    """Recency synchronization (Section 3.1): all nodes of an agent's path carry
    the time of its last access, so LRU empties one agent node after node."""
    c = OracleCache(64, PAGE, PAGE, OracleCache.LRU)
    c.begin_turn(1, 3 * PAGE + 1); c.end_turn(1)   # node 3 pages
    c.begin_turn(1, 6 * PAGE + 1); c.end_turn(1)   # node 3 more
    c.begin_turn(2, 4 * PAGE + 1); c.end_turn(2)   # node 4 pages
    assert c.agents[1].nodes == [3, 3]
    c.begin_turn(1, 6 * PAGE + 1)  # agent 1 resumes: its whole path is now the newest
    c.end_turn(1)
    free = c.free
    c.begin_turn(3, (free + 5) * PAGE)  # reclaim 5: agent 2 (4, oldest), then agent 1's leaf (3)
    assert c.cached_tokens(2) == 0 and c.agents[1].nodes == [3]


def test_turns_reuse_whole_pages_and_compute_at_least_one_token():
    c = OracleCache(64, PAGE, PAGE, OracleCache.RR)
    assert c.begin_turn(1, 40) == 0
    c.end_turn(1)
    assert c.cached_tokens(1) == 32             # the partial page is not kept
    assert c.begin_turn(1, 100) == 32
    c.end_turn(1)
    assert c.cached_tokens(1) == 96
    assert c.begin_turn(1, 96) == 80            # at least one token computed: page 5 recomputed
    c.end_turn(1)
    assert c.cached_tokens(1) == 96
    c.complete(1)
    assert c.free == 64 and c.cached_tokens(1) == 0


# ------------------------------------------------------------------ host tier

def test_host_tier_hand_trace():
    """Toy history of test_algorithm1_hand_trace with a 3-record host tier: the 9
    pages Algorithm 1 evicts are spilled farthest page first, and each spill that
    finds the tier full drops the oldest idle-owned record (its owner's farthest
    host page).  Traced by hand:
      agent 1 loses pages 5, 4 -> records r1 (p5), r2 (p4)
      agent 2 loses page 1     -> r3
      agent 3 loses pages 4, 3 -> drop r1, r2; r4 (p4), r5 (p3)
      agent 1 loses pages 3, 2 -> drop r3, r4; r6 (p3), r7 (p2)
      agent 3 loses pages 2, 1 -> drop r5, r6; r8 (p2), r9 (p1)
    leaving agent 1 = device p1 + host p2, agent 2 = nothing, agent 3 = host p1, p2.
    r1 .. r6 were written and dropped within this one turn start, so their spills
    are void: only r7, r8, r9 are written."""
    c = OracleCache(12, PAGE, 2 * PAGE, OracleCache.RR, host_pages=3)
    _fill(c, 1, 5)
    _fill(c, 2, 1)
    _fill(c, 3, 4)
    assert c.begin_turn(9, 11 * PAGE) == 0
    assert [c.cached_tokens(i) // PAGE for i in (1, 2, 3)] == [1, 0, 0]
    assert [c.host_tokens(i) // PAGE for i in (1, 2, 3)] == [1, 0, 2]
    assert c.last_moves == (3, 0)
    assert (c.spilled_pages, c.host_dropped_pages, c.host_used) == (3, 0, 3)
    c.end_turn(9)
    # agent 3 returns with a 5-page prompt: both host pages come back, 3 new pages
    free_before = c.free
    assert c.begin_turn(3, 5 * PAGE) == 2 * PAGE
    assert c.last_moves[1] == 2 and c.host_tokens(3) == 0 and c.reloaded_pages == 2
    assert c.host_used == 1


@pytest.mark.parametrize("policy", [OracleCache.RR, OracleCache.LRU])
@pytest.mark.parametrize("n,na,m", REGIME)
def test_a_host_tier_as_large_as_the_histories_loses_nothing(policy, n, na, m):
    """Equation 3 with a host tier holding every idle page: X = 0 for every
    returning agent (each reuses its whole history: device pages + reloads)."""
    ns = n - na
    u = 8 * ns
    c = OracleCache(m * u, PAGE, PAGE, policy, host_pages=n * u)
    for i in range(ns):
        _fill(c, i, u)
    for j in range(na):
        c.begin_turn(1000 + j, u * PAGE)
    assert all(c.cached_tokens(i) + c.host_tokens(i) == u * PAGE for i in range(ns))
    assert c.host_dropped_pages == 0 and c.spilled_pages == (n - m) * u
    for j in range(na):  # the active turns end and their agents finish
        c.end_turn(1000 + j)
        c.complete(1000 + j)
    for i in range(ns):
        host = c.host_tokens(i) // PAGE
        assert c.begin_turn(i, u * PAGE + 1) == u * PAGE
        assert c.last_moves[1] == host
        c.end_turn(i)
    assert c.reloaded_pages == c.spilled_pages


def test_a_host_tier_of_size_zero_changes_nothing():
    runs = []
    for host in (0, None):
        c = OracleCache(12, PAGE, 2 * PAGE, OracleCache.RR) if host is None else \
            OracleCache(12, PAGE, 2 * PAGE, OracleCache.RR, host_pages=0)
        _fill(c, 1, 5)
        _fill(c, 2, 1)
        _fill(c, 3, 4)
        c.begin_turn(9, 11 * PAGE)
        runs.append(([c.cached_tokens(i) for i in (1, 2, 3)], c.evictions, c.free, c.spilled_pages))
    assert runs[0] == runs[1] and runs[0][3] == 0


def test_reuse_past_the_prompt_drops_host_pages_first():
    c = OracleCache(8, PAGE, PAGE, OracleCache.RR, host_pages=8)
    _fill(c, 1, 6)
    c.begin_turn(2, 4 * PAGE)          # 2 free, evicts 2 of agent 1's pages -> host
    assert (c.cached_tokens(1), c.host_tokens(1)) == (4 * PAGE, 2 * PAGE)
    c.end_turn(2)
    c.complete(2)
    assert c.begin_turn(1, 5 * PAGE + 1) == 5 * PAGE  # limit 5: 4 device + 1 reloaded, 1 host dropped
    assert c.last_moves == (0, 1) and c.host_used == 0
    c.end_turn(1)
    assert c.begin_turn(1, 3 * PAGE) == 2 * PAGE       # limit 2: device pages dropped past it
    assert c.last_moves == (0, 0)


def test_records_of_an_agent_inside_a_turn_are_never_dropped():
    """Agent 1 returns and must reload 2 host pages while its own allocation
    evicts a page of agent 2: the tier is full of agent 1's pinned records, so
    agent 2's page is dropped, not spilled."""
    c = OracleCache(7, PAGE, 2 * PAGE, OracleCache.RR, host_pages=2)
    _fill(c, 1, 4)                     # 4 pages kept, 3 free
    _fill(c, 2, 2)                     # 2 kept, 1 free
    c.begin_turn(3, 3 * PAGE)          # reclaims one 2-page chunk: agent 1's pages 4, 3 -> host (tier full)
    assert (c.cached_tokens(1), c.host_tokens(1), c.host_used) == (2 * PAGE, 2 * PAGE, 2)
    c.end_turn(3)
    c.complete(3)
    assert c.free == 3
    assert c.begin_turn(1, 6 * PAGE) == 4 * PAGE  # 2 reloads + 2 new pages: 3 free + 1 of agent 2's
    assert c.last_moves == (0, 2) and c.host_dropped_pages == 0
    assert (c.cached_tokens(2), c.host_tokens(2)) == (PAGE, 0)


# ------------------------------------------------------------------ recency tiers

@pytest.mark.parametrize("seed", range(3))
def test_one_wide_tier_is_plain_round_robin(seed):
    """A tier wider than the whole clock puts every idle agent in one tier:
    Algorithm 1 exactly."""
    import numpy as np
    rng = np.random.default_rng(seed)
    a = OracleCache(300, PAGE, 2 * PAGE, OracleCache.RR)
    b = OracleCache(300, PAGE, 2 * PAGE, OracleCache.RR, tier_width=10 ** 9)
    ctx, active = {}, set()
    for _ in range(400):
        ag = int(rng.integers(10))
        if ag in active:
            a.end_turn(ag), b.end_turn(ag)
            active.discard(ag)
            ctx[ag] += int(rng.integers(0, 100))
            continue
        prompt = ctx.get(ag, 0) + int(rng.integers(1, 300))
        try:
            ra = a.begin_turn(ag, prompt)
        except NoMemory:
            ra = None
        try:
            rb = b.begin_turn(ag, prompt)
        except NoMemory:
            rb = None
        assert ra == rb
        if ra is not None:
            active.add(ag)
            ctx[ag] = prompt
    assert a.evictions == b.evictions > 0


@pytest.mark.parametrize("n,na,m", REGIME)
def test_unit_tiers_turn_round_robin_into_whole_agent_eviction(n, na, m):
    """Tiers one clock tick wide hold one agent each: the oldest idle agent loses
    its whole prefix before the next is touched -- Equation 3's LRU outcome."""
    ns = n - na
    u = 8 * ns
    c = OracleCache(m * u, PAGE, PAGE, OracleCache.RR, tier_width=1)
    for i in range(ns):
        _fill(c, i, u)
    for j in range(na):
        c.begin_turn(1000 + j, u * PAGE)
    kept = [c.cached_tokens(i) / (u * PAGE) for i in range(ns)]
    assert kept == [0.0] * (n - m) + [1.0] * (m - na)


def test_tiers_evict_stale_agents_first():
    """Agents 1 and 2 finished long ago without a completion signal; agents 3 and 4
    are recent.  With tiers the stale pair loses its pages first (round-robin
    between them); plain round robin spreads the loss over all four."""
    def run(width):
        c = OracleCache(64, PAGE, PAGE, OracleCache.RR, tier_width=width)
        for a in (1, 2):
            _fill(c, a, 8)
        for k in range(20):          # time passes: other agents' short turns
            c.begin_turn(100 + k, PAGE)
            c.end_turn(100 + k)
            c.complete(100 + k)
        for a in (3, 4):
            _fill(c, a, 8)
        c.begin_turn(9, (c.free + 6) * PAGE)   # reclaim 6 pages
        return [c.cached_tokens(a) // PAGE for a in (1, 2, 3, 4)]
    assert run(8) == [5, 5, 8, 8]
    assert sorted(run(0)) != [5, 5, 8, 8] and sum(run(0)) == 26


# ------------------------------------------------------------------ shared prefixes

def _join_fill(c, agent, group, S, private):
    """A member whose first turn leaves S shared + `private` private pages cached."""
    c.join(agent, group, S * PAGE)
    c.begin_turn(agent, (S + private) * PAGE + 1)
    c.end_turn(agent)


def test_a_shared_prefix_is_stored_once():
    c = OracleCache(64, PAGE, PAGE, OracleCache.RR)
    _join_fill(c, 1, 7, 4, 3)           # creates the group node (4 pages) + 3 private
    assert c.group_tokens(7) == 4 * PAGE and c.cached_tokens(1) == 3 * PAGE
    used = 64 - c.free
    _join_fill(c, 2, 7, 4, 5)           # reuses the 4 shared pages, computes 5 private
    assert 64 - c.free == used + 5
    assert c.begin_turn(2, 9 * PAGE + 1) == 9 * PAGE   # shared + private reused
    c.end_turn(2)


def test_concurrent_first_turns_keep_one_copy():
    c = OracleCache(64, PAGE, PAGE, OracleCache.RR)
    for a in (1, 2):
        c.join(a, 0, 3 * PAGE)
    assert c.begin_turn(1, 5 * PAGE + 1) == 0
    assert c.begin_turn(2, 6 * PAGE + 1) == 0   # both compute the shared span
    assert c.free == 64 - 6 - 7
    c.end_turn(1)                               # creates the node from agent 1's pages
    c.end_turn(2)                               # agent 2's copies of the span are freed
    assert c.group_tokens(0) == 3 * PAGE
    assert (c.cached_tokens(1), c.cached_tokens(2)) == (2 * PAGE, 3 * PAGE)
    assert c.free == 64 - 3 - 2 - 3


@pytest.mark.parametrize("n,na,m", REGIME)
def test_round_robin_closed_form_holds_for_private_histories(n, na, m):
    """Equation 2 with a shared system prompt: the idle agents' private prefixes of
    u pages each keep h = (m - na) / ns of their pages; the shared node (one copy)
    is never touched while any member holds private pages."""
    ns = n - na
    u = 8 * ns
    S = 5
    c = OracleCache(m * u + S, PAGE, PAGE, OracleCache.RR)
    for i in range(ns):
        _join_fill(c, i, 0, S, u)
    for j in range(na):
        c.begin_turn(1000 + j, u * PAGE)
    kept = [c.cached_tokens(i) / (u * PAGE) for i in range(ns)]
    h = (m - na) / ns
    assert all(abs(k - h) < 1e-12 for k in kept), kept
    assert c.group_tokens(0) == S * PAGE


@pytest.mark.parametrize("policy", [OracleCache.RR, OracleCache.LRU])
def test_the_shared_node_goes_only_as_a_whole_leaf(policy):
    c = OracleCache(20, PAGE, PAGE, policy)
    _join_fill(c, 1, 0, 4, 3)
    _join_fill(c, 2, 0, 4, 2)
    assert c.free == 20 - 4 - 3 - 2
    c.begin_turn(9, (c.free + 5) * PAGE)        # needs all 5 private pages, not the node
    assert (c.cached_tokens(1), c.cached_tokens(2), c.group_tokens(0)) == (0, 0, 4 * PAGE)
    c.end_turn(9)
    c.complete(9)
    free = c.free
    c.begin_turn(8, (free + 2) * PAGE)          # now the node is a leaf: evicted whole
    assert c.group_tokens(0) == 0 and c.free == 4 - 2
    # members of an absent group reuse nothing; their next turn recreates the node
    c.end_turn(8)
    c.complete(8)
    assert c.begin_turn(1, 6 * PAGE + 1) == 0
    c.end_turn(1)
    assert c.group_tokens(0) == 4 * PAGE and c.cached_tokens(1) == 2 * PAGE
