"""Pins of the radix-tree prefix-cache oracle (oracle/radix.py) against the paper
and against brute force: the closed forms of the homogeneous analysis (Section
3.3, Equations 1-3) on private histories under a shared system prompt,
hand-traced runs of Algorithm 1 and of LRU on branching toy trees, and the
longest-prefix match against a brute-force search over every cached sequence."""

import numpy as np
import pytest

from oracle import radix as R

PAGE = 16


def toks(*ranges):
    """Token ids: concatenated ranges (each a (start, pages) pair, whole pages)."""
    out = []
    for start, pages in ranges:
        out += list(range(start, start + pages * PAGE))
    return out


SYS = (1_000_000, 5)  # a 5-page system prompt shared by every agent


def priv(agent, pages):
    return (10_000 * (agent + 1), pages)


def _homogeneous(policy, n, na, m, u, chunk_pages, S=5):
    """Section 3.3's model under a shared prompt: ns = n - na idle agents cached first
    (the prompt once, then u private pages each), then na fresh agents start requests
    of u private pages each; capacity m * u + S pages."""
    ns = n - na
    c = R.OracleRadix(m * u + S, PAGE, chunk_pages * PAGE, policy)
    for i in range(ns):
        c.begin(i, toks((1_000_000, S), priv(i, u)) + [7])
        c.end(i)
    for j in range(na):
        c.begin(1000 + j, toks(priv(1000 + j, u)))  # u whole pages, nothing reused
    return c, [c.agent_pages(i) / u for i in range(1, ns)], c.agent_pages(0)


REGIME = [(10, 4, 7), (12, 4, 9), (20, 8, 15), (6, 2, 5)]


@pytest.mark.parametrize("n,na,m", REGIME)
def test_round_robin_keeps_the_same_fraction_of_every_private_prefix(n, na, m):
    """Equation 2: h = (m - na) / (n s) of each idle private prefix survives, with
    1-page chunks exactly; the shared prompt (an inner node while any agent keeps a
    private page under it) survives whole.  Agent 0 owns the prompt node as well as
    its private pages; the others own only private pages."""
    ns = n - na
    u = 8 * ns
    c, kept, agent0 = _homogeneous(R.RR, n, na, m, u, 1)
    h = (m - na) / ns
    assert all(abs(k - h) < 1e-12 for k in kept), (kept, h)
    assert abs((agent0 - 5) / u - h) < 1e-12
    assert c.match(toks(SYS))[0] == 5 * PAGE
    q = 1 - h
    assert abs(q - (n - m) / ns) < 1e-12  # X_RR = q for every returning idle agent


@pytest.mark.parametrize("n,na,m", REGIME)
def test_round_robin_with_coarse_chunks_stays_within_one_chunk(n, na, m):
    ns = n - na
    u, chunk = 64, 8
    c, kept, _ = _homogeneous(R.RR, n, na, m, u, chunk)
    h = (m - na) / ns
    assert all(abs(k - h) <= chunk / u + 1e-12 for k in kept), (kept, h)


@pytest.mark.parametrize("n,na,m", REGIME)
def test_lru_removes_whole_private_prefixes_of_a_fraction_q(n, na, m):
    """Equation 3: LRU keeps m - na idle prefixes whole and loses n - m whole, the
    least recent first, and E[X_LRU] = q; the shared prompt stays (an inner node)."""
    ns = n - na
    u = 16
    c, kept, agent0 = _homogeneous(R.LRU, n, na, m, u, 1)
    full = [agent0 - 5 == u] + [k == 1.0 for k in kept]
    gone = [agent0 - 5 == 0] + [k == 0.0 for k in kept]
    assert sum(full) == m - na and sum(gone) == n - m and all(f or g for f, g in zip(full, gone))
    assert gone[: n - m] == [True] * (n - m)  # oldest first
    assert c.match(toks(SYS))[0] == 5 * PAGE


@pytest.mark.parametrize("policy", [R.RR, R.LRU])
def test_no_eviction_when_everything_fits(policy):
    """Equation 1's upper bound: with m >= n nothing is reclaimed."""
    c, kept, _ = _homogeneous(policy, 6, 2, 6, 16, 1)
    assert c.evictions == 0 and all(k == 1.0 for k in kept)


@pytest.mark.parametrize("policy", [R.RR, R.LRU])
def test_active_demand_above_capacity_cannot_be_met(policy):
    """Equation 1's lower bound: when active demand exceeds capacity, a request
    fails even after every idle page is reclaimed."""
    c = R.OracleRadix(20, PAGE, PAGE, policy)
    c.begin(1, toks(priv(1, 8)) + [1])
    c.end(1)
    c.begin(2, toks(priv(2, 12)) + [1])  # 13 pages: reclaims agent 1's history
    with pytest.raises(R.NoMemory):
        c.begin(3, toks(priv(3, 10)))
    assert c.match(toks(priv(1, 8)))[0] == 0
    assert 3 not in c.running


# ------------------------------------------------------------------ hand traces

def test_branching_tree_hand_trace():
    """A shared prompt, two agents under it, and a second branch of agent 1 (a retry
    from an earlier point of its history), traced page by page."""
    c = R.OracleRadix(32, PAGE, 2 * PAGE, R.RR)
    a1 = toks((500, 2), (100, 3))                      # prompt 2 pages + 3 private
    assert c.begin(1, a1 + [9]) == (0, [0, 1, 2, 3, 4, 5])
    c.end(1)                                          # page 5 (partial) back
    st = c.stats()
    assert (st["nodes"], st["cached_pages"], st["free_pages"]) == (1, 5, 27)
    a2 = toks((500, 2), (200, 1))
    p, table = c.begin(2, a2 + [9, 9])
    assert (p, table) == (32, [0, 1, 5, 6])           # the prompt's pages shared; node split
    assert c.stats()["nodes"] == 3                    # [prompt] -> {agent 1's 3, agent 2's 1}
    c.end(2)
    # agent 1 branches after its first private page
    b1 = toks((500, 2), (100, 1), (300, 2))
    p, table = c.begin(1, b1 + [4])
    assert (p, table) == (48, [0, 1, 2, 6, 7, 8])     # split again: [100] -> {[101,102], [300..]}
    c.end(1)
    st = c.stats()
    assert (st["nodes"], st["leaves"], st["cached_pages"]) == (5, 3, 8)
    assert c.match(a1) == (5 * PAGE, [0, 1, 2, 3, 4])
    assert c.match(b1) == (5 * PAGE, [0, 1, 2, 6, 7])
    assert c.match(a2) == (3 * PAGE, [0, 1, 5])


def test_algorithm1_visits_trajectories_in_turn_on_a_branching_tree():
    """Round-robin tail chunks of 2 pages over three idle agents (one of them holding
    two branches): each visit takes one chunk from the agent's oldest leaf, the queue
    rotates across reclamations, and a leaf emptied exposes its parent."""
    c = R.OracleRadix(24, PAGE, 2 * PAGE, R.RR)
    c.begin(1, toks((500, 2), (100, 4)) + [1]); c.end(1)        # pages 0-5 (+6 temp)
    c.begin(2, toks((500, 2), (200, 3)) + [1]); c.end(2)        # 6-8 (+9 temp)
    c.begin(3, toks((700, 4)) + [1]); c.end(3)                  # 9-12 (+13 temp)
    c.begin(1, toks((500, 2), (100, 1), (300, 2)) + [1]); c.end(1)  # branch 13, 14 (+15)
    assert c.stats()["free_pages"] == 24 - 15
    # a request of 13 pages needs 4 more than the 9 free
    c.begin(4, toks((900, 12)) + [1])
    # queue [1, 2, 3]: agent 1's oldest leaf is the 3-page tail [101..103] (stamped at
    # its first request's end; the branch was stamped later) and loses 2 pages, then
    # agent 2's leaf loses 2
    assert c.match(toks((500, 2), (100, 4)))[0] == 4 * PAGE
    assert c.match(toks((500, 2), (200, 3)))[0] == 3 * PAGE
    assert c.match(toks((700, 4)))[0] == 4 * PAGE
    assert c.last_rr == 2 and c.evictions == 2
    c.end(4)
    # 23 pages cached, 1 free; agent 5 needs 4.  The queue continues after agent 2:
    # agent 3 loses a 2-page chunk, then agent 4 (now idle) the last page needed
    c.begin(5, toks((950, 3)) + [1])
    assert c.last_rr == 4 and c.evictions == 4
    assert c.match(toks((700, 4)))[0] == 2 * PAGE
    assert c.match(toks((900, 12)))[0] == 11 * PAGE
    assert c.match(toks((500, 2), (100, 4)))[0] == 4 * PAGE


def test_algorithm1_skips_running_trajectories():
    c = R.OracleRadix(12, PAGE, PAGE, R.RR)
    c.begin(1, toks(priv(1, 4)) + [1]); c.end(1)
    c.begin(2, toks(priv(2, 4)) + [1]); c.end(2)
    c.begin(1, toks(priv(1, 4), (55, 1)) + [1])       # agent 1 running again (6 pages, 4 reused)
    c.begin(3, toks(priv(3, 3)) + [1])                # needs 4: only agent 2 may lose pages
    assert c.match(toks(priv(1, 4)))[0] == 4 * PAGE
    assert c.match(toks(priv(2, 4)))[0] < 4 * PAGE


def test_lru_takes_whole_leaves_and_exposes_parents():
    """LRU removes the oldest unpinned leaf whole; the shared prompt becomes a leaf
    only when both private leaves under it are gone."""
    c = R.OracleRadix(16, PAGE, PAGE, R.LRU)
    c.begin(1, toks((500, 2), (100, 3)) + [1]); c.end(1)   # 0-4
    c.begin(2, toks((500, 2), (200, 3)) + [1]); c.end(2)   # 5-7 after the split
    c.begin(3, toks((900, 10)) + [1])                      # needs 11 of 16 - 8 free: agent 1's leaf
    assert c.match(toks((500, 2), (100, 3)))[0] == 2 * PAGE
    assert c.match(toks((500, 2), (200, 3)))[0] == 5 * PAGE
    c.end(3)
    c.begin(4, toks((990, 15)) + [1])                      # everything idle goes, oldest first
    assert c.match(toks((500, 2)))[0] == 0
    assert c.stats()["cached_pages"] == 15


def test_completion_frees_only_the_agents_unshared_pages():
    c = R.OracleRadix(32, PAGE, PAGE, R.RR)
    c.begin(1, toks((500, 2), (100, 3)) + [1]); c.end(1)
    c.begin(2, toks((500, 2), (200, 3)) + [1]); c.end(2)
    c.complete(1)                                     # agent 1 owns the prompt node too
    assert c.match(toks((500, 2), (100, 3)))[0] == 2 * PAGE  # the prompt stays: agent 2 is below it
    c.complete(2)
    assert c.match(toks((500, 2)))[0] == 2 * PAGE     # still agent 1's node
    c.complete(1)
    assert c.stats()["cached_pages"] == 0


def test_requests_reuse_whole_pages_and_compute_at_least_one_token():
    c = R.OracleRadix(16, PAGE, PAGE, R.RR)
    c.begin(1, toks(priv(1, 3))); c.end(1)            # 48 tokens: 3 whole pages cached
    p, table = c.begin(2, toks(priv(1, 3)))           # the same 48 tokens again
    assert p == 2 * PAGE and table[:2] == [0, 1] and table[2] != 2  # the last page is recomputed
    c.end(2)
    assert c.stats()["cached_pages"] == 3 and c.stats()["free_pages"] == 13
    p, _ = c.begin(3, toks(priv(1, 3)) + [5])         # one more token: all 3 pages reused
    assert p == 3 * PAGE


# ------------------------------------------------------------------ brute force

def _cached_sequences(c):
    """Every root-to-node token sequence of the tree."""
    out = []

    def rec(x, prefix):
        seq = prefix + x.tokens
        if x is not c.root:
            out.append(seq)
        for ch in x.children:
            rec(ch, seq)
    rec(c.root, [])
    return out


@pytest.mark.parametrize("seed", range(6))
def test_match_is_the_longest_whole_page_prefix_of_any_cached_sequence(seed):
    """The walk (with splits along the way) against brute force over every cached
    sequence, after a random branching trace; and no page is lost or duplicated."""
    rng = np.random.default_rng([41, seed])
    c = R.OracleRadix(400, PAGE, 2 * PAGE, [R.RR, R.LRU][seed % 2])
    pool = [list(rng.integers(0, 3, 6 * PAGE)) for _ in range(4)]  # few distinct tokens: many shared pages
    for step in range(40):
        base = pool[int(rng.integers(0, 4))]
        cut = int(rng.integers(1, len(base)))
        prompt = base[:cut] + list(rng.integers(0, 3, int(rng.integers(1, 40))))
        agent = int(rng.integers(0, 6))
        if agent in c.running:
            c.end(agent)
            continue
        try:
            c.begin(agent, prompt)
        except R.NoMemory:
            pass
        q = base[: int(rng.integers(1, len(base)))]
        best = 0
        for seq in _cached_sequences(c):
            k = 0
            while (k + 1) * PAGE <= min(len(q), len(seq)) and q[k * PAGE:(k + 1) * PAGE] == seq[k * PAGE:(k + 1) * PAGE]:
                k += 1
            best = max(best, k)
        assert c.match(q)[0] == best * PAGE
        st = c.stats()
        assert st["free_pages"] + st["cached_pages"] + st["temp_pages"] == 400
        seen = [pg for x in c._nodes() for pg in x.pages] + [pg for _, own in c.running.values() for pg in own]
        assert len(seen) == len(set(seen)) and not (set(seen) & c.free)
        for x in c._nodes():  # siblings differ in their first page
            firsts = [tuple(ch.tokens[:PAGE]) for ch in x.children]
            assert len(firsts) == len(set(firsts)) and all(len(ch.pages) > 0 for ch in x.children)
