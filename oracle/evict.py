"""CPU oracle of the prefix cache's eviction policies -- TEST INFRASTRUCTURE ONLY.

Only ``tests/`` may import this module.  Plain Python, written from the paper,
sharing no code with the library's cache (``kvx_cache.cpp``):

* round-robin tail eviction follows Algorithm 1 (Section 3.2) step by step:
  one queue of idle trajectories with evictable suffixes, pop the front,
  recheck eligibility, evict one tail chunk (SelectTailChunk), push the
  trajectory back while it still holds an evictable suffix, until enough is
  freed or the queue is empty;
* the LRU baseline (Section 3.1) drops the whole leaf node with the oldest
  access time among idle trajectories, which exposes the parent as a new leaf;
* completion signals (Section 3.2, stale trajectories) free an agent at once.

Sizes are counted in pages; no physical page ids are tracked (which page a
policy hands out is the library's choice, and tests check it separately).

Readings where the paper leaves the backend open (the same ones the library
takes; each is listed in the design doc):

1. A trajectory is one agent's private history; nothing is shared between
   agents (the analysis of Section 3.3 assumes no sharing).
2. Each finished turn adds one node: the whole pages its prompt added.  Turn
   start and turn end both stamp every node of the agent's path with the
   current logical time (matching and inserting touch the whole path).
3. A turn of P tokens reuses min(cached, 16 * floor((P - 1) / 16)) tokens: whole
   pages, and at least one prompt token is computed.  Cached pages past that
   are dropped; the prompt's partial last page is not kept after the turn.
4. SelectTailChunk(tau, M - M_freed) = the last min(chunk, leaf pages,
   M - M_freed) pages of tau's leaf node (a suffix of one leaf, never more than
   is still needed).
5. The queue of each reclamation lists idle agents in agent-id order, starting
   after the agent that lost the previous chunk, so the rotation continues from
   one reclamation to the next.
6. LRU ties (equal stamps cannot happen with a strictly increasing clock) would
   go to the smaller agent id.

Host tier (the paper's future work, Section 6: spill idle state to CPU memory
instead of dropping it), when ``host_pages`` > 0:

7. An idle agent's history is its device pages followed by its host pages, in
   logical order; the host pages continue the device prefix without a gap.
8. Pages the device policy evicts are spilled to host records, farthest page
   first (so within an agent, older records are always farther pages).  A
   spill that finds no free record first drops the oldest record whose owner
   is idle -- that owner's farthest host page.  If every record belongs to an
   active agent, the page is dropped instead.  A record spilled into earlier in
   the same turn start and dropped again before it ends voids that spill: the
   page counts as dropped, not spilled (the moves never write it).
9. A turn start reuses device pages, then host pages, up to reading 3's limit;
   the reused host pages are reloaded into freshly allocated device pages (they
   are pinned while the turn allocates) and their records freed.  Pages past
   the limit are dropped, host pages first.  An agent inside a turn holds no
   host pages.

Recency tiering (Section 3.2, stale trajectories without completion signals;
the paper describes it and does not evaluate it), when ``tier_width`` > 0:

10. Idle agents with evictable pages fall into tiers by age = now - stamp in
    the cache's logical clock (one tick per turn start and turn end): tier =
    age // tier_width.  A reclamation visits tiers from the oldest to the
    newest and runs Algorithm 1's round robin within each (queue in agent-id
    order after the agent that lost the last chunk), moving to the next tier
    once the current one holds nothing evictable.

Shared prefixes (Section 2: agents typically share a short common prefix, such
as a system prompt, in the serving system's radix tree; Section 3.1: eviction
starts at idle leaves and exposes parents):

11. An agent may join a group before it holds any pages; the group's shared
    prefix is its first S whole pages, the same for every member.  The group
    node is all or nothing: present (S pages, one copy, read by every member's
    page table) or absent.  A member's history is the group's pages, then its
    private pages, then its host pages; a member of an absent group holds no
    private pages.
12. A member's turn end creates the absent group node from the turn's own
    pages of the shared span (the turn computed them: nothing was reused);
    if the node appeared meanwhile, the turn's copies of the span are freed.
    Private pages are kept only while the group node is present.
13. The group node is a leaf -- evictable -- only while no member is inside a
    turn and no member holds private or host pages; it is then evicted whole and
    never spilled.  Its stamp is the last turn start or end of any member.  LRU
    weighs it among the other leaves by that stamp; round robin visits it after
    the agents' queue (it is the parent of every member's path), oldest first.
"""

from __future__ import annotations

from collections import deque


class NoMemory(Exception):
    """Active demand exceeds the capacity even after evicting every idle page."""


class _Group:
    def __init__(self, shared_pages: int) -> None:
        self.S = shared_pages
        self.present = False
        self.stamp = 0
        self.members: set[int] = set()


class _Agent:
    def __init__(self) -> None:
        self.nodes: list[int] = []  # pages per node, root .. leaf
        self.host: list[int] = []   # host record ids, nearest page first
        self.group = None           # group id, or None
        self.turn_start = 0         # logical page of the running turn's first page
        self.active = False
        self.stamp = 0
        self.prompt_len = 0
        self.turn_pages = 0

    @property
    def pages(self) -> int:
        return sum(self.nodes)


class OracleCache:
    LRU = 0
    RR = 1

    def __init__(self, num_pages: int, page_size: int, chunk_tokens: int, policy: int, host_pages: int = 0,
                 tier_width: int = 0) -> None:
        assert page_size == 16 and chunk_tokens % page_size == 0 and chunk_tokens > 0 and host_pages >= 0
        assert tier_width >= 0
        self.tier_width = tier_width
        self.host_pages = host_pages
        self.records: list[tuple[int, int]] = []  # live host records (id, owner), oldest first
        self.next_record = 0
        self.spilled_pages = 0
        self.reloaded_pages = 0
        self.host_dropped_pages = 0
        self.last_moves = (0, 0)  # (spills, reloads) of the last turn start
        self.num_pages = num_pages
        self.page_size = page_size
        self.chunk = chunk_tokens // page_size
        self.policy = policy
        self.free = num_pages
        self.agents: dict[int, _Agent] = {}
        self.groups: dict[int, _Group] = {}
        self.clock = 0
        self.rr_last = None
        self.evicted_pages = 0
        self.evictions = 0

    # -- helpers -------------------------------------------------------------
    def _drop_tail(self, a: _Agent, n: int) -> None:
        while n > 0:
            k = min(n, a.nodes[-1])
            a.nodes[-1] -= k
            if a.nodes[-1] == 0:
                a.nodes.pop()
            self.free += k
            n -= k

    def _forget(self, rec: int) -> None:
        self.records = [(r, o) for r, o in self.records if r != rec]

    def _host_record(self) -> int | None:
        """A free host record, dropping the oldest idle-owned one if none is free."""
        if len(self.records) < self.host_pages:
            self.next_record += 1
            return self.next_record
        for rec, owner in self.records:
            o = self.agents[owner]
            if not o.active:
                assert o.host[-1] == rec  # the owner's farthest host page
                o.host.pop()
                self._forget(rec)
                if rec in self.call_spills:  # written earlier in this turn start: that spill is void
                    self.call_spills.discard(rec)
                    self.spilled_pages -= 1
                    self.moves_spill -= 1
                else:
                    self.host_dropped_pages += 1
                self.next_record += 1
                return self.next_record
        return None

    def _evict(self, agent_id: int, a: _Agent, n: int) -> None:
        """Device eviction of a's last n pages; spilled to the host tier if there is one."""
        self._drop_tail(a, n)
        if self.host_pages == 0:
            return
        for _ in range(n):  # farthest page first
            rec = self._host_record()
            if rec is None:
                continue  # dropped (the agent has no host pages: nothing past it is lost)
            a.host.insert(0, rec)
            self.records.append((rec, agent_id))
            self.call_spills.add(rec)
            self.spilled_pages += 1
            self.moves_spill += 1

    def join(self, agent_id: int, group: int, shared_tokens: int) -> None:
        S = shared_tokens // self.page_size
        assert S >= 1
        a = self.agents.setdefault(agent_id, _Agent())
        assert not a.active and a.pages == 0 and not a.host and a.group is None
        g = self.groups.setdefault(group, _Group(S))
        assert g.S == S
        a.group = group
        g.members.add(agent_id)

    def _group_leaf(self, gid: int) -> bool:
        g = self.groups[gid]
        return g.present and all(not self.agents[m].active and self.agents[m].pages == 0 and not self.agents[m].host
                                 for m in g.members)

    def _evict_group(self, gid: int) -> int:
        g = self.groups[gid]
        g.present = False
        self.free += g.S
        self.evicted_pages += g.S
        self.evictions += 1
        return g.S

    def _evictable(self, agent_id: int) -> bool:
        a = self.agents.get(agent_id)
        return a is not None and not a.active and a.pages > 0

    # -- Algorithm 1 ---------------------------------------------------------
    def _reclaim_rr(self, M: int) -> None:
        ids = sorted(i for i in self.agents if self._evictable(i))
        if self.tier_width == 0:
            groups = [ids]
        else:  # recency tiers, oldest first
            tiers: dict[int, list[int]] = {}
            for i in ids:
                tiers.setdefault((self.clock - self.agents[i].stamp) // self.tier_width, []).append(i)
            groups = [tiers[k] for k in sorted(tiers, reverse=True)]
        freed = 0
        for group in groups:
            freed = self._round_robin(group, M, freed)
            if freed >= M:
                return
        for _, gid in sorted((g.stamp, gid) for gid, g in self.groups.items() if self._group_leaf(gid)):
            freed += self._evict_group(gid)
            if freed >= M:
                return

    def _round_robin(self, ids: list[int], M: int, freed: int) -> int:
        """Algorithm 1 over the idle agents `ids` (in id order); returns M_freed."""
        if self.rr_last is None:
            order = ids
        else:
            order = [i for i in ids if i > self.rr_last] + [i for i in ids if i <= self.rr_last]
        Q = deque(order)
        while freed < M and Q:
            tau = Q.popleft()
            if not self._evictable(tau):  # active, or no evictable suffix
                continue
            a = self.agents[tau]
            c = min(self.chunk, a.nodes[-1], M - freed)  # SelectTailChunk(tau, M - M_freed)
            self._evict(tau, a, c)  # Evict(c)
            freed += c
            self.evicted_pages += c
            self.evictions += 1
            self.rr_last = tau
            if self._evictable(tau):
                Q.append(tau)
        return freed

    # -- LRU baseline ----------------------------------------------------------
    def _reclaim_lru(self, M: int) -> None:
        freed = 0
        while freed < M:
            leaves = [(self.agents[i].stamp, i) for i in self.agents if self._evictable(i)]
            leaves += [(g.stamp, ("group", gid)) for gid, g in self.groups.items() if self._group_leaf(gid)]
            if not leaves:
                return
            _, victim = min(leaves, key=lambda x: x[0])
            if isinstance(victim, tuple):
                freed += self._evict_group(victim[1])
                continue
            a = self.agents[victim]
            n = a.nodes[-1]
            self._evict(victim, a, n)
            freed += n
            self.evicted_pages += n
            self.evictions += 1

    # -- turns -----------------------------------------------------------------
    def begin_turn(self, agent_id: int, prompt_len: int) -> int:
        assert prompt_len >= 1
        a = self.agents.setdefault(agent_id, _Agent())
        assert not a.active
        self.clock += 1
        a.stamp = self.clock
        g = self.groups.get(a.group) if a.group is not None else None
        if g is not None:
            g.stamp = self.clock
        self.moves_spill = 0
        self.call_spills: set[int] = set()
        self.last_moves = (0, 0)
        limit = (prompt_len - 1) // self.page_size
        gp = g.S if g is not None and g.present else 0  # group pages on the agent's path
        reuse = min(gp + a.pages + len(a.host), limit)
        if reuse < gp:  # the prompt ends inside the shared span
            used_group = reuse
            for rec in a.host:
                self._forget(rec)
            a.host = []
            self._drop_tail(a, a.pages)
        else:
            used_group = gp
            r2 = reuse - gp
            if r2 < a.pages:  # past the limit: host pages go first, then device pages
                for rec in a.host:
                    self._forget(rec)
                a.host = []
                self._drop_tail(a, a.pages - r2)
            else:
                for rec in a.host[r2 - a.pages:]:
                    self._forget(rec)
                a.host = a.host[: r2 - a.pages]
        reload = len(a.host)
        a.turn_start = used_group + a.pages
        need = -(-prompt_len // self.page_size) - a.turn_start  # reloaded pages + new pages
        a.active = True
        if self.free < need:
            if self.policy == self.RR:
                self._reclaim_rr(need - self.free)
            else:
                self._reclaim_lru(need - self.free)
        if self.free < need:
            a.active = False
            self.last_moves = (self.moves_spill, 0)
            raise NoMemory(agent_id)
        self.free -= need
        for rec in a.host:
            self._forget(rec)
        a.host = []
        self.reloaded_pages += reload
        self.last_moves = (self.moves_spill, reload)
        a.turn_pages = need
        a.prompt_len = prompt_len
        return reuse * self.page_size

    def end_turn(self, agent_id: int) -> None:
        a = self.agents[agent_id]
        assert a.active
        g = self.groups.get(a.group) if a.group is not None else None
        whole = a.prompt_len // self.page_size
        kept = 0       # turn pages that stay: the new private node, or the new group node
        new_node = 0
        if g is None:
            new_node = whole - a.pages
        else:
            if not g.present and whole >= g.S:
                assert a.turn_start == 0
                g.present = True   # this turn's pages of the shared span become the group node
                kept += g.S
            if g.present:
                new_node = max(0, whole - max(g.S, a.turn_start))
        kept += new_node
        self.free += a.turn_pages - kept
        if new_node > 0:
            a.nodes.append(new_node)
        a.turn_pages = 0
        a.active = False
        self.clock += 1
        a.stamp = self.clock
        if g is not None:
            g.stamp = self.clock

    def complete(self, agent_id: int) -> None:
        a = self.agents[agent_id]
        assert not a.active
        self._drop_tail(a, a.pages)
        for rec in a.host:
            self._forget(rec)
        if a.group is not None:
            self.groups[a.group].members.discard(agent_id)
        del self.agents[agent_id]

    def cached_tokens(self, agent_id: int) -> int:
        a = self.agents.get(agent_id)
        return 0 if a is None else a.pages * self.page_size

    def host_tokens(self, agent_id: int) -> int:
        a = self.agents.get(agent_id)
        return 0 if a is None else len(a.host) * self.page_size

    def group_tokens(self, gid: int) -> int:
        g = self.groups.get(gid)
        return 0 if g is None or not g.present else g.S * self.page_size

    @property
    def host_used(self) -> int:
        return len(self.records)
