"""CPU oracle of the token-content prefix cache (a radix tree) -- TEST INFRASTRUCTURE ONLY.

Only ``tests/`` may import this module.  Plain Python written from the paper,
sharing no code with the library's tree (``kvx_radix.cpp``):

* Section 2 ("Prefix caching for multi-turn agents"): a request reuses the KV of
  its longest matching prefix in a radix tree whose nodes hold variable-length
  token spans; agents may share a short prefix (a system prompt) while their
  longer histories stay private.
* Section 3.1: nodes used by running requests are active and cannot be
  reclaimed; eviction starts at idle leaves and exposes their parents; LRU
  orders the eligible leaves by last access time, and a request start touches
  every node on its matched path (recency synchronization).
* Section 3.2, Algorithm 1: the eligible leaves are grouped by agent trajectory
  and visited in round-robin order, one tail chunk per visit, rechecking
  eligibility at every pop; SelectTailChunk picks a whole leaf or a suffix of
  one.

Readings where the paper leaves the backend open (the library takes the same
ones; the design doc lists them):

R1. The tree indexes whole pages of ``page_size`` tokens: a node holds a span of
    pages (token ids) and one pool page per span page; children differ in their
    first page; matching compares whole pages.
R2. A request of n tokens reuses the matched pages up to the last whole page
    before its final token: min(matched, floor((n - 1) / page_size)) pages.
R3. At the request start, the prompt's whole pages past the match become one
    new leaf owned by the agent, under the match point (a node the match ends
    inside is split there; both parts keep owner, stamp and pins).  Fresh pages
    of whole pages the tree already holds (past the reuse limit) and of a
    partial last page are the request's own and go back at its end.
R4. One logical clock ticks at every request start and end; the start stamps
    and pins every node of the matched path, the end stamps and unpins the
    path (new leaf included).
R5. A node belongs to the agent whose request created it.  An agent's evictable
    suffix is the set of its leaves that no running request pins.
R6. SelectTailChunk(tau, M - freed): the agent's evictable leaf with the oldest
    stamp (ties: the node created first), its last min(chunk, leaf pages,
    M - freed) pages.  A leaf left empty is removed.
R7. The queue holds idle agents with an evictable suffix in agent-id order,
    starting after the agent that lost the previous chunk (of any earlier
    reclamation).  If it runs empty before M pages are freed, a new queue is
    formed, so that parents exposed meanwhile are reached.
R8. LRU removes the whole unpinned leaf with the oldest stamp (ties: the node
    created first), repeatedly.
R9. Completion: an idle agent's unpinned leaves that it owns are removed,
    repeatedly, until none is left (its unshared cache).
R10. Free pages are handed out lowest id first; a request that cannot get its
    pages after reclaiming everything evictable fails (evictions stay) and the
    agent stays idle.
"""

from __future__ import annotations

RR = 1
LRU = 0


class NoMemory(Exception):
    pass


class _Node:
    def __init__(self, nid, parent, tokens, pages, owner, stamp):
        self.id = nid
        self.parent = parent
        self.tokens = list(tokens)  # whole pages of token ids
        self.pages = list(pages)
        self.owner = owner
        self.stamp = stamp
        self.pins = 0
        self.children = []  # nodes


class OracleRadix:
    def __init__(self, num_pages: int, page_size: int, chunk_tokens: int, policy: int):
        self.ps = page_size
        self.chunk = chunk_tokens // page_size
        self.policy = policy
        self.free = set(range(num_pages))
        self.root = _Node(0, None, [], [], None, 0)
        self.next_id = 1
        self.clock = 0
        self.running = {}  # agent -> (path of nodes, own pages)
        self.last_rr = None
        self.evictions = 0
        self.evicted_pages = 0

    # ---------------------------------------------------------------- the tree
    def _nodes(self):
        out, stack = [], [self.root]
        while stack:
            x = stack.pop()
            out.append(x)
            stack.extend(x.children)
        return out

    def _page(self, tokens, i):
        return list(tokens[i * self.ps:(i + 1) * self.ps])

    def _walk(self, tokens, whole):
        """Matched nodes (root excluded) and pages; a last node matched only in part
        is returned with the number of its pages that matched."""
        x, got, path = self.root, 0, []
        while got < whole:
            nxt = None
            for c in x.children:
                if c.tokens[:self.ps] == self._page(tokens, got):
                    nxt = c
            if nxt is None:
                return path, got, None, 0
            k = 0
            while k < len(nxt.pages) and got + k < whole and nxt.tokens[k * self.ps:(k + 1) * self.ps] == \
                    self._page(tokens, got + k):
                k += 1
            if k < len(nxt.pages):
                return path, got + k, nxt, k
            path.append(nxt)
            got += k
            x = nxt
        return path, got, None, 0

    def _split(self, node, k):
        tail = _Node(self.next_id, node, node.tokens[k * self.ps:], node.pages[k:], node.owner, node.stamp)
        self.next_id += 1
        tail.pins = node.pins
        tail.children = node.children
        for c in tail.children:
            c.parent = tail
        node.tokens = node.tokens[:k * self.ps]
        node.pages = node.pages[:k]
        node.children = [tail]
        for path, own in self.running.values():
            if node in path:
                path.insert(path.index(node) + 1, tail)

    def _evictable_leaves(self, agent=None):
        return [x for x in self._nodes() if x is not self.root and not x.children and x.pins == 0
                and (agent is None or x.owner == agent)]

    def _remove_tail(self, leaf, k):
        self.free.update(leaf.pages[len(leaf.pages) - k:])
        leaf.pages = leaf.pages[:len(leaf.pages) - k]
        leaf.tokens = leaf.tokens[:len(leaf.pages) * self.ps]
        if not leaf.pages:
            leaf.parent.children.remove(leaf)

    # ---------------------------------------------------------------- policies
    def _select_tail_chunk(self, agent, want):
        leaves = self._evictable_leaves(agent)
        leaf = min(leaves, key=lambda x: (x.stamp, x.id))
        return leaf, min(self.chunk, len(leaf.pages), want)

    def _reclaim_rr(self, M):
        freed = 0
        while freed < M:
            owners = sorted({x.owner for x in self._evictable_leaves()})
            queue = [a for a in owners if a not in self.running]
            if not queue:
                return freed
            if self.last_rr is not None:
                after = [a for a in queue if a > self.last_rr]
                queue = after + [a for a in queue if a <= self.last_rr]
            while freed < M and queue:
                tau = queue.pop(0)
                if tau in self.running or not self._evictable_leaves(tau):
                    continue
                leaf, k = self._select_tail_chunk(tau, M - freed)
                self._remove_tail(leaf, k)
                freed += k
                self.evictions += 1
                self.evicted_pages += k
                self.last_rr = tau
                if self._evictable_leaves(tau):
                    queue.append(tau)
        return freed

    def _reclaim_lru(self, M):
        freed = 0
        while freed < M:
            leaves = self._evictable_leaves()
            if not leaves:
                return freed
            leaf = min(leaves, key=lambda x: (x.stamp, x.id))
            k = len(leaf.pages)
            self._remove_tail(leaf, k)
            freed += k
            self.evictions += 1
            self.evicted_pages += k
        return freed

    # ---------------------------------------------------------------- requests
    def begin(self, agent, tokens):
        """Returns (prefix_len, page table); raises NoMemory."""
        tokens = list(tokens)
        n = len(tokens)
        assert n >= 1 and agent not in self.running
        whole, total = n // self.ps, -(-n // self.ps)
        path, matched, part, k = self._walk(tokens, whole)
        if part is not None:
            self._split(part, k)
            path.append(part)
        reuse = min(matched, (n - 1) // self.ps)
        self.clock += 1
        for x in path:
            x.pins += 1
            x.stamp = self.clock
        self.running[agent] = (path, [])
        need = total - reuse
        if len(self.free) < need:
            if self.policy == RR:
                self._reclaim_rr(need - len(self.free))
            else:
                self._reclaim_lru(need - len(self.free))
        if len(self.free) < need:
            for x in path:
                x.pins -= 1
            del self.running[agent]
            raise NoMemory(agent)
        fresh = sorted(self.free)[:need]
        self.free.difference_update(fresh)
        reused = [pg for x in path for pg in x.pages][:reuse]
        table = reused + fresh
        own = []
        if whole > matched:
            leaf = _Node(self.next_id, path[-1] if path else self.root, tokens[matched * self.ps:whole * self.ps],
                         table[matched:whole], agent, self.clock)
            self.next_id += 1
            leaf.pins = 1
            leaf.parent.children.append(leaf)
            path.append(leaf)
        own += table[reuse:matched]           # recomputed pages the tree already holds
        if total > whole:
            own.append(table[whole])          # the partial last page
        self.running[agent] = (path, own)
        return reuse * self.ps, table

    def end(self, agent):
        path, own = self.running.pop(agent)
        self.clock += 1
        for x in path:
            x.pins -= 1
            x.stamp = self.clock
        self.free.update(own)

    def complete(self, agent):
        assert agent not in self.running
        while True:
            leaves = self._evictable_leaves(agent)
            if not leaves:
                return
            leaf = min(leaves, key=lambda x: x.id)
            self._remove_tail(leaf, len(leaf.pages))

    # ---------------------------------------------------------------- probes
    def match(self, tokens):
        path, matched, part, k = self._walk(list(tokens), len(tokens) // self.ps)
        pages = [pg for x in path for pg in x.pages] + (part.pages[:k] if part is not None else [])
        return matched * self.ps, pages

    def stats(self):
        nodes = [x for x in self._nodes() if x is not self.root]
        return {"free_pages": len(self.free), "cached_pages": sum(len(x.pages) for x in nodes),
                "temp_pages": sum(len(own) for _, own in self.running.values()), "nodes": len(nodes),
                "leaves": sum(1 for x in nodes if not x.children), "evicted_pages": self.evicted_pages,
                "evictions": self.evictions, "active": len(self.running)}

    def agent_pages(self, agent):
        """Pages of the nodes an agent owns (for the analytical pins)."""
        return sum(len(x.pages) for x in self._nodes() if x is not self.root and x.owner == agent)
