"""Seeded synthetic workloads for prefix-extend attention.

This module only *generates inputs*: per-request (prefix_len, extend_len) pairs,
the physical placement of every request's KV pages in the pool, fp8 scales and
bf16 Q/K/V values.  It holds none of the attention arithmetic and none of the
KV-store arithmetic, so both the CPU oracle (tests) and the HIP path draw their
inputs from it without sharing any of the method's code.

The workload shapes stand in for the agent traces of the paper (Section 4,
Experimental setup), which are not available: a returning agent reuses a cached
prefix and prefills only the uncached suffix (Section 1; Section 2, "Prefix
caching for multi-turn agents"); a fully evicted agent recomputes its whole
context (Section 3.1); round-robin tail eviction leaves partial prefixes whose
lost tail chunks are recomputed (Section 3.2, Algorithm 1).

Generation order (fixed, so every draw is reproducible):
  * ``numpy.random.default_rng([config_id, 0, seed])`` draws the lengths, then
    one permutation of the pool's pages, then the fp8 K scales and V scales.
  * Each request's values come from torch generators seeded by
    ``SeedSequence([config_id, 1, seed, kind, r])`` with kind 0 = Q, 1 = K, 2 = V;
    the RMS-norm weights of the fused RoPE store from ``SeedSequence([config_id,
    2, seed, kind])`` with kind 0 = Q, 1 = K, uniform in [0.5, 1.5].
    Values are drawn as fp32 N(0, sigma^2) and rounded to bf16 (RNE); the bf16
    values *are* the inputs.  The values depend on the device type the
    generator runs on (torch's CPU and GPU generators differ), so a test always
    hands the same tensors to both sides.
"""

from __future__ import annotations

import dataclasses
import math
from typing import Optional, Sequence

import numpy as np
import torch

PAGE_SIZE = 16

KV_BF16 = 0
KV_FP8_E4M3 = 1

# Named synthetic configurations (prefix-extend batches of agent-shaped requests).
CONFIG_IDS = {
    "tiny": 1,          # 4 requests, 4/2 heads, head_dim 64
    "llama8b": 2,       # 16 returning agents, Llama-3-8B-shaped layer
    "tail_outlier": 3,  # one fully evicted 131072-token recompute + 31 partial hits
    "rr_partial": 4,    # 64 agents that lost 1-4 tail chunks of 2048 tokens
    "wide70b": 5,       # 48 requests, 64/8 heads, bf16 K/V pool
    "wide70b_fp8": 5,   # same batch, fp8 e4m3 K/V pool with per-head scales
    "decode_llama8b": 8,  # decode step: 128 agents, one new token each, Llama-3-8B-shaped
    "decode_long": 9,     # decode step: 32 agents with 64k-128k contexts
}


@dataclasses.dataclass
class Workload:
    """Shapes and page placement of one prefix-extend batch (host arrays)."""

    name: str
    config_id: int
    seed: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    prefix_lens: np.ndarray           # int32 [R]
    extend_lens: np.ndarray           # int32 [R]
    num_pages: int                    # pool capacity in pages
    page_indptr: np.ndarray           # int32 [R+1]: request r owns page_ids[indptr[r]:indptr[r+1]]
    page_ids: np.ndarray              # int32: logical page j of request r -> physical page
    kv_dtype: int = KV_BF16
    k_scale: Optional[np.ndarray] = None  # float32 [Hkv] for the fp8 pool
    v_scale: Optional[np.ndarray] = None
    sigma: float = 1.0                # std of K and V values
    q_sigma: float = 1.0              # std of Q values
    page_size: int = PAGE_SIZE
    orig_req: Optional[np.ndarray] = None  # request ids in the batch a subset was taken from

    def value_id(self, r: int) -> int:
        """The request id that seeds request r's values (stable under ``subset``)."""
        return int(r if self.orig_req is None else self.orig_req[r])

    @property
    def num_reqs(self) -> int:
        return int(self.prefix_lens.shape[0])

    @property
    def seq_lens(self) -> np.ndarray:
        return (self.prefix_lens.astype(np.int64) + self.extend_lens).astype(np.int64)

    @property
    def qo_indptr(self) -> np.ndarray:
        out = np.zeros(self.num_reqs + 1, dtype=np.int32)
        np.cumsum(self.extend_lens, out=out[1:])
        return out

    @property
    def total_extend(self) -> int:
        return int(self.extend_lens.astype(np.int64).sum())

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def sm_scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)

    def pages_of(self, r: int) -> np.ndarray:
        return self.page_ids[self.page_indptr[r]:self.page_indptr[r + 1]]

    def visible_pairs(self) -> int:
        """Number of (query row, key) pairs a causal prefix-extend pass visits, per q-head."""
        p = self.prefix_lens.astype(np.int64)
        e = self.extend_lens.astype(np.int64)
        return int((e * p + e * (e + 1) // 2).sum())

    def flops(self) -> float:
        """Algorithmic FLOPs of one attention pass: 4*d*Hq per visible causal pair."""
        return 4.0 * self.head_dim * self.num_q_heads * self.visible_pairs()

    def subset(self, reqs: Sequence[int], compact_pages: bool = True) -> "Workload":
        """Restrict to some requests.  With ``compact_pages`` their pages are renumbered
        0..n-1 in order of appearance (a smaller pool with the same logical contents)."""
        reqs = [int(r) for r in reqs]
        pages = [self.pages_of(r) for r in reqs]
        indptr = np.zeros(len(reqs) + 1, dtype=np.int32)
        np.cumsum([len(p) for p in pages], out=indptr[1:])
        ids = np.concatenate(pages).astype(np.int32) if pages else np.zeros(0, np.int32)
        num_pages = self.num_pages
        if compact_pages:
            ids = np.arange(len(ids), dtype=np.int32)
            num_pages = max(1, len(ids))
        return dataclasses.replace(
            self, prefix_lens=self.prefix_lens[reqs].copy(), extend_lens=self.extend_lens[reqs].copy(),
            page_indptr=indptr, page_ids=ids, num_pages=num_pages,
            orig_req=np.array([self.value_id(r) for r in reqs], dtype=np.int64))


def _pages_needed(prefix_lens: np.ndarray, extend_lens: np.ndarray, page_size: int) -> np.ndarray:
    total = prefix_lens.astype(np.int64) + extend_lens.astype(np.int64)
    return (total + page_size - 1) // page_size


def _round_to(x: np.ndarray, m: int) -> np.ndarray:
    return (np.round(x / m) * m).astype(np.int64)


def _place_pages(need: np.ndarray, num_pages: int, perm: np.ndarray):
    indptr = np.zeros(len(need) + 1, dtype=np.int32)
    np.cumsum(need, out=indptr[1:])
    total = int(indptr[-1])
    if total > num_pages:
        raise ValueError(f"pool of {num_pages} pages cannot hold {total} pages")
    return indptr, perm[:total].astype(np.int32)


def make_custom(prefix_lens, extend_lens, num_q_heads, num_kv_heads, head_dim, *,
                num_pages: Optional[int] = None, pool_factor: float = 1.5,
                placement: str = "random", kv_dtype: int = KV_BF16,
                k_scale=None, v_scale=None, sigma: float = 1.0, q_sigma: Optional[float] = None,
                seed: int = 0, config_id: int = 99, name: str = "custom") -> Workload:
    """A workload with explicit lengths.  ``placement`` is ``random`` (seeded shuffle of
    the pool) or ``linear`` (pages 0, 1, 2, ... in request order)."""
    p = np.asarray(prefix_lens, dtype=np.int32)
    e = np.asarray(extend_lens, dtype=np.int32)
    if p.shape != e.shape or (p < 0).any() or (e < 0).any():
        raise ValueError("prefix_lens / extend_lens must be non-negative and equal length")
    need = _pages_needed(p, e, PAGE_SIZE)
    if num_pages is None:
        num_pages = max(1, int(math.ceil(pool_factor * max(1, int(need.sum())))))
    rng = np.random.default_rng([config_id, 0, seed])
    if placement == "random":
        perm = rng.permutation(num_pages)
    elif placement == "linear":
        perm = np.arange(num_pages)
    else:
        raise ValueError(placement)
    indptr, ids = _place_pages(need, num_pages, perm)
    if kv_dtype == KV_FP8_E4M3:
        if k_scale is None:
            k_scale = rng.uniform(0.01, 0.1, num_kv_heads)
        if v_scale is None:
            v_scale = rng.uniform(0.01, 0.1, num_kv_heads)
        k_scale = np.asarray(k_scale, dtype=np.float32)
        v_scale = np.asarray(v_scale, dtype=np.float32)
    return Workload(name=name, config_id=config_id, seed=seed, num_q_heads=num_q_heads,
                    num_kv_heads=num_kv_heads, head_dim=head_dim, prefix_lens=p, extend_lens=e,
                    num_pages=int(num_pages), page_indptr=indptr, page_ids=ids, kv_dtype=kv_dtype,
                    k_scale=k_scale, v_scale=v_scale, sigma=sigma,
                    q_sigma=sigma if q_sigma is None else q_sigma)


def make_workload(name: str, seed: int = 0) -> Workload:
    """The five named agent-shaped batches (lengths and page placement only)."""
    if name not in CONFIG_IDS:
        raise KeyError(f"unknown workload {name!r}; known: {sorted(CONFIG_IDS)}")
    cid = CONFIG_IDS[name]
    rng = np.random.default_rng([cid, 0, seed])
    kv_dtype = KV_BF16
    sigma = 1.0
    if name == "tiny":
        hq, hkv, d = 4, 2, 64
        p = np.array([0, 64, 208, 512])
        e = np.array([32, 16, 100, 8])
        num_pages = 256
    elif name == "llama8b":
        hq, hkv, d = 32, 8, 128
        p = _round_to(rng.integers(4096, 32768 + 1, 16), PAGE_SIZE)
        e = rng.integers(64, 2048 + 1, 16)
        sigma = 0.5
        num_pages = None
    elif name == "tail_outlier":
        hq, hkv, d = 32, 8, 128
        p = np.concatenate([[0], _round_to(rng.integers(32768, 98304 + 1, 31), PAGE_SIZE)])
        e = np.concatenate([[131072], rng.integers(256, 1024 + 1, 31)])
        num_pages = None
    elif name == "rr_partial":
        hq, hkv, d = 32, 8, 128
        ctx = np.exp(rng.uniform(math.log(8192), math.log(196608), 64))
        ctx = (np.floor(ctx / PAGE_SIZE) * PAGE_SIZE).astype(np.int64)
        k = rng.integers(1, 4 + 1, 64)
        new = rng.integers(128, 4096 + 1, 64)
        p = ctx - 2048 * k
        e = 2048 * k + new
        num_pages = None
    elif name == "decode_llama8b":
        hq, hkv, d = 32, 8, 128
        p = _round_to(rng.integers(4096, 32768 + 1, 128), PAGE_SIZE)
        e = np.ones(128, np.int64)
        sigma = 0.5
        num_pages = None
    elif name == "decode_long":
        hq, hkv, d = 32, 8, 128
        p = _round_to(rng.integers(65536, 131072 + 1, 32), PAGE_SIZE)
        e = np.ones(32, np.int64)
        num_pages = None
    else:  # wide70b, wide70b_fp8
        hq, hkv, d = 64, 8, 128
        p = _round_to(np.exp(rng.uniform(math.log(16384), math.log(262144), 48)), PAGE_SIZE)
        e = rng.integers(512, 8192 + 1, 48)
        num_pages = None
        if name == "wide70b_fp8":
            kv_dtype = KV_FP8_E4M3
    p = p.astype(np.int32)
    e = e.astype(np.int32)
    need = _pages_needed(p, e, PAGE_SIZE)
    if num_pages is None:
        num_pages = int(math.ceil(1.5 * int(need.sum())))
    perm = rng.permutation(num_pages)
    indptr, ids = _place_pages(need, num_pages, perm)
    k_scale = v_scale = None
    if name.startswith("wide70b"):
        # drawn for both wide70b runs so the two share lengths, pages and seeds
        k_scale = rng.uniform(0.01, 0.1, hkv).astype(np.float32)
        v_scale = rng.uniform(0.01, 0.1, hkv).astype(np.float32)
        if kv_dtype == KV_BF16:
            k_scale = v_scale = None
    return Workload(name=name, config_id=cid, seed=seed, num_q_heads=hq, num_kv_heads=hkv,
                    head_dim=d, prefix_lens=p, extend_lens=e, num_pages=num_pages,
                    page_indptr=indptr, page_ids=ids, kv_dtype=kv_dtype, k_scale=k_scale,
                    v_scale=v_scale, sigma=sigma, q_sigma=sigma)


# ----------------------------------------------------------------------------- values

def _torch_seed(*parts: int) -> int:
    state = np.random.SeedSequence([int(x) for x in parts]).generate_state(2, dtype=np.uint32)
    return int((int(state[0]) << 31) ^ int(state[1])) & ((1 << 62) - 1)


def _randn_bf16(shape, sigma: float, seed: int, device) -> torch.Tensor:
    dev = torch.device(device)
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    x = torch.randn(shape, generator=g, device=dev, dtype=torch.float32)
    if sigma != 1.0:
        x.mul_(sigma)
    return x.to(torch.bfloat16)


def request_q(w: Workload, r: int, device="cpu") -> torch.Tensor:
    """Q rows of request r's uncached suffix: bf16 [E_r, Hq, d]."""
    e = int(w.extend_lens[r])
    return _randn_bf16((e, w.num_q_heads, w.head_dim), w.q_sigma,
                       _torch_seed(w.config_id, 1, w.seed, 0, w.value_id(r)), device)


def request_kv(w: Workload, r: int, device="cpu"):
    """The logical K and V sequences of request r (cached prefix then suffix): bf16 [L_r, Hkv, d]."""
    n = int(w.prefix_lens[r]) + int(w.extend_lens[r])
    shape = (n, w.num_kv_heads, w.head_dim)
    k = _randn_bf16(shape, w.sigma, _torch_seed(w.config_id, 1, w.seed, 1, w.value_id(r)), device)
    v = _randn_bf16(shape, w.sigma, _torch_seed(w.config_id, 1, w.seed, 2, w.value_id(r)), device)
    return k, v


@dataclasses.dataclass(frozen=True)
class RopeSpec:
    """Rotary-embedding and Q/K-norm settings of the fused store (plain data).
    The default is shaped like the Qwen3 models the paper serves: half-layout
    rotation of the whole head with base 10^6, and an RMS norm of every Q and K
    head before it."""
    theta: float = 1e6
    rotary_dim: int = 128
    style: int = 0          # 0: half layout, 1: interleaved
    norm: bool = True
    eps: float = 1e-6


def norm_weights(w: Workload, device="cpu"):
    """RMS-norm weights (q_norm, k_norm), bf16 [d] each, uniform in [0.5, 1.5]."""
    out = []
    for kind in (0, 1):
        g = torch.Generator(device=torch.device(device))
        g.manual_seed(_torch_seed(w.config_id, 2, w.seed, kind))
        x = torch.rand((w.head_dim,), generator=g, device=torch.device(device), dtype=torch.float32)
        out.append((0.5 + x).to(torch.bfloat16))
    return out[0], out[1]


def batch_tensors(w: Workload, device="cpu", reqs: Optional[Sequence[int]] = None):
    """Concatenated inputs of one prefix-extend call.

    Returns a dict with
      ``q``        bf16 [T, Hq, d]    suffix queries (T = sum of extend_lens)
      ``k_ext``    bf16 [T, Hkv, d]   suffix keys   (written by the KV store)
      ``v_ext``    bf16 [T, Hkv, d]   suffix values
      ``k_hist``   bf16 [sum P, Hkv, d] cached-prefix keys (written by an earlier turn)
      ``v_hist``   bf16 [sum P, Hkv, d]
    """
    reqs = range(w.num_reqs) if reqs is None else reqs
    qs, ke, ve, kh, vh = [], [], [], [], []
    for r in reqs:
        p = int(w.prefix_lens[r])
        qs.append(request_q(w, r, device))
        k, v = request_kv(w, r, device)
        kh.append(k[:p])
        vh.append(v[:p])
        ke.append(k[p:])
        ve.append(v[p:])
        del k, v
    def cat(xs, heads):
        if xs:
            return torch.cat(xs, 0)
        return torch.zeros((0, heads, w.head_dim), dtype=torch.bfloat16, device=device)
    return dict(q=cat(qs, w.num_q_heads), k_ext=cat(ke, w.num_kv_heads), v_ext=cat(ve, w.num_kv_heads),
                k_hist=cat(kh, w.num_kv_heads), v_hist=cat(vh, w.num_kv_heads))


def history_batch(w: Workload) -> Workload:
    """The earlier turn that produced the cached prefixes: each request with prefix 0 and
    extend = its cached prefix_len, on the same pages (the leading ceil(P/16) of them)."""
    need = (w.prefix_lens.astype(np.int64) + w.page_size - 1) // w.page_size
    indptr = np.zeros(w.num_reqs + 1, dtype=np.int32)
    np.cumsum(need, out=indptr[1:])
    ids = np.concatenate([w.pages_of(r)[:int(need[r])] for r in range(w.num_reqs)]
                         ).astype(np.int32) if w.num_reqs else np.zeros(0, np.int32)
    return dataclasses.replace(w, prefix_lens=np.zeros_like(w.prefix_lens),
                               extend_lens=w.prefix_lens.copy(), page_indptr=indptr, page_ids=ids)


def sample_rows(w: Workload, per_req: int, seed: int = 0, reqs: Optional[Sequence[int]] = None):
    """Seeded rows (r, i) to check at full size: always the first and last suffix row and
    a page-boundary row, plus random rows, ``per_req`` per request (fewer if E is small)."""
    rng = np.random.default_rng([w.config_id, 2, seed])
    reqs = range(w.num_reqs) if reqs is None else reqs
    out = []
    for r in reqs:
        e = int(w.extend_lens[r])
        p = int(w.prefix_lens[r])
        if e == 0:
            continue
        chosen = {0, e - 1}
        nb = (-p) % w.page_size  # first suffix row whose absolute position starts a page
        if nb < e:
            chosen.add(nb)
        if e > 1 and nb + w.page_size - 1 < e:
            chosen.add(nb + w.page_size - 1)
        want = min(per_req, e)
        while len(chosen) < want:
            chosen.add(int(rng.integers(0, e)))
        out.extend((r, i) for i in sorted(chosen))
    return np.array(out, dtype=np.int32).reshape(-1, 2)


# ----------------------------------------------------------------------------- agents

AGENT_CONFIG_ID = 7  # seed domain of the multi-agent traces below


@dataclasses.dataclass
class AgentTrace:
    """A synthetic multi-turn agent workload (stand-in for replayed agent traces,
    Section 4): agent i starts at tick start[i]; turn k appends new[i][k] tokens
    (user input or tool output) to its context, its reply adds reply[i][k] tokens,
    and it then waits idle[i][k] ticks (tool or user latency) before the next turn.
    The first `shared` tokens of every context are the same (a common system
    prompt, Section 2); the first prompt always covers them."""
    seed: int
    start: list
    new: list
    reply: list
    idle: list
    num_q_heads: int = 8
    num_kv_heads: int = 2
    head_dim: int = 64
    sigma: float = 1.0
    shared: int = 0

    @property
    def num_agents(self) -> int:
        return len(self.start)

    def max_context(self, i: int) -> int:
        return int(sum(self.new[i]) + sum(self.reply[i]))

    @property
    def sm_scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)


def make_agent_trace(num_agents: int, turns: int, *, seed: int = 0, first=(2048, 8192), new=(64, 1024),
                     reply=(32, 256), idle=(1, 8), spread: int = 8, num_q_heads: int = 8, num_kv_heads: int = 2,
                     head_dim: int = 64, shared: int = 0) -> AgentTrace:
    """Lengths only: integer uniforms (inclusive) from default_rng([7, 0, seed]).
    `shared` tokens (at most the smallest first prompt) open every context."""
    if not 0 <= shared <= first[0]:
        raise ValueError("the shared prefix must fit in every first prompt")
    rng = np.random.default_rng([AGENT_CONFIG_ID, 0, seed])
    start = rng.integers(0, spread + 1, num_agents).tolist()
    news, replies, idles = [], [], []
    for _ in range(num_agents):
        n = rng.integers(new[0], new[1] + 1, turns)
        n[0] = rng.integers(first[0], first[1] + 1)  # the first prompt carries the task
        news.append(n.tolist())
        replies.append(rng.integers(reply[0], reply[1] + 1, turns).tolist())
        idles.append(rng.integers(idle[0], idle[1] + 1, turns).tolist())
    return AgentTrace(seed, start, news, replies, idles, num_q_heads, num_kv_heads, head_dim, shared=shared)


def agent_kv(tr: AgentTrace, agent: int, length: int, device="cpu"):
    """The logical K and V of an agent's context (positions 0 .. length-1): bf16
    [length, Hkv, d].  A position's values never change between turns, so a
    recomputed suffix writes the same K/V its evicted copy held."""
    shape = (tr.max_context(agent), tr.num_kv_heads, tr.head_dim)
    k = _randn_bf16(shape, tr.sigma, _torch_seed(AGENT_CONFIG_ID, 1, tr.seed, 1, agent), device)
    v = _randn_bf16(shape, tr.sigma, _torch_seed(AGENT_CONFIG_ID, 1, tr.seed, 2, agent), device)
    if tr.shared:  # the common prefix: one generator for every agent
        sh = (tr.shared, tr.num_kv_heads, tr.head_dim)
        k[: tr.shared] = _randn_bf16(sh, tr.sigma, _torch_seed(AGENT_CONFIG_ID, 3, tr.seed, 1), device)
        v[: tr.shared] = _randn_bf16(sh, tr.sigma, _torch_seed(AGENT_CONFIG_ID, 3, tr.seed, 2), device)
    return k[:length], v[:length]


def agent_q(tr: AgentTrace, agent: int, turn: int, rows: int, device="cpu") -> torch.Tensor:
    """Queries of the uncached rows of one turn: bf16 [rows, Hq, d]."""
    return _randn_bf16((rows, tr.num_q_heads, tr.head_dim), tr.sigma,
                       _torch_seed(AGENT_CONFIG_ID, 1, tr.seed, 0, agent * 4096 + turn), device)


# ----------------------------------------------------------------------------- token content

TOKEN_CONFIG_ID = 11  # seed domain of the token-keyed K/V below
_HASH_MOD = (1 << 61) - 1


def prefix_hashes(tokens) -> list:
    """Rolling hash of every prefix: h_t = (h_{t-1} * 1000003 + token_t + 1) mod (2^61 - 1)."""
    h, out = 0, []
    for x in tokens:
        h = (h * 1_000_003 + int(x) + 1) % _HASH_MOD
        out.append(h)
    return out


def content_kv(tokens, num_kv_heads: int, head_dim: int, sigma: float = 1.0, device="cpu", _memo={}):
    """K and V [n, Hkv, d] (bf16) of a token sequence in which row t depends only on
    tokens[0 .. t] -- the way a model's KV depends on the context so far -- drawn
    N(0, sigma^2) from a generator seeded by the prefix's hash.  Sequences that share
    a prefix share its rows, whichever request computes them."""
    rows = []
    per = 2 * num_kv_heads * head_dim
    for h in prefix_hashes(tokens):
        key = (h, per, sigma)
        r = _memo.get(key)
        if r is None:
            r = np.random.default_rng([TOKEN_CONFIG_ID, h & 0xFFFFFFFF, h >> 32]).standard_normal(per) * sigma
            _memo[key] = r
        rows.append(r)
    x = torch.from_numpy(np.asarray(rows, dtype=np.float32).reshape(len(rows), 2, num_kv_heads, head_dim))
    x = x.to(torch.bfloat16).to(device)
    return x[:, 0].contiguous(), x[:, 1].contiguous()
