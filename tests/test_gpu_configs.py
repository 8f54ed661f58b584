"""The five agent-shaped configurations, and two decode steps, at full size on the GPU.

The whole batch runs through store_kv + extend_attention exactly as the benchmark
launches it; the oracle then checks sampled rows (first, last, page-boundary and
seeded random rows of seeded requests, always including the longest-prefix and
longest-extend requests), every output row is checked to be written and finite,
and the sampled requests' pool pages are compared bit for bit with the oracle's
KV store.
"""

import numpy as np
import pytest
import torch

from gpu_harness import GpuRun, compare, oracle_rows
from helpers import oracle_pool_for
from paper_2609_32278_amd import workloads as wl

pytestmark = pytest.mark.gpu

# name -> (requests sampled, rows per request)
SAMPLING = {
    "llama8b": (16, 16),
    "tail_outlier": (32, 16),
    "rr_partial": (8, 8),
    "wide70b": (8, 8),
    "wide70b_fp8": (8, 8),
    # decode steps (one row per request; the planner splits every long key range)
    "decode_llama8b": (32, 1),
    "decode_long": (12, 1),
}


def _sample_requests(w, k, seed=0):
    rng = np.random.default_rng([w.config_id, 3, seed])
    must = {int(np.argmax(w.prefix_lens)), int(np.argmax(w.extend_lens))}
    rest = [r for r in range(w.num_reqs) if r not in must]
    extra = rng.choice(rest, size=max(0, min(len(rest), k - len(must))), replace=False)
    return sorted(must | set(int(x) for x in extra))


@pytest.mark.parametrize("name,scaled_q", [(n, False) for n in SAMPLING] + [("wide70b", True)])
def test_full_config_parity(name, scaled_q):
    w = wl.make_workload(name)
    k, per = SAMPLING[name]
    reqs = _sample_requests(w, k)
    rows = wl.sample_rows(w, per, reqs=reqs)
    if name == "tail_outlier":
        # 32 rows spread over the 131072-token recompute
        e0 = int(w.extend_lens[0])
        extra = np.stack([np.zeros(32, np.int32), np.linspace(0, e0 - 1, 32).astype(np.int32)], 1)
        rows = np.unique(np.concatenate([rows, extra]), axis=0)
    print(f"[config] {name}: R={w.num_reqs} T={w.total_extend} pages={w.num_pages} sampled reqs={reqs} "
          f"rows={len(rows)} scaled_q={int(scaled_q)}", flush=True)
    run = GpuRun(w, scaled_q=scaled_q)
    try:
        run.store()
        out = run.attend()
        assert not torch.isnan(out).any(), "some output rows were not written"
        assert torch.isfinite(out.float()).all()
        print(f"[config] {name}: GPU done, running the oracle", flush=True)
        ref, gidx = oracle_rows(w, run.q, rows, scaled_q=scaled_q)
        got = out[torch.from_numpy(gidx).to(out.device)].float().cpu().numpy().astype(np.float64)
        compare(got, ref, name)
        # KV store: the sampled requests' pages, bit for bit
        sub = w.subset(reqs)
        t = {"k_hist": [], "v_hist": [], "k_ext": [], "v_ext": []}
        for r in reqs:
            kk, vv = wl.request_kv(w, r, "cuda")
            p = int(w.prefix_lens[r])
            t["k_hist"].append(kk[:p].cpu())
            t["v_hist"].append(vv[:p].cpu())
            t["k_ext"].append(kk[p:].cpu())
            t["v_ext"].append(vv[p:].cpu())
        t = {key: torch.cat(val) for key, val in t.items()}
        ref_pool = oracle_pool_for(sub, t)
        pages = np.concatenate([w.pages_of(r) for r in reqs]).astype(np.int32)
        gk, gv = run.read_pages(pages)
        assert np.array_equal(gk, ref_pool.k[sub.page_ids]), f"{name}: K pages differ"
        assert np.array_equal(gv, ref_pool.v[sub.page_ids]), f"{name}: V pages differ"
    finally:
        run.close()


def test_row_offsets_past_two_to_the_31():
    """Q and O of 300,000 suffix tokens x 64 query heads x 128 dims hold 2.46e9 elements,
    so the last rows' offsets pass 2^31: rows at both ends of both requests must
    match the oracle (64-bit row indexing in the kernel, the binding and the plan)."""
    w = wl.make_custom([0, 4096], [150000, 150000], 64, 8, 128, seed=31, name="offsets64")
    assert w.total_extend * w.num_q_heads * w.head_dim > 2 ** 31
    rows = np.array([[0, 0], [0, 149999], [1, 0], [1, 77777], [1, 149998], [1, 149999]], np.int32)
    print(f"[config] offsets64: T={w.total_extend} pages={w.num_pages} rows={len(rows)}", flush=True)
    run = GpuRun(w)
    try:
        run.store()
        out = run.attend()
        assert not torch.isnan(out[-1]).any() and not torch.isnan(out[0]).any()
        print("[config] offsets64: GPU done, running the oracle", flush=True)
        ref, gidx = oracle_rows(w, run.q, rows)
        got = out[torch.from_numpy(gidx).to(out.device)].float().cpu().numpy().astype(np.float64)
        compare(got, ref, "offsets64")
    finally:
        run.close()
