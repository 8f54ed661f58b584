"""The seeded workload generator: determinism, length recipes, page placement."""

import math

import numpy as np
import pytest
import torch

from paper_2609_32278_amd import workloads as wl

NAMES = ["tiny", "llama8b", "tail_outlier", "rr_partial", "wide70b", "wide70b_fp8"]


@pytest.mark.parametrize("name", NAMES)
@pytest.mark.parametrize("seed", [0, 1, 7])
def test_shapes_placement_and_determinism(name, seed):
    a = wl.make_workload(name, seed)
    b = wl.make_workload(name, seed)
    assert np.array_equal(a.prefix_lens, b.prefix_lens)
    assert np.array_equal(a.extend_lens, b.extend_lens)
    assert np.array_equal(a.page_ids, b.page_ids)
    need = (a.prefix_lens.astype(np.int64) + a.extend_lens + 15) // 16
    assert np.array_equal(np.diff(a.page_indptr), need)
    ids = a.page_ids
    assert ids.min() >= 0 and ids.max() < a.num_pages
    assert len(np.unique(ids)) == len(ids)            # no page shared between requests
    if name != "tiny":
        assert a.num_pages == math.ceil(1.5 * int(need.sum()))


def test_length_recipes():
    t = wl.make_workload("tiny")
    assert t.prefix_lens.tolist() == [0, 64, 208, 512] and t.extend_lens.tolist() == [32, 16, 100, 8]
    assert t.num_pages == 256 and (t.num_q_heads, t.num_kv_heads, t.head_dim) == (4, 2, 64)
    for seed in range(5):
        c2 = wl.make_workload("llama8b", seed)
        assert ((c2.prefix_lens % 16) == 0).all()
        assert c2.prefix_lens.min() >= 4096 and c2.prefix_lens.max() <= 32768
        assert c2.extend_lens.min() >= 64 and c2.extend_lens.max() <= 2048
        assert c2.sigma == 0.5 and c2.num_reqs == 16
        c3 = wl.make_workload("tail_outlier", seed)
        assert c3.prefix_lens[0] == 0 and c3.extend_lens[0] == 131072 and c3.num_reqs == 32
        assert ((c3.prefix_lens[1:] >= 32768) & (c3.prefix_lens[1:] <= 98304)).all()
        assert ((c3.extend_lens[1:] >= 256) & (c3.extend_lens[1:] <= 1024)).all()
        c4 = wl.make_workload("rr_partial", seed)
        # context floored to the page size, minus k whole 2048-token tail chunks
        assert (c4.prefix_lens >= 0).all() and ((c4.prefix_lens % 16) == 0).all()
        assert (c4.prefix_lens + c4.extend_lens >= 8192 + 128).all()
        assert c4.num_reqs == 64 and c4.extend_lens.min() >= 2048 + 128
        assert c4.extend_lens.max() <= 4 * 2048 + 4096
        c5 = wl.make_workload("wide70b", seed)
        c5f = wl.make_workload("wide70b_fp8", seed)
        assert np.array_equal(c5.prefix_lens, c5f.prefix_lens)
        assert np.array_equal(c5.page_ids, c5f.page_ids)
        assert c5.prefix_lens.min() >= 16384 and c5.prefix_lens.max() <= 262144
        assert c5f.kv_dtype == wl.KV_FP8_E4M3 and c5.kv_dtype == wl.KV_BF16
        assert ((c5f.k_scale >= 0.01) & (c5f.k_scale <= 0.1)).all() and c5f.v_scale.shape == (8,)
        assert (c5.num_q_heads, c5.num_kv_heads) == (64, 8)


def test_values_are_seeded_bf16_and_per_request():
    w = wl.make_workload("tiny")
    q1 = wl.request_q(w, 2)
    q2 = wl.request_q(w, 2)
    assert q1.dtype == torch.bfloat16 and q1.shape == (100, 4, 64)
    assert torch.equal(q1, q2)
    k, v = wl.request_kv(w, 3)
    assert k.shape == (520, 2, 64) and not torch.equal(k, v)
    t = wl.batch_tensors(w)
    assert t["q"].shape == (156, 4, 64) and t["k_hist"].shape == (784, 2, 64)
    assert torch.equal(t["k_ext"][-8:], k[512:])
    # the value distribution is N(0, sigma^2) rounded to bf16
    x = t["k_hist"].float()
    assert abs(float(x.mean())) < 0.05 and abs(float(x.std()) - 1.0) < 0.05


def test_history_batch_and_subset():
    w = wl.make_workload("tiny")
    h = wl.history_batch(w)
    assert h.extend_lens.tolist() == w.prefix_lens.tolist() and (h.prefix_lens == 0).all()
    for r in range(w.num_reqs):
        n = len(h.pages_of(r))
        assert np.array_equal(h.pages_of(r), w.pages_of(r)[:n])
    s = w.subset([3, 1])
    assert s.prefix_lens.tolist() == [512, 64]
    assert s.page_ids.tolist() == list(range(len(s.page_ids)))
    # a subset regenerates the same values for the same requests
    assert torch.equal(wl.request_q(s, 0), wl.request_q(w, 3))
    assert torch.equal(wl.request_kv(s, 1)[1], wl.request_kv(w, 1)[1])


def test_sample_rows_cover_ends_and_page_boundaries():
    w = wl.make_workload("llama8b")
    rows = wl.sample_rows(w, 16)
    for r in range(w.num_reqs):
        mine = rows[rows[:, 0] == r, 1]
        assert 0 in mine and (w.extend_lens[r] - 1) in mine and len(mine) == 16


def test_flops_formula_matches_pair_count():
    w = wl.make_custom([3, 0], [2, 4], 2, 1, 8)
    # request 0 rows see 4 and 5 keys; request 1 rows see 1..4 keys
    assert w.visible_pairs() == 4 + 5 + 1 + 2 + 3 + 4
    assert w.flops() == 4 * 8 * 2 * w.visible_pairs()
