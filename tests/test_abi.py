"""The C ABI on the CPU: the library loads, exports every declared symbol, rejects
bad arguments before touching the device, and its work plan covers every visible
(query row, key) pair exactly once."""

import os
import re

import numpy as np
import pytest
from hypothesis import assume, given, settings, strategies as st

from paper_2609_32278_amd import kvx
from paper_2609_32278_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
TILE_ROWS = int(re.search(r"#define KVX_TILE_ROWS (\d+)", open(os.path.join(ROOT, "include", "kvx.h")).read()).group(1))


@pytest.fixture(scope="module", autouse=True)
def _built():
    if not os.path.exists(kvx.LIB_PATH):
        from paper_2609_32278_amd import build
        build.build()


def _declared_functions():
    names = set()
    for h in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if not h.endswith(".h"):
            continue
        text = open(os.path.join(ROOT, "include", h)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"^\s*(?:int|const char\s*\*)\s*(\w+)\s*\(", text, flags=re.M))
    return sorted(names)


def test_every_declared_symbol_is_exported():
    names = _declared_functions()
    assert set(names) == set(kvx.EXPORTS), names
    lib = kvx.lib()
    for n in names:
        assert hasattr(lib, n), n


def _err(fn, *a):
    with pytest.raises(kvx.KvxError) as e:
        fn(*a)
    assert kvx.kvx_last_error() != ""
    return e.value.status


def test_pool_argument_errors():
    assert _err(kvx.kv_pool_create, 0, 16, 2, 64) == kvx.KVX_EINVAL
    assert _err(kvx.kv_pool_create, 10, 8, 2, 64) == kvx.KVX_EUNSUPPORTED
    assert _err(kvx.kv_pool_create, 10, 16, 2, 96) == kvx.KVX_EUNSUPPORTED
    assert _err(kvx.kv_pool_create, 10, 16, 0, 64) == kvx.KVX_EINVAL
    assert _err(kvx.kv_pool_create, 10, 16, 2, 64, kvx.KVX_KV_FP8_E4M3) == kvx.KVX_EUNSUPPORTED
    assert _err(kvx.kv_pool_create, 10, 16, 2, 64, kvx.KVX_KV_FP8_E4M3, [1.0, 0.0], [1.0, 1.0]) == kvx.KVX_EINVAL
    assert _err(kvx.kv_pool_create, 10, 16, 2, 64, 7) == kvx.KVX_EINVAL
    assert _err(kvx.kv_pool_set_split_keys, None, 64) == kvx.KVX_EINVAL
    assert _err(kvx.kv_pool_set_scaled_q, None, True) == kvx.KVX_EINVAL
    assert _err(kvx.kv_pool_layout, None) == kvx.KVX_EINVAL


def test_hot_path_argument_errors_before_any_device_work():
    b = kvx.Batch([16], [4], [0, 2], 0x1000)
    assert _err(kvx.store_kv, None, b, 1, 1) == kvx.KVX_EINVAL
    assert _err(lambda: kvx.store_kv_rope(None, b, 1, 1, rotary_dim=64)) == kvx.KVX_EINVAL
    assert _err(kvx.extend_attention, None, b, 1, 4, 0.125, 1) == kvx.KVX_EINVAL
    # plan-level checks
    assert _err(kvx.extend_attention_plan, b, 6, 4, 128) == kvx.KVX_EINVAL      # 6 % 4 != 0
    assert _err(kvx.extend_attention_plan, b, 4, 2, 80) == kvx.KVX_EUNSUPPORTED  # head_dim
    assert _err(kvx.extend_attention_plan, b, 1024, 2, 128) == kvx.KVX_EUNSUPPORTED  # > 256 q heads per kv head
    short = kvx.Batch([16], [17], [0, 2], 0x1000)                                # 33 tokens need 3 pages
    assert _err(kvx.extend_attention_plan, short, 4, 2, 128) == kvx.KVX_EINVAL
    neg = kvx.Batch([-1], [4], [0, 1], 0x1000)
    assert _err(kvx.extend_attention_plan, neg, 4, 2, 128) == kvx.KVX_EINVAL
    bad0 = kvx.Batch([0], [4], [1, 2], 0x1000)
    assert _err(kvx.extend_attention_plan, bad0, 4, 2, 128) == kvx.KVX_EINVAL
    ok = kvx.Batch([16], [4], [0, 2], 0x1000)
    assert _err(kvx.extend_attention_plan, ok, 4, 2, 128, 100) == kvx.KVX_EINVAL  # split not a multiple of 64
    assert _err(kvx.extend_attention_plan, ok, 4, 2, 128, -64) == kvx.KVX_EINVAL


def test_binding_rejects_short_buffers_and_ragged_lengths():
    import torch
    kvx._need(torch.empty(8, dtype=torch.int16), 16, "x")  # exactly enough
    with pytest.raises(ValueError):
        kvx._need(torch.empty(7, dtype=torch.int16), 16, "x")
    kvx._need(0x1000, 1 << 40, "raw address")  # raw addresses are not checked
    kvx._need(None, 16, "absent")
    with pytest.raises(ValueError):
        kvx.Batch([16, 0], [4], [0, 2, 2], 0x1000)  # extend_lens one short
    with pytest.raises(ValueError):
        kvx.Batch([16], [4], [0, 2, 2], 0x1000)  # page_indptr one too long
    with pytest.raises(ValueError, match="int32"):
        kvx.Batch([16], [4], [0, 2], torch.zeros(2, dtype=torch.int64))  # int64 page ids


def _check_plan(w, split=0):
    b = kvx.Batch(w.prefix_lens, w.extend_lens, w.page_indptr, 0)
    items = kvx.extend_attention_plan(b, w.num_q_heads, w.num_kv_heads, w.head_dim, split)
    g = w.group
    tile_tok = TILE_ROWS // g
    real = items[items["req"] >= 0]
    # dispatch position i runs on XCD i % 8
    assert (items["xcd"] == np.arange(len(items)) % 8).all()
    # every (request, kv head, suffix token) covered by exactly one tile; every tile's
    # key range [0, P + last token] partitioned by its parts at multiples of 64
    seen = {}
    parts = set()
    for it in real:
        key = (int(it["req"]), int(it["kv_head"]), int(it["tok_begin"]))
        seen.setdefault(key, []).append((int(it["key_begin"]), int(it["key_end"]), int(it["part"]),
                                         int(it["tok_count"])))
        if it["part"] >= 0:
            assert it["part"] not in parts
            parts.add(int(it["part"]))
    if parts:
        assert parts == set(range(len(parts)))
    for r in range(w.num_reqs):
        P, E = int(w.prefix_lens[r]), int(w.extend_lens[r])
        for h in range(w.num_kv_heads):
            covered = np.zeros(E, np.int32)
            for t0 in range(0, E, tile_tok):
                rng = sorted(seen.pop((r, h, t0)))
                ntok = min(tile_tok, E - t0)
                assert all(x[3] == ntok for x in rng)
                covered[t0:t0 + ntok] += 1
                assert rng[0][0] == 0 and rng[-1][1] == P + t0 + ntok
                for (a, b_, pa, _), (c, _, pc, _) in zip(rng, rng[1:]):
                    assert b_ == c and b_ % 64 == 0
                    # earlier parts hold keys every row of the tile sees, so each part's first
                    # key is visible to all its rows (the attention kernel takes that key's
                    # tile maximum as its softmax reference)
                    assert b_ <= P + t0
                assert (len(rng) == 1) == (rng[0][2] == -1)
            assert (covered == 1).all()
    assert not seen
    # longest first within an XCD, by request then by tile
    return items


@settings(max_examples=40, deadline=None, derandomize=True)
@given(st.data())
def test_plan_covers_drawn_batches(data):
    """The coverage check of the work plan on ragged batches hypothesis draws, with
    and without forced key splits."""
    r = data.draw(st.integers(1, 6), label="requests")
    prefix = data.draw(st.lists(st.integers(0, 3000), min_size=r, max_size=r), label="prefix_lens")
    extend = data.draw(st.lists(st.integers(0, 600), min_size=r, max_size=r), label="extend_lens")
    assume(sum(extend) > 0)
    hkv = data.draw(st.sampled_from([1, 2, 3, 8]), label="kv_heads")
    g = data.draw(st.sampled_from([1, 4, 8]), label="group")
    split = data.draw(st.sampled_from([0, 0, 64, 1024]), label="split_keys")
    w = wl.make_custom(prefix, extend, hkv * g, hkv, 128, seed=1)
    _check_plan(w, split)


@pytest.mark.parametrize("name", ["tiny", "llama8b", "tail_outlier", "rr_partial", "wide70b", "decode_llama8b",
                                  "decode_long"])
def test_plan_covers_every_visible_pair_once(name):
    _check_plan(wl.make_workload(name))


def test_decode_steps_get_key_chunks_of_one_token():
    """A batch of one-token suffixes (a decode step) is planned as key chunks of
    (request, KV head), split so that the step fills the chip."""
    w = wl.make_workload("decode_long")
    b = kvx.Batch(w.prefix_lens, w.extend_lens, w.page_indptr, 0)
    items = kvx.extend_attention_plan(b, w.num_q_heads, w.num_kv_heads, w.head_dim)
    assert (items["tok_count"] == 1).all() and (items["tok_begin"] == 0).all()
    assert len(items) >= 1024 and (items["part"] >= 0).all()
    # a batch with a longer suffix anywhere goes through the prefill tiles instead
    w2 = wl.make_custom([5000, 300], [1, 2], 32, 8, 128)
    b2 = kvx.Batch(w2.prefix_lens, w2.extend_lens, w2.page_indptr, 0)
    items2 = kvx.extend_attention_plan(b2, 32, 8, 128)
    assert (items2["tok_count"] == 2).any()


@pytest.mark.parametrize("split", [64, 1024])
def test_plan_with_forced_splits(split):
    w = wl.make_custom([3000, 129, 0, 77], [70, 200, 300, 1], 12, 2, 128)
    items = _check_plan(w, split)
    assert (items["part"] >= 0).any()


def test_plan_splits_decode_like_batches_automatically():
    w = wl.make_custom([32768], [64], 32, 8, 128)
    items = _check_plan(w)
    real = items[items["req"] >= 0]
    # one round that fills at least 90% of the 256 workgroup slots (not 264 units,
    # whose last 8 would run as a second round)
    assert 0.9 * 256 <= len(real) <= 256 and (real["part"] >= 0).all()


def test_plan_balances_xcds_for_eight_kv_heads():
    w = wl.make_workload("rr_partial")
    b = kvx.Batch(w.prefix_lens, w.extend_lens, w.page_indptr, 0)
    items = kvx.extend_attention_plan(b, w.num_q_heads, w.num_kv_heads, w.head_dim)
    real = items[items["req"] >= 0]
    assert (real["xcd"] == real["kv_head"] % 8).all()
    cost = np.zeros(8)
    np.add.at(cost, real["xcd"], (real["key_end"] - real["key_begin"]).astype(np.float64))
    assert cost.max() / cost.min() < 1.0001


@pytest.mark.parametrize("hkv,extend", [(1, [53, 200]), (2, [53, 200]), (1, [1, 1])])
def test_plan_spreads_few_long_requests_over_all_xcds(hkv, extend):
    """Two requests with 4M- and 1M-token prefixes and 1-2 KV heads: the planner
    splits their key ranges, and binds each (request, KV head, part) rather than
    each (request, KV head), so all eight XCDs carry work; units that read the same
    key range of one (request, KV head) stay on one XCD."""
    w = wl.make_custom([4194319, 1048577], extend, 8 * hkv, hkv, 128, seed=41)
    items = _check_plan(w)
    real = items[items["req"] >= 0]
    assert (real["part"] >= 0).all()
    cost = np.zeros(8)
    np.add.at(cost, real["xcd"], (real["key_end"] - real["key_begin"]).astype(np.float64))
    assert cost.max() / cost.mean() < 1.15, cost
    if extend[0] > 1:
        xcd_of = {}
        for it in real:
            key = (int(it["req"]), int(it["kv_head"]), int(it["key_begin"]))
            assert xcd_of.setdefault(key, int(it["xcd"])) == int(it["xcd"])


@pytest.mark.parametrize("prefix,extend,hq,hkv", [
    ([131072], [512], 32, 8),                    # one returning agent
    ([200000], [300], 64, 8),
    ([4194319, 1048577], [53, 200], 8, 1),
    ([4194319, 1048577], [53, 200], 16, 2),
])
def test_split_parts_fill_whole_rounds(prefix, extend, hq, hkv):
    """A few tiles with long key ranges: the automatic split would leave a unit count
    a little past two rounds of the 256 workgroup slots (519-576 units); the planner
    lengthens the parts just enough to fit two rounds, and every visible pair is
    still covered once."""
    w = wl.make_custom(prefix, extend, hq, hkv, 128, seed=41)
    items = _check_plan(w)
    real = items[items["req"] >= 0]
    assert (real["part"] >= 0).any()
    assert 256 < len(real) <= 512, len(real)
    # a forced split length is kept as given: parts start at its multiples, and every
    # part but a tile's last is exactly that long
    f = 30720
    forced = _check_plan(w, f)
    fr = forced[(forced["req"] >= 0) & (forced["part"] >= 0)]
    lens = fr["key_end"] - fr["key_begin"]
    assert (fr["key_begin"] % f == 0).all() and (lens == f).any() and (lens <= f + 256).all()


def test_headers_compile_as_c99_and_work_from_c(tmp_path):
    """A C99 program (tests/c_abi/consumer.c) includes both public headers with
    -pedantic -Werror, links libkvx.so and calls the host-only entry points."""
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("gcc not installed")
    exe = str(tmp_path / "consumer")
    lib_dir = os.path.dirname(kvx.LIB_PATH)
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror", "-I" + os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "c_abi", "consumer.c"), "-L" + lib_dir, "-l:libkvx.so",
           "-Wl,-rpath," + lib_dir, "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    run = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "cache cycle ok" in run.stdout


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    """With no built libkvx.so the binding raises KvxNotBuilt on first use: there
    is no CPU or torch fallback on the product path."""
    monkeypatch.setattr(kvx, "_lib", None)
    monkeypatch.setattr(kvx, "LIB_PATH", str(tmp_path / "libkvx.so"))
    with pytest.raises(kvx.KvxNotBuilt):
        kvx.lib()
    with pytest.raises(kvx.KvxNotBuilt):
        kvx.extend_attention_plan(kvx.Batch([0], [4], [0, 1], 0x1000), 4, 2, 128)
