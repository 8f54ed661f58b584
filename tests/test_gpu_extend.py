"""extend_attention on the GPU against the CPU oracle: small cases run in full
(several tiles and ragged tails), plus the invariances prefix reuse relies on."""

import math

import numpy as np
import pytest
import torch

from gpu_harness import DEV, GpuRun, compare, oracle_rows
from paper_2609_32278_amd import kvx
from paper_2609_32278_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _f64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def _run_and_compare(w, tag, want_lse=False, fill=None, split_keys=0, scaled_q=False):
    print(f"[extend] {tag}: R={w.num_reqs} T={w.total_extend} Hq={w.num_q_heads} Hkv={w.num_kv_heads} "
          f"d={w.head_dim} fp8={w.kv_dtype} split={split_keys} scaled_q={int(scaled_q)}", flush=True)
    run = GpuRun(w, fill_bits=fill, split_keys=split_keys, scaled_q=scaled_q)
    try:
        run.store()
        res = run.attend(want_lse=want_lse)
        out, lse = (res if want_lse else (res, None))
        # an fp8 pool's prefill kernel always scales Q; its reference stays the exact
        # attention over the dequantised pool
        ref, gidx = oracle_rows(w, run.q, None, want_lse=want_lse, scaled_q=scaled_q and w.kv_dtype == wl.KV_BF16)
        if want_lse:
            ref, ref_lse = ref
        got = _f64(out)[gidx]
        compare(got, ref, tag)
        if want_lse:
            lerr = np.abs(lse.cpu().numpy()[gidx] - ref_lse).max()
            print(f"[parity] {tag}: lse max err {lerr:.3e}", flush=True)
            assert lerr <= 2e-3 * max(1.0, float(np.abs(ref_lse).max()))
        return out
    finally:
        run.close()


def test_tiny_config_every_row():
    _run_and_compare(wl.make_workload("tiny"), "tiny", want_lse=True)


CASES = {
    # unaligned prefixes, an empty suffix, single-token suffixes, ragged tails
    "ragged_g4_d128": ([0, 5, 16, 37, 100, 3, 1000], [7, 0, 1, 29, 18, 40, 200], 8, 2, 128, wl.KV_BF16),
    "g1_d64": ([0, 64, 129], [130, 17, 64], 4, 4, 64, wl.KV_BF16),
    "g6_d128": ([33, 0], [45, 70], 12, 2, 128, wl.KV_BF16),
    "g16_d64": ([80, 1], [19, 33], 32, 2, 64, wl.KV_BF16),
    "g8_fp8_d128": ([300, 16, 0], [57, 129, 40], 16, 2, 128, wl.KV_FP8_E4M3),
    "g2_fp8_d64": ([7, 200], [99, 3], 4, 2, 64, wl.KV_FP8_E4M3),
    "decode_like": ([5000, 3001, 64], [1, 1, 1], 8, 1, 128, wl.KV_BF16),
    # decode steps on the decode kernel: fp8 pool, 16 heads per KV head, an empty
    # prefix (a single key), a request with no suffix at all
    "decode_fp8_g8_d128": ([3000, 77, 1025], [1, 1, 1], 16, 2, 128, wl.KV_FP8_E4M3),
    "decode_g16_d64": ([700, 16, 0, 4100], [1, 1, 1, 0], 32, 2, 64, wl.KV_BF16),
    "decode_fp8_d64": ([9000, 33], [1, 1], 8, 4, 64, wl.KV_FP8_E4M3),
    "long_causal": ([0], [1000], 4, 1, 128, wl.KV_BF16),
    # wide groups: 32 and the maximum 256 query heads per KV head (8 and 1 tokens per
    # tile); a one-token batch above the decode kernel's group limit (prefill path)
    "g32_d128": ([100, 3, 0], [40, 9, 17], 32, 1, 128, wl.KV_BF16),
    "g256_d64": ([50, 0], [5, 3], 256, 1, 64, wl.KV_BF16),
    "decode_g32_fp8": ([500, 20], [1, 1], 64, 2, 128, wl.KV_FP8_E4M3),
    # KV head counts off the XCD count: 3 (greedy XCD binding) and 16
    "hkv3_fp8_d128": ([129, 40, 0, 700], [60, 1, 33, 90], 6, 3, 128, wl.KV_FP8_E4M3),
    "hkv16_d64": ([16, 250], [70, 31], 32, 16, 64, wl.KV_BF16),
}


@pytest.mark.parametrize("name", list(CASES))
def test_edge_cases_every_row(name):
    p, e, hq, hkv, d, dt = CASES[name]
    w = wl.make_custom(p, e, hq, hkv, d, kv_dtype=dt, seed=len(name))
    _run_and_compare(w, name, want_lse=True)


def test_sharpened_queries():
    w = wl.make_custom([40, 300, 0], [90, 33, 77], 8, 2, 128, q_sigma=4.0, seed=9)
    _run_and_compare(w, "sharpened")


# The scaled-Q mode (kv_pool_set_scaled_q): the folded softmax on bf16 pools,
# every row against the oracle's definition of the mode (queries rounded to bf16
# after scaling, scores in base 2) at the same gate.
SCALED = ["ragged_g4_d128", "g1_d64", "g6_d128", "g16_d64", "long_causal", "g32_d128", "g256_d64", "hkv16_d64"]


@pytest.mark.parametrize("name", SCALED)
def test_scaled_q_mode_every_row(name):
    p, e, hq, hkv, d, dt = CASES[name]
    w = wl.make_custom(p, e, hq, hkv, d, kv_dtype=dt, seed=len(name))
    _run_and_compare(w, f"scaled_{name}", want_lse=True, scaled_q=True)


@pytest.mark.parametrize("q_sigma", [1.0, 4.0])
def test_scaled_q_mode_sharpened_queries(q_sigma):
    w = wl.make_custom([40, 300, 0], [90, 33, 77], 8, 2, 128, q_sigma=q_sigma, seed=9)
    _run_and_compare(w, f"scaled_sharp{q_sigma:g}", want_lse=True, scaled_q=True)


def test_scaled_q_mode_with_forced_splits():
    w = wl.make_custom([1000, 77], [130, 64], 8, 2, 128, seed=21)
    _run_and_compare(w, "scaled_split", want_lse=True, split_keys=128, scaled_q=True)


def test_scaled_q_setting_leaves_fp8_prefill_and_decode_steps_unchanged():
    """An fp8 pool's prefill kernel always takes the folded form, and decode steps
    are always exact: the setting changes no bit of their outputs.  A value other
    than 0 or 1 is rejected."""
    for name in ["g8_fp8_d128", "decode_like"]:
        p, e, hq, hkv, d, dt = CASES[name]
        w = wl.make_custom(p, e, hq, hkv, d, kv_dtype=dt, seed=len(name))
        run = GpuRun(w)
        try:
            run.store()
            a = run.attend()
            kvx.kv_pool_set_scaled_q(run.pool, True)
            b = run.attend()
            assert kvx.lib().kv_pool_set_scaled_q(run.pool, 2) == kvx.KVX_EINVAL
        finally:
            run.close()
        assert torch.equal(a.view(torch.int16), b.view(torch.int16)), name


@pytest.mark.parametrize("split", [64, 128, 1024])
def test_forced_key_split_matches_oracle(split):
    w = wl.make_custom([3000, 129, 0], [70, 200, 300], 8, 2, 128, seed=10)
    _run_and_compare(w, f"split{split}", want_lse=True, split_keys=split)


def test_single_key_returns_value_bits():
    for dt in (wl.KV_BF16, wl.KV_FP8_E4M3):
        w = wl.make_custom([0], [1], 4, 2, 128, kv_dtype=dt, seed=2)
        print(f"[extend] single key fp8={dt}", flush=True)
        run = GpuRun(w)
        try:
            run.store()
            out = run.attend().cpu()
            v0 = run.v_ext[0].cpu()  # [Hkv, d]
            if dt == wl.KV_FP8_E4M3:
                s = torch.from_numpy(w.v_scale)
                code = (v0.float() * (1.0 / s)[:, None]).clamp(-448, 448).to(torch.float8_e4m3fn)
                v0 = (code.float() * s[:, None]).to(torch.bfloat16)
            expect = v0.repeat_interleave(2, dim=0)
            assert torch.equal(out[0].view(torch.int16), expect.view(torch.int16))
        finally:
            run.close()


def test_page_permutation_gives_bitwise_identical_outputs():
    outs = []
    for seed in (1, 2, 3):
        w = wl.make_custom([300, 17, 64], [100, 60, 5], 8, 2, 128, seed=seed, num_pages=128)
        w.seed = 0  # same values, different placement
        print(f"[extend] placement {seed}", flush=True)
        run = GpuRun(w)
        try:
            run.store()
            outs.append(run.attend().cpu())
        finally:
            run.close()
    assert torch.equal(outs[0].view(torch.int16), outs[1].view(torch.int16))
    assert torch.equal(outs[0].view(torch.int16), outs[2].view(torch.int16))


@pytest.mark.parametrize("kv_dtype", [wl.KV_BF16, wl.KV_FP8_E4M3])
def test_poisoned_unused_slots_do_not_change_outputs(kv_dtype):
    """Slots past a request's last key (in its last page) hold whatever the pool held;
    zero, NaN and large values there must leave every output bit unchanged.  On an fp8
    pool the poison is a code: 0, NaN (0x7F) and the largest finite value (0x7E)."""
    outs = []
    fills = (0x0000, 0x7FC0, 0x461C) if kv_dtype == wl.KV_BF16 else (0x00, 0x7F, 0x7E)
    for fill in fills:
        w = wl.make_custom([21, 130], [30, 9], 4, 1, 128, kv_dtype=kv_dtype, seed=6, num_pages=40)
        print(f"[extend] poison {fill:#x} fp8={kv_dtype}", flush=True)
        run = GpuRun(w, fill_bits=fill)
        try:
            run.store()
            outs.append(run.attend().cpu())
        finally:
            run.close()
    assert not torch.isnan(outs[1].float()).any()
    assert torch.equal(outs[0].view(torch.int16), outs[1].view(torch.int16))
    assert torch.equal(outs[0].view(torch.int16), outs[2].view(torch.int16))


def test_constant_values_give_the_constant():
    c = 0.71875
    w = wl.make_custom([100, 0], [40, 300], 8, 2, 128, seed=7)
    shapes = {r: (int(w.prefix_lens[r] + w.extend_lens[r]), 2, 128) for r in range(w.num_reqs)}
    run = GpuRun(w, overrides={"kv": lambda r: (wl.request_kv(w, r, DEV)[0],
                                                  torch.full(shapes[r], c, dtype=torch.bfloat16, device=DEV))})
    try:
        run.store()
        out = run.attend().float().cpu()
        assert (out - c).abs().max().item() <= c * 2.0 ** -7
    finally:
        run.close()


@pytest.mark.parametrize("where", ["prefix", "page_boundary", "diagonal"])
def test_needle_key_dominates(where):
    P, E, d = 200, 50, 128
    w = wl.make_custom([P], [E], 4, 1, d, seed=12, sigma=0.05)
    i = E - 1
    j = {"prefix": 7, "page_boundary": 192, "diagonal": P + i}[where]
    q = wl.request_q(w, 0, DEV)
    k, v = wl.request_kv(w, 0, DEV)
    qv = q[i, 0].double()
    needle = (qv * (60.0 * math.sqrt(d) / float(qv.norm()) ** 2)).to(torch.bfloat16)
    k = k.clone()
    v = v.clone()
    k[j, 0] = needle
    v[j, 0] = 3.0
    run = GpuRun(w, overrides={"kv": lambda r: (k, v), "q": lambda r: q})
    try:
        run.store()
        out = run.attend().float().cpu()
        # query head 0 sees the needle with a logit margin of ~60: output = V_j
        assert (out[i, 0] - 3.0).abs().max().item() <= 3.0 * 2.0 ** -7
    finally:
        run.close()


# A few query rows are aimed at one key far past the unit's first tile, with a
# logit margin of about 200 (natural units) over every other key: exponentials
# against the first tile's maximum overflow fp32 there, and the rows must still
# come out as the oracle's (nearly one-hot) softmax of that key.
FAR_ABOVE = {
    "bf16_tile3": (wl.KV_BF16, False, 128, "tile3", 0),
    "bf16_diagonal": (wl.KV_BF16, False, 128, "diagonal", 0),
    "bf16_d64_tile3": (wl.KV_BF16, False, 64, "tile3", 0),
    "scaled_q_tile3": (wl.KV_BF16, True, 128, "tile3", 0),
    "scaled_q_diagonal": (wl.KV_BF16, True, 128, "diagonal", 0),
    "fp8_tile3": (wl.KV_FP8_E4M3, False, 128, "tile3", 0),
    "fp8_diagonal": (wl.KV_FP8_E4M3, False, 128, "diagonal", 0),
    "bf16_split": (wl.KV_BF16, False, 128, "tile3", 128),
    "fp8_split": (wl.KV_FP8_E4M3, False, 128, "diagonal", 128),
    "fp8_d64_tile3": (wl.KV_FP8_E4M3, False, 64, "tile3", 0),
}


@pytest.mark.parametrize("name", sorted(FAR_ABOVE))
def test_scores_far_above_the_first_tile(name):
    kv_dtype, scaled_q, d, where, split = FAR_ABOVE[name]
    P, E, B = 200, 60, 12.0
    w = wl.make_custom([P, 90], [E, 50], 8, 2, d, kv_dtype=kv_dtype, seed=31)
    g = torch.Generator().manual_seed(5)
    u = torch.randn(d, generator=g, dtype=torch.float64)
    u /= u.norm()
    a = 200.0 * math.sqrt(d) / B  # logit A B / sqrt(d) = 200
    hot = [10, 33, E - 1]
    q0 = wl.request_q(w, 0, DEV).clone()
    k0, v0 = (t.clone() for t in wl.request_kv(w, 0, DEV))
    for i in hot:
        j = {"tile3": 3 * 64 + 5, "diagonal": P + i}[where]
        q0[i, 0] = (a * u).to(torch.bfloat16).to(DEV)
        k0[j, 0] = (B * u).to(torch.bfloat16).to(DEV)
        v0[j, 0] = 3.0
    kv = lambda r: (k0, v0) if r == 0 else wl.request_kv(w, r, DEV)
    qq = lambda r: q0 if r == 0 else wl.request_q(w, r, DEV)
    print(f"[extend] far_above {name}: d={d} fp8={kv_dtype} scaled_q={int(scaled_q)} split={split}", flush=True)
    run = GpuRun(w, overrides={"kv": kv, "q": qq}, split_keys=split, scaled_q=scaled_q)
    try:
        run.store()
        out, lse = run.attend(want_lse=True)
        ref, gidx = oracle_rows(w, run.q, None, want_lse=True, kv_override=kv,
                                scaled_q=scaled_q and kv_dtype == wl.KV_BF16)
        ref, ref_lse = ref
        compare(_f64(out)[gidx], ref, f"far_above_{name}")
        lerr = np.abs(lse.cpu().numpy()[gidx] - ref_lse).max()
        print(f"[parity] far_above_{name}: lse max err {lerr:.3e}", flush=True)
        assert lerr <= 2e-3 * max(1.0, float(np.abs(ref_lse).max()))
        # the aimed rows really are dominated by the key they aim at
        assert float(ref_lse[hot, 0].min()) > 150.0
    finally:
        run.close()


@pytest.mark.parametrize("kv_dtype", [wl.KV_BF16, wl.KV_FP8_E4M3])
def test_split_invariance_across_page_boundaries(kv_dtype):
    """One logical sequence, cut into cached prefix + suffix at several page
    boundaries: the rows past the last cut agree with each other within the gate.
    On an fp8 pool the suffix is read back dequantised like the prefix, so the cut
    does not change what any row sees either (one set of per-head scales)."""
    total, hq, hkv, d = 700, 8, 2, 128
    base = wl.make_custom([0], [total], hq, hkv, d, seed=13, kv_dtype=kv_dtype)
    q_all = wl.request_q(base, 0, DEV)
    k_all, v_all = wl.request_kv(base, 0, DEV)
    cuts = [0, 16, 320, 640]
    rows = []
    for cut in cuts:
        w = wl.make_custom([cut], [total - cut], hq, hkv, d, seed=13 + cut, kv_dtype=kv_dtype,
                           k_scale=base.k_scale, v_scale=base.v_scale)
        print(f"[extend] cut {cut} fp8={kv_dtype}", flush=True)
        run = GpuRun(w, overrides={"kv": lambda r: (k_all, v_all), "q": lambda r: q_all[cut:]})
        try:
            run.store()
            out = run.attend()
            rows.append(_f64(out)[cuts[-1] - cut:])
        finally:
            run.close()
    for r in rows[1:]:
        err = np.abs(r - rows[0])
        assert err.max() <= 2e-2 and err.mean() <= 2e-3


def test_empty_batches_are_no_ops():
    pool = kvx.kv_pool_create(8, 16, 2, 64)
    try:
        out = torch.full((4, 4, 64), 7.0, dtype=torch.bfloat16, device=DEV)
        ids = torch.zeros(2, dtype=torch.int32, device=DEV)
        b0 = kvx.Batch([], [], [0], ids)
        kvx.extend_attention(pool, b0, out, 4, 0.125, out)
        b1 = kvx.Batch([16, 3], [0, 0], [0, 1, 2], ids)
        kvx.store_kv(pool, b1, out, out)
        kvx.extend_attention(pool, b1, out, 4, 0.125, out)
        torch.cuda.synchronize()
        assert (out.float() == 7.0).all()
    finally:
        kvx.kv_pool_destroy(pool)


def test_validation_mode_rejects_out_of_range_pages(monkeypatch):
    monkeypatch.setenv("KVX_VALIDATE", "1")
    pool = kvx.kv_pool_create(8, 16, 1, 64)
    try:
        ids = torch.tensor([3, 8], dtype=torch.int32, device=DEV)  # 8 is outside the pool
        b = kvx.Batch([16], [4], [0, 2], ids)
        x = torch.zeros((4, 1, 64), dtype=torch.bfloat16, device=DEV)
        with pytest.raises(kvx.KvxError) as e:
            kvx.store_kv(pool, b, x, x)
        assert e.value.status == kvx.KVX_ERANGE
        q = torch.zeros((4, 2, 64), dtype=torch.bfloat16, device=DEV)
        with pytest.raises(kvx.KvxError) as e:
            kvx.extend_attention(pool, b, q, 2, 0.125, q)
        assert e.value.status == kvx.KVX_ERANGE
    finally:
        kvx.kv_pool_destroy(pool)


def test_binding_rejects_buffers_smaller_than_the_call():
    """The Python binding checks tensor sizes against the batch and the pool before
    the C call, so an undersized tensor raises instead of reaching a kernel."""
    pool = kvx.kv_pool_create(8, 16, 2, 64)
    try:
        ids = torch.arange(2, dtype=torch.int32, device=DEV)
        b = kvx.Batch([16], [4], [0, 2], ids)
        q = torch.zeros((4, 4, 64), dtype=torch.bfloat16, device=DEV)
        kv = torch.zeros((4, 2, 64), dtype=torch.bfloat16, device=DEV)
        with pytest.raises(ValueError):
            kvx.extend_attention(pool, b, q[:3], 4, 0.125, q)
        with pytest.raises(ValueError):
            kvx.extend_attention(pool, b, q, 4, 0.125, q, lse=torch.zeros(15, device=DEV))
        with pytest.raises(ValueError):
            kvx.store_kv(pool, b, kv, kv[:3])
        with pytest.raises(ValueError):
            kvx.store_kv_rope(pool, b, kv, kv, rotary_dim=64, q=q, num_q_heads=4, q_out=q[:2])
        with pytest.raises(ValueError):
            kvx.kv_pool_read_pages(pool, [0, 1], torch.zeros((1, 2, 16, 64), dtype=torch.int16, device=DEV),
                                   torch.zeros((2, 2, 16, 64), dtype=torch.int16, device=DEV))
        with pytest.raises(ValueError):
            kvx.Batch([16], [4], [0, 2], ids[:1])
        with pytest.raises(ValueError, match="bf16"):  # float32 Q of enough bytes is still refused
            kvx.extend_attention(pool, b, q.float(), 4, 0.125, q)
        # the same calls with whole buffers go through
        kvx.store_kv(pool, b, kv, kv)
        kvx.extend_attention(pool, b, q, 4, 0.125, torch.empty_like(q), lse=torch.zeros(16, device=DEV))
        torch.cuda.synchronize()
    finally:
        kvx.kv_pool_destroy(pool)


@pytest.mark.parametrize("seed", range(12))
def test_seeded_random_batches(seed):
    """Seeded random small batches (1-5 requests, ragged and empty suffixes, prefixes
    up to 700 tokens, GQA groups 1-8, head_dim 64/128, bf16 or fp8 pools, optional
    forced splits), every row against the oracle with LSE."""
    rng = np.random.default_rng([17, seed])
    r = int(rng.integers(1, 6))
    prefix = rng.integers(0, 700, r).tolist()
    extend = [int(x) if rng.random() > 0.15 else 0 for x in rng.integers(1, 260, r)]
    if sum(extend) == 0:
        extend[0] = 1
    hkv = int(rng.choice([1, 2, 3, 4]))
    g = int(rng.choice([1, 2, 4, 8]))
    d = int(rng.choice([64, 128]))
    dt = wl.KV_FP8_E4M3 if rng.random() < 0.3 else wl.KV_BF16
    split = int(rng.choice([0, 0, 64, 256]))
    w = wl.make_custom(prefix, extend, hkv * g, hkv, d, kv_dtype=dt, seed=100 + seed)
    print(f"[random] seed={seed} P={prefix} E={extend} Hq={hkv * g} Hkv={hkv} d={d} fp8={dt} split={split}",
          flush=True)
    _run_and_compare(w, f"random{seed}", want_lse=True, split_keys=split)
