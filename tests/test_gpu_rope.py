"""The fused RoPE store (store_kv_rope) on the GPU against the oracle
(oracle/rope.py): rotated Q and K are the bf16 / e4m3 values nearest to the
oracle's exact ones (either neighbour where the exact value sits within float32
error of a rounding midpoint), V and every slot the batch does not write are
bit-exact, and attention over the rotated pool passes the standard gate."""

import numpy as np
import pytest
import torch

import oracle
from gpu_harness import DEV, compare, fresh_batch
from helpers import check_nearest_bf16, check_nearest_e4m3, plane_scale
from oracle import rope as R
from paper_2609_32278_amd import kvx
from paper_2609_32278_amd import workloads as wl

pytestmark = pytest.mark.gpu

RAGGED_P = [0, 5, 16, 37, 100, 3, 1000]
RAGGED_E = [7, 0, 1, 29, 18, 40, 200]

# name: (prefix_lens, extend_lens, Hq, Hkv, d, kv dtype, rope settings)
CASES = {
    "half_d128_norm": (RAGGED_P, RAGGED_E, 8, 2, 128, wl.KV_BF16, wl.RopeSpec(1e6, 128, R.HALF, True)),
    "interleaved_d64": (RAGGED_P, RAGGED_E, 4, 2, 64, wl.KV_BF16, wl.RopeSpec(1e4, 64, R.INTERLEAVED, False)),
    "partial_half_norm": (RAGGED_P, RAGGED_E, 8, 4, 128, wl.KV_BF16, wl.RopeSpec(5e5, 64, R.HALF, True)),
    "partial_interleaved_d128": (RAGGED_P, RAGGED_E, 4, 4, 128, wl.KV_BF16,
                                 wl.RopeSpec(1e4, 96, R.INTERLEAVED, False)),
    "fp8_half_norm": (RAGGED_P, RAGGED_E, 8, 2, 128, wl.KV_FP8_E4M3, wl.RopeSpec(1e6, 128, R.HALF, True)),
    "fp8_interleaved_partial_d64": (RAGGED_P, RAGGED_E, 8, 2, 64, wl.KV_FP8_E4M3,
                                    wl.RopeSpec(1e4, 32, R.INTERLEAVED, True)),
    "gqa16_half_d64": ([0, 33, 250], [300, 64, 9], 16, 1, 64, wl.KV_BF16, wl.RopeSpec(1e4, 48, R.HALF, True)),
    "long_positions": ([131000, 262000, 65535], [40, 17, 3], 4, 1, 64, wl.KV_BF16,
                       wl.RopeSpec(5e5, 64, R.HALF, False)),
}


def _workload(name, seed=0):
    p, e, hq, hkv, d, kvd, spec = CASES[name]
    pool_factor = 1.0 if name == "long_positions" else 1.5
    w = wl.make_custom(p, e, hq, hkv, d, kv_dtype=kvd, seed=seed, pool_factor=pool_factor)
    return w, spec


def _pool(w, fill):
    pool = kvx.kv_pool_create(w.num_pages, w.page_size, w.num_kv_heads, w.head_dim, w.kv_dtype, w.k_scale,
                              w.v_scale)
    dt = torch.int16 if w.kv_dtype == wl.KV_BF16 else torch.uint8
    val = fill if w.kv_dtype != wl.KV_BF16 else (fill - 65536 if fill >= 32768 else fill)
    for p0 in range(0, w.num_pages, 4096):
        ids = np.arange(p0, min(w.num_pages, p0 + 4096), dtype=np.int32)
        buf = torch.full((len(ids), w.num_kv_heads, w.page_size, w.head_dim), val, dtype=dt, device=DEV)
        kvx.kv_pool_write_pages(pool, ids, buf, buf)
    torch.cuda.synchronize()
    return pool


def _read(w, pool, page_ids):
    dt = torch.int16 if w.kv_dtype == wl.KV_BF16 else torch.uint8
    k = torch.empty((len(page_ids), w.num_kv_heads, w.page_size, w.head_dim), dtype=dt, device=DEV)
    v = torch.empty_like(k)
    kvx.kv_pool_read_pages(pool, np.asarray(page_ids, np.int32), k, v)
    torch.cuda.synchronize()
    npdt = np.uint16 if w.kv_dtype == wl.KV_BF16 else np.uint8
    return k.cpu().numpy().view(npdt), v.cpu().numpy().view(npdt)


def _pages_near_suffix(w):
    """The pages holding suffix slots, plus the prefix page before each suffix."""
    out = set()
    for r in range(w.num_reqs):
        P, E = int(w.prefix_lens[r]), int(w.extend_lens[r])
        if E == 0:
            continue
        pages = w.pages_of(r)
        out.update(int(x) for x in pages[max(P // 16 - 1, 0):(P + E + 15) // 16])
    return np.array(sorted(out), np.int32)


def _suffix_places(w, pages_read):
    """(index into pages_read, slot) of every suffix row, in row order."""
    where = {int(p): i for i, p in enumerate(pages_read)}
    idx, slot = [], []
    for r in range(w.num_reqs):
        pages = w.pages_of(r)
        for t in range(int(w.prefix_lens[r]), int(w.prefix_lens[r]) + int(w.extend_lens[r])):
            idx.append(where[int(pages[t // 16])])
            slot.append(t % 16)
    return np.array(idx, np.int64), np.array(slot, np.int64)


def _rope_kwargs(spec, qn, kn, freqs):
    return dict(theta=spec.theta, rotary_dim=spec.rotary_dim, style=spec.style, q_norm=qn, k_norm=kn,
                norm_eps=spec.eps, inv_freq=freqs)


def _check_store(name, in_place=False, with_q=True, freqs=None, seed=0):
    print(f"[rope] {name} in_place={in_place} with_q={with_q} freqs={freqs is not None}", flush=True)
    w, spec = _workload(name, seed)
    fill = 0x5A if w.kv_dtype == wl.KV_FP8_E4M3 else 0x5A5A
    t = wl.batch_tensors(w, device=DEV)
    qn, kn = wl.norm_weights(w, DEV) if spec.norm else (None, None)
    q_in = t["q"].cpu()
    pool = _pool(w, fill)
    try:
        batch, ids = fresh_batch(w, w.page_ids, w.prefix_lens, w.extend_lens, w.page_indptr)
        q = t["q"]
        q_out = q if in_place else torch.full_like(q, float("nan"))
        kvx.store_kv_rope(pool, batch, t["k_ext"], t["v_ext"], q=q if with_q else None,
                          num_q_heads=w.num_q_heads if with_q else 0, q_out=q_out if with_q else None,
                          **_rope_kwargs(spec, qn, kn, freqs))
        torch.cuda.synchronize()
        touched = _pages_near_suffix(w)
        k, v = _read(w, pool, touched)
    finally:
        kvx.kv_pool_destroy(pool)
    opool = oracle.OraclePool(w.num_pages, w.num_kv_heads, w.head_dim, w.kv_dtype, w.page_size, w.k_scale,
                              w.v_scale, fill=fill)
    cpu = (lambda x: None if x is None else x.cpu())
    kx = R.store_kv_rope(opool, w.prefix_lens, w.extend_lens, w.page_indptr, w.page_ids, t["k_ext"].cpu(),
                         t["v_ext"].cpu(), spec.theta, spec.rotary_dim, spec.style, cpu(kn), spec.eps, freqs)
    assert np.array_equal(v, opool.v[touched]), "V pool differs"
    idx, slot = _suffix_places(w, touched)
    written = np.zeros(k.shape[:1] + (16,), bool)
    written[idx, slot] = True
    ok = opool.k[touched]
    assert np.array_equal(k.transpose(0, 2, 1, 3)[~written], ok.transpose(0, 2, 1, 3)[~written]), \
        "slots outside the batch changed"
    got = k[idx, :, slot, :]
    scale = plane_scale(kx, spec.rotary_dim, spec.style)
    if w.kv_dtype == wl.KV_BF16:
        flips = check_nearest_bf16(got, kx, scale)
    else:
        inv = (np.float32(1.0) / np.asarray(w.k_scale, np.float32))[None, :, None]
        flips = check_nearest_e4m3(got, kx, inv, scale)
    print(f"[rope] {name}: K rows {kx.shape[0]}, other-neighbour roundings {flips}", flush=True)
    if with_q:
        qx, _ = R.rotate_q(q_in, w.prefix_lens, w.extend_lens, spec.theta, spec.rotary_dim, spec.style,
                           cpu(qn), spec.eps, freqs)
        qflips = check_nearest_bf16(q_out.cpu(), qx, plane_scale(qx, spec.rotary_dim, spec.style))
        print(f"[rope] {name}: Q other-neighbour roundings {qflips} of {qx.size}", flush=True)


@pytest.mark.parametrize("name", list(CASES))
def test_rotated_store_matches_the_oracle(name):
    _check_store(name)


def test_rotation_in_place_of_the_queries():
    _check_store("half_d128_norm", in_place=True, seed=1)


def test_keys_only():
    _check_store("fp8_half_norm", with_q=False, seed=2)


def test_given_frequency_table():
    # a band-scaled table: the slow half of the planes turns 8x slower
    f = R.frequencies(5e5, 128)
    f[32:] /= 8.0
    _check_store("half_d128_norm", freqs=f, seed=3)


def test_positions_past_float32_integers():
    """Positions up to 2^27 + 600: every logical page of the prefixes points at
    page 0, which the store never writes (only suffix slots are written)."""
    print("[rope] positions past 2^24", flush=True)
    P, E = [16777200, 134217000, 99999999], [20, 40, 600]
    hq, hkv, d = 4, 2, 128
    spec = wl.RopeSpec(1e6, 128, R.HALF, True)
    indptr, ids, nxt = [0], [], 1
    for p, e in zip(P, E):
        n = (p + e + 15) // 16
        first = p // 16
        ids.extend([0] * first)
        ids.extend(range(nxt, nxt + n - first))
        nxt += n - first
        indptr.append(len(ids))
    ids = np.array(ids, np.int32)
    num_pages = nxt
    T = sum(E)
    g = torch.Generator(device=DEV).manual_seed(77)
    q = torch.randn((T, hq, d), generator=g, device=DEV).to(torch.bfloat16)
    k = torch.randn((T, hkv, d), generator=g, device=DEV).to(torch.bfloat16)
    v = torch.randn((T, hkv, d), generator=g, device=DEV).to(torch.bfloat16)
    qn = (0.5 + torch.rand((d,), generator=g, device=DEV)).to(torch.bfloat16)
    kn = (0.5 + torch.rand((d,), generator=g, device=DEV)).to(torch.bfloat16)
    pool = kvx.kv_pool_create(num_pages, 16, hkv, d, kvx.KVX_KV_BF16)
    try:
        ids_d = torch.from_numpy(ids).to(DEV)
        batch = kvx.Batch(P, E, indptr, ids_d)
        zero = torch.zeros((num_pages, hkv, 16, d), dtype=torch.int16, device=DEV)
        kvx.kv_pool_write_pages(pool, np.arange(num_pages, dtype=np.int32), zero, zero)
        q_out = torch.empty_like(q)
        kvx.store_kv_rope(pool, batch, k, v, q=q, num_q_heads=hq, q_out=q_out,
                          **_rope_kwargs(spec, qn, kn, None))
        kk = torch.empty_like(zero)
        vv = torch.empty_like(zero)
        kvx.kv_pool_read_pages(pool, np.arange(num_pages, dtype=np.int32), kk, vv)
        torch.cuda.synchronize()
        kk = kk.cpu().numpy().view(np.uint16)
    finally:
        kvx.kv_pool_destroy(pool)
    opool = oracle.OraclePool(num_pages, hkv, d, oracle.KV_BF16)
    kx = R.store_kv_rope(opool, P, E, indptr, ids, k.cpu(), v.cpu(), spec.theta, spec.rotary_dim, spec.style,
                         kn.cpu(), spec.eps)
    assert (kk[0] == 0).all()
    pos = R.positions(P, E)
    pg = np.array([ids[indptr[r] + t // 16] for r, (p, e) in enumerate(zip(P, E)) for t in range(p, p + e)])
    got = kk[pg, :, pos % 16, :]
    check_nearest_bf16(got, kx, plane_scale(kx, 128, R.HALF))
    qx, _ = R.rotate_q(q.cpu(), P, E, spec.theta, spec.rotary_dim, spec.style, qn.cpu(), spec.eps)
    check_nearest_bf16(q_out.cpu(), qx, plane_scale(qx, 128, R.HALF))


def test_argument_errors():
    w, spec = _workload("interleaved_d64")
    pool = _pool(w, 0)
    try:
        batch, ids = fresh_batch(w, w.page_ids, w.prefix_lens, w.extend_lens, w.page_indptr)
        t = wl.batch_tensors(w, device=DEV)

        def err(**kw):
            args = dict(theta=1e4, rotary_dim=64, style=0, q=t["q"], num_q_heads=w.num_q_heads, q_out=t["q"])
            args.update(kw)
            with pytest.raises(kvx.KvxError) as e:
                kvx.store_kv_rope(pool, batch, t["k_ext"], t["v_ext"], **args)
            return e.value.status

        for rd in (0, 8, 72, 128):
            assert err(rotary_dim=rd) == kvx.KVX_EINVAL
        assert err(style=2) == kvx.KVX_EINVAL
        assert err(theta=0.0) == kvx.KVX_EINVAL
        assert err(theta=float("inf")) == kvx.KVX_EINVAL
        assert err(inv_freq=np.full(32, np.nan)) == kvx.KVX_EINVAL
        assert err(norm_eps=-1.0) == kvx.KVX_EINVAL
        assert err(q=None) == kvx.KVX_EINVAL
        assert err(num_q_heads=-1) == kvx.KVX_EINVAL
        assert err(q_out=t["q"].data_ptr() + 2) == kvx.KVX_EINVAL          # not 16-byte aligned
        with pytest.raises(kvx.KvxError) as e:
            kvx.store_kv(pool, batch, t["k_ext"].data_ptr() + 8, t["v_ext"])
        assert e.value.status == kvx.KVX_EINVAL
        out = torch.empty_like(t["q"])
        with pytest.raises(kvx.KvxError) as e:
            kvx.extend_attention(pool, batch, t["q"].data_ptr() + 4, w.num_q_heads, w.sm_scale, out)
        assert e.value.status == kvx.KVX_EINVAL
        torch.cuda.synchronize()
    finally:
        kvx.kv_pool_destroy(pool)


@pytest.mark.parametrize("name", ["half_d128_norm", "fp8_half_norm", "interleaved_d64", "gqa16_half_d64"])
def test_attention_over_the_rotated_pool(name):
    """History turn and suffix both go through the fused store; attention of the
    rotated queries over the pool against the oracle's rotated pool and queries."""
    print(f"[rope-attn] {name}", flush=True)
    w, spec = _workload(name, seed=4)
    t = wl.batch_tensors(w, device=DEV)
    qn, kn = wl.norm_weights(w, DEV) if spec.norm else (None, None)
    kw = _rope_kwargs(spec, qn, kn, None)
    h = wl.history_batch(w)
    pool = _pool(w, 0)
    try:
        hb, hids = fresh_batch(h, h.page_ids, h.prefix_lens, h.extend_lens, h.page_indptr)
        kvx.store_kv_rope(pool, hb, t["k_hist"], t["v_hist"], **kw)
        batch, ids = fresh_batch(w, w.page_ids, w.prefix_lens, w.extend_lens, w.page_indptr)
        q_rot = torch.empty_like(t["q"])
        kvx.store_kv_rope(pool, batch, t["k_ext"], t["v_ext"], q=t["q"], num_q_heads=w.num_q_heads, q_out=q_rot,
                          **kw)
        out = torch.full_like(q_rot, float("nan"))
        lse = torch.full((w.total_extend, w.num_q_heads), float("nan"), dtype=torch.float32, device=DEV)
        kvx.extend_attention(pool, batch, q_rot, w.num_q_heads, w.sm_scale, out, lse)
        torch.cuda.synchronize()
    finally:
        kvx.kv_pool_destroy(pool)
    cpu = (lambda x: None if x is None else x.cpu())
    opool = oracle.OraclePool(w.num_pages, w.num_kv_heads, w.head_dim, w.kv_dtype, w.page_size, w.k_scale,
                              w.v_scale)
    R.store_kv_rope(opool, h.prefix_lens, h.extend_lens, h.page_indptr, h.page_ids, t["k_hist"].cpu(),
                    t["v_hist"].cpu(), spec.theta, spec.rotary_dim, spec.style, cpu(kn), spec.eps)
    R.store_kv_rope(opool, w.prefix_lens, w.extend_lens, w.page_indptr, w.page_ids, t["k_ext"].cpu(),
                    t["v_ext"].cpu(), spec.theta, spec.rotary_dim, spec.style, cpu(kn), spec.eps)
    _, q_bits = R.rotate_q(t["q"].cpu(), w.prefix_lens, w.extend_lens, spec.theta, spec.rotary_dim, spec.style,
                           cpu(qn), spec.eps)
    rr, rp = oracle.all_rows(w.extend_lens)
    ref, ref_lse = oracle.extend_attention(opool, w.prefix_lens, w.extend_lens, w.page_indptr, w.page_ids,
                                           q_bits.reshape(t["q"].shape), rr, rp, w.num_q_heads, w.sm_scale,
                                           want_lse=True)
    compare(out.cpu().to(torch.float64).numpy(), ref, f"rope-attn {name}")
    assert np.abs(lse.cpu().numpy() - ref_lse).max() <= 2e-2


def test_full_size_llama8b_with_fused_rope():
    """The llama8b batch at full size, launched as `bench.py --rope` launches it
    (history and suffix through store_kv_rope, attention on the rotated queries):
    sampled rows of sampled requests against the oracle -- rotated queries,
    rotated keys and values in the pool, and attention outputs."""
    import bench
    name = "llama8b"
    s = bench.setup(name, rope=True)
    w, pool, batch = s["w"], s["pool"], s["batch"]
    try:
        q_rot = torch.full_like(s["q"], float("nan"))
        kvx.store_kv_rope(pool, batch, s["k_ext"], s["v_ext"], q=s["q"], num_q_heads=w.num_q_heads, q_out=q_rot,
                          **s["rope"])
        out = torch.full_like(q_rot, float("nan"))
        kvx.extend_attention(pool, batch, q_rot, w.num_q_heads, w.sm_scale, out)
        torch.cuda.synchronize()
        assert torch.isfinite(out.float()).all() and torch.isfinite(q_rot.float()).all()
        rng = np.random.default_rng([w.config_id, 5])
        must = {int(np.argmax(w.prefix_lens)), int(np.argmax(w.extend_lens))}
        reqs = sorted(must | set(int(x) for x in rng.choice(w.num_reqs, 2, replace=False)))
        rows = wl.sample_rows(w, 8, reqs=reqs)
        print(f"[rope-full] {name}: T={w.total_extend} sampled reqs={reqs} rows={len(rows)}", flush=True)
        sub = w.subset(reqs)
        pages = np.concatenate([w.pages_of(r) for r in reqs]).astype(np.int32)
        gk, gv = _read(w, pool, pages)
    finally:
        kvx.kv_pool_destroy(pool)
    spec = wl.RopeSpec(rotary_dim=w.head_dim)
    qn, kn = (x.cpu() for x in wl.norm_weights(w, DEV))
    t = {"k_hist": [], "v_hist": [], "k_ext": [], "v_ext": [], "q": []}
    for r in reqs:
        kk, vv = wl.request_kv(w, r, DEV)
        p = int(w.prefix_lens[r])
        t["k_hist"].append(kk[:p].cpu())
        t["v_hist"].append(vv[:p].cpu())
        t["k_ext"].append(kk[p:].cpu())
        t["v_ext"].append(vv[p:].cpu())
        t["q"].append(wl.request_q(w, r, DEV).cpu())
    t = {key: torch.cat(val) for key, val in t.items()}
    opool = oracle.OraclePool(sub.num_pages, sub.num_kv_heads, sub.head_dim, sub.kv_dtype, sub.page_size)
    h = wl.history_batch(sub)
    kh = R.store_kv_rope(opool, h.prefix_lens, h.extend_lens, h.page_indptr, h.page_ids, t["k_hist"], t["v_hist"],
                         spec.theta, spec.rotary_dim, spec.style, kn, spec.eps)
    ke = R.store_kv_rope(opool, sub.prefix_lens, sub.extend_lens, sub.page_indptr, sub.page_ids, t["k_ext"],
                         t["v_ext"], spec.theta, spec.rotary_dim, spec.style, kn, spec.eps)
    # pool: V bit for bit, every rotated key the nearest bf16
    assert np.array_equal(gv, opool.v[sub.page_ids]), "V pages differ"
    ok_bits = opool.k[sub.page_ids]
    same = gk == ok_bits
    if not same.all():
        # the pages hold history keys then suffix keys, in logical order per request
        exact = np.zeros(gk.shape, np.float64)
        ph = pe = 0
        base = 0
        for j, r in enumerate(reqs):
            P, E = int(w.prefix_lens[r]), int(w.extend_lens[r])
            for tok in range(P + E):
                src = kh[ph + tok] if tok < P else ke[pe + tok - P]
                exact[base + tok // 16, :, tok % 16, :] = src
            ph += P
            pe += E
            base += len(w.pages_of(r))
        mask = ~same
        check_nearest_bf16(gk[mask], exact[mask], plane_scale(exact, spec.rotary_dim, spec.style)[mask])
    # rotated queries of the sampled rows
    qo = w.qo_indptr.astype(np.int64)
    sqo = sub.qo_indptr.astype(np.int64)
    remap = {r: k for k, r in enumerate(reqs)}
    gidx = np.array([qo[r] + i for r, i in rows], np.int64)
    lidx = np.array([sqo[remap[int(r)]] + i for r, i in rows], np.int64)
    pos = np.array([int(w.prefix_lens[r]) + int(i) for r, i in rows], np.int64)
    qx = R.transform(t["q"][torch.from_numpy(lidx)], pos, spec.theta, spec.rotary_dim, spec.style, qn, spec.eps)
    check_nearest_bf16(q_rot[torch.from_numpy(gidx).to(DEV)].cpu(), qx, plane_scale(qx, spec.rotary_dim, spec.style))
    # attention of the sampled rows with the oracle's own rotated queries
    rr = np.array([remap[int(r)] for r in rows[:, 0]], np.int32)
    ref = oracle.extend_attention(opool, sub.prefix_lens, sub.extend_lens, sub.page_indptr, sub.page_ids,
                                  oracle.bf16_round(qx), rr, rows[:, 1].astype(np.int32), w.num_q_heads,
                                  w.sm_scale)
    got = out[torch.from_numpy(gidx).to(DEV)].float().cpu().numpy().astype(np.float64)
    compare(got, ref, f"rope-full {name}")
