"""KV spill to pinned host memory and reload (kv_pool_spill / kv_pool_reload):
records hold exactly the pool's bytes of a page (checked against the canonical
page read-out), and spill + reload into other pages is a bit-exact round trip."""

import numpy as np
import pytest
import torch

from gpu_harness import DEV
from paper_2609_32278_amd import kvx

pytestmark = pytest.mark.gpu


def _pool_with_random_pages(num_pages, hkv, d, dtype, seed):
    scales = {}
    if dtype == kvx.KVX_KV_FP8_E4M3:
        scales = dict(k_scale=np.full(hkv, 0.05, np.float32), v_scale=np.full(hkv, 0.02, np.float32))
    pool = kvx.kv_pool_create(num_pages, 16, hkv, d, dtype, **scales)
    g = torch.Generator(device=DEV).manual_seed(seed)
    tdt = torch.int16 if dtype == kvx.KVX_KV_BF16 else torch.uint8
    lo, hi = (-32768, 32767) if dtype == kvx.KVX_KV_BF16 else (0, 255)
    k = torch.randint(lo, hi, (num_pages, hkv, 16, d), generator=g, device=DEV, dtype=torch.int32).to(tdt)
    v = torch.randint(lo, hi, (num_pages, hkv, 16, d), generator=g, device=DEV, dtype=torch.int32).to(tdt)
    kvx.kv_pool_write_pages(pool, np.arange(num_pages, dtype=np.int32), k, v)
    torch.cuda.synchronize()
    return pool, k, v


@pytest.mark.parametrize("dtype,hkv,d", [(kvx.KVX_KV_BF16, 8, 128), (kvx.KVX_KV_FP8_E4M3, 2, 64),
                                         (kvx.KVX_KV_BF16, 1, 64)])
def test_spill_records_and_round_trip(dtype, hkv, d):
    print(f"[spill] dtype={dtype} hkv={hkv} d={d}", flush=True)
    pool, k, v = _pool_with_random_pages(48, hkv, d, dtype, seed=hkv * 100 + d)
    try:
        rb = kvx.kv_pool_record_bytes(pool)
        eb = 2 if dtype == kvx.KVX_KV_BF16 else 1
        assert rb == 2 * hkv * 16 * d * eb
        host_slots = 9
        host = torch.empty(host_slots * rb, dtype=torch.uint8, pin_memory=True)
        host.fill_(0xA5)
        pages = np.array([7, 0, 47, 12, 30], np.int32)
        slots = np.array([3, 0, 8, 1, 5], np.int32)
        kvx.kv_pool_spill(pool, pages, slots, host, host_slots)
        torch.cuda.synchronize()
        hb = host.numpy().reshape(host_slots, 2, -1)
        kc = k.cpu().numpy().view(np.uint8 if eb == 1 else np.uint16)
        vc = v.cpu().numpy().view(np.uint8 if eb == 1 else np.uint16)
        npdt = np.uint8 if eb == 1 else np.uint16
        for p, s in zip(pages, slots):
            # K block: [head][slot][dim], the canonical order; V block: [head][dim][slot]
            assert np.array_equal(hb[s, 0].view(npdt).reshape(hkv, 16, d), kc[p])
            assert np.array_equal(hb[s, 1].view(npdt).reshape(hkv, d, 16), vc[p].transpose(0, 2, 1))
        untouched = sorted(set(range(host_slots)) - set(slots.tolist()))
        assert (hb[untouched] == 0xA5).all()
        # reload into other pages, some of them spilled ones (read before overwritten: other call)
        dst = np.array([1, 2, 3, 4, 7], np.int32)
        kvx.kv_pool_reload(pool, dst, slots, host, host_slots)
        k2 = torch.empty((len(dst), hkv, 16, d), dtype=k.dtype, device=DEV)
        v2 = torch.empty_like(k2)
        kvx.kv_pool_read_pages(pool, dst, k2, v2)
        torch.cuda.synchronize()
        assert torch.equal(k2, k[torch.from_numpy(pages).long().to(DEV)])
        assert torch.equal(v2, v[torch.from_numpy(pages).long().to(DEV)])
        # pages outside the reload keep their contents
        rest = np.array(sorted(set(range(48)) - set(dst.tolist())), np.int32)
        k3 = torch.empty((len(rest), hkv, 16, d), dtype=k.dtype, device=DEV)
        v3 = torch.empty_like(k3)
        kvx.kv_pool_read_pages(pool, rest, k3, v3)
        torch.cuda.synchronize()
        idx = torch.from_numpy(rest).long().to(DEV)
        assert torch.equal(k3, k[idx]) and torch.equal(v3, v[idx])
    finally:
        kvx.kv_pool_destroy(pool)


def test_spill_argument_errors():
    pool, _, _ = _pool_with_random_pages(8, 2, 64, kvx.KVX_KV_BF16, seed=1)
    try:
        rb = kvx.kv_pool_record_bytes(pool)
        pinned = torch.empty(4 * rb, dtype=torch.uint8, pin_memory=True)
        pageable = torch.empty(4 * rb, dtype=torch.uint8)

        def err(fn, pages, slots, host=pinned, n=4):
            with pytest.raises(kvx.KvxError) as e:
                fn(pool, pages, slots, host, n)
            return e.value.status

        assert err(kvx.kv_pool_spill, [0], [0], pageable) == kvx.KVX_EINVAL
        assert err(kvx.kv_pool_spill, [8], [0]) == kvx.KVX_ERANGE
        assert err(kvx.kv_pool_spill, [0], [4]) == kvx.KVX_ERANGE
        assert err(kvx.kv_pool_spill, [0, 1], [2, 2]) == kvx.KVX_EINVAL
        assert err(kvx.kv_pool_reload, [3, 3], [0, 1]) == kvx.KVX_EINVAL
        assert err(kvx.kv_pool_spill, [0], [0], pinned.data_ptr() + 8) == kvx.KVX_EINVAL  # alignment
        with pytest.raises(ValueError):  # the tensor holds 4 records, not 5
            kvx.kv_pool_spill(pool, [0], [0], pinned, 5)
        kvx.kv_pool_spill(pool, [0, 0], [0, 1], pinned, 4)   # reading a page twice is fine
        kvx.kv_pool_reload(pool, [5, 6], [0, 0], pinned, 4)  # so is reading a record twice
        torch.cuda.synchronize()
    finally:
        kvx.kv_pool_destroy(pool)


def test_host_pointer_inside_a_pinned_allocation():
    """A host buffer that starts inside a larger pinned allocation (a tensor view)
    addresses its records from its own start."""
    print("[spill] host view at a record offset", flush=True)
    pool, k, v = _pool_with_random_pages(8, 2, 64, kvx.KVX_KV_BF16, seed=7)
    try:
        rb = kvx.kv_pool_record_bytes(pool)
        whole = torch.zeros(6 * rb, dtype=torch.uint8, pin_memory=True)
        view = whole[2 * rb:]  # 4 records, starting at the allocation's third record
        kvx.kv_pool_spill(pool, [5, 1], [0, 3], view, 4)
        torch.cuda.synchronize()
        hb = whole.numpy().reshape(6, 2, -1)
        kc = k.cpu().numpy().view(np.uint16)
        assert np.array_equal(hb[2, 0].view(np.uint16).reshape(2, 16, 64), kc[5])
        assert np.array_equal(hb[5, 0].view(np.uint16).reshape(2, 16, 64), kc[1])
        assert (hb[[0, 1, 3, 4]] == 0).all()
        kvx.kv_pool_reload(pool, [6, 7], [3, 0], view, 4)
        k2 = torch.empty((2, 2, 16, 64), dtype=k.dtype, device=DEV)
        v2 = torch.empty_like(k2)
        kvx.kv_pool_read_pages(pool, [6, 7], k2, v2)
        torch.cuda.synchronize()
        assert torch.equal(k2, k[[1, 5]]) and torch.equal(v2, v[[1, 5]])
    finally:
        kvx.kv_pool_destroy(pool)
