"""Test helpers: an independent brute-force attention (numpy/scipy, no page table)
and builders that run the oracle over a generated workload.

The brute force is deliberately formulated differently from the oracle: it
materialises the whole (suffix x context) score matrix of a request from the
*logical* K/V sequence (never from a pool), expands KV heads to query heads with
``numpy.repeat`` and applies softmax/logsumexp from scipy.
"""

from __future__ import annotations

import numpy as np
import scipy.special
import torch

import oracle
from paper_2609_32278_amd import workloads as wl


def to_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().to(torch.float64).numpy()


def brute_force(q: np.ndarray, k: np.ndarray, v: np.ndarray, prefix_len: int, sm_scale: float):
    """q [E, Hq, d], k/v [L, Hkv, d] float64 (the logical sequence), L = P + E.
    Returns out [E, Hq, d] and lse [E, Hq] of bottom-right-aligned causal attention."""
    e, hq, d = q.shape
    n, hkv, _ = k.shape
    assert n == prefix_len + e
    g = hq // hkv
    if e == 0:  # no suffix rows (the request may have no keys at all)
        return np.zeros((0, hq, d)), np.zeros((0, hq))
    kx = np.repeat(k, g, axis=1)  # [L, Hq, d]: query head h reads kv head h // g
    vx = np.repeat(v, g, axis=1)
    s = np.einsum("ihc,jhc->hij", q, kx) * sm_scale  # [Hq, E, L]
    rows = np.arange(e)[:, None] + prefix_len
    cols = np.arange(n)[None, :]
    s = np.where(cols <= rows, s, -np.inf)
    p = scipy.special.softmax(s, axis=-1)
    out = np.einsum("hij,jhc->ihc", p, vx)
    lse = scipy.special.logsumexp(s, axis=-1).T  # [E, Hq]
    return out, lse


def oracle_pool_for(w: wl.Workload, t: dict, fill=None) -> oracle.OraclePool:
    """An oracle pool holding the workload's cached prefixes (stored by an earlier
    turn, the history batch) and then its suffix rows (this turn's KV store)."""
    pool = oracle.OraclePool(w.num_pages, w.num_kv_heads, w.head_dim, w.kv_dtype, w.page_size,
                             w.k_scale, w.v_scale, fill=fill)
    h = wl.history_batch(w)
    oracle.store_kv(pool, h.prefix_lens, h.extend_lens, h.page_indptr, h.page_ids,
                    t["k_hist"], t["v_hist"])
    oracle.store_kv(pool, w.prefix_lens, w.extend_lens, w.page_indptr, w.page_ids,
                    t["k_ext"], t["v_ext"])
    return pool


def oracle_all_rows(w: wl.Workload, pool: oracle.OraclePool, q: torch.Tensor, mutant="none",
                    want_lse=False, num_threads=0, scaled_q=False):
    rr, rp = oracle.all_rows(w.extend_lens)
    return oracle.extend_attention(pool, w.prefix_lens, w.extend_lens, w.page_indptr, w.page_ids,
                                   q, rr, rp, w.num_q_heads, w.sm_scale, mutant=mutant,
                                   want_lse=want_lse, num_threads=num_threads, scaled_q=scaled_q)


def brute_force_all(w: wl.Workload, dequant=None):
    """Brute-force outputs for every suffix row of every request, from the generator's
    logical sequences.  ``dequant(k, v)`` maps the float64 logical K/V to what the pool
    holds (identity for bf16)."""
    outs, lses = [], []
    for r in range(w.num_reqs):
        q = to_f64(wl.request_q(w, r))
        k, v = wl.request_kv(w, r)
        k, v = to_f64(k), to_f64(v)
        if dequant is not None:
            k, v = dequant(k, v)
        o, l = brute_force(q, k, v, int(w.prefix_lens[r]), w.sm_scale)
        outs.append(o)
        lses.append(l)
    return np.concatenate(outs, 0), np.concatenate(lses, 0)


def fp8_dequant_torch(w: wl.Workload):
    """Dequantisation of the fp8 pool computed with torch's float8_e4m3fn cast of the
    pre-clamped fp32 product (a library routine, independent of the oracle's codec)."""
    ks = torch.from_numpy(np.asarray(w.k_scale, np.float32))
    vs = torch.from_numpy(np.asarray(w.v_scale, np.float32))

    def q8(x64: np.ndarray, scale: torch.Tensor) -> np.ndarray:
        x = torch.from_numpy(x64).to(torch.float32)  # exact: values are bf16
        inv = (1.0 / scale).to(torch.float32)  # fp32 reciprocal, as stored
        y = (x * inv[None, :, None]).clamp(-448.0, 448.0)
        code = y.to(torch.float8_e4m3fn)
        return (code.to(torch.float64) * scale.to(torch.float64)[None, :, None]).numpy()

    return lambda k, v: (q8(k, ks), q8(v, vs))


def plane_scale(exact: np.ndarray, rotary_dim: int, style: int) -> np.ndarray:
    """Per-element magnitude that bounds the error of a rotation done in single
    precision: the length of the element's rotation plane, or |x| past rotary_dim."""
    from oracle import rope as orope
    s = np.abs(exact).astype(np.float64)
    first, second = orope.planes(rotary_dim, style)
    r = np.hypot(exact[..., first], exact[..., second])
    s[..., first] = r
    s[..., second] = r
    return s


def check_nearest_bf16(got_bits, exact: np.ndarray, scale: np.ndarray, rel: float = 2.0 ** -17) -> int:
    """Assert that every value is the bf16 nearest to some y with
    |y - exact| <= rel * scale (exact: float64).  A computation carried out in
    float32 lands within that distance of the exact value (rel = 2^-17 is several
    times its error bound, relative to the magnitude ``scale`` of the operands),
    so its correctly rounded result may be the nearest bf16 of exact or, when
    exact sits near a rounding midpoint or the result nearly cancels, a value
    between the nearest bf16 of exact - tol and of exact + tol.  Returns how many
    values differ from the nearest bf16 of exact."""
    want = oracle.bf16_round(exact)
    got = oracle.bf16_bits(got_bits).reshape(want.shape)
    bad = got != want
    if not bad.any():
        return 0
    tol = rel * scale[bad]
    lo = oracle.bf16_value(oracle.bf16_round(exact[bad] - tol))
    hi = oracle.bf16_value(oracle.bf16_round(exact[bad] + tol))
    g = oracle.bf16_value(got[bad])
    ok = (lo <= g) & (g <= hi)
    assert ok.all(), (f"{int((~ok).sum())} of {want.size} values are off: got {g[~ok][:4]}, exact "
                      f"{exact[bad][~ok][:4]}, scale {scale[bad][~ok][:4]}")
    return int(bad.sum())


def check_nearest_e4m3(got_codes, exact: np.ndarray, inv_scale: np.ndarray, scale: np.ndarray,
                       rel: float = 2.0 ** -17) -> int:
    """The fp8 counterpart of check_nearest_bf16 for a quantised store: the code
    must be encode(float32(y) * inv_scale) (inv_scale float32, broadcast to
    exact) for some y within rel * scale of exact."""
    inv32 = np.broadcast_to(np.asarray(inv_scale, np.float32), exact.shape)

    def enc(x, inv):
        return oracle.e4m3_encode((x.astype(np.float32) * inv).astype(np.float32))

    want = enc(exact, inv32)
    got = np.asarray(got_codes, np.uint8).reshape(want.shape)
    bad = got != want
    if not bad.any():
        return 0
    tol = rel * scale[bad]
    lo = oracle.e4m3_decode(enc(exact[bad] - tol, inv32[bad]))
    hi = oracle.e4m3_decode(enc(exact[bad] + tol, inv32[bad]))
    g = oracle.e4m3_decode(got[bad])
    ok = (lo <= g) & (g <= hi)
    assert ok.all(), (f"{int((~ok).sum())} of {want.size} codes are off: got {got[bad][~ok][:4]}, want "
                      f"{want[bad][~ok][:4]}")
    return int(bad.sum())
