"""Pins of the CPU oracle to things other than itself (no GPU).

The paper prints no worked example of the attention it reuses KV for, so the
oracle is pinned by mathematics and library routines:
  (a) a brute-force score-matrix computation over the logical sequence (no page
      table, numpy repeat for GQA, scipy softmax/logsumexp);
  (b) prefix_len = 0 reduces to ordinary causal attention (torch SDPA, fp64);
  (c) the output of a row does not depend on where its context is split into a
      cached prefix and a recomputed suffix -- the property prefix reuse relies on
      (Section 1: the cached prefix is reused and only the suffix is computed);
  (d) physical page placement does not matter;
  (e) a single key returns its value exactly; constant V returns the constant;
      Q = 0 averages the visible values; a planted needle key dominates;
  plus the fp8 codec against torch's float8_e4m3fn cast, store round trips, and
  planted mistakes that must each fail a pin and the parity gate;
  (f) the scaled-Q mode of the kernels (queries times the softmax scale in log2
      units, rounded to bf16, scores in base 2): its rounding step against torch's
      float32 product and bf16 cast, the brute force on the rounded queries, and
      exact attention wherever that product is exact.
"""

import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F
from hypothesis import assume, given, settings, strategies as st

import oracle
from helpers import (brute_force, brute_force_all, fp8_dequant_torch, oracle_all_rows,
                     oracle_pool_for, to_f64)
from paper_2609_32278_amd import workloads as wl

TOL = 1e-12


def _oracle_outputs(w, want_lse=False, mutant="none", fill=None):
    t = wl.batch_tensors(w)
    pool = oracle_pool_for(w, t, fill=fill)
    return oracle_all_rows(w, pool, t["q"], mutant=mutant, want_lse=want_lse), t, pool


# ------------------------------------------------------------------ (a) brute force

def test_brute_force_tiny_config():
    w = wl.make_workload("tiny")
    (out, lse), _, _ = _oracle_outputs(w, want_lse=True)
    ref, ref_lse = brute_force_all(w)
    assert out.shape == ref.shape == (156, 4, 64)
    assert np.abs(out - ref).max() <= TOL
    assert np.abs(lse - ref_lse).max() <= TOL


@settings(max_examples=30, deadline=None, derandomize=True)
@given(st.data())
def test_brute_force_on_drawn_shapes(data):
    """(a) on shapes hypothesis draws: ragged prefixes and suffixes (empty ones too),
    one to four KV heads, GQA groups of 1-4, random page placement and pool slack."""
    r = data.draw(st.integers(1, 4), label="requests")
    prefix = data.draw(st.lists(st.integers(0, 70), min_size=r, max_size=r), label="prefix_lens")
    extend = data.draw(st.lists(st.integers(0, 40), min_size=r, max_size=r), label="extend_lens")
    assume(sum(extend) > 0)
    hkv = data.draw(st.integers(1, 4), label="kv_heads")
    g = data.draw(st.sampled_from([1, 2, 4]), label="group")
    d = data.draw(st.sampled_from([8, 16, 32]), label="head_dim")
    w = wl.make_custom(prefix, extend, hkv * g, hkv, d, seed=data.draw(st.integers(0, 9999), label="seed"),
                       pool_factor=data.draw(st.sampled_from([1.0, 1.5, 3.0]), label="pool_factor"))
    (out, lse), _, _ = _oracle_outputs(w, want_lse=True)
    ref, ref_lse = brute_force_all(w)
    assert np.abs(out - ref).max() <= TOL
    assert np.abs(lse - ref_lse).max() <= TOL


@pytest.mark.parametrize("hq,hkv,d", [(1, 1, 16), (4, 2, 32), (8, 2, 16), (6, 3, 8)])
def test_brute_force_unaligned_and_ragged(hq, hkv, d):
    # prefixes that do not end on a page boundary, empty suffixes, suffixes that
    # end mid-page and a prefix-free request
    w = wl.make_custom([0, 5, 16, 37, 100, 3], [7, 0, 1, 29, 18, 40], hq, hkv, d, seed=hq * 10 + d)
    (out, lse), _, _ = _oracle_outputs(w, want_lse=True)
    ref, ref_lse = brute_force_all(w)
    assert np.abs(out - ref).max() <= TOL
    assert np.abs(lse - ref_lse).max() <= TOL


def test_brute_force_sharpened_queries():
    # large logits (Q sigma 4) make the softmax peaky; the definition still agrees
    w = wl.make_custom([48, 13], [20, 35], 4, 1, 32, q_sigma=4.0, seed=5)
    out, _, _ = _oracle_outputs(w)
    ref, _ = brute_force_all(w)
    assert np.abs(out - ref).max() <= 1e-11


# ------------------------------------------------------- (b) prefix 0 = causal SDPA

@pytest.mark.parametrize("e,hq,hkv,d", [(1, 2, 1, 16), (33, 4, 2, 32), (70, 8, 8, 16)])
def test_prefix_zero_is_causal_attention(e, hq, hkv, d):
    w = wl.make_custom([0], [e], hq, hkv, d, seed=e)
    out, _, _ = _oracle_outputs(w)
    q = wl.request_q(w, 0).to(torch.float64).permute(1, 0, 2)[None]   # [1, Hq, E, d]
    k, v = wl.request_kv(w, 0)
    g = hq // hkv
    k = k.to(torch.float64).repeat_interleave(g, dim=1).permute(1, 0, 2)[None]
    v = v.to(torch.float64).repeat_interleave(g, dim=1).permute(1, 0, 2)[None]
    ref = F.scaled_dot_product_attention(q, k, v, is_causal=True, scale=w.sm_scale)
    ref = ref[0].permute(1, 0, 2).numpy()
    assert np.abs(out - ref).max() <= TOL


# ---------------------------------------------------------- (c) split invariance

@pytest.mark.parametrize("total", [40, 97])
def test_split_invariance_at_every_page_boundary(total):
    """Same logical sequence, cut into (prefix, suffix) at every page boundary: rows at
    absolute positions >= the largest cut agree exactly."""
    hq, hkv, d = 4, 2, 16
    base = wl.make_custom([0], [total], hq, hkv, d, seed=77, placement="linear")
    q_all = wl.request_q(base, 0)
    k_all, v_all = wl.request_kv(base, 0)
    cuts = list(range(0, total, 16))
    last = cuts[-1]
    results = []
    for cut in cuts:
        w = wl.make_custom([cut], [total - cut], hq, hkv, d, seed=77, placement="random")
        t = dict(q=q_all[cut:], k_ext=k_all[cut:], v_ext=v_all[cut:], k_hist=k_all[:cut],
                 v_hist=v_all[:cut])
        pool = oracle_pool_for(w, t)
        out = oracle_all_rows(w, pool, t["q"])
        results.append(out[last - cut:])
    for r in results[1:]:
        assert np.array_equal(r, results[0])


# ------------------------------------------------------ (d) page permutation

def test_page_permutation_invariance_is_bitwise():
    p, e = [30, 64, 7], [20, 5, 44]
    outs = []
    for seed in (1, 2, 3):
        w = wl.make_custom(p, e, 4, 2, 32, seed=seed, num_pages=64)
        # same values for every placement: generator values come from the config id
        # and request index, not from the placement seed
        w.seed = 0
        t = wl.batch_tensors(w)
        pool = oracle_pool_for(w, t, fill=0x3F80)  # unused slots hold 1.0
        outs.append(oracle_all_rows(w, pool, t["q"]))
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


def test_unused_slots_and_pages_do_not_matter():
    w = wl.make_custom([5, 40], [9, 3], 2, 1, 16, seed=3, num_pages=32)
    a, _, _ = _oracle_outputs(w, fill=0)
    b, _, _ = _oracle_outputs(w, fill=0x461C)      # 1e4-ish poison
    c, _, _ = _oracle_outputs(w, fill=0x7FC0)      # NaN poison
    assert np.array_equal(a, b) and np.array_equal(a, c)


# ------------------------------------------------------------ (e) closed forms

@pytest.mark.parametrize("kv_dtype", [wl.KV_BF16, wl.KV_FP8_E4M3])
def test_single_key_returns_its_value(kv_dtype):
    w = wl.make_custom([0], [1], 4, 2, 32, kv_dtype=kv_dtype, seed=11)
    out, t, pool = _oracle_outputs(w)
    v0 = to_f64(t["v_ext"])[0]                     # [Hkv, d]
    if kv_dtype == wl.KV_FP8_E4M3:
        _, v0 = fp8_dequant_torch(w)(v0[None], v0[None])
        v0 = v0[0]
    expect = np.repeat(v0, 2, axis=0)
    assert np.array_equal(out[0], expect)


def test_constant_values_give_the_constant():
    w = wl.make_custom([21, 0], [11, 30], 4, 2, 16, seed=4)
    t = wl.batch_tensors(w)
    c = 0.71875  # exactly representable in bf16
    t["v_ext"] = torch.full_like(t["v_ext"], c)
    t["v_hist"] = torch.full_like(t["v_hist"], c)
    pool = oracle_pool_for(w, t)
    out = oracle_all_rows(w, pool, t["q"])
    assert np.abs(out - c).max() <= 1e-14


def test_zero_queries_average_the_visible_values():
    w = wl.make_custom([19, 32], [14, 6], 2, 2, 16, seed=8)
    t = wl.batch_tensors(w)
    t["q"] = torch.zeros_like(t["q"])
    pool = oracle_pool_for(w, t)
    out = oracle_all_rows(w, pool, t["q"])
    row = 0
    for r in range(w.num_reqs):
        _, v = wl.request_kv(w, r)
        v = to_f64(v)
        for i in range(int(w.extend_lens[r])):
            n = int(w.prefix_lens[r]) + i + 1
            expect = v[:n].mean(axis=0)               # [Hkv, d], g = 1
            assert np.abs(out[row] - expect).max() <= 1e-14
            row += 1


@pytest.mark.parametrize("where", ["prefix", "page_boundary", "diagonal"])
def test_needle_key_dominates(where):
    """A key aligned with the query and a logit margin >= 20 over every other key makes
    the output that key's value, to within exp(-20) of the value spread."""
    P, E, d = 48, 24, 32
    w = wl.make_custom([P], [E], 1, 1, d, seed=21, sigma=0.05, q_sigma=1.0)
    t = wl.batch_tensors(w)
    i = E - 1                      # the last suffix row sees every key
    j = {"prefix": 7, "page_boundary": 32, "diagonal": P + i}[where]
    q = t["q"][i, 0].to(torch.float64)
    alpha = 60.0 * math.sqrt(d) / float(q.norm())   # logit of the needle = 60 * |q|/|q| ...
    needle = (q * alpha / float(q.norm())).to(torch.bfloat16)
    k_all = torch.cat([t["k_hist"], t["k_ext"]])
    v_all = torch.cat([t["v_hist"], t["v_ext"]])
    k_all[j, 0] = needle
    v_all[j, 0] = 3.0
    t.update(k_hist=k_all[:P], k_ext=k_all[P:], v_hist=v_all[:P], v_ext=v_all[P:])
    logits = (k_all[:, 0].to(torch.float64) @ t["q"][i, 0].to(torch.float64)) * w.sm_scale
    others = torch.cat([logits[:j], logits[j + 1:P + i + 1]])
    assert float(logits[j] - others.max()) >= 20.0
    pool = oracle_pool_for(w, t)
    out = oracle_all_rows(w, pool, t["q"])
    spread = float((v_all[:P + i + 1, 0].to(torch.float64) - 3.0).abs().max())
    assert np.abs(out[i, 0] - 3.0).max() <= math.exp(-20.0) * spread * (P + E)


def test_two_key_closed_form():
    """Hand-derived: q = (a, 0), keys (0, 0) and (1, 0), values e0 and e1, scale 1:
    weights are 1/(1+e^a) and e^a/(1+e^a); lse = ln(1 + e^a)."""
    a = 1.09375  # bf16-exact, close to ln 3
    pool = oracle.OraclePool(2, 1, 2, oracle.KV_BF16)
    k_ext = torch.tensor([[[0.0, 0.0]], [[1.0, 0.0]]], dtype=torch.bfloat16)
    v_ext = torch.tensor([[[1.0, 0.0]], [[0.0, 1.0]]], dtype=torch.bfloat16)
    oracle.store_kv(pool, [0], [2], [0, 1], [1], k_ext, v_ext)
    q = torch.tensor([[[0.0, 0.0]], [[a, 0.0]]], dtype=torch.bfloat16)
    out, lse = oracle.extend_attention(pool, [0], [2], [0, 1], [1], q, [0, 0], [0, 1], 1, 1.0,
                                       want_lse=True)
    w1 = math.exp(a) / (1.0 + math.exp(a))
    assert out[0, 0].tolist() == [1.0, 0.0] and lse[0, 0] == 0.0
    assert abs(out[1, 0, 0] - (1.0 - w1)) <= 1e-15 and abs(out[1, 0, 1] - w1) <= 1e-15
    assert abs(lse[1, 0] - math.log1p(math.exp(a))) <= 1e-15


# ----------------------------------------------------------------- fp8 codec

def test_e4m3_decode_matches_torch_for_all_codes():
    codes = np.arange(256, dtype=np.uint8)
    ours = oracle.e4m3_decode(codes)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan) and nan.sum() == 2
    assert np.array_equal(ours[~nan], ref[~nan])
    assert ours[0x7E] == 448.0 and ours[0x01] == 2.0 ** -9


@pytest.mark.parametrize("scale", [1.0, 0.01, 0.0371, 0.1, 0.0125, 3.3e-5])
def test_e4m3_encode_all_bf16_inputs_matches_torch_cast(scale):
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    x = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float32)
    finite_or_inf = ~torch.isnan(x)
    inv = 1.0 / torch.tensor(scale, dtype=torch.float32)   # fp32 reciprocal
    y = x * inv
    ours = oracle.e4m3_encode(y.numpy())
    ref = y.clamp(-448.0, 448.0).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    m = finite_or_inf.numpy()
    assert np.array_equal(ours[m], ref[m])
    assert (ours[~m] & 0x7F == 0x7F).all()


def test_e4m3_encode_ties_and_saturation():
    enc = oracle.e4m3_encode
    # 2^-10 is halfway between 0 and the smallest subnormal: ties to the even code 0
    assert enc(np.array([2.0 ** -10], np.float32))[0] == 0x00
    assert enc(np.array([3 * 2.0 ** -10], np.float32))[0] == 0x02   # 1.5 sub -> even 2
    assert enc(np.array([464.0, 470.0, 1e30, -1e30], np.float32)).tolist() == [0x7E, 0x7E, 0x7E, 0xFE]
    assert enc(np.array([-0.0], np.float32))[0] == 0x80


# ----------------------------------------------------------------- store

@pytest.mark.parametrize("kv_dtype", [wl.KV_BF16, wl.KV_FP8_E4M3])
def test_store_then_read_through_page_table(kv_dtype):
    w = wl.make_custom([0, 17, 64], [40, 15, 3], 4, 2, 16, kv_dtype=kv_dtype, seed=9, num_pages=40)
    t = wl.batch_tensors(w)
    fill = 0x5A
    pool = oracle_pool_for(w, t, fill=fill)
    touched = np.zeros(w.num_pages, bool)
    for r in range(w.num_reqs):
        k, v = wl.request_kv(w, r)
        if kv_dtype == wl.KV_BF16:
            ek = k.view(torch.int16).numpy().view(np.uint16)
            ev = v.view(torch.int16).numpy().view(np.uint16)
        else:
            ks = torch.from_numpy(w.k_scale)
            vs = torch.from_numpy(w.v_scale)
            def codes(x, s):
                y = (x.to(torch.float32) * (1.0 / s)[None, :, None]).clamp(-448, 448)
                return y.to(torch.float8_e4m3fn).view(torch.uint8).numpy()
            ek, ev = codes(k, ks), codes(v, vs)
        pages = w.pages_of(r)
        for j in range(ek.shape[0]):
            pg, sl = pages[j // 16], j % 16
            touched[pg] = True
            assert np.array_equal(pool.k[pg, :, sl, :], ek[j])
            assert np.array_equal(pool.v[pg, :, sl, :], ev[j])
    assert (pool.k[~touched] == fill).all() and (pool.v[~touched] == fill).all()


@pytest.mark.parametrize("seed", [0, 1])
def test_fp8_attention_matches_brute_force_on_dequantised_pool(seed):
    w = wl.make_custom([16, 45, 0], [20, 7, 33], 8, 2, 32, kv_dtype=wl.KV_FP8_E4M3, seed=seed)
    out, _, _ = _oracle_outputs(w)
    ref, _ = brute_force_all(w, dequant=fp8_dequant_torch(w))
    assert np.abs(out - ref).max() <= TOL


# ------------------------------------------------------------ planted mistakes

GATE_MAX, GATE_MEAN = 2e-2, 2e-3


def _fails_gate(a, b):
    err = np.abs(a - b)
    return err.max() > GATE_MAX or err.mean() > GATE_MEAN


@pytest.mark.parametrize("mutant", [m for m in oracle.MUTANTS if m != "none"])
def test_each_planted_mistake_fails_the_parity_gate_and_a_pin(mutant):
    # the parity gate's own small inputs: the tiny config and a sharpened ragged batch
    cases = [wl.make_workload("tiny"),
             wl.make_custom([0, 37, 64], [1, 29, 40], 4, 2, 32, q_sigma=4.0, seed=12)]
    gate_fails = False
    pin_fails = False
    for w in cases:
        t = wl.batch_tensors(w)
        pool = oracle_pool_for(w, t)
        good = oracle_all_rows(w, pool, t["q"])
        bad = oracle_all_rows(w, pool, t["q"], mutant=mutant)
        gate_fails |= _fails_gate(bad, good)
        ref, _ = brute_force_all(w)
        pin_fails |= not (np.abs(bad - ref).max() <= TOL)
    assert gate_fails, f"mutant {mutant} passes the parity gate"
    assert pin_fails, f"mutant {mutant} passes the brute-force pin"


# ------------------------------------------------- (f) the scaled-Q mode (kernel option)

@pytest.mark.parametrize("sm_scale", [1 / math.sqrt(64), 1 / math.sqrt(128), 0.3])
def test_scaled_queries_match_torch_float32_product_and_bf16_cast(sm_scale):
    g = torch.Generator().manual_seed(3)
    q = (torch.randn(7, 5, 64, generator=g) * 3).to(torch.bfloat16)
    q[0, 0, :4] = torch.tensor([0.0, -0.0, 3.0e38, -1.0e-38]).to(torch.bfloat16)
    c = torch.tensor(sm_scale, dtype=torch.float32) * torch.tensor(math.log2(math.e), dtype=torch.float32)
    want = (q.float() * c).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(oracle.scaled_queries(q, sm_scale), want)


@pytest.mark.parametrize("q_sigma", [1.0, 4.0])
def test_scaled_mode_is_base_two_attention_of_the_rounded_queries(q_sigma):
    """The mode's output is the brute force over the logical sequence with the
    rounded queries bf16(q c) and scores ln 2 * q'.k (exp2 of the base-2 scores)."""
    w = wl.make_custom([48, 13, 0], [20, 35, 9], 4, 2, 32, q_sigma=q_sigma, seed=11)
    t = wl.batch_tensors(w)
    pool = oracle_pool_for(w, t)
    out, lse = oracle_all_rows(w, pool, t["q"], want_lse=True, scaled_q=True)
    outs, lses = [], []
    for r in range(w.num_reqs):
        q = oracle.bf16_value(oracle.scaled_queries(wl.request_q(w, r), w.sm_scale))
        k, v = wl.request_kv(w, r)
        o, l = brute_force(q, to_f64(k), to_f64(v), int(w.prefix_lens[r]), math.log(2.0))
        outs.append(o)
        lses.append(l)
    assert np.abs(out - np.concatenate(outs)).max() <= TOL
    assert np.abs(lse - np.concatenate(lses)).max() <= TOL
    # and it differs from the exact attention by the rounding of q only
    exact = oracle_all_rows(w, pool, t["q"])
    assert 0 < np.abs(out - exact).max() < 0.05


def test_scaled_mode_reduces_to_exact_attention_when_the_product_is_exact():
    """With a float32 scale whose product with float32(log2 e) is exactly 1/8, every
    bf16(q / 8) is q / 8, and the mode is exact attention with softmax scale
    ln 2 / 8 (a relative 2^-24 from the scale passed)."""
    l2e = np.float32(math.log2(math.e))
    sm = np.float32(0.125 / float(l2e))
    for _ in range(8):
        prod = np.float32(sm * l2e)
        if prod == np.float32(0.125):
            break
        sm = np.nextafter(sm, np.float32(np.inf) if prod < 0.125 else np.float32(0), dtype=np.float32)
    assert np.float32(sm * l2e) == np.float32(0.125)
    w = wl.make_custom([40, 7], [25, 30], 4, 2, 32, seed=12)
    t = wl.batch_tensors(w)
    pool = oracle_pool_for(w, t)
    rr, rp = oracle.all_rows(w.extend_lens)

    def run(scale, scaled_q):
        return oracle.extend_attention(pool, w.prefix_lens, w.extend_lens, w.page_indptr, w.page_ids, t["q"],
                                       rr, rp, w.num_q_heads, scale, scaled_q=scaled_q)

    assert np.abs(run(float(sm), True) - run(math.log(2.0) / 8.0, False)).max() <= TOL
    # a scale whose product is not exact does change the result
    assert np.abs(run(0.3, True) - run(0.3, False)).max() > 1e-6
