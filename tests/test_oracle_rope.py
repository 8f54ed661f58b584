"""Pins of the RoPE / RMS-norm oracle (oracle/rope.py), of the oracle's one-step
bf16 rounding and of its value store -- no GPU.

The rotation is pinned by what fixes rotary embeddings independently of any
code: the identity at position 0, plane lengths kept, attention scores that
depend only on the relative position (RoFormer's defining property), the
complex-number form of a plane rotation, and the geometric progression of the
plane frequencies read back through the rotation itself.  The norm is pinned by
its closed forms, the rounding by torch's float32 -> bf16 cast and by exact
ties, and every planted mistake must break a pin and the GPU parity check.
"""

import numpy as np
import pytest
import torch

import oracle
from helpers import check_nearest_bf16, plane_scale
from oracle import rope as R

STYLES = [R.HALF, R.INTERLEAVED]


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def _complex_planes(x, rd, style):
    first, second = R.planes(rd, style)
    return x[..., first] + 1j * x[..., second]


# ------------------------------------------------------------------ rotation

@pytest.mark.parametrize("style", STYLES)
@pytest.mark.parametrize("rd", [128, 64, 16])
def test_position_zero_is_the_identity(style, rd):
    x = _rand((3, 2, 128), 0)
    assert np.array_equal(R.rope(x, np.zeros(3, np.int64), 1e4, rd, style), x)


@pytest.mark.parametrize("style", STYLES)
def test_rotation_keeps_every_plane_length_and_the_rest(style):
    rd = 96
    x = _rand((6, 4, 128), 1)
    pos = np.array([1, 2, 77, 4095, 131072, 262143])
    y = R.rope(x, pos, 5e5, rd, style)
    first, second = R.planes(rd, style)
    assert np.allclose(np.hypot(y[..., first], y[..., second]), np.hypot(x[..., first], x[..., second]),
                       rtol=1e-14, atol=0)
    assert np.array_equal(y[..., rd:], x[..., rd:])
    assert not np.allclose(y[..., :rd], x[..., :rd])


@pytest.mark.parametrize("style", STYLES)
@pytest.mark.parametrize("theta", [1e4, 5e5, 1e6])
def test_scores_depend_only_on_the_relative_position(style, theta):
    """<R(m) q, R(n) k> is a function of q, k and m - n (RoFormer, Section 3.1)."""
    q, k = _rand((1, 1, 128), 2), _rand((1, 1, 128), 3)
    tol = 1e-8 * np.linalg.norm(q) * np.linalg.norm(k)

    def score(m, n):
        return float(np.sum(R.rope(q, [m], theta, 128, style) * R.rope(k, [n], theta, 128, style)))

    for m, n in [(5, 3), (1000, 10), (0, 7)]:
        base = score(m, n)
        for s in [1, 17, 4096, 200000]:
            assert abs(score(m + s, n + s) - base) <= tol
    assert abs(score(5, 3) - score(6, 3)) > 1e-3


@pytest.mark.parametrize("style", STYLES)
@pytest.mark.parametrize("rd", [128, 32])
def test_each_plane_is_multiplied_by_a_unit_complex_number(style, rd):
    """Plane j of a vector at position p, read as a + ib, becomes (a + ib) e^(i p f_j)
    with f_j = theta^(-2j/rd) (RoFormer, Section 3.2)."""
    theta = 1e4
    x = _rand((5, 3, 128), 4)
    pos = np.array([0, 1, 2, 1000, 131071])
    f = theta ** (-np.arange(0, rd, 2, dtype=np.float64) / rd)
    want = _complex_planes(x, rd, style) * np.exp(1j * pos[:, None, None] * f[None, None, :])
    got = _complex_planes(R.rope(x, pos, theta, rd, style), rd, style)
    assert np.abs(got - want).max() <= 1e-10


@pytest.mark.parametrize("rd", [128, 64])
def test_plane_frequencies_form_a_geometric_progression(rd):
    """Read back through the rotation: plane 0 turns one radian per position and
    each plane turns theta^(-2/rd) times as fast as the one before."""
    theta, half = 1e4, rd // 2
    x = np.zeros((1, 1, 128))
    first, second = R.planes(rd, R.HALF)
    x[..., first] = 1.0
    y = R.rope(x, [1], theta, rd, R.HALF)[0, 0]
    ang = np.arctan2(y[second], y[first])
    assert abs(ang[0] - 1.0) <= 1e-15
    assert np.allclose(ang[1:] / ang[:-1], theta ** (-2.0 / rd), rtol=1e-12, atol=0)
    assert abs(ang[half - 1] - theta ** (-(rd - 2) / rd)) <= 1e-15


def test_the_two_layouts_differ_by_a_permutation_of_dims():
    rd = 64
    x = _rand((4, 2, 128), 5)
    pos = np.array([3, 100, 9999, 65536])
    perm = np.concatenate([np.arange(0, rd, 2), np.arange(1, rd, 2), np.arange(rd, 128)])
    a = R.rope(x[..., perm], pos, 1e4, rd, R.HALF)
    b = R.rope(x, pos, 1e4, rd, R.INTERLEAVED)[..., perm]
    assert np.array_equal(a, b)


def test_given_frequencies_scale_positions():
    """Frequencies divided by 4 at position 4p give the rotation at position p
    (the caller-given table is used as a per-plane angle rate)."""
    x = _rand((3, 2, 64), 6)
    f = R.frequencies(1e4, 64)
    a = R.rope(x, np.array([4, 400, 40000]), 0.0, 64, R.HALF, freqs=f / 4)
    b = R.rope(x, np.array([1, 100, 10000]), 1e4, 64, R.HALF)
    assert np.abs(a - b).max() <= 1e-12


# ------------------------------------------------------------------ RMS norm

def test_rms_norm_gives_unit_mean_square():
    x = _rand((7, 3, 128), 7) * 5
    y = R.rms_norm(x, np.ones(128), 0.0)
    assert np.allclose(np.mean(y * y, axis=-1), 1.0, rtol=1e-14, atol=0)


def test_rms_norm_is_scale_invariant_and_applies_the_weight_per_dim():
    x = _rand((4, 2, 64), 8)
    w = np.linspace(0.5, 1.5, 64)
    a = R.rms_norm(3.7 * x, w, 0.0)
    b = R.rms_norm(x, w, 0.0)
    assert np.allclose(a, b, rtol=1e-14, atol=1e-15)
    assert np.allclose(a / R.rms_norm(x, np.ones(64), 0.0), w[None, None, :], rtol=1e-14)


@pytest.mark.parametrize("c,eps", [(2.0, 0.0), (0.01, 1e-6), (-3.0, 1e-2)])
def test_rms_norm_of_a_constant_vector(c, eps):
    x = np.full((1, 1, 32), c)
    w = np.arange(1, 33, dtype=np.float64) / 8
    assert np.allclose(R.rms_norm(x, w, eps)[0, 0], c / np.sqrt(c * c + eps) * w, rtol=1e-15)


def test_rms_norm_and_rotation_commute_with_a_unit_weight():
    x = _rand((3, 2, 128), 9)
    pos = np.array([5, 60, 70000])
    a = R.rope(R.rms_norm(x, np.ones(128), 1e-6), pos, 1e6, 128)
    b = R.rms_norm(R.rope(x, pos, 1e6, 128), np.ones(128), 1e-6)
    assert np.allclose(a, b, rtol=1e-13, atol=1e-14)


# ------------------------------------------------------------------ bf16 rounding

def test_bf16_round_keeps_every_bf16_value():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    v = oracle.bf16_value(bits)
    m = ~np.isnan(v)
    assert np.array_equal(oracle.bf16_round(v[m]), bits[m])


def test_bf16_round_matches_torch_on_float32_inputs():
    rng = np.random.default_rng(10)
    mant = rng.uniform(1, 2, 200000)
    x = (mant * np.exp2(rng.integers(-140, 128, mant.size)) * rng.choice([-1, 1], mant.size)).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(oracle.bf16_round(x.astype(np.float64)), ref)


def test_bf16_round_ties_to_even_and_rounds_once():
    r = oracle.bf16_round
    one = 1.0
    ulp = 2.0 ** -7
    assert r(np.array([one + ulp / 2]))[0] == 0x3F80            # tie -> even (1.0)
    assert r(np.array([one + 3 * ulp / 2]))[0] == 0x3F82        # tie -> even (1 + 2 ulp)
    # just above the tie: a detour through float32 would round to the tie and then down
    x = one + ulp / 2 + 2.0 ** -30
    assert np.float32(x) == np.float32(one + ulp / 2)
    assert r(np.array([x]))[0] == 0x3F81
    assert r(np.array([-(one + ulp / 2) - 2.0 ** -30]))[0] == 0xBF81


# ------------------------------------------------------------------ value store

@pytest.mark.parametrize("kv_dtype", [oracle.KV_BF16, oracle.KV_FP8_E4M3])
def test_value_store_equals_bit_store_on_bf16_values(kv_dtype):
    rng = np.random.default_rng(11)
    P, E = [0, 21, 48], [30, 5, 17]
    T, H, d = sum(E), 2, 32
    indptr = np.array([0, 2, 4, 9])
    ids = rng.permutation(12)[:9].astype(np.int32)
    kb = oracle.bf16_round(rng.standard_normal((T, H, d)))
    vb = oracle.bf16_round(rng.standard_normal((T, H, d)))
    scales = dict(k_scale=np.array([0.02, 0.07], np.float32), v_scale=np.array([0.05, 0.03], np.float32))
    pools = [oracle.OraclePool(12, H, d, kv_dtype, fill=0x33, **scales) for _ in range(2)]
    oracle.store_kv(pools[0], P, E, indptr, ids, kb, vb)
    oracle.store_kv_values(pools[1], P, E, indptr, ids, oracle.bf16_value(kb), vb)
    assert np.array_equal(pools[0].k, pools[1].k) and np.array_equal(pools[0].v, pools[1].v)


def _e4m3_codes_f32(vals, inv):
    """torch's float8_e4m3fn cast of float32(float32(x) * inv[h]), pre-clamped to +-448."""
    y = torch.from_numpy(np.asarray(vals, np.float64).astype(np.float32)) * torch.from_numpy(inv)[None, :, None]
    return y.clamp(-448.0, 448.0).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def _e4m3_codes_f64(vals, inv):
    """The same code with the product taken in double and rounded to float32 once."""
    y = torch.from_numpy(np.asarray(vals, np.float64) * inv.astype(np.float64)[None, :, None])
    return y.clamp(-448.0, 448.0).to(torch.float32).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_fp8_value_store_matches_torch_cast_on_non_bf16_values():
    """The fp8 branch of the value store on doubles that are not bf16 values (the
    rotated keys of the fused store): each stored code must equal torch's
    float8_e4m3fn cast of float32(float32(x) * float32(1/scale)), pre-clamped to
    +-448 (the store's fp8 reading), placed through the page table.  Two plausible
    mistakes must each change some code: rounding x to bf16 before quantising,
    and scaling in double before the one rounding to float32."""
    rng = np.random.default_rng(21)
    P, E = [0, 21, 48], [30, 5, 17]
    T, H, d = sum(E), 2, 64
    indptr = np.array([0, 2, 4, 9])
    ids = rng.permutation(12)[:9].astype(np.int32)
    k_scale = np.array([0.03, 0.07], np.float32)
    inv = (np.float32(1.0) / k_scale).astype(np.float32)
    kd = rng.standard_normal((T, H, d)) * 2.0
    kd[0, 0, :8] = [5.0, -5.0, 6.0, -7.0, 1e-6, -3e-7, 0.0, 4.6]  # saturating and subnormal codes
    # keys next to the e4m3 tie points 1.0625 and -2.625 (after scaling): the float32 and
    # the double product land on opposite sides of the tie for some of them
    cand = []
    for tie in (1.0625, -2.625, 0.15625):
        for h in range(H):
            base = tie / float(inv[h])
            for k in range(-400, 400):
                x = base + k * 2.0 ** -34
                a = _e4m3_codes_f32(np.full((1, H, 1), x), inv)[0, h, 0]
                b = _e4m3_codes_f64(np.full((1, H, 1), x), inv)[0, h, 0]
                if a != b:
                    cand.append((h, x))
                    break
    assert len(cand) >= 4, "no value separates the float32 and double products"
    for j, (h, x) in enumerate(cand):
        kd[1 + j, h, 0] = x
    vb = oracle.bf16_round(rng.standard_normal((T, H, d)))
    pool = oracle.OraclePool(12, H, d, oracle.KV_FP8_E4M3, fill=0x33, k_scale=k_scale,
                             v_scale=np.array([0.05, 0.03], np.float32))
    oracle.store_kv_values(pool, P, E, indptr, ids, kd, vb)

    want = _e4m3_codes_f32(kd, inv)
    # the placement written out: token P+i of request r -> page ids[indptr[r] + (P+i)//16], slot (P+i)%16
    got = np.empty_like(want)
    row = 0
    for r in range(3):
        for i in range(E[r]):
            t = P[r] + i
            got[row] = pool.k[ids[indptr[r] + t // 16], :, t % 16, :]
            row += 1
    assert np.array_equal(got, want)
    # planted mistakes: a bf16 detour, and the product taken in double
    assert not np.array_equal(_e4m3_codes_f32(oracle.bf16_value(oracle.bf16_round(kd)), inv), want)
    assert not np.array_equal(_e4m3_codes_f64(kd, inv), want)


# ------------------------------------------------------------------ planted mistakes

@pytest.mark.parametrize("mutant", [m for m in R.MUTANTS if m != "none"])
def test_each_planted_mistake_fails_the_gpu_check(mutant):
    """A rotation with the mistake, rounded to bf16, must be rejected by the
    nearest-bf16 check the GPU tests apply (on a batch with a partial rotary
    dim, unit-free norm weights and positions up to 131k)."""
    rng = np.random.default_rng(12)
    rd, d = 64, 128
    x = oracle.bf16_round(rng.standard_normal((40, 4, d)))
    pos = np.concatenate([np.arange(20), 131000 + np.arange(20)])
    w = oracle.bf16_round(rng.uniform(0.5, 1.5, d))
    exact = R.transform(x, pos, 1e6, rd, R.HALF, w, 1e-6)
    bad = oracle.bf16_round(R.transform(x, pos, 1e6, rd, R.HALF, w, 1e-6, mutant=mutant))
    assert check_nearest_bf16(oracle.bf16_round(exact), exact, plane_scale(exact, rd, R.HALF)) == 0
    with pytest.raises(AssertionError):
        check_nearest_bf16(bad, exact, plane_scale(exact, rd, R.HALF))


def test_planted_rotation_mistakes_break_a_pin():
    x = _rand((5, 3, 128), 13)
    pos = np.array([0, 1, 2, 1000, 131071])
    f = 1e4 ** (-np.arange(0, 128, 2, dtype=np.float64) / 128)
    want = _complex_planes(x, 128, R.HALF) * np.exp(1j * pos[:, None, None] * f[None, None, :])
    for m in ("sin_sign", "other_layout"):
        got = _complex_planes(R.rope(x, pos, 1e4, 128, R.HALF, mutant=m), 128, R.HALF)
        assert np.abs(got - want).max() > 1e-3, m
    assert not np.array_equal(R.rope(x, np.zeros(5), 1e4, 128, mutant="position_plus_one"), x)
    xs = np.zeros((1, 1, 128))
    xs[..., :32] = 1.0
    y = R.rope(xs, [1], 1e4, 64, R.HALF, mutant="freq_over_head_dim")[0, 0]
    ang = np.arctan2(y[32:64], y[:32])
    assert not np.allclose(ang[1:] / ang[:-1], 1e4 ** (-2.0 / 64), rtol=1e-12, atol=0)
