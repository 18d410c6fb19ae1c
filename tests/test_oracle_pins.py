"""Pins for the CPU oracle against facts that do not come from the oracle itself.

- number formats: torch's float8_e4m3fn / bfloat16 converters (library routines);
- compression: the defining round trip (decompress(compress(W, mask)) == W * mask,
  bitwise), the 2:4 bound of Eq. (1), exhaustive masks on one group, brute force on tiny
  matrices, and hand-worked fixtures under tests/golden/;
- GEMM: numpy fp64 matmul within the Higham bound for fp32 summation, exact integers,
  and the linearity of the two split variants of sec. 3.2 (output-split concatenates
  disjoint outputs, input-split sums two partial products).
"""
import itertools
import json
import os

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

import gen
import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
U32 = 2.0 ** -24


def tdec(codes, dtype):
    """Decode via torch (an implementation independent of the oracle)."""
    if dtype == oracle.FP8:
        return torch.from_numpy(np.ascontiguousarray(codes, np.uint8)).view(torch.float8_e4m3fn).to(
            torch.float64).numpy()
    return torch.from_numpy(np.ascontiguousarray(codes, np.uint16).view(np.int16)).view(torch.bfloat16).to(
        torch.float64).numpy()


def higham(K):
    return K * U32 / (1 - K * U32)


def same_bits(a, b):
    return np.array_equal(np.asarray(a).view(np.uint8), np.asarray(b).view(np.uint8))


# ------------------------------------------------------------------ number formats
def test_e4m3fn_decode_all_codes_match_torch():
    codes = np.arange(256, dtype=np.uint8)
    mine = oracle.decode_e4m3fn(codes)
    ref = tdec(codes, oracle.FP8)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(mine), nan)
    assert np.array_equal(mine[~nan], ref[~nan])
    assert np.array_equal(np.signbit(mine[~nan]), np.signbit(ref[~nan]))
    # format facts: NaN only at 0x7f / 0xff, max 448, smallest subnormal 2^-9
    assert set(np.nonzero(nan)[0]) == {0x7F, 0xFF}
    assert mine[0x7E] == 448.0 and mine[0x01] == 2.0 ** -9 and mine[0x08] == 2.0 ** -6


def test_bf16_decode_all_patterns_match_torch():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    mine = oracle.decode_bf16(bits).astype(np.float64)
    ref = tdec(bits, oracle.BF16)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(mine), nan)
    assert np.array_equal(mine[~nan], ref[~nan])


def test_bf16_rne_matches_torch():
    r = np.random.default_rng(5)
    u = r.integers(0, 2 ** 32, size=200000, dtype=np.uint64).astype(np.uint32)
    # exact ties with both parities of the kept bit, and values next to overflow
    ties = (r.integers(0, 2 ** 16, size=2000, dtype=np.uint64).astype(np.uint32) << 16) | 0x8000
    special = np.array([0x7F7FFFFF, 0x7F7F8000, 0x7F7F7FFF, 0x00008000, 0x00018000, 0x80008000, 0x3F808000,
                        0x3F818000, 0x7F800000, 0xFF800000], np.uint32)
    u = np.concatenate([u, ties, special])
    f = u.view(np.float32)
    mine = oracle.bf16_rne(f)
    ref = torch.from_numpy(f.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    nan = np.isnan(f)
    assert np.array_equal(mine[~nan], ref[~nan])
    assert np.all(np.isnan(oracle.decode_bf16(mine[nan])))


# ------------------------------------------------------------------ hand-worked fixtures
def _golden():
    with open(os.path.join(HERE, "golden", "hand_examples.json")) as f:
        return json.load(f)["cases"]


@pytest.mark.parametrize("case", _golden(), ids=lambda c: c["name"])
def test_golden_hand_examples(case):
    dt = oracle.FP8 if case["dtype"] == "fp8" else oracle.BF16
    ax = oracle.AXIS_OUTPUT if case["axis"] == "output" else oracle.AXIS_INPUT
    vt = np.uint8 if dt == oracle.FP8 else np.uint16
    W = np.array(case["W_codes"], vt)
    # the fixture's codes encode its stated values (checked with torch)
    assert np.array_equal(tdec(W, dt), np.array(case["W_values"], np.float64))
    mask = np.array(case["mask"], np.uint8)
    v, m, d, bad = oracle.compress(W, mask, dt, ax, case["dense_begin"])
    assert bad == 0
    assert np.array_equal(v, np.array(case["values"], vt))
    assert np.array_equal(m, np.array(case["meta"], np.uint32))
    assert np.array_equal(d, np.array(case["dense"], vt))
    X = np.array(case["X_codes"], vt)
    assert np.array_equal(tdec(X, dt), np.array(case["X_values"], np.float64))
    sw = None if case["sw"] is None else np.array(case["sw"], np.float32)
    sx = None if case["sx"] is None else np.array(case["sx"], np.float32)
    out = oracle.spense_gemm(X, v, m, d, case["N"], case["K"], dt, ax, case["dense_begin"], sw, sx)
    assert np.array_equal(out["acc"], np.array(case["acc"], np.float32))
    assert np.array_equal(out["y_f32"], np.array(case["y_exact"], np.float32))
    assert np.array_equal(out["y_bf16"], np.array(case["y_bf16_bits"], np.uint16))


# ------------------------------------------------------------------ compression
def test_compress_exhaustive_single_group():
    """All 16 masks of one group of 4: >2 kept is rejected, <=2 round-trips and is
    stored in the canonical way (ascending positions, padding holds +0)."""
    W = np.array([[0x38, 0x40, 0x44, 0xC0]], np.uint8)  # 1, 2, 3, -2
    for bits in range(16):
        mask = np.array([[(bits >> i) & 1 for i in range(4)]], np.uint8)
        v, m, d, bad = oracle.compress(W, mask, oracle.FP8, oracle.AXIS_OUTPUT, 1)
        kept = [i for i in range(4) if mask[0, i]]
        if len(kept) > 2:
            assert bad == 1
            continue
        assert bad == 0
        code = int(m[0, 0])
        i0, i1 = code & 3, (code >> 2) & 3
        assert i0 < i1 and code >> 4 == 0
        assert set(kept) <= {i0, i1}
        for j, pos in enumerate((i0, i1)):
            assert v[0, j] == (W[0, pos] if pos in kept else 0)
        # padding takes the smallest non-kept positions
        pad = sorted({i0, i1} - set(kept))
        free = [i for i in range(4) if i not in kept]
        assert pad == free[: len(pad)]
        back = oracle.decompress(v, m, d, 1, 4, oracle.FP8, oracle.AXIS_OUTPUT, 1)
        assert np.array_equal(back, W * mask)


def test_compress_bruteforce_tiny_all_two_of_four_masks():
    """N=2, K=16: every exactly-2-of-4 mask on row 0 (6^4 of them), random on row 1."""
    r = np.random.default_rng(0)
    pats = [(0, 1), (0, 2), (0, 3), (1, 2), (1, 3), (2, 3)]
    W = r.integers(1, 256, size=(2, 16)).astype(np.uint8)
    W[W == 0x80] = 0x81
    import itertools
    for combo in itertools.product(range(6), repeat=4):
        mask = np.zeros((2, 16), np.uint8)
        for g, c in enumerate(combo):
            a, b = pats[c]
            mask[0, 4 * g + a] = mask[0, 4 * g + b] = 1
            a, b = pats[r.integers(0, 6)]
            mask[1, 4 * g + a] = mask[1, 4 * g + b] = 1
        v, m, d, bad = oracle.compress(W, mask, oracle.FP8, oracle.AXIS_OUTPUT, 2)
        assert bad == 0
        back = oracle.decompress(v, m, d, 2, 16, oracle.FP8, oracle.AXIS_OUTPUT, 2)
        assert np.array_equal(back, W * mask)
        # the stored codes are exactly the kept pairs
        for g, c in enumerate(combo):
            assert (int(m[0, 0]) >> (4 * g)) & 15 == pats[c][0] | (pats[c][1] << 2)


def test_round_trip_all_byte_patterns_including_nan():
    codes = np.arange(256, dtype=np.uint8)
    W = np.tile(codes, 4).reshape(8, 128)
    r = np.random.default_rng(1)
    for axis, db in ((oracle.AXIS_OUTPUT, 6), (oracle.AXIS_INPUT, 96)):
        mask = gen.random_mask_24(r, 8, 128, gen.OUTPUT if axis == 0 else gen.INPUT, db, allow_fewer=False)
        v, m, d, bad = oracle.compress(W, mask, oracle.FP8, axis, db)
        assert bad == 0
        back = oracle.decompress(v, m, d, 8, 128, oracle.FP8, axis, db)
        assert np.array_equal(back, W * mask)


def test_second_round_trip_from_packed():
    r = np.random.default_rng(2)
    N, K, db = 24, 96, 16
    W = r.integers(0, 65536, size=(N, K)).astype(np.uint16)
    mask = gen.random_mask_24(r, N, K, gen.OUTPUT, db)
    v, m, d, _ = oracle.compress(W, mask, oracle.BF16, oracle.AXIS_OUTPUT, db)
    Wd = oracle.decompress(v, m, d, N, K, oracle.BF16, oracle.AXIS_OUTPUT, db)
    # the metadata names the positions that hold the stored values
    mask2 = np.ones((N, K), np.uint8)
    mask2[:db] = 0
    for row in range(db):
        for g in range(K // 4):
            code = (int(m[row, g // 8]) >> (4 * (g % 8))) & 15
            mask2[row, 4 * g + (code & 3)] = 1
            mask2[row, 4 * g + (code >> 2)] = 1
    v2, m2, d2, bad = oracle.compress(Wd, mask2, oracle.BF16, oracle.AXIS_OUTPUT, db)
    assert bad == 0 and np.array_equal(v2, v) and np.array_equal(m2, m) and np.array_equal(d2, d)


def test_null_mask_keeps_nonzero_bit_patterns():
    W = np.array([[0x38, 0, 0x80, 0, 0, 0, 0, 0x44]], np.uint8)  # 1, 0, -0, 0 | 0, 0, 0, 3
    v, m, d, bad = oracle.compress(W, None, oracle.FP8, oracle.AXIS_OUTPUT, 1)
    assert bad == 0
    assert list(v[0]) == [0x38, 0x80, 0x00, 0x44]
    assert int(m[0, 0]) == (0 | 2 << 2) | ((0 | 3 << 2) << 4)
    W3 = np.array([[0x38, 0x38, 0x38, 0]], np.uint8)
    assert oracle.compress(W3, None, oracle.FP8, oracle.AXIS_OUTPUT, 1)[3] == 1


@settings(max_examples=60, deadline=None)
@given(st.integers(1, 40), st.integers(1, 24), st.sampled_from([0, 1]), st.floats(0.0, 1.0),
       st.sampled_from([1, 2]), st.integers(0, 2 ** 31))
def test_property_round_trip_and_eq1(N, k4, axis, frac, dtype, seed):
    K = 4 * k4
    r = np.random.default_rng(seed)
    vt = np.uint8 if dtype == 1 else np.uint16
    W = r.integers(0, 256 if dtype == 1 else 65536, size=(N, K)).astype(vt)
    if axis == 0:
        db = int(round(frac * N))
        mask = gen.random_mask_24(r, N, K, gen.OUTPUT, db)
    else:
        db = 4 * int(round(frac * k4))
        mask = gen.random_mask_24(r, N, K, gen.INPUT, db)
    v, m, d, bad = oracle.compress(W, mask, dtype, axis, db)
    assert bad == 0
    back = oracle.decompress(v, m, d, N, K, dtype, axis, db)
    assert np.array_equal(back, W * mask.astype(vt))
    # Eq. (1): every group of 4 in the sparse region has at most 2 non-zero patterns
    reg = back[:db] if axis == 0 else back[:, :db]
    if reg.size:
        nz = (reg != 0).reshape(reg.shape[0], -1, 4).sum(-1)
        assert nz.max() <= 2


def test_bad_groups_are_counted():
    W = np.full((4, 64), 0x38, np.uint8)
    mask = np.ones((4, 64), np.uint8)
    _, _, _, bad = oracle.compress(W, mask, oracle.FP8, oracle.AXIS_INPUT, 32)
    assert bad == 4 * 8
    _, _, _, bad = oracle.compress(W, mask, oracle.FP8, oracle.AXIS_OUTPUT, 0)
    assert bad == 0  # everything is dense


# ------------------------------------------------------------------ GEMM
def _rand_fp8(r, shape, scale=1.0):
    return gen.to_e4m3fn(r.standard_normal(shape).astype(np.float32) * np.float32(scale))


@pytest.mark.parametrize("dtype", [oracle.FP8, oracle.BF16])
def test_gemm_within_higham_bound_of_fp64_matmul(dtype):
    r = np.random.default_rng(3)
    M, N, K = 7, 33, 1024
    if dtype == oracle.FP8:
        X, W = _rand_fp8(r, (M, K)), _rand_fp8(r, (N, K), 8.0)
    else:
        X = gen.to_bf16(r.standard_normal((M, K)).astype(np.float32))
        W = gen.to_bf16(r.standard_normal((N, K)).astype(np.float32) * 0.02)
    xd, wd = tdec(X, dtype), tdec(W, dtype)
    exact = xd @ wd.T
    absd = np.abs(xd) @ np.abs(wd).T
    out = oracle.gemm(X, W, dtype)
    err = np.abs(out["acc"].astype(np.float64) - exact)
    assert np.all(err <= higham(K) * absd)
    assert np.any(err > 0)  # the fp32 oracle really rounds
    o64 = oracle.gemm_f64(X, W, dtype)
    assert np.all(np.abs(o64["acc"] - exact) <= 2 * K * 2.0 ** -53 * absd)
    assert np.allclose(o64["abs_dot"], absd, rtol=1e-12, atol=0)


def test_gemm_exact_integers_and_pow2_epilogue():
    r = np.random.default_rng(4)
    M, N, K = 5, 19, 4096
    Wv, Xv = r.integers(-3, 4, size=(N, K)), r.integers(-3, 4, size=(M, K))
    W, X = gen.int_codes(Wv, gen.FP8), gen.int_codes(Xv, gen.FP8)
    sw = (2.0 ** r.integers(-4, 3, size=N)).astype(np.float32)
    sx = (2.0 ** r.integers(-4, 3, size=M)).astype(np.float32)
    out = oracle.gemm(X, W, oracle.FP8, sw, sx)
    exact = (Xv @ Wv.T).astype(np.int64)
    assert np.array_equal(out["acc"].astype(np.int64), exact)
    y = exact * sw[None, :].astype(np.float64) * sx[:, None].astype(np.float64)
    assert np.array_equal(out["y_f32"].astype(np.float64), y)
    ref = torch.from_numpy(y.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(out["y_bf16"], ref)


def test_epilogue_two_fp32_roundings_then_bf16():
    r = np.random.default_rng(6)
    M, N, K = 9, 21, 256
    X, W = _rand_fp8(r, (M, K)), _rand_fp8(r, (N, K))
    sw = r.uniform(1e-4, 1e-2, N).astype(np.float32)
    sx = r.uniform(1e-3, 1e-1, M).astype(np.float32)
    out = oracle.gemm(X, W, oracle.FP8, sw, sx)
    t = (out["acc"] * sw[None, :]).astype(np.float32)
    t = (t * sx[:, None]).astype(np.float32)
    assert np.array_equal(out["y_f32"], t)
    ref = torch.from_numpy(t).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(out["y_bf16"], ref)


def _packed(r, N, K, axis, db, dtype):
    if dtype == oracle.FP8:
        W = _rand_fp8(r, (N, K), 4.0)
    else:
        W = gen.to_bf16(r.standard_normal((N, K)).astype(np.float32))
    mask = gen.random_mask_24(r, N, K, gen.OUTPUT if axis == 0 else gen.INPUT, db)
    v, m, d, bad = oracle.compress(W, mask, dtype, axis, db)
    assert bad == 0
    return W, mask, v, m, d


@pytest.mark.parametrize("dtype", [oracle.FP8, oracle.BF16])
def test_output_split_is_concatenation_of_two_gemms(dtype):
    """Sec. 3.2: the sparse GEMM produces one block of output columns, the dense GEMM
    the other; checked against numpy on the stored pieces directly."""
    r = np.random.default_rng(7)
    M, N, K, Ns = 6, 40, 256, 24
    W, mask, v, m, d = _packed(r, N, K, 0, Ns, dtype)
    X = _rand_fp8(r, (M, K)) if dtype == oracle.FP8 else gen.to_bf16(r.standard_normal((M, K)).astype(np.float32))
    out = oracle.spense_gemm(X, v, m, d, N, K, dtype, 0, Ns)
    xd = tdec(X, dtype)
    # sparse block from the values + metadata by numpy indexing, dense block as stored
    vals = tdec(v, dtype)
    ws = np.zeros((Ns, K))
    for g in range(K // 4):
        code = (m[:, g // 8] >> np.uint32(4 * (g % 8))) & np.uint32(15)
        ws[np.arange(Ns), 4 * g + (code & 3).astype(np.int64)] = vals[:, 2 * g]
        ws[np.arange(Ns), 4 * g + (code >> 2).astype(np.int64)] = vals[:, 2 * g + 1]
    y_s = xd @ ws.T
    y_d = xd @ tdec(d, dtype).T
    ref = np.concatenate([y_s, y_d], axis=1)
    absd = np.abs(xd) @ np.abs(np.concatenate([ws, tdec(d, dtype)])).T
    assert np.all(np.abs(out["acc"] - ref) <= higham(K) * absd)


@pytest.mark.parametrize("dtype", [oracle.FP8, oracle.BF16])
def test_input_split_is_sum_of_two_partial_gemms(dtype):
    r = np.random.default_rng(8)
    M, N, K, Ks = 5, 17, 384, 256
    W, mask, v, m, d = _packed(r, N, K, 1, Ks, dtype)
    X = _rand_fp8(r, (M, K)) if dtype == oracle.FP8 else gen.to_bf16(r.standard_normal((M, K)).astype(np.float32))
    out = oracle.spense_gemm(X, v, m, d, N, K, dtype, 1, Ks)
    xd = tdec(X, dtype)
    wm = tdec(W, dtype) * mask
    part_s = xd[:, :Ks] @ wm[:, :Ks].T
    part_d = xd[:, Ks:] @ tdec(d, dtype).T
    absd = np.abs(xd) @ np.abs(wm).T
    assert np.all(np.abs(out["acc"] - (part_s + part_d)) <= higham(K) * absd)
    # the dense region ignores the mask: it equals the unpruned W columns
    assert np.array_equal(d, W[:, Ks:])


@pytest.mark.parametrize("axis", [0, 1])
def test_dense_fraction_zero_and_one(axis):
    r = np.random.default_rng(9)
    M, N, K = 4, 32, 256
    X = _rand_fp8(r, (M, K))
    W = _rand_fp8(r, (N, K))
    full = N if axis == 0 else K
    # fraction 1: sparse region empty -> plain GEMM on W
    v, m, d, _ = oracle.compress(W, None, oracle.FP8, axis, 0)
    assert v.size == 0 and m.size == 0 and np.array_equal(d, W)
    out = oracle.spense_gemm(X, v, m, d, N, K, oracle.FP8, axis, 0)
    assert np.array_equal(out["acc"], oracle.gemm(X, W, oracle.FP8)["acc"])
    # fraction 0: dense region empty -> pure 2:4 GEMM on W * mask
    mask = gen.random_mask_24(r, N, K, gen.OUTPUT if axis == 0 else gen.INPUT, full, allow_fewer=False)
    v, m, d, _ = oracle.compress(W, mask, oracle.FP8, axis, full)
    assert d.size == 0
    out = oracle.spense_gemm(X, v, m, d, N, K, oracle.FP8, axis, full)
    xd, wm = tdec(X, oracle.FP8), tdec(W, oracle.FP8) * mask
    absd = np.abs(xd) @ np.abs(wm).T
    assert np.all(np.abs(out["acc"] - xd @ wm.T) <= higham(K) * absd)


def test_empty_shapes():
    W = np.zeros((0, 64), np.uint8)
    v, m, d, bad = oracle.compress(W, None, oracle.FP8, 0, 0)
    assert bad == 0 and v.shape == (0, 32) and d.shape == (0, 64)
    X = np.zeros((0, 64), np.uint8)
    out = oracle.gemm(X, np.zeros((3, 64), np.uint8), oracle.FP8)
    assert out["y_bf16"].shape == (0, 3)
    out = oracle.gemm(np.zeros((2, 0), np.uint8), np.zeros((3, 0), np.uint8), oracle.FP8)
    assert np.array_equal(out["acc"], np.zeros((2, 3), np.float32))


# ------------------------------------------------------------------ input generators
def test_magnitude_mask_keeps_two_largest_and_row_absmax():
    r = np.random.default_rng(10)
    Wf = gen.draw_weight(r, 64, 128)
    Wf[0, :4] = [0.5, -0.5, 0.5, 0.1]  # tie: the lower indices win
    mask = gen.magnitude_mask_24(Wf, gen.OUTPUT, 48)
    assert list(mask[0, :4]) == [1, 1, 0, 0]
    kept = mask[:48].reshape(48, -1, 4).sum(-1)
    assert np.all(kept == 2) and np.all(mask[48:] == 1)
    a = np.abs(Wf[:48]).reshape(48, -1, 4)
    kmin = np.where(mask[:48].reshape(48, -1, 4) == 1, a, np.inf).min(-1)
    dmax = np.where(mask[:48].reshape(48, -1, 4) == 0, a, -np.inf).max(-1)
    assert np.all(kmin >= dmax)
    # pruning keeps every group's maximum, so the row absmax (the fp8 scale) is unchanged
    assert np.array_equal(np.abs(Wf[:48] * mask[:48]).max(1), np.abs(Wf[:48]).max(1))


def test_quantize_rows_fp8_scale_and_saturation():
    r = np.random.default_rng(11)
    A = r.standard_normal((8, 64)).astype(np.float32)
    A[3] = 0
    codes, s = gen.quantize_rows_fp8(A)
    assert s[3] == 1.0 and np.all(codes[3] == 0)
    d = tdec(codes, oracle.FP8)
    assert np.all(np.abs(d).max(1)[[0, 1, 2, 4, 5, 6, 7]] == 448.0)
    assert not np.any(np.isnan(d))


# ------------------------------------------------------------------ activation quantisation and GLU
def _finite_codes():
    return np.array([c for c in range(256) if c & 0x7F != 0x7F], np.uint8)


def test_encode_e4m3fn_round_trips_every_finite_code():
    c = _finite_codes()
    v = tdec(c, oracle.FP8).astype(np.float32)
    assert np.array_equal(oracle.encode_e4m3fn(v), c)  # -0 included (0x80)


def test_encode_e4m3fn_ties_go_to_even_mantissa_and_neighbours_to_nearest():
    pos = np.arange(0, 0x7F, dtype=np.uint8)  # 0 .. 448
    v = tdec(pos, oracle.FP8)
    mid = ((v[:-1] + v[1:]) / 2).astype(np.float32)  # dyadic, exact in fp32
    assert np.array_equal(mid.astype(np.float64), (v[:-1] + v[1:]) / 2)
    want = np.where(pos[:-1] % 2 == 0, pos[:-1], pos[1:])
    assert np.array_equal(oracle.encode_e4m3fn(mid), want)
    assert np.array_equal(oracle.encode_e4m3fn(-mid), want | 0x80)
    below = np.nextafter(mid, np.float32(0))
    above = np.nextafter(mid, np.float32(np.inf))
    assert np.array_equal(oracle.encode_e4m3fn(below), pos[:-1])
    assert np.array_equal(oracle.encode_e4m3fn(above), pos[1:])


def test_encode_e4m3fn_saturates_and_keeps_nan():
    big = np.array([448.0, 449.0, 463.99, 464.0, 480.0, 1e6, 3.4e38, np.inf], np.float32)
    assert np.all(oracle.encode_e4m3fn(big) == 0x7E)
    assert np.all(oracle.encode_e4m3fn(-big) == 0xFE)
    assert oracle.encode_e4m3fn(np.array([np.nan], np.float32))[0] & 0x7F == 0x7F


def test_encode_e4m3fn_matches_torch_in_range():
    r = np.random.default_rng(21)
    x = np.concatenate([r.uniform(-448, 448, 20000), r.standard_normal(20000) * 0.05,
                        r.uniform(-2 ** -6, 2 ** -6, 5000)]).astype(np.float32)
    want = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(oracle.encode_e4m3fn(x), want)


def test_quantize_rows_matches_generator_and_its_invariants():
    r = np.random.default_rng(22)
    A = (r.standard_normal((12, 300)) * np.exp(r.uniform(-6, 6, (12, 1)))).astype(np.float32)
    A[4] = 0
    A[7, 5] = -A[7].__abs__().max() * 3  # a single dominant negative entry
    q, s = oracle.quantize_rows(A)
    gq, gs = gen.quantize_rows_fp8(A)  # torch's converter, independent of the oracle
    assert np.array_equal(q, gq) and np.array_equal(s.view(np.uint32), gs.view(np.uint32))
    d = tdec(q, oracle.FP8)
    assert s[4] == 1.0 and np.all(q[4] == 0)
    nz = [i for i in range(12) if i != 4]
    assert np.all(np.abs(d[nz]).max(axis=1) == 448.0)
    # every entry is within half a step of its code (relative 2^-4 for normals, 2^-10 * s
    # absolute in the subnormal range)
    err = np.abs(d * s[:, None].astype(np.float64) - A.astype(np.float64))
    bound = np.maximum(2.0 ** -4 * np.abs(A), 2.0 ** -10 * s[:, None]) * (1 + 1e-6)
    assert np.all(err <= bound)
    # scaling a row by a power of two leaves the codes and scales the scale
    q2, s2 = oracle.quantize_rows(A * np.float32(2.0 ** 5))
    assert np.array_equal(q2, q) and np.array_equal(s2[nz], s[nz] * np.float32(32.0))


def test_glu_silu_odd_and_even_parts_and_linearity():
    g = np.linspace(-30, 30, 4001)
    one = np.ones_like(g)
    h = oracle.glu_f64(g, one)
    hn = oracle.glu_f64(-g, one)
    assert np.allclose(h - hn, g, rtol=0, atol=1e-13)  # silu(x) - silu(-x) = x
    assert np.allclose(h + hn, g * np.tanh(g / 2), rtol=1e-13, atol=1e-300)  # = x tanh(x/2)
    u = np.random.default_rng(23).standard_normal(g.size)
    assert np.array_equal(oracle.glu_f64(g, 2 * u), 2 * oracle.glu_f64(g, u))
    assert oracle.glu_f64(np.zeros(1), np.ones(1))[0] == 0.0


def test_mlp_is_invariant_under_a_permutation_of_intermediate_indices():
    """Eq. (4): permuting the intermediate dimension (rows of gate and up, columns of
    down) consistently leaves the MLP output unchanged; with every weight dense only the
    fp32 summation order of the down GEMM changes."""
    r = np.random.default_rng(24)
    M, D, I = 3, 64, 96
    X, sx = gen.quantize_rows_fp8(r.standard_normal((M, D)).astype(np.float32))

    Wg, Wu, Wd = [(r.standard_normal(shape) * 0.05).astype(np.float32) for shape in ((I, D), (I, D), (D, I))]
    p = r.permutation(I)

    def pack(Wf, axis):  # every entry dense (dense_begin 0 on either axis)
        q, s = gen.quantize_rows_fp8(Wf)
        N, K = q.shape
        v, m, d, bad = oracle.compress(q, np.ones_like(q), oracle.FP8, axis, 0)
        return (v, m, d, N, K, axis, 0, s)

    a = oracle.mlp(X, sx, pack(Wg, 0), pack(Wu, 0), pack(Wd, 1))
    b = oracle.mlp(X, sx, pack(Wg[p], 0), pack(Wu[p], 0), pack(Wd[:, p], 1))
    assert np.array_equal(b["Hq"], a["Hq"][:, p]) and np.array_equal(b["sh"], a["sh"])
    assert np.allclose(b["Y"], a["Y"], rtol=1e-5, atol=1e-6 * np.abs(a["Y"]).max())


def _torch_decode_e4m3fn(codes):
    """e4m3fn codes -> fp64 through torch's converter (independent of the oracle's decoder)."""
    return torch.from_numpy(np.ascontiguousarray(codes)).view(torch.float8_e4m3fn).to(torch.float64).numpy()


def _independent_mlp(X, sx, Wg, sg, Wu, su, Wd, sd):
    """Eq. (4) composed with numpy and torch only: inputs and weights decoded by torch,
    G and U as fp64 matmuls of the scaled values, H = U * G / (1 + exp(-G)), its per-token
    fp8 quantisation by torch's converter (the generator's), Y = (Hq sh) (Wd sd)^T in fp64.
    Returns the pieces and, per output, sum |h w| * |sh sd| for the error bound."""
    Xs = _torch_decode_e4m3fn(X) * sx.astype(np.float64)[:, None]
    G = Xs @ (_torch_decode_e4m3fn(Wg) * sg.astype(np.float64)[:, None]).T
    U = Xs @ (_torch_decode_e4m3fn(Wu) * su.astype(np.float64)[:, None]).T
    H = U * G / (1.0 + np.exp(-G))
    Hq, sh = gen.quantize_rows_fp8(H.astype(np.float32))
    hd, wd = _torch_decode_e4m3fn(Hq), _torch_decode_e4m3fn(Wd)
    scale = sh.astype(np.float64)[:, None] * sd.astype(np.float64)[None, :]
    Y = (hd @ wd.T) * scale
    absdot = (np.abs(hd) @ np.abs(wd).T) * np.abs(scale)
    return {"G": G, "U": U, "H": H, "Hq": Hq, "sh": sh, "Y": Y, "absdot": absdot}


def test_mlp_matches_an_independent_composition():
    """Eq. (4) through the oracle (Spense-packed weights with 2:4 and dense regions)
    against the same MLP composed with numpy and torch's converters from the decompressed
    weights: G, U and H agree to fp64 rounding, the codes and token scales of H bit for
    bit, and Y (fp32 sums, two fp32 scale roundings) is inside the Higham bound of the
    fp64 Y.  The check tells the plausible mistakes apart: gate and up swapped, or the
    down GEMM scaled by the input's token scales instead of H's, land far outside it."""
    r = np.random.default_rng(25)
    M, D, I = 5, 128, 192
    X, sx = gen.quantize_rows_fp8(r.standard_normal((M, D)).astype(np.float32))
    Wg, Wu, Wd = [(r.standard_normal(shape) * 0.05).astype(np.float32) for shape in ((I, D), (I, D), (D, I))]
    dbg, dbd = 144, 160  # the last 48 rows of gate / up and the last 32 columns of down dense

    def pack(Wf, axis, db):
        q, s = gen.quantize_rows_fp8(Wf)
        N, K = q.shape
        mask = gen.magnitude_mask_24(Wf, gen.OUTPUT if axis == 0 else gen.INPUT, db)
        v, m, d, bad = oracle.compress(q, mask, oracle.FP8, axis, db)
        assert bad == 0
        dense = np.where(mask.astype(bool), q, np.uint8(0))  # masked-out entries are +0
        return (v, m, d, N, K, axis, db, s), dense, s

    pg, qg, sg = pack(Wg, 0, dbg)
    pu, qu, su = pack(Wu, 0, dbg)
    pd, qd, sd = pack(Wd, 1, dbd)
    o = oracle.mlp(X, sx, pg, pu, pd)
    ind = _independent_mlp(X, sx, qg, sg, qu, su, qd, sd)
    for k in ("G", "U", "H"):
        assert np.allclose(o[k], ind[k], rtol=1e-12, atol=1e-14 * np.abs(ind[k]).max()), k
    assert np.array_equal(o["Hq"], ind["Hq"]) and np.array_equal(o["sh"].view(np.uint32), ind["sh"].view(np.uint32))
    gamma = I * 2.0 ** -24 / (1 - I * 2.0 ** -24)
    bound = 2 * gamma * ind["absdot"] + 4 * 2.0 ** -24 * np.abs(ind["Y"]) + 1e-30
    assert np.all(np.abs(o["Y"].astype(np.float64) - ind["Y"]) <= bound)
    # sensitivity of the check: two plausible mistakes fall outside the same bound
    swapped = _independent_mlp(X, sx, qu, su, qg, sg, qd, sd)["Y"]
    assert np.abs(o["Y"] - swapped).max() > 100 * bound.max()
    wrong_scale = ind["Y"] / ind["sh"].astype(np.float64)[:, None] * sx.astype(np.float64)[:, None]
    assert np.abs(o["Y"] - wrong_scale).max() > 100 * bound.max()


def test_reconstruction_loss_is_eq2_with_explicit_activations():
    """Eq. (2) evaluated from an explicit calibration matrix X, ||X W^T - X W_hat^T||_F^2,
    equals the oracle's form through H = X^T X; zero for W_hat = W; a single changed
    weight w[n, k] -> w[n, k] + d costs d^2 ||X[:, k]||^2; losses of disjoint row sets add."""
    r = np.random.default_rng(26)
    n, N, K = 300, 12, 40
    X = r.standard_normal((n, K)) * np.exp(r.uniform(-1, 1, K))[None, :]
    W = r.standard_normal((N, K))
    W_hat = W * (r.random((N, K)) > 0.5)
    H = X.T @ X
    want = float(np.sum((X @ W.T - X @ W_hat.T) ** 2))
    assert abs(oracle.reconstruction_loss(W, W_hat, H) - want) <= 1e-10 * want
    assert oracle.reconstruction_loss(W, W, H) == 0.0
    W2 = W.copy()
    W2[3, 7] += 0.25
    assert np.isclose(oracle.reconstruction_loss(W, W2, H), 0.0625 * np.sum(X[:, 7] ** 2), rtol=1e-12, atol=0)
    a, b = oracle.reconstruction_loss(W[:5], W_hat[:5], H), oracle.reconstruction_loss(W[5:], W_hat[5:], H)
    assert np.isclose(a + b, want, rtol=1e-12, atol=0)
    # transposing W (an N x K vs K x N mix-up) is caught: the shapes no longer fit H
    with pytest.raises(ValueError):
        oracle.reconstruction_loss(W.T, W_hat.T, H)


# ------------------------------------------------------------------ dense-index selection (sec. 3.3.1)
def test_index_scores_closed_forms():
    I, D = 6, 8
    ones = np.ones((I, D))
    r = oracle.index_scores(ones, ones, np.ones((D, I)), np.full(D, 4.0), np.full(I, 9.0), eps=0.0)
    assert np.allclose(r["gate"], 2.0) and np.allclose(r["up"], 2.0) and np.allclose(r["down"], 3.0)
    assert np.allclose(r["total"], 3.0)  # each normalised vector is all ones
    # one row / column scaled: its raw score scales, the normalised sum keeps mean 3 (eps 0)
    Wg = ones.copy()
    Wg[2] *= 5
    Wd = np.ones((D, I))
    Wd[:, 4] *= -7  # signs do not matter
    r = oracle.index_scores(Wg, ones, Wd, np.full(D, 4.0), np.full(I, 9.0), eps=0.0)
    assert r["gate"][2] == 10.0 and r["down"][4] == 21.0
    assert np.isclose(r["total"].mean(), 3.0)
    assert np.argmax(r["total"]) in (2, 4)


def test_index_scores_wanda_identity_against_activations():
    """With h = diag(X^T X), the score is the mean over j of |W_ij| * ||X[:, j]||_2."""
    rng = np.random.default_rng(70)
    I, D, T = 20, 12, 30
    X = rng.standard_normal((T, D))
    Hm = rng.standard_normal((T, I))
    Wg, Wu, Wd = rng.standard_normal((I, D)), rng.standard_normal((I, D)), rng.standard_normal((D, I))
    r = oracle.index_scores(Wg, Wu, Wd, np.einsum("td,td->d", X, X), np.einsum("ti,ti->i", Hm, Hm))
    colnorm = np.linalg.norm(X, axis=0)
    assert np.allclose(r["gate"], (np.abs(Wg) @ colnorm) / D, rtol=1e-12)
    assert np.allclose(r["down"], np.abs(Wd).mean(axis=0) * np.linalg.norm(Hm, axis=0), rtol=1e-12)


def test_dense_index_permutation_brute_force():
    rng = np.random.default_rng(71)
    for trial in range(50):
        n = int(rng.integers(1, 12))
        k = int(rng.integers(0, n + 1))
        t = rng.integers(0, 4, n).astype(np.float64)  # many ties
        r = oracle.dense_index_permutation(t, k)
        # brute force over every k-subset: the largest score sum, then the lexicographically
        # smallest index list (ties keep lower indices)
        best = min(itertools.combinations(range(n), k), key=lambda c: (-sum(t[i] for i in c), c))
        assert np.array_equal(r["dense"], np.array(sorted(best), dtype=r["dense"].dtype))
        perm = r["perm"]
        assert sorted(perm.tolist()) == list(range(n))  # a permutation
        assert set(perm[n - k:].tolist()) == set(best)  # dense indices at the back
        assert np.all(np.diff(perm[: n - k]) > 0) and np.all(np.diff(perm[n - k:]) > 0)


# ---------------------------------------------------------------- SparseGPT 2:4 with a protected dense region
def _spd(seed, K, M=None, corr=0.3):
    """H = X^T X of correlated synthetic activations (M x K)."""
    r = np.random.default_rng(seed)
    M = M or 4 * K
    X = r.standard_normal((M, K)) @ (np.eye(K) + corr * r.standard_normal((K, K)) / np.sqrt(K))
    return X.T @ X


def test_obs_factor_rows_are_the_sequential_inverse_hessians():
    """Row j of U (scaled by U_jj) is row 0 of inv(Hd[j:, j:]), the inverse Hessian of the
    columns not yet frozen when column j is processed: the OBS quantities of Eq. (3)."""
    H = _spd(1, 14)
    U, _ = oracle.obs_factor(H, 0.01)
    Hd, _ = oracle.obs_damp(H, 0.01)
    assert np.allclose(np.tril(U, -1), 0)
    for j in range(14):
        row = np.linalg.inv(Hd[j:, j:])[0]
        assert np.allclose(U[j, j] * U[j, j:], row, rtol=1e-10, atol=1e-14)


def _explicit_obs(W, H, dense_begin, percdamp=0.01):
    """Eq. (3) written out with an explicit inverse per step: before column j is processed
    the free set is F = {j, ..., K-1}; the denominator of column m is [inv(Hd[m:, m:])]_00."""
    Hd, dead = oracle.obs_damp(H, percdamp)
    W = np.array(W, np.float64)
    W[:, dead] = 0
    N, K = W.shape
    keep = np.ones((N, K), bool)
    d = [np.linalg.inv(Hd[m:, m:])[0, 0] for m in range(K)]
    for j in range(dense_begin):
        if j % 4 == 0:
            for n in range(N):
                errs = [(W[n, j + c] ** 2 / d[j + c], c) for c in range(4)]
                for _, c in sorted(errs)[:2]:
                    keep[n, j + c] = False
        Hinv = np.linalg.inv(Hd[j:, j:])
        for n in range(N):
            q = W[n, j] if keep[n, j] else 0.0
            W[n, j:] -= (W[n, j] - q) / Hinv[0, 0] * Hinv[0]
            W[n, j] = q
    return W, keep


def test_obs_sweep_matches_eq3_with_explicit_inverses():
    H = _spd(2, 24)
    W = np.random.default_rng(3).standard_normal((6, 24))
    ref_W, ref_keep = _explicit_obs(W, H, 16)
    out = oracle.obs_prune_24(W, H, 16)
    assert np.array_equal(out["keep"], ref_keep)
    assert np.allclose(out["W"], ref_W, rtol=1e-9, atol=1e-12)


def test_obs_with_a_diagonal_hessian_is_magnitude_pruning():
    """Uncorrelated inputs: no compensation (U is diagonal); each group keeps the two
    weights with the largest |w| sqrt(h_jj + lambda), unchanged; the rest become 0."""
    r = np.random.default_rng(4)
    K, N = 32, 7
    h = r.uniform(0.1, 5.0, K)
    W = r.standard_normal((N, K))
    out = oracle.obs_prune_24(W, np.diag(h), 24)
    hd = h + 0.01 * h.mean()
    for n in range(N):
        for g in range(6):
            s = [abs(W[n, 4 * g + c]) * np.sqrt(hd[4 * g + c]) for c in range(4)]
            top = sorted(range(4), key=lambda c: -s[c])[:2]
            for c in range(4):
                want = W[n, 4 * g + c] if c in top else 0.0
                assert out["W"][n, 4 * g + c] == want and out["keep"][n, 4 * g + c] == (c in top)
    assert np.array_equal(out["W"][:, 24:], W[:, 24:])


def test_obs_dense_buffer_is_the_least_squares_compensation():
    """After the sweep the dense columns hold the best compensation for the frozen 2:4
    columns: w_D - Hd_DD^{-1} Hd_DS (w_hat_S - w_S) minimises Eq. (2) over the dense
    entries (damped Hessian)."""
    H = _spd(5, 40)
    W = np.random.default_rng(6).standard_normal((5, 40))
    out = oracle.obs_prune_24(W, H, 24)
    Hd, _ = oracle.obs_damp(H, 0.01)
    S, D = slice(0, 24), slice(24, 40)
    want = W[:, D] - np.linalg.solve(Hd[D, D], Hd[D, S] @ (out["W"][:, S] - W[:, S]).T).T
    assert np.allclose(out["W"][:, D], want, rtol=1e-9, atol=1e-11)


def test_obs_edge_cases():
    H = _spd(7, 16)
    W = np.random.default_rng(8).standard_normal((3, 16))
    out = oracle.obs_prune_24(W, H, 0)  # all dense: nothing changes
    assert np.array_equal(out["W"], W) and out["keep"].all()
    out = oracle.obs_prune_24(W, H, 16)  # all 2:4
    assert (out["keep"].reshape(3, 4, 4).sum(-1) == 2).all()
    assert np.array_equal(out["W"] != 0, out["keep"])
    H2 = H.copy()
    H2[5, :] = 0
    H2[:, 5] = 0  # a column no input excites
    out = oracle.obs_prune_24(W, H2, 8)
    assert (out["W"][:, 5] == 0).all() and np.isfinite(out["W"]).all()


def test_back_placement_keeps_the_dense_columns_as_a_compensation_buffer():
    """Sec. 3.3.1 (Table "front_back"): with the same dense columns, processing them last
    (they absorb the compensation) reconstructs better than processing them first (they
    are frozen before any 2:4 column is pruned).  Front placement is the sweep over the
    2:4 columns alone (their inverse Hessians involve only unprocessed 2:4 columns) with
    the dense columns unchanged.  An observed property on seeded correlated data."""
    K, nd = 64, 16
    H = _spd(9, K, corr=1.0)
    W = np.random.default_rng(10).standard_normal((16, K))
    back = oracle.obs_prune_24(W, H, K - nd)["W"]
    S = slice(0, K - nd)
    front = W.copy()
    front[:, S] = oracle.obs_prune_24(W[:, S], H[S, S], K - nd)["W"]
    lb, lf = oracle.reconstruction_loss(W, back, H), oracle.reconstruction_loss(W, front, H)
    assert lb < 0.9 * lf, (lb, lf)
