"""Pins of the oracle's FP8 E4M3 cache support (a quantised KV cache, which
the paper treats as complementary to SANTA: Sec. 1 and Related Work).

- The code -> value decode against torch's float8_e4m3fn conversion (a
  library routine with the OCP definition) on all 256 codes, and against
  values the format fixes (largest finite 448, smallest subnormal 2^-9,
  smallest normal 2^-6, the two NaN codes, signed zeros).
- The batch driver on an FP8 cache equals, bit for bit, the driver on a
  bfloat16 cache holding the decoded values times the scales, with scales
  that are powers of two (so the bfloat16 values are exact) and differ by
  KV head, batch, and between K and V: a driver that applies the wrong
  scale, another row's scale or no scale fails.
"""

import math

import numpy as np
import pytest
import torch

from oracle import oracle as O
from workload import f32_to_bf16_bits, make_workload


def test_every_code_matches_torch_float8_e4m3fn():
    codes = np.arange(256, dtype=np.uint8)
    ours = O.fp8_e4m3_decode(codes)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan], ref[~nan])
    assert np.array_equal(np.signbit(ours[~nan]), np.signbit(ref[~nan]))


def test_values_the_format_fixes():
    dec = lambda c: float(O.fp8_e4m3_decode(np.array([c], np.uint8))[0])  # noqa: E731
    assert dec(0x7E) == 448.0 and dec(0xFE) == -448.0          # largest finite
    assert dec(0x01) == 2.0 ** -9 and dec(0x07) == 7 * 2.0 ** -9  # subnormals
    assert dec(0x08) == 2.0 ** -6                               # smallest normal
    assert dec(0x38) == 1.0 and dec(0xC0) == -2.0 and dec(0x3C) == 1.5
    assert math.isnan(dec(0x7F)) and math.isnan(dec(0xFF))      # no infinities
    assert dec(0x00) == 0.0 and math.copysign(1.0, dec(0x80)) == -1.0
    pos = O.fp8_e4m3_decode(np.arange(0x7F, dtype=np.uint8))
    assert np.all(np.diff(pos) > 0)                              # codes 0..126 increase


def _pow2_scales(shape, rng, lo=-4, hi=4):
    return np.ldexp(np.float32(1.0), rng.integers(lo, hi, size=shape)).astype(np.float32)


@pytest.mark.parametrize("kind", ["dense", "systematic", "stratified", "iid"])
def test_fp8_driver_equals_driver_on_decoded_values(kind):
    gen_kind = "systematic" if kind == "dense" else kind
    w = make_workload(2, B=2, n=700, ctx_len=[700, 311], kind=gen_kind, S=64, kv_dtype="fp8",
                      seed=7)
    rng = np.random.default_rng(8)
    w.k_scale = _pow2_scales((w.B, w.Hkv), rng)
    w.v_scale = _pow2_scales((w.B, w.Hkv), rng)
    assert not np.array_equal(w.k_scale, w.v_scale)
    r8 = O.decode_workload(w, kind, want_cdf=kind != "dense")
    # the same cache as bfloat16 values: scale * e4m3(code), exact in bfloat16
    kf = O.fp8_e4m3_decode(w.k) * w.k_scale[:, None, :, None]
    vf = O.fp8_e4m3_decode(w.v) * w.v_scale[:, None, :, None]
    kb, vb = f32_to_bf16_bits(kf.astype(np.float32)), f32_to_bf16_bits(vf.astype(np.float32))
    assert np.array_equal(kb.astype(np.uint32) << 16, kf.astype(np.float32).view(np.uint32))
    w.k, w.v, w.kv_dtype, w.k_scale, w.v_scale = kb, vb, "", None, None
    rb = O.decode_workload(w, kind, want_cdf=kind != "dense")
    assert np.array_equal(r8.out, rb.out)
    if kind != "dense":
        assert np.array_equal(r8.idx, rb.idx)
        assert np.array_equal(r8.cdf, rb.cdf, equal_nan=True)


def test_fp8_paged_and_flash_drivers_equal_decoded_values():
    w = make_workload(4, B=2, len_lo=300, len_hi=900, kv_dtype="fp8", seed=9)
    rng = np.random.default_rng(10)
    w.k_scale = _pow2_scales((w.B, w.Hkv), rng)
    w.v_scale = _pow2_scales((w.B, w.Hkv), rng)
    r8 = O.decode_workload(w)
    ks, vs = w.k_scale, w.v_scale
    w.k_seq = [f32_to_bf16_bits((O.fp8_e4m3_decode(w.k_seq[b]) * ks[b][None, :, None]).astype(np.float32))
               for b in range(w.B)]
    w.v_seq = [f32_to_bf16_bits((O.fp8_e4m3_decode(w.v_seq[b]) * vs[b][None, :, None]).astype(np.float32))
               for b in range(w.B)]
    w.kv_dtype, w.k_scale, w.v_scale = "", None, None
    rb = O.decode_workload(w)
    assert np.array_equal(r8.out, rb.out) and np.array_equal(r8.idx, rb.idx)

    wf = make_workload(2, B=2, n=600, ctx_len=[600, 257], kind="flash", tile=64, S_tile=4,
                       kv_dtype="fp8", seed=11)
    wf.k_scale = _pow2_scales((wf.B, wf.Hkv), rng)
    wf.v_scale = _pow2_scales((wf.B, wf.Hkv), rng)
    f8 = O.decode_workload(wf)
    wf.k = f32_to_bf16_bits((O.fp8_e4m3_decode(wf.k) * wf.k_scale[:, None, :, None]).astype(np.float32))
    wf.v = f32_to_bf16_bits((O.fp8_e4m3_decode(wf.v) * wf.v_scale[:, None, :, None]).astype(np.float32))
    wf.kv_dtype, wf.k_scale, wf.v_scale = "", None, None
    fb = O.decode_workload(wf)
    assert np.array_equal(f8.out, fb.out) and np.array_equal(f8.idx, fb.idx)


def test_fp8_workload_quantisation_is_round_to_nearest():
    """The generator's codes are the nearest E4M3 values of x / scale (input
    construction, checked here so that the FP8 workloads mean what they say)."""
    w = make_workload(2, B=1, Hq=4, Hkv=2, n=64, kind="systematic", S=8, kv_dtype="fp8", seed=12)
    grid = O.fp8_e4m3_decode(np.arange(0x7F, dtype=np.uint8))
    vals = O.fp8_e4m3_decode(w.k)
    assert np.all(np.isfinite(vals)) and np.abs(vals).max() == 448.0
    assert np.all(np.isin(np.abs(vals), grid))
