"""Pins of the oracle's KV-cache append and its OCP E4M3 encoder.

Checked against: torch's float8_e4m3fn cast (a library routine) on clamped
float32 values, the exact round trip of every finite E4M3 code, ties and
saturation worked out by hand from the format, and an element-by-element
scalar restatement of the append on small pools.
"""
import numpy as np
import torch

from oracle import append, numerics


def torch_e4m3(x32):
    x32 = np.clip(np.asarray(x32, np.float32), -448.0, 448.0)
    return torch.from_numpy(x32).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_encode_matches_torch_cast_over_all_magnitudes():
    rng = np.random.default_rng(21)
    mant = rng.random(200000) + 1.0
    expo = rng.integers(-14, 11, 200000)
    sign = np.where(rng.random(200000) < 0.5, -1.0, 1.0)
    x = (sign * mant * np.exp2(expo)).astype(np.float32)
    x = np.concatenate([x, np.float32([0.0, -0.0, 448.0, -448.0, 500.0, -1e30, 1e-30, -1e-30])])
    assert np.array_equal(append.e4m3_encode(x.astype(np.float64)), torch_e4m3(x))


def test_encode_round_trips_every_finite_code():
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], np.uint8)
    vals = numerics.decode_e4m3(codes)
    assert np.array_equal(append.e4m3_encode(vals), codes)


def test_encode_ties_and_saturation_by_hand():
    cases = {
        1.0625: 0x38,           # midway 1.0 (0x38) / 1.125 (0x39): even mantissa -> 1.0
        1.1875: 0x3A,           # midway 1.125 (0x39) / 1.25 (0x3A) -> 1.25
        2.0 ** -10: 0x00,       # midway 0 / 2^-9 (smallest subnormal) -> 0
        3 * 2.0 ** -10: 0x02,   # midway 2^-9 (0x01) / 2^-8 (0x02) -> 0x02
        464.0: 0x7E,            # beyond the largest finite value: saturates to 448
        -1e30: 0xFE,
        -0.0: 0x80,
        -2.0 ** -11: 0x80,      # rounds to zero, keeps the sign
        0.5: 0x30,
    }
    for x, c in cases.items():
        assert int(append.e4m3_encode(np.array([x]))[0]) == c, (x, c)


def scalar_append(knew, vnew, kp, vp, bt, pos, fmt, ks, vs):
    kp, vp = kp.copy(), vp.copy()
    for s in range(knew.shape[0]):
        t = int(pos[s])
        if t < 0 or t >= bt.shape[1] * 16:
            continue
        b = int(bt[s, t // 16])
        if b < 0 or b >= kp.shape[0]:
            continue
        for g in range(knew.shape[1]):
            for d in range(knew.shape[2]):
                for src, dst, sc, is_v in ((knew, kp, ks, False), (vnew, vp, vs, True)):
                    bits = int(src[s, g, d])
                    if fmt == "bf16":
                        code = bits
                    else:
                        q = np.float32(numerics.bf16_value(bits)) / np.float32(sc[g])
                        code = int(append.e4m3_encode(np.array([float(q)]))[0])
                    if is_v:
                        dst[b, g, d, t % 16] = code
                    else:
                        dst[b, g, t % 16, d] = code
    return kp, vp


def test_append_equals_scalar_restatement():
    rng = np.random.default_rng(22)
    for fmt in ("bf16", "fp8_e4m3"):
        B, Hkv, nb = 5, 2, 12
        dt = np.uint16 if fmt == "bf16" else np.uint8
        kp = rng.integers(0, 1 << (16 if fmt == "bf16" else 8), (nb, Hkv, 16, 128)).astype(dt)
        vp = rng.integers(0, 1 << (16 if fmt == "bf16" else 8), (nb, Hkv, 128, 16)).astype(dt)
        knew = np.frombuffer(rng.standard_normal((B, Hkv, 128)).astype(np.float32).tobytes(), np.uint32)
        knew = (knew >> 16).astype(np.uint16).reshape(B, Hkv, 128)
        vnew = (np.frombuffer(rng.standard_normal((B, Hkv, 128)).astype(np.float32).tobytes(), np.uint32)
                >> 16).astype(np.uint16).reshape(B, Hkv, 128)
        bt = rng.permutation(nb)[:B * 2].reshape(B, 2).astype(np.int32)
        bt[3, 1] = -1
        pos = np.array([0, 15, 31, 17, -1], np.int32)           # seq 3 hits the -1 block; seq 4 skipped
        ks = np.array([0.01, 0.02], np.float32) if fmt != "bf16" else None
        vs = np.array([0.015, 0.005], np.float32) if fmt != "bf16" else None
        got = append.kv_cache_append(knew, vnew, kp, vp, bt, pos, fmt, ks, vs)
        ref = scalar_append(knew, vnew, kp, vp, bt, pos, fmt, ks, vs)
        assert np.array_equal(got[0], ref[0]) and np.array_equal(got[1], ref[1])
        assert np.array_equal(got[0][bt[4]], kp[bt[4]])          # untouched
