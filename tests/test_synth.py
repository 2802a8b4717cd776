"""Synthetic input generators: determinism, torch == numpy bit-exactness, distribution sanity."""
import numpy as np
import torch

from synth import values as sv
from synth import traces as st


def test_torch_cpu_matches_numpy_reference():
    key = sv.mix_key(1234, 5, st.KIND_K, 0)
    for start, count in [(0, 1000), (123456789, 4097), (2**40 + 3, 513)]:
        t = sv.bf16_tensor(key, (count,), start=start)
        a = sv.bf16_bits(t)
        b = sv.bf16_bits_numpy(key, start, count)
        assert np.array_equal(a, b)


def test_scaled_heads_match_numpy():
    key = sv.mix_key(7, 1, st.KIND_V, 0)
    scales = np.array([0.5, 1.25, 2.0], dtype=np.float32)
    t = sv.bf16_tensor(key, (5, 3, 8), head_scale=scales)
    bits = sv.bf16_bits(t).reshape(5, 3, 8)
    for h in range(3):
        ref = sv.bf16_bits_numpy(key, 0, 5 * 3 * 8, scale=float(scales[h])).reshape(5, 3, 8)
        assert np.array_equal(bits[:, h], ref[:, h])


def test_slices_regenerate():
    key = sv.mix_key(99, 0, st.KIND_Q, 0)
    full = sv.bf16_bits(sv.bf16_tensor(key, (64, 4, 16)))
    part = sv.bf16_bits(sv.bf16_tensor(key, (3, 4, 16), start=10 * 4 * 16))
    assert np.array_equal(full.reshape(64, 4, 16)[10:13], part.reshape(3, 4, 16))


def test_chunked_generation_is_seamless():
    key = sv.mix_key(1, 2, 3)
    a = sv.bf16_bits(sv.bf16_tensor(key, (10000,), chunk=777))
    b = sv.bf16_bits(sv.bf16_tensor(key, (10000,)))
    assert np.array_equal(a, b)


def test_distribution_is_roughly_standard_normal():
    x = sv.bf16_to_f64(sv.bf16_tensor(sv.mix_key(5), (1 << 20,)))
    assert abs(x.mean()) < 5e-3
    assert abs(x.std() - 1.0) < 5e-3
    assert np.abs(x).max() <= 2 * np.sqrt(3) + 1e-2      # Irwin-Hall(4) support, +-2 sqrt(3)


def test_bf16_rounding_is_nearest_even():
    vals = torch.tensor([1.0, 1.00390625, 1.005859375, -3.14159, 123.456, 1e-3], dtype=torch.float32)
    bits = sv._f32_to_bf16_bits_t(vals).numpy().astype(np.uint16)
    ref = sv.bf16_bits(vals.to(torch.bfloat16))        # torch's own fp32 -> bf16 is RNE
    assert np.array_equal(bits, ref)


def test_trace_shapes():
    assert st.TinyTrace().final_len() == 256 + 16 + 2 * (32 + 16)
    L = st.DecodeBatch().lengths()
    assert L.shape == (64,) and L.min() >= 8192 and L.max() <= 32768
    p, n = st.ExtendBatch().lengths()
    assert p.min() >= 16384 and p.max() <= 65536 and n.min() >= 128 and n.max() <= 4096
    assert 600 < np.median(n) < 1700
    L4 = st.PrefillTransfer().lengths()
    assert L4.min() >= 32768 and L4.max() <= 131072
    convs = st.MixedTrace().conversations()
    assert len(convs) == 256
    assert all(5 <= c.turns <= 30 and 1024 <= c.turn1 <= 65536 for c in convs)
    assert all(len(c.appends) == c.turns - 1 for c in convs)
    # deterministic
    assert [c.turn1 for c in convs] == [c.turn1 for c in st.MixedTrace().conversations()]


def test_row_batched_generation_matches_streams():
    keys = [sv.mix_key(3, c, st.KIND_K, l) for c in range(3) for l in range(2)]
    starts = [17 * 64 * i for i in range(6)]
    rows = sv.bf16_rows(keys, starts, 64 * 5)
    for r, (k, s0) in enumerate(zip(keys, starts)):
        ref = sv.bf16_tensor(k, (5, 64), start=s0)
        assert torch.equal(rows[r].view(5, 64), ref)
