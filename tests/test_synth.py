"""The seeded generator: published Philox known answers, determinism, distributions."""
import numpy as np

import synth
from synth.workloads import WORKLOADS, SHAPE_8B, SHAPE_14B


def test_philox_known_answers():
    # Known-answer vectors of Philox-4x32-10 from the Random123 distribution (Salmon et al., SC'11).
    assert list(synth.philox4x32_10([0, 0, 0, 0], [0, 0])) == [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]
    assert list(synth.philox4x32_10([0xFFFFFFFF] * 4, [0xFFFFFFFF] * 2)) == [0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD]
    assert list(synth.philox4x32_10([0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344], [0xA4093822, 0x299F31D0])) == \
        [0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1]


def test_fnv1a():
    # FNV-1a 32-bit test values: "" -> offset basis, "a" -> 0xE40C292C.
    assert synth.stream_id("") == 0x811C9DC5
    assert synth.stream_id("a") == 0xE40C292C


def test_normals_moments_and_offsets():
    z = synth.normal_f64(7, "w", (400000,))
    assert abs(z.mean()) < 0.01 and abs(z.std() - 1.0) < 0.01
    b = synth.normal_bf16(7, "w", (1001,), 0.02)
    assert np.array_equal(synth.normal_bf16(7, "w", (13,), 0.02, offset=5), b[5:18])
    assert np.array_equal(synth.normal_bf16(7, "w", (1001,), 0.02), b)           # deterministic
    assert not np.array_equal(synth.normal_bf16(8, "w", (1001,), 0.02), b)       # seed matters
    assert not np.array_equal(synth.normal_bf16(7, "w2", (1001,), 0.02), b)      # stream matters
    # bf16 values are the float32 RNE of z*std, then bf16 RNE
    f = (b.astype(np.uint32) << 16).view(np.float32)
    ref = (z[:1001] * 0.02).astype(np.float32)
    assert np.max(np.abs(f - ref) / np.abs(ref)) <= 2.0 ** -8


def test_bf16_rounding_ties_to_even():
    assert synth.f32_to_bf16(1.0) == 0x3F80
    # 1 + 2^-8 is exactly halfway between bf16 1.0 and 1.0078125: ties to even (1.0)
    assert synth.f32_to_bf16(1.0 + 2.0 ** -8) == 0x3F80
    # 1 + 3*2^-8 is halfway between 1.0078125 (odd mantissa) and 1.015625: rounds up to even
    assert synth.f32_to_bf16(1.0 + 3 * 2.0 ** -8) == 0x3F82
    assert synth.f32_to_bf16(-2.0) == 0xC000


def test_uniform_int_range():
    u = synth.uniform_int(3, "lengths", (200000,), 512, 8192)
    assert u.min() == 512 and u.max() == 8192
    assert abs(u.mean() - (512 + 8192) / 2) < 30


def test_workload_weight_bytes():
    # algorithmic bf16 weight bytes streamed per pass for the 8B and 14B shapes
    assert SHAPE_8B.weight_bytes() == 15136194560
    assert SHAPE_14B.weight_bytes() == 27979939840
    r = WORKLOADS["8b_batch32"].prefix_lengths()
    assert len(r) == 32 and r.min() >= 512 and r.max() <= 8192


def test_gain_vectors():
    """RMSNorm gains bf16(1 + std z): float32 RNE to bf16 of the stream's normals, one stream per name,
    exact ones at std 0."""
    g = synth.gain_bf16(2, "layer3.ffn_norm", 4096, 0.1)
    z = synth.normal_f64(2, "layer3.ffn_norm", (4096,))
    ref = np.array([synth.f32_to_bf16(float(np.float32(1.0 + 0.1 * v))) for v in z[:512]], dtype=np.uint16)
    assert np.array_equal(g[:512], ref)
    f = (g.astype(np.uint32) << 16).view(np.float32)
    assert abs(f.mean() - 1.0) < 0.01 and abs(f.std() - 0.1) < 0.01
    assert not np.array_equal(g, synth.gain_bf16(2, "layer3.attn_norm", 4096, 0.1))
    assert np.array_equal(synth.gain_bf16(2, "x", 7, 0.0), synth.bf16_ones(7))
    # the array rounding agrees with the scalar one on ties and near-ties
    x = np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -2.0, 0.5 + 2.0 ** -10, 3.1415927], dtype=np.float32)
    assert synth.f32_array_to_bf16(x).tolist() == [synth.f32_to_bf16(float(v)) for v in x]
