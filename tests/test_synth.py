"""The seeded input generator: determinism, shapes and the stated structure."""
import numpy as np

import synth
from synth import bf16_bits_to_f64, to_bf16_bits


def test_bf16_round_to_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 3.0e-5], np.float64)
    b = to_bf16_bits(x)
    y = bf16_bits_to_f64(b)
    assert y[0] == 1.0
    assert y[1] == 1.0                       # tie -> even
    assert y[2] == 1.0 + 4 * 2 ** -8         # tie -> even (up)
    assert y[3] == -2.5
    assert abs(y[4] - 3.0e-5) <= 3.0e-5 * 2 ** -8


def test_tiny_workload_shapes_and_determinism():
    a = synth.workload_inputs("tiny")
    b = synth.workload_inputs("tiny")
    assert a.q.shape == (1024, 2, 64) and a.v.shape == (1024, 2, 64)
    assert a.g.shape == (1024, 2) and a.cu_seqlens.tolist() == [0, 1024]
    assert np.array_equal(a.q, b.q) and np.array_equal(a.g, b.g)
    k = bf16_bits_to_f64(a.k)
    np.testing.assert_allclose(np.linalg.norm(k, axis=-1), 1.0, atol=4e-3)
    assert np.all(a.g < 0) and np.all((a.beta > 0) & (a.beta < 1))
    assert a.n_frames() == 4


def test_novelty_structure_small():
    x = synth.workload_inputs("single_layer", T=4 * 256, frame_len=256, H_k=2, H_v=4)
    k = bf16_bits_to_f64(x.k)
    # frame 0 keys of a head lie in a 32-dim subspace
    s = np.linalg.svd(k[:256, 0], compute_uv=False)
    assert s[31] > 1e-2 and s[32] < 1e-2
    # frame 1 re-presents frame-0 keys plus small noise: every key has a close
    # neighbour in the previous frame
    sim = k[256:512, 0] @ k[:256, 0].T
    assert np.median(sim.max(axis=1)) > 0.8


def test_varlen_lengths_in_range():
    ls = synth.varlen_lengths(8, 16384, 131072)
    assert len(ls) == 8 and all(16384 <= x <= 131072 for x in ls)


def test_kv_rows_numpy_torch_agree():
    import torch
    pos = np.array([0, 1, 5, 1000, 2 ** 20 + 3])
    a = synth.kv_row_bits(2, 1, pos, 64)
    b = synth.kv_row_bits_torch(2, 1, torch.tensor(pos), 64).numpy().view(np.uint16)
    assert np.array_equal(a, b)
    f = bf16_bits_to_f64(a)
    assert np.all(np.isfinite(f)) and np.all(np.abs(f) < 2)
