"""Host checks of the seeded input generators (no method arithmetic here)."""
import numpy as np

from paper_2508_19078_amd import workloads as W


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.00390625, 1.01171875, -2.5, 3.0e-3], dtype=np.float32)
    # 1+2^-8 is halfway between 1 and 1+2^-7 -> even (1.0); 1+3*2^-8 -> 1+2^-6
    np.testing.assert_array_equal(W.bf16_bits_to_f32(W.round_to_bf16_bits(x))[:3],
                                  np.array([1.0, 1.0, 1.015625], dtype=np.float32))
    y = W.bf16_bits_to_f32(W.round_to_bf16_bits(x))
    assert np.all(np.abs(y - x) <= np.abs(x) * 2.0 ** -8)


def test_draws_are_deterministic_and_scaled():
    w = W.WORKLOADS["deepseek_moe"]
    a = W.draw([3, 0, W.TID_WR], (64, 2048), 1 / np.sqrt(2048), "bf16")
    b = W.draw([3, 0, W.TID_WR], (64, 2048), 1 / np.sqrt(2048), "bf16")
    np.testing.assert_array_equal(a.store, b.store)
    assert abs(a.f64().std() * np.sqrt(2048) - 1) < 0.01
    assert np.all(W.draw_router(w).f64() == a.f64())


def test_linear_merge_schedule_and_biases():
    m = [W.merge_count_linear(l) for l in range(28)]
    assert m[0] == 0 and m[27] == 48 and sum(m) // 4 == 168
    assert all(b >= a for a, b in zip(m, m[1:]))
    z = W.router_bias(W.WORKLOADS["stress"])
    assert sorted(np.round(np.exp(-z / 1.2)).astype(int)) == list(range(1, 65))
    nb = W.router_bias(W.WORKLOADS["llama_moe"])
    assert nb.shape == (16,) and nb.std() > 0.5
    assert W.layer_merge_spec(W.WORKLOADS["deepseek_stack"], 0) == ("frequency", 0, 4)
    assert W.layer_merge_spec(W.WORKLOADS["deepseek_stack"], 27) == ("frequency", 48, 4)
