"""Pins of the oracle's quantised profiling pass over a layer stack
(Section 4.1): lossless quantisation reduces it to the full-precision stack
(with torch's RMSNorm in front of each layer), a stack whose experts output
nothing keeps its input, and one layer is the int8 histogram of the normalised
input; the RMS normalisation itself against torch's."""
import numpy as np
import torch

import oracle as O


def torch_rms_norm(X, eps=1e-6):
    """torch's RMSNorm (unit weight) in float64."""
    x = torch.from_numpy(np.asarray(X, dtype=np.float64))
    return torch.nn.functional.rms_norm(x, (x.shape[-1],), eps=eps).numpy()


def test_rms_norm_rows_against_torch_and_invariants():
    rng = np.random.default_rng(3)
    X = rng.standard_normal((50, 24)) * rng.uniform(0.01, 100, size=(50, 1))
    Xn = O.rms_norm_rows(X)
    np.testing.assert_allclose(Xn, torch_rms_norm(X), rtol=1e-13, atol=0)
    # unit root mean square (up to eps), scale invariance, a zero row stays zero
    rms = np.sqrt(np.mean(Xn ** 2, axis=1))
    np.testing.assert_allclose(rms, np.sqrt(np.mean(X ** 2, axis=1) / (np.mean(X ** 2, axis=1) + 1e-6)), rtol=1e-13)
    np.testing.assert_allclose(O.rms_norm_rows(X * 1e3, eps=0.0), O.rms_norm_rows(X, eps=0.0), rtol=1e-13)
    Z = np.zeros((2, 8))
    assert np.array_equal(O.rms_norm_rows(Z), Z) and np.array_equal(O.rms_norm_rows(Z, eps=0.0), Z)
    np.testing.assert_allclose(O.rms_norm_rows(X, eps=0.5), torch_rms_norm(X, eps=0.5), rtol=1e-13)


def _representable(rng, shape, scale_exp=-6):
    """Rows of int8 codes times 2^scale_exp whose row maximum |code| is 127, so
    that per-row int8 quantisation returns exactly these codes and scale."""
    q = rng.integers(-127, 128, size=shape).astype(np.float64)
    rows = q.reshape(-1, shape[-1])
    rows[np.arange(len(rows)), rng.integers(0, shape[-1], size=len(rows))] = 127.0
    return rows.reshape(shape) * 2.0 ** scale_exp


def _stack(rng, L, E, d, I, representable, shared=0):
    layers = []
    for _ in range(L):
        mk = (lambda shape, exp: _representable(rng, shape, exp)) if representable else \
            (lambda shape, exp: rng.standard_normal(shape) * 2.0 ** (exp + 6) / np.sqrt(shape[-1]))
        lay = dict(Wr=mk((E, d), -6), bias=rng.standard_normal(E) * 0.3,
                   wg=mk((E, I, d), -9), wu=mk((E, I, d), -9), wd=mk((E, d, I), -9))
        if shared:
            lay.update(sg=mk((shared, I, d), -9), su=mk((shared, I, d), -9), sd=mk((shared, d, I), -9))
        layers.append(lay)
    return layers


def test_lossless_quantisation_is_the_full_precision_stack():
    rng = np.random.default_rng(0)
    T, d, E, k, I, L = 40, 16, 6, 2, 12, 3
    layers = _stack(rng, L, E, d, I, representable=True, shared=1)
    X0 = rng.standard_normal((T, d))
    counts, idxs, gates, Xs = O.quantized_stack_profile(X0, layers, k)
    X = X0.copy()
    for l, lay in enumerate(layers):
        Xn = torch_rms_norm(X)
        idx, gate, _ = O.route_topk(Xn, lay["Wr"], lay["bias"], k)
        assert np.array_equal(idx, idxs[l])
        np.testing.assert_allclose(gate, gates[l], rtol=1e-12, atol=1e-14)
        assert np.array_equal(np.bincount(idx.ravel(), minlength=E), counts[l])
        slots = O.SlotWeights(list(lay["wg"]) + list(lay["sg"]), list(lay["wu"]) + list(lay["su"]),
                              list(lay["wd"]) + list(lay["sd"]), [False] * (E + 1), n_shared=1)
        X = X + O.moe_forward(Xn, idx, gate, np.arange(E), slots)
        np.testing.assert_allclose(Xs[l + 1], X, rtol=1e-12, atol=1e-12)


def test_silent_experts_keep_the_stream_and_one_layer_is_the_histogram():
    rng = np.random.default_rng(1)
    T, d, E, k, I, L = 64, 16, 8, 3, 8, 3
    layers = _stack(rng, L, E, d, I, representable=False)
    for lay in layers:
        lay["wd"] = np.zeros_like(lay["wd"])
    X0 = rng.standard_normal((T, d))
    counts, idxs, gates, Xs = O.quantized_stack_profile(X0, layers, k)
    for l, lay in enumerate(layers):
        np.testing.assert_array_equal(Xs[l + 1], X0)
        q, s = O.quantize_int8_rows(lay["Wr"])
        c, idx, _ = O.profile_hist(torch_rms_norm(X0), q, s, lay["bias"], k)
        assert np.array_equal(c, counts[l]) and np.array_equal(idx, idxs[l])
        assert counts[l].sum() == T * k
        np.testing.assert_allclose(gates[l].sum(axis=1), 1.0, rtol=0, atol=1e-12)


def test_dequantised_experts_within_half_a_step():
    """The experts a layer runs differ from the stored ones by at most half a
    quantisation step per element, and the layer's update stays close to (but
    is not) the full-precision update on the same routing."""
    rng = np.random.default_rng(2)
    T, d, E, k, I = 32, 16, 4, 2, 8
    lay = _stack(rng, 1, E, d, I, representable=False)[0]
    X0 = rng.standard_normal((T, d))
    _, idxs, gates, Xs = O.quantized_stack_profile(X0, [lay], k)
    for name in ("wg", "wu", "wd"):
        W = lay[name]
        q, s = O.quantize_int8_rows(W.reshape(-1, W.shape[-1]))
        err = np.abs(O.dequantize_rows(q, s).reshape(W.shape) - W)
        assert np.all(err <= s.reshape(W.shape[:-1] + (1,)) / 2 * (1 + 1e-6))
    full = O.moe_forward(O.rms_norm_rows(X0), idxs[0], gates[0], np.arange(E),
                         O.SlotWeights(lay["wg"], lay["wu"], lay["wd"], [False] * E))
    rel = np.linalg.norm(Xs[1] - X0 - full) / np.linalg.norm(full)
    assert 0 < rel < 0.05
