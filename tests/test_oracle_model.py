"""Pins of the oracle's transformer step (sparse input of Section 3.2 over a
LLaDA/Dream-style bidirectional decoder) and of its output statistics."""
import math

import numpy as np
import pytest

from oracle import model as M
from oracle import selection as S
from oracle.generate import NumpyWeights
from synthetic import TINY, make_weights
import dataclasses

rng = np.random.default_rng(7)


def brute_attention(q, k, v):
    """Triple loop, scalar float64 arithmetic, explicit GQA head map."""
    n_q, H, dh = q.shape
    n_k, Hkv, _ = k.shape
    out = np.zeros((n_q, H * dh))
    for i in range(n_q):
        for h in range(H):
            g = h * Hkv // H
            s = []
            for j in range(n_k):
                acc = 0.0
                for c in range(dh):
                    acc += float(q[i, h, c]) * float(k[j, g, c])
                s.append(acc / math.sqrt(dh))
            m = max(s)
            e = [math.exp(x - m) for x in s]
            z = sum(e)
            for c in range(dh):
                out[i, h * dh + c] = sum(e[j] / z * float(v[j, g, c]) for j in range(n_k))
    return out


@pytest.mark.parametrize("H,Hkv", [(2, 2), (4, 2), (4, 1)])
def test_attention_matches_brute_force(H, Hkv):
    q = rng.normal(size=(5, H, 4))
    k = rng.normal(size=(7, Hkv, 4))
    v = rng.normal(size=(7, Hkv, 4))
    assert np.max(np.abs(M.attention(q, k, v) - brute_attention(q, k, v))) < 1e-12


def test_attention_special_cases():
    q = rng.normal(size=(3, 2, 4))
    # one key: output is that key's value
    k1 = rng.normal(size=(1, 2, 4))
    v1 = rng.normal(size=(1, 2, 4))
    assert np.allclose(M.attention(q, k1, v1), np.broadcast_to(v1.reshape(1, 8), (3, 8)))
    # identical values: output is that value whatever the scores
    k = rng.normal(size=(6, 2, 4))
    v = np.broadcast_to(rng.normal(size=(1, 2, 4)), (6, 2, 4))
    assert np.allclose(M.attention(q, k, v), np.broadcast_to(v[0].reshape(1, 8), (3, 8)))
    # zero queries: uniform average of the values (no causal mask)
    out = M.attention(np.zeros((2, 2, 4)), k, rng.normal(size=(6, 2, 4)) * 0 + np.arange(6)[:, None, None])
    assert np.allclose(out, 2.5)


def test_rms_norm():
    x = rng.normal(size=(4, 64)) * 3
    y = M.rms_norm(x, np.ones(64), 0.0)
    assert np.allclose(np.sqrt(np.mean(y * y, axis=-1)), 1.0, atol=1e-12)
    assert np.allclose(M.rms_norm(5 * x, np.ones(64), 0.0), y, atol=1e-12)
    g = rng.normal(size=64)
    assert np.allclose(M.rms_norm(x, g, 0.0), y * g, atol=1e-12)
    # eps enters under the root: a zero row stays zero, a tiny row is damped
    assert np.all(M.rms_norm(np.zeros((1, 64)), np.ones(64), 1e-5) == 0)


def test_rope_complex_form():
    """Rotate-half RoPE == multiplying z_i = x_i + i x_{i+d/2} by exp(i p theta_i)."""
    dh, base = 16, 10000.0
    x = rng.normal(size=(6, 3, dh))
    pos = np.array([0, 1, 5, 17, 300, 4095])
    y = M.apply_rope(x, pos, base)
    half = dh // 2
    theta = base ** (-np.arange(half) * 2.0 / dh)
    z = x[..., :half] + 1j * x[..., half:]
    zr = z * np.exp(1j * pos[:, None, None] * theta[None, None, :])
    assert np.allclose(y[..., :half], zr.real, atol=1e-12)
    assert np.allclose(y[..., half:], zr.imag, atol=1e-12)
    assert np.array_equal(M.apply_rope(x[:1], np.array([0]), base), x[:1])


def test_rope_relative_shift_invariance():
    dh = 32
    q = rng.normal(size=(1, 1, dh))
    k = rng.normal(size=(1, 1, dh))
    dots = []
    for c in (0, 11, 1000):
        qa = M.apply_rope(q, np.array([40 + c]), 10000.0)
        ka = M.apply_rope(k, np.array([3 + c]), 10000.0)
        dots.append(float(np.sum(qa * ka)))
    assert np.allclose(dots, dots[0], atol=1e-10)


def _tiny(norm_jitter=0.1):
    shape = dataclasses.replace(TINY, n_layers=2)
    return shape, NumpyWeights(make_weights(shape, seed=3, norm_jitter=norm_jitter))


def test_layer_special_cases():
    shape, w = _tiny()
    lw = w.layers[0]
    x = rng.normal(size=(9, shape.d_model))
    pos = np.arange(9)
    # with W_o and W_down zero the layer is the identity
    class Z:  # noqa: E306
        pass
    z = Z()
    for name in ("attn_norm", "wq", "wk", "wv", "ffn_norm", "w_gate", "w_up"):
        setattr(z, name, getattr(lw, name))
    z.wo = np.zeros_like(lw.wo)
    z.w_down = np.zeros_like(lw.w_down)
    assert np.array_equal(M.layer_forward(x, pos, z, shape).x, x)
    # with W_v zero only the FFN acts (test_ffn_against_scalar_loops writes it out)


def test_permutation_invariance_with_positions_fixed():
    shape, w = _tiny()
    n = 23
    x = rng.normal(size=(n, shape.d_model)) * 0.05
    pos = np.sort(rng.choice(200, size=n, replace=False))
    ref = M.forward(x, pos, w, shape).hidden
    perm = rng.permutation(n)
    out = M.forward(x[perm], pos[perm], w, shape).hidden
    assert np.max(np.abs(out - ref[perm])) < 1e-12


def test_prefix_cache_equals_uncached():
    """Reusing the prefix keys/values of a full pass gives the full pass's rows."""
    shape, w = _tiny()
    n, P = 30, 12
    x = rng.normal(size=(n, shape.d_model)) * 0.05
    pos = np.arange(n) + 3
    full = M.forward(x, pos, w, shape)
    prefix_kv = [(k[:P], v[:P]) for (k, v) in full.kv]
    cached = M.forward(x[P:], pos[P:], w, shape, prefix_kv)
    assert np.max(np.abs(cached.hidden - full.hidden[P:])) < 1e-12


def test_output_stats_brute_force():
    shape, w = _tiny()
    h = rng.normal(size=(6, shape.d_model))
    st = M.output_stats(h, w, shape, k=5)
    hn = M.rms_norm(h, w.final_norm, shape.rms_eps)
    for r in range(6):
        logits = [float(np.dot(hn[r], w.lm_head[v])) for v in range(shape.vocab)]
        cand = sorted((-logits[v], v) for v in range(shape.vocab) if v != shape.mask_id)
        z = sum(math.exp(logits[v] - (-cand[0][0])) for v in range(shape.vocab) if v != shape.mask_id)
        assert st.argmax[r] == cand[0][1]
        assert abs(st.conf[r] - 1.0 / z) < 1e-12
        assert list(st.topk_ids[r]) == [v for _, v in cand[:5]]
        assert abs(st.p_sorted2[r, 1] - math.exp(-cand[1][0] + cand[0][0]) / z) < 1e-12


def _silu_scalar(v: float) -> float:
    """x * logistic(x), with the logistic written through math.exp."""
    return v / (1.0 + math.exp(-v))


def test_silu_values_and_limits():
    """SiLU (the gate of the SwiGLU FFN of the LLaDA/Dream decoder): known
    values, the identity silu(x) - silu(-x) = x (logistic(x) + logistic(-x)
    = 1), the slope 1/2 at 0, and its limits."""
    assert M.silu(np.array(0.0)) == 0.0
    assert abs(float(M.silu(np.array(1.0))) - 0.7310585786300049) < 1e-15
    assert abs(float(M.silu(np.array(-1.0))) + 0.2689414213699951) < 1e-15
    xs = np.linspace(-12.0, 12.0, 97)
    got = M.silu(xs)
    assert np.max(np.abs(got - np.array([_silu_scalar(float(v)) for v in xs]))) < 1e-14
    assert np.max(np.abs((got - M.silu(-xs)) - xs)) < 1e-13
    h = 1e-6
    assert abs((float(M.silu(np.array(h))) - float(M.silu(np.array(-h)))) / (2 * h) - 0.5) < 1e-9
    assert abs(float(M.silu(np.array(40.0))) - 40.0) < 1e-12          # -> x as x -> +inf
    assert 0.0 > float(M.silu(np.array(-40.0))) > -1e-15               # -> 0- as x -> -inf
    with np.errstate(over="ignore"):                                  # exp(745) = inf
        assert float(M.silu(np.array(-745.0))) == 0.0


def test_ffn_against_scalar_loops():
    """The feed-forward half of a layer, written out with scalar loops: RMSNorm,
    gate and up projections, silu(gate) * up, down projection, residual add.
    With W_v = 0 the attention branch adds nothing, so the layer output is
    x + FFN(x)."""
    shape, w = _tiny()
    lw = w.layers[1]

    class Z:  # noqa: E306
        pass
    z = Z()
    for name in ("attn_norm", "wq", "wk", "wo", "ffn_norm", "w_gate", "w_up", "w_down"):
        setattr(z, name, getattr(lw, name))
    z.wv = np.zeros_like(lw.wv)
    x = rng.normal(size=(2, shape.d_model))
    got = M.layer_forward(x, np.array([3, 40]), z, shape).x
    d, F = shape.d_model, shape.ffn_dim
    for r in range(2):
        xr = [float(v) for v in x[r]]
        inv = 1.0 / math.sqrt(sum(v * v for v in xr) / d + shape.rms_eps)
        hn = [xr[c] * inv * float(lw.ffn_norm[c]) for c in range(d)]
        act = []
        for j in range(F):
            g = sum(hn[c] * float(lw.w_gate[j, c]) for c in range(d))
            u = sum(hn[c] * float(lw.w_up[j, c]) for c in range(d))
            act.append(_silu_scalar(g) * u)
        for c in range(d):
            want = xr[c] + sum(act[j] * float(lw.w_down[c, j]) for j in range(F))
            assert abs(float(got[r, c]) - want) < 1e-12
