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
    # with W_v zero only the FFN acts, and it sees x itself
    z.wv = np.zeros_like(lw.wv)
    z.wo, z.w_down = lw.wo, lw.w_down
    hn = M.rms_norm(x, lw.ffn_norm, shape.rms_eps)
    f = M.silu(hn @ lw.w_gate.T) * (hn @ lw.w_up.T)
    assert np.allclose(M.layer_forward(x, pos, z, shape).x, x + f @ lw.w_down.T, atol=1e-12)


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
