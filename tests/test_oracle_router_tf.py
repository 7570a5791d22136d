"""Pins of the router oracle (oracle/router_tf.py): RoPE against its closed
form and the algebra of rotations, causal attention against a pure-Python
brute force and its special cases, and the whole router's independence of
requests.  CPU only."""
import math

import numpy as np
import pytest

from oracle import router_tf as R


def test_rope_is_identity_at_position_zero():
    x = np.random.default_rng(0).standard_normal((3, 256))
    assert np.array_equal(R.rope_f64(x, np.zeros(3, np.int64)), x)


def test_rope_closed_form():
    """Pair (i, i + 64) of a head turns by p * 10000^(-2i/128)."""
    x = np.zeros((2, 128))
    x[0, 0] = 1.0                 # pair 0 at position 1: angle 1 rad
    x[1, 5] = 2.0                 # pair 5 at position 3
    x[1, 5 + 64] = -1.0
    out = R.rope_f64(x, np.array([1, 3]))
    assert out[0, 0] == pytest.approx(math.cos(1.0), abs=1e-15)
    assert out[0, 64] == pytest.approx(math.sin(1.0), abs=1e-15)
    th = 3 * 10000.0 ** (-2 * 5 / 128)
    assert out[1, 5] == pytest.approx(2 * math.cos(th) + math.sin(th), abs=1e-14)
    assert out[1, 5 + 64] == pytest.approx(-math.cos(th) + 2 * math.sin(th), abs=1e-14)
    others = np.ones(128, bool)
    others[[5, 69]] = False
    assert np.all(out[1, others] == 0)


def test_rope_rotations_compose_and_keep_norms():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((4, 256))
    p1, p2 = np.array([0, 5, 17, 300]), np.array([3, 0, 40, 7])
    both = R.rope_f64(R.rope_f64(x, p1), p2)
    assert np.allclose(both, R.rope_f64(x, p1 + p2), atol=1e-12)
    y = R.rope_f64(x, p1)
    for h in range(2):
        a, b = x[:, h * 128:h * 128 + 64], x[:, h * 128 + 64:(h + 1) * 128]
        c, d = y[:, h * 128:h * 128 + 64], y[:, h * 128 + 64:(h + 1) * 128]
        assert np.allclose(a * a + b * b, c * c + d * d, atol=1e-12)
    # the inverse rotation (negative positions) restores the input
    assert np.allclose(R.rope_f64(y, -p1), x, atol=1e-12)


def _attention_brute(q, k, v, ro):
    T, HD = len(q), len(q[0])
    out = [[0.0] * HD for _ in range(T)]
    for r in range(len(ro) - 1):
        for t in range(ro[r], ro[r + 1]):
            for h in range(HD // 128):
                base = h * 128
                scores = []
                for j in range(ro[r], t + 1):
                    s = sum(q[t][base + i] * k[j][base + i] for i in range(128))
                    scores.append(s / math.sqrt(128))
                m = max(scores)
                w = [math.exp(s - m) for s in scores]
                z = sum(w)
                for i in range(128):
                    out[t][base + i] = sum(w[n] * v[ro[r] + n][base + i]
                                           for n in range(len(w))) / z
    return np.array(out)


def test_attention_equals_brute_force():
    rng = np.random.default_rng(2)
    ro = np.array([0, 3, 3, 7])              # an empty request in the middle
    q, k, v = (rng.standard_normal((7, 256)) for _ in range(3))
    got = R.attention_f64(q, k, v, ro)
    assert np.allclose(got, _attention_brute(q.tolist(), k.tolist(), v.tolist(), ro),
                       atol=1e-12)


def test_attention_special_cases():
    rng = np.random.default_rng(3)
    ro = np.array([0, 4, 9])
    q, k, v = (rng.standard_normal((9, 128)) for _ in range(3))
    out = R.attention_f64(q, k, v, ro)
    # a request's first token sees only itself
    assert np.array_equal(out[0], v[0]) and np.array_equal(out[4], v[4])
    # equal keys: uniform weights, the mean of the prefix's values
    k2 = np.tile(k[:1], (9, 1))
    out2 = R.attention_f64(q, k2, v, ro)
    assert np.allclose(out2[6], v[4:7].mean(axis=0), atol=1e-12)
    # causality: later tokens do not change earlier outputs
    v3 = v.copy()
    v3[8] += 100.0
    assert np.array_equal(R.attention_f64(q, k, v3, ro)[:8], out[:8])


def _weights(rng, V=50, D=256, F=128, E=5):
    def b(*shape, std):
        return R.bf16(rng.standard_normal(shape) * std)
    return dict(emb=b(V, D, std=1.0), wq=b(D, D, std=0.05), wk=b(D, D, std=0.05),
                wv=b(D, D, std=0.05), wo=b(D, D, std=0.05), w1=b(F, D, std=0.05),
                w3=b(F, D, std=0.05), w2=b(D, F, std=0.05), w_router=b(E, D, std=0.05),
                bias=rng.standard_normal(E).astype(np.float32))


def _run(w, tokens, ro):
    return R.router_tf(tokens, ro, w["emb"], w["wq"], w["wk"], w["wv"], w["wo"], w["w1"],
                       w["w3"], w["w2"], w["w_router"], w["bias"])


def test_router_requests_are_independent(oracle_mod):
    rng = np.random.default_rng(4)
    w = _weights(rng)
    t1, t2 = rng.integers(0, 50, 6), rng.integers(0, 50, 4)
    both = _run(w, np.concatenate([t1, t2]), np.array([0, 6, 10]))
    a = _run(w, t1, np.array([0, 6]))
    b = _run(w, t2, np.array([0, 4]))
    assert np.array_equal(both["ids"], np.concatenate([a["ids"], b["ids"]]))
    assert np.array_equal(both["logits"], np.concatenate([a["logits"], b["logits"]]))
    assert np.array_equal(both["x2"], np.concatenate([a["x2"], b["x2"]]))


def test_router_single_token_request_attends_to_itself(oracle_mod):
    """A one-token request: the attention output is its own value row."""
    rng = np.random.default_rng(5)
    w = _weights(rng)
    out = _run(w, np.array([7, 3, 9]), np.array([0, 1, 3]))
    assert np.array_equal(out["o"][0], out["v"][0])
    assert np.array_equal(out["pos"], [0, 0, 1])
    # and the token's position 0 leaves q, k unrotated
    af = R._f(out["a"][:1])
    assert np.array_equal(out["q"][0], R.bf16(af @ R._f(w["wq"]).T)[0])


def test_embedding_of_out_of_range_ids_is_zero():
    emb = R.bf16(np.random.default_rng(6).standard_normal((10, 256)))
    x = R.embed(np.array([0, -1, 10, 9]), emb)
    assert np.all(x[1] == 0) and np.all(x[2] == 0)
    assert np.array_equal(x[3], R._f(emb[9]).astype(np.float32))


def test_mlp_hidden_agrees_with_the_layer_oracle(oracle_mod):
    """W2 mlp_hidden(m) is the C oracle's FFN layer output on the same
    residual rows (one expert covering every row)."""
    rng = np.random.default_rng(7)
    D, F, T = 128, 96, 5
    x = rng.standard_normal((T, D)).astype(np.float32)
    w1, w3 = (R.bf16(rng.standard_normal((F, D)) * 0.05) for _ in range(2))
    w2 = R.bf16(rng.standard_normal((D, F)) * 0.05)
    m = R.rmsnorm_bf16(x)
    ours = R.mlp_hidden(m, w1, w3) @ R._f(w2).T
    ref, xn = oracle_mod.layer(x, np.array([0, T], np.int32), w1[None], w3[None], w2[None],
                               want_xn=True)
    assert np.array_equal(xn, m)
    assert np.allclose(ours, ref, rtol=1e-12, atol=1e-12)


def test_router_with_zero_output_projections_is_the_gate_of_the_embedding(oracle_mod):
    """Wo = 0 and W2 = 0: both residual branches add exact zeros, so the
    block's output is the embedding itself and the logits are the gate of
    its norm."""
    rng = np.random.default_rng(8)
    w = _weights(rng)
    w["wo"] = np.zeros_like(w["wo"])
    w["w2"] = np.zeros_like(w["w2"])
    tokens = rng.integers(0, 50, 9)
    out = _run(w, tokens, np.array([0, 4, 9]))
    x0 = R.embed(tokens, w["emb"])
    assert np.array_equal(out["x1"], x0) and np.array_equal(out["x2"], x0)
    ids, logits = oracle_mod.route(R.rmsnorm_bf16(x0), w["w_router"], w["bias"])
    assert np.array_equal(out["ids"], ids) and np.array_equal(out["logits"], logits)


def test_router_with_zero_queries_averages_the_prefix(oracle_mod):
    """Wq = 0: every score is 0, so each token's attention output is the
    plain mean of its request's value rows up to itself."""
    rng = np.random.default_rng(9)
    w = _weights(rng)
    w["wq"] = np.zeros_like(w["wq"])
    tokens = rng.integers(0, 50, 11)
    ro = np.array([0, 5, 5, 11])
    out = _run(w, tokens, ro)
    v = R._f(out["v"])
    mean = np.empty_like(v)
    for r in range(len(ro) - 1):
        a, b = ro[r], ro[r + 1]
        mean[a:b] = np.cumsum(v[a:b], axis=0) / np.arange(1, b - a + 1)[:, None]
    assert np.allclose(R._f(out["o"]), mean, rtol=2.0 ** -8, atol=1e-30)


def test_router_mlp_reads_the_attention_residual(oracle_mod):
    """The MLP branch is the layer oracle applied to x1 (the residual after
    attention), not to the embedding."""
    rng = np.random.default_rng(10)
    w = _weights(rng)
    tokens = rng.integers(0, 50, 7)
    out = _run(w, tokens, np.array([0, 7]))
    x1 = out["x1"]
    assert not np.array_equal(x1, R.embed(tokens, w["emb"]))
    delta = oracle_mod.layer(x1, np.array([0, 7], np.int32), w["w1"][None], w["w3"][None],
                             w["w2"][None])
    assert np.array_equal(out["x2"], (x1.astype(np.float64) + delta).astype(np.float32))
