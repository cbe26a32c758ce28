"""Pins of the fp64 oracle's prefix + causal attention against facts that do not
come from the oracle itself: closed forms, invariances, and a library routine
(torch's float64 scaled_dot_product_attention on the CPU) for special cases.

The attention is the prefill form of the transition F (Eq. (1), Section 3.1)
over the replayed suffix; queries sit at absolute positions pos0 + i and see
keys 0 .. pos0 + i.
"""
import numpy as np
import pytest
import torch

import oracle
from workloads import workload, single_episode


def _rand(rng, *shape):
    return rng.standard_normal(shape)


def test_single_key_returns_its_value():
    # P = 0, S = 1: the only key gets weight 1, so o = v_0 exactly.
    rng = np.random.default_rng(10)
    q, k, v = _rand(rng, 1, 4, 16), _rand(rng, 1, 2, 16), _rand(rng, 1, 2, 16)
    o = oracle.attention(q, k, v, pos0=0, scale=0.25)
    np.testing.assert_array_equal(o[0, :2], np.repeat(v[0, :1], 2, axis=0))
    np.testing.assert_array_equal(o[0, 2:], np.repeat(v[0, 1:], 2, axis=0))


def test_constant_values_give_that_constant():
    rng = np.random.default_rng(11)
    n, P = 9, 5
    q, k = _rand(rng, n, 4, 8), _rand(rng, P + n, 4, 8)
    c = _rand(rng, 4, 8)
    v = np.broadcast_to(c, (P + n, 4, 8)).copy()
    o = oracle.attention(q, k, v, pos0=P, scale=0.3)
    np.testing.assert_allclose(o, np.broadcast_to(c, o.shape), rtol=0, atol=1e-14)


def test_equal_keys_give_the_causal_prefix_mean():
    # All logits of a row are equal, so the weights are uniform over keys 0..p.
    rng = np.random.default_rng(12)
    n, P, hq, hkv, d = 7, 6, 4, 2, 8
    q = _rand(rng, n, hq, d)
    k = np.broadcast_to(_rand(rng, 1, hkv, d), (P + n, hkv, d)).copy()
    v = _rand(rng, P + n, hkv, d)
    o = oracle.attention(q, k, v, pos0=P, scale=0.5)
    for i in range(n):
        for h in range(hq):
            want = v[: P + i + 1, h // (hq // hkv)].mean(axis=0)
            np.testing.assert_allclose(o[i, h], want, rtol=0, atol=1e-13)


def test_dominant_logit_selects_its_value():
    rng = np.random.default_rng(13)
    n, P, d = 3, 10, 16
    q = np.zeros((n, 1, d))
    q[:, 0, 0] = 1.0
    k = _rand(rng, P + n, 1, d) * 0.01
    star = 4
    k[star, 0, 0] = 100.0          # logit at least ~99 above every other key
    v = _rand(rng, P + n, 1, d)
    o = oracle.attention(q, k, v, pos0=P, scale=1.0)
    for i in range(n):
        np.testing.assert_allclose(o[i, 0], v[star, 0], rtol=0, atol=1e-30)


def test_gqa_mapping_against_torch_enable_gqa():
    # torch's GQA groups contiguous query heads: head h reads KV head h // G.
    rng = np.random.default_rng(14)
    T, hq, hkv, d = 24, 8, 2, 16
    q, k, v = _rand(rng, T, hq, d), _rand(rng, T, hkv, d), _rand(rng, T, hkv, d)
    o = oracle.attention(q, k, v, pos0=0, scale=d ** -0.5)
    tq, tk, tv = (torch.from_numpy(a).permute(1, 0, 2).unsqueeze(0) for a in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True, enable_gqa=True)
    np.testing.assert_allclose(o, ref[0].permute(1, 0, 2).numpy(), rtol=0, atol=1e-13)


def test_gqa_equals_mha_on_replicated_kv():
    rng = np.random.default_rng(15)
    n, P, hq, hkv, d = 5, 7, 6, 3, 8
    q, k, v = _rand(rng, n, hq, d), _rand(rng, P + n, hkv, d), _rand(rng, P + n, hkv, d)
    G = hq // hkv
    o_gqa = oracle.attention(q, k, v, P, 0.4)
    o_mha = oracle.attention(q, np.repeat(k, G, axis=1), np.repeat(v, G, axis=1), P, 0.4)
    np.testing.assert_array_equal(o_gqa, o_mha)


@pytest.mark.parametrize("P,S", [(0, 17), (13, 5), (32, 1)])
def test_prefix_mask_matches_torch_sdpa(P, S):
    rng = np.random.default_rng(100 + P)
    hq, hkv, d = 4, 4, 16
    q, k, v = _rand(rng, S, hq, d), _rand(rng, P + S, hkv, d), _rand(rng, P + S, hkv, d)
    scale = 0.21
    o = oracle.attention(q, k, v, pos0=P, scale=scale)
    mask = torch.arange(P + S)[None, :] <= (P + torch.arange(S))[:, None]
    tq, tk, tv = (torch.from_numpy(a).permute(1, 0, 2).unsqueeze(0) for a in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask, scale=scale)
    np.testing.assert_allclose(o, ref[0].permute(1, 0, 2).numpy(), rtol=0, atol=1e-13)


def test_tiny_workload_matches_torch_sdpa():
    """The tiny fp32 episode at its real shape: P = 512, S = 128, 8 heads, d = 64."""
    w = workload("tiny_mha8_d64_p512_s128_f32")
    ep = single_episode(w)
    q = ep.q[ep.prefix:].astype(np.float64)
    k, v = ep.k.astype(np.float64), ep.v.astype(np.float64)
    o = oracle.attention(q, k, v, pos0=ep.prefix, scale=w.scale)
    T, S = ep.t_sanitized, ep.suffix
    mask = torch.arange(T)[None, :] <= (ep.prefix + torch.arange(S))[:, None]
    tq, tk, tv = (torch.from_numpy(a).permute(1, 0, 2).unsqueeze(0) for a in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask, scale=w.scale)
    np.testing.assert_allclose(o, ref[0].permute(1, 0, 2).numpy(), rtol=0, atol=1e-12)


def test_row_subset_equals_full_rows():
    rng = np.random.default_rng(16)
    n, P, hq, hkv, d = 6, 4, 4, 2, 8
    q, k, v = _rand(rng, n, hq, d), _rand(rng, P + n, hkv, d), _rand(rng, P + n, hkv, d)
    full = oracle.attention(q, k, v, P, 0.3)
    rows = np.array([0, 5, 23, 9, 17])
    sub = oracle.attention(q, k, v, P, 0.3, rows=rows)
    np.testing.assert_array_equal(sub, full.reshape(n * hq, d)[rows])


def test_key_shift_invariance():
    # Adding one vector u to every key shifts all logits of a row by q.u:
    # softmax is unchanged.
    rng = np.random.default_rng(17)
    n, P, d = 5, 9, 8
    q, k, v = _rand(rng, n, 2, d), _rand(rng, P + n, 1, d), _rand(rng, P + n, 1, d)
    u = _rand(rng, 1, 1, d) * 3
    a = oracle.attention(q, k, v, P, 0.5)
    b = oracle.attention(q, k + u, v, P, 0.5)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_last_row_is_invariant_to_key_order():
    # The last query sees every key; permuting (key, value) pairs jointly keeps it.
    rng = np.random.default_rng(18)
    n, P, d = 4, 11, 8
    q, k, v = _rand(rng, n, 2, d), _rand(rng, P + n, 2, d), _rand(rng, P + n, 2, d)
    perm = rng.permutation(P + n)
    a = oracle.attention(q, k, v, P, 0.5)[-1]
    b = oracle.attention(q, k[perm], v[perm], P, 0.5)[-1]
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-13)


def test_causality_future_keys_do_not_matter():
    # Changing key/value p+1 .. leaves row p unchanged (inclusive causal mask).
    rng = np.random.default_rng(19)
    n, P, d = 6, 3, 8
    q, k, v = _rand(rng, n, 1, d), _rand(rng, P + n, 1, d), _rand(rng, P + n, 1, d)
    a = oracle.attention(q, k, v, P, 0.5)
    k2, v2 = k.copy(), v.copy()
    k2[P + 3:] += 5.0
    v2[P + 3:] -= 7.0
    b = oracle.attention(q, k2, v2, P, 0.5)
    np.testing.assert_array_equal(a[:3], b[:3])
    assert np.abs(a[3:] - b[3:]).max() > 0.1


def test_rejects_bad_shapes():
    q = np.zeros((4, 2, 8)); k = np.zeros((3, 2, 8))
    with pytest.raises(ValueError):
        oracle.attention(q, k, k, pos0=0, scale=1.0)   # pos0 + n_q > n_kv
    with pytest.raises(ValueError):
        oracle.attention(np.zeros((1, 3, 8)), np.zeros((1, 2, 8)), np.zeros((1, 2, 8)), 0, 1.0)
