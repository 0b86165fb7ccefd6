"""Pins for the oracle's building blocks: BCE (Eq. 1), the per-row clip and
its backward, embedding lookup and its gradient, and the storage rounding of
the emulation modes."""
import numpy as np
import pytest
import torch
from scipy import special

from oracle import layers as L
from oracle.rounding import round_bf16, round_f32


# ------------------------------------------------------------------ BCE
def test_bce_special_values():
    y = np.array([0.0, 1.0])
    np.testing.assert_allclose(L.bce_with_logits(np.zeros(2), y), np.log(2.0), rtol=0, atol=1e-16)
    np.testing.assert_allclose(L.bce_dlogit(np.zeros(2), y), 0.5 - y, atol=0)
    big = L.bce_with_logits(np.array([100.0, -100.0, 100.0, -100.0]),
                            np.array([0.0, 1.0, 1.0, 0.0]))
    assert np.all(np.isfinite(big))
    np.testing.assert_allclose(big[:2], 100.0, rtol=1e-15)
    assert np.all(big[2:] < 1e-40)


def test_bce_symmetry_and_eq1():
    rng = np.random.default_rng(0)
    l = rng.normal(0, 4, 1000)
    y = (rng.random(1000) < 0.5).astype(np.float64)
    np.testing.assert_allclose(L.bce_with_logits(l, y), L.bce_with_logits(-l, 1 - y), rtol=1e-14)
    # Eq. (1) written directly on yhat = sigmoid(l), for moderate logits
    np.testing.assert_allclose(L.bce_with_logits(l, y), L.bce_direct(special.expit(l), y),
                               rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(L.sigmoid(l), special.expit(l), rtol=1e-15)
    # derivative: central differences of the per-row loss
    h = 1e-6
    fd = (L.bce_with_logits(l + h, y) - L.bce_with_logits(l - h, y)) / (2 * h)
    np.testing.assert_allclose(L.bce_dlogit(l, y), fd, atol=1e-8)


# ------------------------------------------------------------------ clip
def test_clip_invariants():
    rng = np.random.default_rng(1)
    v = rng.normal(0, 1, (500, 7)) * rng.uniform(0.01, 3, (500, 1))
    v[0] = 0.0
    C = 1.0
    out, n, c = L.clip_rows(v, C)
    assert np.all(np.linalg.norm(out, axis=1) <= C * (1 + 1e-12))
    small = n <= C
    assert np.array_equal(out[small], v[small])           # unchanged bitwise
    np.testing.assert_allclose(np.linalg.norm(out[~small], axis=1), C, rtol=1e-14)
    same, _, _ = L.clip_rows(v, np.inf)
    assert np.array_equal(same, v)


def test_clip_backward_is_jacobian_transpose():
    rng = np.random.default_rng(2)
    C = 1.0
    v = rng.normal(0, 1, (40, 5)) * rng.uniform(0.05, 2.0, (40, 1))
    g = rng.normal(0, 1, (40, 5))
    _, n, c = L.clip_rows(v, C)
    got = L.clip_rows_backward(g, v, n, c, C)
    h = 1e-6
    fd = np.zeros_like(v)
    for j in range(5):
        e = np.zeros(5)
        e[j] = h
        fp = L.clip_rows(v + e, C)[0]
        fm = L.clip_rows(v - e, C)[0]
        fd[:, j] = np.sum(g * (fp - fm), axis=1) / (2 * h)
    keep = np.abs(n - C) > 1e-4       # away from the clip boundary
    np.testing.assert_allclose(got[keep], fd[keep], rtol=1e-6, atol=1e-8)


# ------------------------------------------------------------ embeddings
def test_embedding_lookup_and_grad_equal_one_hot():
    rng = np.random.default_rng(3)
    V, F, E, n = 7, 3, 4, 11
    table = rng.normal(size=(F * V, E))
    ids = rng.integers(0, V, size=(n, F)).astype(np.int32)
    ids[:4, 0] = 2                              # repeated ids
    got = L.gather_embeddings(table, ids, V)
    oh = np.zeros((n, F, F * V))
    for i in range(n):
        for f in range(F):
            oh[i, f, f * V + ids[i, f]] = 1.0
    ref = np.einsum("nft,te->nfe", oh, table).reshape(n, F * E)
    np.testing.assert_array_equal(got, ref)
    g = rng.normal(size=(n, F * E))
    ref_grad = np.einsum("nft,nfe->te", oh, g.reshape(n, F, E))
    np.testing.assert_allclose(L.embedding_grad(g, ids, V, table.shape), ref_grad, rtol=1e-14)


# --------------------------------------------------------------- rounding
def test_round_bf16_matches_library_on_float32_values():
    rng = np.random.default_rng(4)
    x = np.concatenate([rng.normal(0, 1, 100000), rng.normal(0, 1e-3, 1000),
                        rng.normal(0, 1e3, 1000)]).astype(np.float32)
    # ties: float32 values exactly half-way between two bf16 values
    base = rng.normal(0, 1, 1000).astype(np.float32)
    bits = base.view(np.uint32) & np.uint32(0xFFFF0000) | np.uint32(0x8000)
    x = np.concatenate([x, bits.view(np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(round_bf16(x.astype(np.float64)), ref)


def test_round_bf16_direct_from_float64_brute_force():
    """float64 inputs: the result is the nearest 8-significant-bit value,
    ties to even, found by brute force over the neighbouring candidates."""
    rng = np.random.default_rng(6)
    x = rng.normal(0, 1, 2000)
    got = round_bf16(x)
    for xi, gi in zip(x, got):
        e = np.floor(np.log2(abs(xi)))
        ulp = 2.0 ** (e - 7)
        lo = np.floor(xi / ulp) * ulp
        cands = [lo, lo + ulp]
        d = [abs(xi - c) for c in cands]
        best = cands[int(np.argmin(d))]
        assert gi == best
    assert np.array_equal(round_f32(x), x.astype(np.float32).astype(np.float64))
