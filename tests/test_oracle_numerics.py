"""Pins of the oracle's numeric building blocks against library routines."""
import numpy as np
import pytest
import torch
import scipy.special

from oracle.numerics import attend, logsumexp, rmsnorm, round_bf16, softmax


def test_round_bf16_matches_torch_bfloat16():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(
        -6, 6, 20000), [0.0, -0.0, 1.0, 1.00390625, 1.01171875, -3.5]])
    # values exactly half-way between two bf16 neighbours (ties to even)
    base = rng.standard_normal(1000).astype(np.float32)
    ties = (torch.tensor(base).bfloat16().float().numpy().astype(np.float64)
            * (1 + 2.0 ** -9))
    x = np.concatenate([x, ties])
    ref = torch.tensor(x, dtype=torch.float64).to(torch.bfloat16).to(
        torch.float64).numpy()
    np.testing.assert_array_equal(round_bf16(x), ref)


def test_rmsnorm_matches_torch():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((7, 96))
    g = rng.standard_normal(96)
    ref = torch.nn.functional.rms_norm(torch.tensor(x), (96,), torch.tensor(g),
                                       eps=1e-5).numpy()
    np.testing.assert_allclose(rmsnorm(x, g, 1e-5), ref, rtol=1e-12,
                               atol=1e-12)


def test_softmax_logsumexp_match_scipy():
    rng = np.random.default_rng(2)
    z = rng.standard_normal((5, 1000)) * 4
    np.testing.assert_allclose(softmax(z), scipy.special.softmax(z, axis=-1),
                               rtol=1e-12)
    np.testing.assert_allclose(logsumexp(z),
                               scipy.special.logsumexp(z, axis=-1),
                               rtol=1e-13)


@pytest.mark.parametrize("H,Hkv", [(4, 4), (8, 2), (6, 1)])
def test_attend_matches_sdpa_gqa(H, Hkv):
    rng = np.random.default_rng(3)
    hd, n = 16, 23
    q = rng.standard_normal((H, hd))
    k = rng.standard_normal((n, Hkv, hd))
    v = rng.standard_normal((n, Hkv, hd))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.tensor(q)[None, :, None, :],
        torch.tensor(k).permute(1, 0, 2)[None],
        torch.tensor(v).permute(1, 0, 2)[None], enable_gqa=True)
    np.testing.assert_allclose(attend(q, k, v), ref.reshape(-1).numpy(),
                               rtol=1e-11, atol=1e-12)
