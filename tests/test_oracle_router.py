"""Pins for the oracle's neural routing policy (Sec. 3.3.2; the appendix on
the neural router: d -> d/8 linear, GELU, linear to one scalar; dropout is
inactive at inference).  The MLP is pinned to torch's fp64 linear and exact
GELU, the GELU itself to the normal CDF from scipy, and the architecture
reading to the parameter counts the paper reports."""
import numpy as np
import pytest
import scipy.stats
import torch

import oracle
import workloads as W


def _rand(shape, rng, std):
    return rng.standard_normal(shape) * std


@pytest.mark.parametrize("gamma,d", [(1, 64), (5, 256), (16, 1024)])
def test_matches_torch_mlp(gamma, d):
    rng = np.random.default_rng(gamma + d)
    m = W.router_hidden(d)
    h = _rand((gamma, d), rng, 1.0)
    w1, b1 = _rand((m, d), rng, 0.05), _rand((m,), rng, 0.05)
    w2, b2 = _rand((m,), rng, 0.1), _rand((1,), rng, 0.1)
    got = oracle.router_mlp(h, w1, b1, w2, b2)
    t = torch.nn.functional.linear(torch.from_numpy(h), torch.from_numpy(w1),
                                   torch.from_numpy(b1))
    t = torch.nn.functional.gelu(t, approximate="none")
    ref = torch.nn.functional.linear(t, torch.from_numpy(w2)[None, :],
                                     torch.from_numpy(b2)).numpy()[:, 0]
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_gelu_is_x_times_normal_cdf():
    """W1 = 0 leaves z = b1, so delta = b2 + sum_i w2_i * b1_i * Phi(b1_i)."""
    c = np.array([0.0, 1.0, -1.0, 2.5, -3.0, 0.3, 7.0, -7.0])
    m, d = len(c), 16
    w2 = np.linspace(-1.0, 1.0, m)
    b2 = np.array([0.25])
    got = oracle.router_mlp(np.ones((3, d)), np.zeros((m, d)), c, w2, b2)
    ref = b2[0] + np.sum(w2 * c * scipy.stats.norm.cdf(c))
    np.testing.assert_allclose(got, np.full(3, ref), rtol=1e-14, atol=1e-14)


def test_parameter_counts_match_the_paper():
    """d/8 hidden units with biases on both layers gives the 2.10M (hidden
    4096, the 8B targets) and 0.82M (hidden 2560, the 4B target)
    parameters the router-latency table lists."""
    for d, expect in ((4096, 2_098_177), (2560, 819_841)):
        m = W.router_hidden(d)
        assert m * d + m + m + 1 == expect
    assert round(2_098_177 / 1e6, 2) == 2.10 and round(819_841 / 1e6, 2) == 0.82
    w = W.CONFIGS[3]
    r = W.generate_router(w, device="cpu")
    assert sum(t.numel() for t in r.values()) == 2_098_177


def test_bf16_storage_decodes_exactly():
    rng = np.random.default_rng(3)
    gamma, d = 4, 128
    m = W.router_hidden(d)
    ts = [torch.from_numpy(_rand(s, rng, 0.3)).to(torch.bfloat16)
          for s in ((gamma, d), (m, d), (m,), (m,), (1,))]
    a = oracle.router_mlp(*[W.to_oracle(t) for t in ts])
    b = oracle.router_mlp(*[t.to(torch.float64).numpy() for t in ts])
    np.testing.assert_array_equal(a, b)


def test_route_rule_is_strict():
    delta = np.array([0.2, 1.0, 1.5])
    assert oracle.route_neural(delta, 1, 1.0) == 0
    assert oracle.route_neural(delta, 2, 1.0) == 1
    assert oracle.route_neural(delta, 0, -0.5) == 1
