"""CPU check of the weighted form the mean-of-probabilities kernels take for their
column sums (Sec. 4.1 Eq. 8-9 with the softmax per text query, then the mean over
the queries).

With a per-query reference c_t, x = expm1(s z - c_t) and S_t = N + sum_n x, the
softmax of query t is (1 + x) / S_t, so N P - 1 = (N / S_t) x - E_t / S_t with
E_t = sum_n x.  The kernels sum w_t x over the queries and subtract sum_t E_t / S_t
once per key.  Here the form, evaluated in float64 on seeded logits (near-uniform,
as in the workloads, and spread out, with and without a reference), is compared
with the oracle's support computed from the same logits."""
import numpy as np
import pytest

import oracle as O


def _weighted_u(z, scale, ref):
    """u = N r - 1 of every key by the weighted form; z: [N_T, N] logits."""
    N = z.shape[1]
    c = ref(z)[:, None]
    x = np.expm1(scale * z - c)
    E = x.sum(axis=1, keepdims=True)
    S = N + E
    return ((N / S) * x).sum(axis=0) / z.shape[0] - (E / S).sum() / z.shape[0]


@pytest.mark.parametrize("spread", [0.05, 3.0])
@pytest.mark.parametrize("ref", ["mean16", "zero", "first"])
def test_weighted_form_matches_oracle_supports(spread, ref):
    rng = np.random.default_rng(2608)
    nt, n, d = 37, 437, 64
    q = rng.normal(0.0, spread, (nt, d))
    k = rng.normal(0.0, 1.0, (n, d))
    scale = 1.0 / np.sqrt(d)
    z = q @ k.T
    refs = {"mean16": lambda z: scale * z[:, :16].mean(axis=1),
            "zero": lambda z: np.zeros(z.shape[0]),
            "first": lambda z: scale * z[:, 0]}
    u = _weighted_u(z, scale, refs[ref])
    # the oracle's mean of probabilities: r_n = mean_t softmax_n(s z)
    r = O.normalized_attention(O.text_visual_logits(q, k, scale), "mean_prob")
    np.testing.assert_allclose(1.0 + u, n * r, rtol=0, atol=1e-12)


def test_weighted_form_uniform_is_exactly_zero():
    """Identical keys: x = 0 for every logit (c_t equals each logit), so E = 0,
    S = N, w = 1 and u = 0 exactly."""
    z = np.tile(np.linspace(-1.0, 1.0, 9)[:, None], (1, 40))
    u = _weighted_u(z, 0.5, lambda z: 0.5 * z[:, :16].mean(axis=1))
    assert (u == 0.0).all()
