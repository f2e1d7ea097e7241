"""GPU parity of the point-embedding MLP (matrix cores, bfloat16 with fp32
accumulation) against the oracle's exact sums.

Bar: where every partial sum is exactly representable (quarter-step inputs
and half-step weights) the two sides agree bit for bit.  In general the GPU
accumulates in fp32, so a hidden activation lying within the fp32 rounding
of a bfloat16 tie can round the other way; each output element must then
stay within the bound that such one-ulp changes (2^-7 relative) of the
hidden activations, and fp32 accumulation, can cause, computed from the
magnitudes |x| |W1|, |h1| |W2| and |h2| |W3| of that point, and 99 % of the
elements within fp32 accumulation error alone."""
import numpy as np
import pytest
import torch

import oracle
from paper_2512_00385_amd import ezsp, scenes

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ezsp.load()
    yield


def dev(a):
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).cuda()


def run_both(x, w):
    w1, b1, w2, b2, w3, b3 = w
    ref = oracle.embed_mlp(x, w1, b1, w2, b2, w3, b3)
    got = ezsp.embed_mlp(dev(x), dev(w1), dev(b1), dev(w2), dev(b2), dev(w3),
                         dev(b3)).cpu().numpy().astype(np.float64)
    return got, ref


def bound(x, w):
    f = scenes.bf16_bits_to_f32
    w1, b1, w2, b2, w3, b3 = w
    a1 = np.abs(f(x)) @ np.abs(f(w1)) + np.abs(b1)
    a2 = a1 @ np.abs(f(w2)) + np.abs(b2)
    mag = a2 @ np.abs(f(w3)) + np.abs(b3)
    flips = 2.0 ** -7 * (mag + (a1 @ np.abs(f(w2))) @ np.abs(f(w3)))
    return flips + 2.0 ** -20 * mag, 2.0 ** -20 * mag * 64


def check(x, w):
    got, ref = run_both(x, w)
    tol, tight = bound(x, w)
    err = np.abs(got - ref)
    assert np.all(err <= tol), float((err - tol).max())
    assert np.mean(err <= tight) >= 0.99
    return got, ref


@pytest.mark.parametrize("n", [1, 31, 32, 33, 1000, 4097])
def test_mlp_exact_grid_values(n):
    # quarter-step inputs, half-step weights, eighth-step biases: every
    # partial sum is exact in fp32, so the bfloat16 roundings agree
    rng = np.random.default_rng(n)
    q = lambda shape, step, lim: (rng.integers(-lim, lim + 1, shape) * step)
    x = scenes.to_bf16_bits(q((n, 6), 0.25, 4).astype(np.float32))
    w = (scenes.to_bf16_bits(q((6, 32), 0.5, 2).astype(np.float32)),
         q(32, 0.125, 8).astype(np.float32),
         scenes.to_bf16_bits(q((32, 32), 0.5, 1).astype(np.float32)),
         q(32, 0.125, 8).astype(np.float32),
         scenes.to_bf16_bits(q((32, 16), 0.5, 1).astype(np.float32)),
         q(16, 0.125, 8).astype(np.float32))
    got, ref = run_both(x, w)
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("d_in,d_out", [(1, 1), (6, 16), (8, 32), (3, 5),
                                        (7, 31)])
def test_mlp_random_shapes(d_in, d_out):
    rng = np.random.default_rng(d_in * 40 + d_out)
    x = scenes.to_bf16_bits(rng.uniform(-1, 1, (3001, d_in)).astype(np.float32))
    check(x, scenes.mlp_weights(d_in, (d_in, 32, d_out)))


def test_mlp_sweep_full():
    # the 1.28M-point sweep stand-in with the seed-0 weights
    _, feat, _ = scenes.sweep()
    check(feat, scenes.mlp_weights(0))


def test_mlp_rejects():
    w = [dev(a) for a in scenes.mlp_weights(0)]
    x = dev(scenes.to_bf16_bits(np.zeros((10, 6), np.float32)))
    bad_w2 = dev(scenes.to_bf16_bits(np.zeros((32, 16), np.float32)))
    with pytest.raises(ValueError):
        ezsp.embed_mlp(x, w[0], w[1], bad_w2, w[3], w[4], w[5])
    x9 = dev(scenes.to_bf16_bits(np.zeros((10, 9), np.float32)))
    w9 = dev(scenes.to_bf16_bits(np.zeros((9, 32), np.float32)))
    with pytest.raises(ezsp.EzspError):
        ezsp.embed_mlp(x9, w9, w[1], w[2], w[3], w[4], w[5])
