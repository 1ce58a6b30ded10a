"""The closed form behind the DDA cell boundaries, checked by brute force.

The device search turns every (candidate scale alpha, set midpoint mu) into the
smallest fp32 X with fl32(X / alpha) >= mu, so that "|x| >= X" decides the cell
of |x| exactly as the projection's IEEE division does (eq. (6), (8)).  It takes
X as the fp32 rounding up of alpha * m, m the real midpoint between mu and the
fp32 just below it (the quotient rounds up to mu from m on, a tie going to mu's
even significand).  Here that rule is evaluated in numpy and compared with the
definition on both sides of the answer: fl32(X / alpha) >= mu and
fl32(pred(X) / alpha) < mu, with numpy's IEEE binary32 division (subnormals
kept), for every midpoint of every format and scales over the whole fp32 range.
"""
import numpy as np

import oracle


def closed_form(alpha, mu):
    """fp32 bits of the rounding up of alpha * (pred(mu) + mu) / 2 (exact in fp64)."""
    mu = np.float32(mu)
    pred = np.frombuffer((np.array([mu]).view(np.uint32) - 1).tobytes(), dtype=np.float32)[0]
    m = 0.5 * (np.float64(pred) + np.float64(mu))
    t = np.float64(alpha) * m
    with np.errstate(over="ignore"):
        f = np.float32(t)
    b = int(np.array([f]).view(np.uint32)[0])
    if np.float64(f) < t:
        b += 1
    return min(b, 0x7F800000)


def f32(bits):
    return np.array([bits], dtype=np.uint32).view(np.float32)[0]


def midpoints(b, k_sig):
    q = np.asarray(oracle.valueset(b, k_sig), dtype=np.float64)
    q = np.unique(q[q >= 0])
    return ((q[:-1] + q[1:]) / 2).astype(np.float32)


def scales(rng, count):
    # log-uniform over normal and subnormal fp32, plus edge values
    e = rng.uniform(-149.0, 127.5, count)
    a = (2.0 ** e * rng.uniform(1.0, 2.0, count)).astype(np.float32)
    a = a[(a > 0) & np.isfinite(a)]
    edge = np.array([1.4e-45, 2.8e-45, 1.1754942e-38, 1.1754944e-38, 1.0, 0.4871, 3.0e38,
                     3.4028235e38], dtype=np.float32)
    return np.concatenate([edge, a])


def test_threshold_rule_brute_force():
    rng = np.random.default_rng(11)
    with np.errstate(over="ignore", under="ignore", divide="ignore"):
        for (b, k_sig) in [(2, 1), (3, 1), (3, 2), (4, 1), (4, 2), (5, 3), (6, 2), (8, 5), (8, 7)]:
            for mu in midpoints(b, k_sig):
                for alpha in scales(rng, 300):
                    X = closed_form(alpha, mu)
                    if X < 0x7F800000:
                        assert f32(X) / alpha >= mu, (b, k_sig, mu, alpha, X)
                    if X > 0:
                        assert f32(X - 1) / alpha < mu, (b, k_sig, mu, alpha, X)
