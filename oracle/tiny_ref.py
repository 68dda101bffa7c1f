"""ORACLE -- test infrastructure, not product code.

A second, independent reference for tiny cases, in pure Python:

* Philox4x32-10 on Python integers (Salmon et al., SC'11), used to cross-check
  the C oracle's fixed-width arithmetic bit for bit;
* an exact rational (``fractions.Fraction``) run of Algorithm 2's local steps
  and synchronizations for K <= 4 workers and a handful of parameters, given the
  noise values as inputs, used to bound the C oracle's rounding.
"""
from __future__ import annotations

from fractions import Fraction
from typing import List, Sequence

MASK = (1 << 32) - 1


def philox4x32_10(ctr: Sequence[int], key: Sequence[int]) -> List[int]:
    c = [int(v) & MASK for v in ctr]
    k0, k1 = int(key[0]) & MASK, int(key[1]) & MASK
    for _ in range(10):
        prod0 = 0xD2511F53 * c[0]
        prod1 = 0xCD9E8D57 * c[2]
        c = [(prod1 >> 32) ^ c[1] ^ k0, prod1 & MASK, (prod0 >> 32) ^ c[3] ^ k1, prod0 & MASK]
        k0 = (k0 + 0x9E3779B9) & MASK
        k1 = (k1 + 0xBB67AE85) & MASK
    return c


def exact_run(K, P, offsets, h, xs, noise, sigma, momentum, wd, lrs, sync_after):
    """Exact Algorithm 2 dynamics with a given sync schedule.

    noise[t][k][i] are the z values (any numbers, converted exactly); lrs[t] the
    learning rate of step t; sync_after is the set of steps after which the
    replicas are averaged.  Returns (x, v, [(t, var_per_tensor)]) as Fractions.
    """
    F = Fraction
    sigma, momentum, wd = F(sigma), F(momentum), F(wd)
    h = [F(a) for a in h]
    xs = [F(a) for a in xs]
    x = [[F(0)] * P for _ in range(K)]
    v = [[F(0)] * P for _ in range(K)]
    syncs = []
    for t, gamma in enumerate(lrs):
        gamma = F(gamma)
        for k in range(K):
            for i in range(P):
                d = h[i] * (x[k][i] - xs[i]) + sigma * F(noise[t][k][i]) + wd * x[k][i]
                v[k][i] = momentum * v[k][i] + d
                x[k][i] = x[k][i] - gamma * v[k][i]
        if t in sync_after:
            xbar = [sum(x[k][i] for k in range(K)) / K for i in range(P)]
            var = []
            for tau in range(len(offsets) - 1):
                acc = F(0)
                for k in range(K):
                    for i in range(offsets[tau], offsets[tau + 1]):
                        acc += (xbar[i] - x[k][i]) ** 2
                var.append(acc / K)
            for k in range(K):
                x[k] = list(xbar)
            syncs.append((t, var))
    return x, v, syncs
