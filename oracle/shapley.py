"""Exact Shapley values by eq. 1 (Sec. 2.3): the weighted mean of every
marginal contribution, |S|!(n-|S|-1)!/n! * (f(S + i) - f(S)).  Brute force
over all 2^n coalitions; only for small n."""
import itertools
import math

import numpy as np


def all_values(game, n):
    """f over every coalition, indexed by the bitmask sum_i m_i 2^i."""
    vals = np.zeros(1 << n, dtype=np.float64)
    for code in range(1 << n):
        m = np.array([(code >> i) & 1 for i in range(n)], dtype=bool)
        vals[code] = game(m)
    return vals


def exact_shapley(vals, n):
    phi = np.zeros(n, dtype=np.float64)
    fact = [math.factorial(i) for i in range(n + 1)]
    for i in range(n):
        others = [j for j in range(n) if j != i]
        for r in range(n):
            coef = fact[r] * fact[n - r - 1] / fact[n]
            for S in itertools.combinations(others, r):
                code = sum(1 << j for j in S)
                phi[i] += coef * (vals[code | (1 << i)] - vals[code])
    return phi
