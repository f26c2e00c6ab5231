"""Brute-force enumeration for tiny mixtures — TEST INFRASTRUCTURE ONLY.

A mixture model gives every point a hidden component z_i in [K].  The
marginal likelihood of the data is the sum over all K^N joint assignments of
prod_i pi_{z_i} N(x_i | z_i), and the posterior probability that point i
came from component k is the share of that sum carried by assignments with
z_i = k (the responsibility of Sec. 2).  This module evaluates both by
literally enumerating the K^N assignments with pure-Python loops, using a
Gaussian density written from its textbook formula, so it pins the checker
in ``oracle.c`` without sharing any of its code.  Only N <= 6, K <= 3 is
practical.
"""
from __future__ import annotations

import itertools
import math


def gauss_pdf_diag(x, mu, var):
    """Product over dimensions of the 1-D normal density (diagonal covariance)."""
    p = 1.0
    for xd, md, vd in zip(x, mu, var):
        p *= math.exp(-(xd - md) ** 2 / (2.0 * vd)) / math.sqrt(2.0 * math.pi * vd)
    return p


def enumerate_posterior(x, weights, means, variances):
    """Returns (marginal likelihood, posterior marginals r[i][k]) by summing over all K^N
    joint component assignments."""
    n, k = len(x), len(weights)
    dens = [[weights[c] * gauss_pdf_diag(x[i], means[c], variances[c]) for c in range(k)]
            for i in range(n)]
    total = 0.0
    marg = [[0.0] * k for _ in range(n)]
    for z in itertools.product(range(k), repeat=n):
        p = 1.0
        for i, c in enumerate(z):
            p *= dens[i][c]
        total += p
        for i, c in enumerate(z):
            marg[i][c] += p
    post = [[marg[i][c] / total for c in range(k)] for i in range(n)]
    return total, post


def expected_complete_loglik(x, post, weights, means, variances):
    """sum_i sum_k r_ik [log pi_k + log N(x_i | mu_k, var_k)] — the quantity the M-step maximises
    for fixed responsibilities."""
    tot = 0.0
    for i, xi in enumerate(x):
        for c, r in enumerate(post[i]):
            if r == 0.0:
                continue
            lp = math.log(weights[c])
            for xd, md, vd in zip(xi, means[c], variances[c]):
                lp += -0.5 * math.log(2.0 * math.pi * vd) - (xd - md) ** 2 / (2.0 * vd)
            tot += r * lp
    return tot
