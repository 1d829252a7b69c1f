"""Pins of the oracle's sampled request lengths (no GPU).

The table tests pin the quantised CDF tables; these pin what the oracle draws
from them, end to end: Philox words -> inverse CDF -> the prompt and output
length of every arrival of a tick (the synthetic workloads of Sections
4.2-4.4).  The expected moments come from each workload's distribution
written out here from its definition, not from the oracle's tables:

* uniform prompt on [lo, hi];
* log-normal prompt, P(len <= n) = Phi((ln(n + 1/2) - mu) / sigma) on
  [lo, hi] with both tails lumped at the bounds;
* geometric output on {1, 2, ...} with the given mean;
* Pareto output min(floor(x_min U^(-1/alpha)), cap), so
  P(out >= n) = (x_min / n)^alpha for x_min <= n <= cap.

Each test draws a few thousand ticks of arrivals on a two-instance cluster
(sampling does not depend on the cluster) and compares the sample mean and
variance with the closed forms at five standard errors, the standard error of
the variance taken from the distribution's fourth central moment.  The prompt
and the output of an arrival come from different Philox words, so their
sample correlation must vanish within five standard errors as well.
"""
import math

import numpy as np
import pytest
from scipy.stats import norm

import oracle
from workloads import preset

Z = 5.0


def _pmf_uniform(lo, hi):
    n = np.arange(lo, hi + 1, dtype=np.float64)
    return n, np.full(len(n), 1.0 / (hi - lo + 1))


def _pmf_lognormal(mu, sigma, lo, hi):
    n = np.arange(lo, hi + 1, dtype=np.float64)
    cdf = norm.cdf((np.log(n + 0.5) - mu) / sigma)
    cdf[-1] = 1.0
    return n, np.diff(np.concatenate([[0.0], cdf]))


def _pmf_geometric(mean, tail=1e-13):
    q = 1.0 / mean
    nmax = int(math.ceil(math.log(tail) / math.log1p(-q))) + 1
    n = np.arange(1, nmax + 1, dtype=np.float64)
    p = q * np.exp((n - 1) * math.log1p(-q))
    return n, p / p.sum()


def _pmf_pareto(alpha, xmin, cap):
    n = np.arange(xmin, cap + 1, dtype=np.float64)
    ge = (xmin / n) ** alpha              # P(out >= n)
    ge_next = np.concatenate([ge[1:], [0.0]])
    return n, ge - ge_next


def _pmf(spec):
    k = spec["kind"]
    if k == "uniform_int":
        return _pmf_uniform(spec["lo"], spec["hi"])
    if k == "lognormal":
        return _pmf_lognormal(spec["mu"], spec["sigma"], spec["lo"], spec["hi"])
    if k == "geometric":
        return _pmf_geometric(spec["mean"])
    if k == "pareto":
        return _pmf_pareto(spec["alpha"], spec["min"], spec["cap"])
    raise ValueError(k)


def _moments(n, p):
    m = float((n * p).sum())
    c = n - m
    var = float((c * c * p).sum())
    mu4 = float((c ** 4 * p).sum())
    return m, var, mu4


def _draws(name, ticks):
    c = preset(name)
    c["n_instances"] = 2
    c["slots_per_instance"] = 64
    c["mig_max_pairs"] = 1
    c["groups"] = [dict(c["groups"][0], n_replicas=1)]
    o = oracle.Oracle(c, 0, 1, check=False)
    prompts, outputs = [], []
    for _ in range(ticks):
        o.step(1)
        a = o.last_arrivals(0)
        prompts.append(a[:, 1].astype(np.float64))
        outputs.append(a[:, 2].astype(np.float64))
    o.close()
    return c, np.concatenate(prompts), np.concatenate(outputs)


def _check(x, spec, what):
    n, p = _pmf(spec)
    assert abs(p.sum() - 1.0) < 1e-9
    m, var, mu4 = _moments(n, p)
    N = len(x)
    assert N > 1000, what
    xm = float(x.mean())
    xv = float(x.var(ddof=1))
    zm = (xm - m) / math.sqrt(var / N)
    zv = (xv - var) / math.sqrt(max(mu4 - var * var, 1e-30) / N)
    assert abs(zm) < Z, "%s mean %.3f vs %.3f (z %.1f)" % (what, xm, m, zm)
    assert abs(zv) < Z, "%s variance %.1f vs %.1f (z %.1f)" % (what, xv, var, zv)
    # every draw lies in the distribution's support
    assert x.min() >= n[0] and x.max() <= n[-1], what


@pytest.mark.parametrize("name,ticks", [("tiny", 4000), ("enterprise", 2000), ("gauss10", 2000),
                                        ("sweep", 1000), ("wide", 300)])
def test_sampled_lengths_match_the_workload_distributions(name, ticks):
    c, pr, out = _draws(name, ticks)
    _check(pr, c["prompt"], "%s prompt" % name)
    _check(out, c["output"], "%s output" % name)
    # distinct Philox words: uncorrelated prompt and output lengths
    r = float(np.corrcoef(pr, out)[0, 1])
    assert abs(r) < Z / math.sqrt(len(pr)), "%s prompt/output correlation %.4f" % (name, r)


def test_closed_forms_of_the_sampling_pins():
    # the closed forms used above, against textbook values
    n, p = _pmf_geometric(256.0)
    m, var, _ = _moments(n, p)
    assert abs(m - 256.0) < 1e-6 and abs(var - 256.0 * 255.0) < 1e-3
    n, p = _pmf_uniform(64, 1024)
    m, var, _ = _moments(n, p)
    assert abs(m - 544.0) < 1e-9 and abs(var - (961.0 ** 2 - 1) / 12) < 1e-6
    # Pareto: E[out] = x_min + sum_{n = x_min + 1}^{cap} (x_min / n)^alpha
    n, p = _pmf_pareto(1.5, 16, 8192)
    m, _, _ = _moments(n, p)
    want = 16 + sum((16 / k) ** 1.5 for k in range(17, 8193))
    assert abs(m - want) < 1e-9 * want
    # log-normal with the clip bounds far out: P(len <= n) = P(X <= n + 1/2)
    # rounds X to the nearest integer, so the mean stays that of the
    # continuous law, exp(mu + sigma^2 / 2), up to the rounding's small bias
    n, p = _pmf_lognormal(6.0, 0.5, 1, 1 << 16)
    m, var, _ = _moments(n, p)
    assert abs(m - math.exp(6.0 + 0.125)) < 0.01
    assert abs(var - (math.exp(0.25) - 1) * math.exp(12.25)) / var < 1e-4
