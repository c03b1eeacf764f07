"""Seeded synthetic workloads shared by the tests, the bench and the oracle
checks.  This module only draws random numbers; it holds none of the method's
arithmetic.

The shapes follow the evaluation's workload families (gradient-, weight- and
KV-cache-like tensors; App. F.1 uses Normal, Lognormal, Student-t and
sparse-outlier vectors and real-model tensors, which are not available here):

  normal_1k      fp32, d = 1024,  Normal(0, 1)
  lognormal_16k  fp32, d = 16384, exp(Normal(0, 1)) with random +-1 signs
  kv_rows        fp16, 4096 x 128, Normal(0, 1); 1% of entries replaced by +-8
  weights_256k   fp32, d = 2^18,  0.9 Normal(0, 0.01) + 0.1 Laplace(0, 0.1)
  student_t_1m   fp32, d = 2^20,  Student-t with 3 degrees of freedom

Every draw uses numpy.random.Generator(PCG64(seed)) in float64 and then rounds
to the storage type (round to nearest even).
"""
import numpy as np

WORKLOADS = {
    "normal_1k": dict(d=1024, s=16, budgets=(2.0,)),
    "lognormal_16k": dict(d=16384, s=32, budgets=(1.5, 2.5, 3.5)),
    "kv_rows": dict(rows=4096, d=128, s=16, budgets=(3.0,)),
    "weights_256k": dict(d=1 << 18, s=32, budgets=(2.0,)),
    "student_t_1m": dict(d=1 << 20, s=64, budgets=(1.0, 2.0, 3.0, 4.0)),
}


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def normal(d, seed=0):
    return _rng(seed).standard_normal(d).astype(np.float32)


def lognormal_signed(d, seed=0):
    g = _rng(seed)
    mag = np.exp(g.standard_normal(d))
    sign = g.choice(np.array([-1.0, 1.0]), size=d)
    return (mag * sign).astype(np.float32)


def kv_rows(rows=4096, d=128, seed=0, outlier_rate=0.01, outlier=8.0):
    g = _rng(seed)
    x = g.standard_normal((rows, d))
    hit = g.random((rows, d)) < outlier_rate
    sign = g.choice(np.array([-1.0, 1.0]), size=(rows, d))
    x = np.where(hit, outlier * sign, x)
    return x.astype(np.float16)


def sparse_outlier(d, seed=0, rate=0.01, scale=8.0):
    """Standard normal entries, a share `rate` of them replaced by +-scale."""
    g = _rng(seed)
    x = g.standard_normal(d)
    hit = g.random(d) < rate
    sign = g.choice(np.array([-1.0, 1.0]), size=d)
    return np.where(hit, scale * sign, x).astype(np.float32)


def weight_mixture(d=1 << 18, seed=0):
    g = _rng(seed)
    pick = g.random(d) < 0.9
    a = g.normal(0.0, 0.01, d)
    b = g.laplace(0.0, 0.1, d)
    return np.where(pick, a, b).astype(np.float32)


def student_t(d=1 << 20, seed=0, nu=3.0):
    return _rng(seed).standard_t(nu, d).astype(np.float32)


def make(name, seed=0, d=None):
    """Input array of a named workload (optionally with a smaller d)."""
    w = WORKLOADS[name]
    if name == "normal_1k":
        return normal(d or w["d"], seed)
    if name == "lognormal_16k":
        return lognormal_signed(d or w["d"], seed)
    if name == "kv_rows":
        return kv_rows(w["rows"], d or w["d"], seed)
    if name == "weights_256k":
        return weight_mixture(d or w["d"], seed)
    if name == "student_t_1m":
        return student_t(d or w["d"], seed)
    raise KeyError(name)
