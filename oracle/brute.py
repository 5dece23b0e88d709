"""Brute-force reference for tiny problems (D <= 4, N <= 8) -- TEST INFRASTRUCTURE ONLY.

A second, literal implementation of one OpenAI-ES generation of the evosax
report (arXiv 2212.04180, Sec. 2.1 ask / evaluate / tell; FD gradient
estimator; centered ranks of Sec. 3.2; Adam), written in pure Python with
integers and exact rationals.  It shares nothing with ``esoracle.c`` (its own
Philox, its own Box-Muller, its own ranking by counting, the population matrix
E built explicitly) and is used only to pin that oracle.

fp32 rounding is done exactly: every fp32 result is the round-to-nearest-even
of the exact rational value (``f32``), so a fused multiply-add is one rounding
by construction.  Transcendentals use Python's fp64 ``math`` functions and
then one fp32 rounding.
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np

M0, M1 = 0xD2511F53, 0xCD9E8D57   # Philox-4x32 multipliers (Salmon et al., SC'11)
W0, W1 = 0x9E3779B9, 0xBB67AE85   # Weyl key increments
MASK = 0xFFFFFFFF


def philox(key, ctr, rounds=10):
    """Philox-4x32-R block: R rounds of two 32x32->64 products and xors with the key."""
    k0, k1 = key
    c0, c1, c2, c3 = ctr
    for i in range(rounds):
        if i:
            k0, k1 = (k0 + W0) & MASK, (k1 + W1) & MASK
        p0, p1 = M0 * c0, M1 * c2
        c0, c1, c2, c3 = ((p1 >> 32) ^ c1 ^ k0, p1 & MASK, (p0 >> 32) ^ c3 ^ k1, p0 & MASK)
    return [c0, c1, c2, c3]


def _q(v) -> Fraction:
    """Exact rational value of an int, float, numpy scalar or Fraction."""
    if isinstance(v, (Fraction, int)):
        return Fraction(v)
    return Fraction(float(v))


def f32(q) -> float:
    """Round an exact rational (or int / float) to the nearest fp32, ties to even."""
    q = _q(q)
    if q == 0:
        return 0.0
    sgn = -1 if q < 0 else 1
    a = abs(q)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    # 2^e <= a < 2^(e+1); fp32 keeps 24 significant bits down to 2^-149
    lsb_exp = max(e - 23, -149)
    scaled = a / Fraction(2) ** lsb_exp
    n = scaled.numerator // scaled.denominator
    rem = scaled - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    val = Fraction(n) * Fraction(2) ** lsb_exp
    if val >= Fraction(2) ** 128 - Fraction(2) ** 103:
        return sgn * math.inf
    return float(np.float32(sgn * float(val)))


def fma32(a, b, c):
    return f32(_q(a) * _q(b) + _q(c))


def normals_block(seed, domain, row, t, b):
    """Four N(0,1) values of Philox block b: Box-Muller on (w0,w1), (w2,w3)."""
    w = philox((seed & MASK, (seed >> 32) & MASK), (b & MASK, row, t, domain))
    out = []
    for h in range(2):
        u = ((w[2 * h] >> 8) + 1) * 2.0 ** -24
        th = (w[2 * h + 1] >> 8) * 2.0 ** -24
        r = math.sqrt(-2.0 * math.log(u))
        a = 2.0 * math.pi * th
        out += [f32(r * math.cos(a)), f32(r * math.sin(a))]
    return out


def eps_vector(seed, domain, row, t, D):
    v = []
    for b in range((D + 3) // 4):
        v += normals_block(seed, domain, row, t, b)
    return v[:D]


def init_uniform(seed, D, lo, hi):
    rng = f32(_q(f32(hi)) - _q(f32(lo)))
    m = []
    for d in range(D):
        w = philox((seed & MASK, (seed >> 32) & MASK), (d // 4, 0, 0, 1))[d % 4]
        m.append(fma32(rng, Fraction(w >> 8, 2 ** 24), f32(lo)))
    return m


def fitness(problem, x, s=None, a=10.0):
    """Benchmark problems on fp32 x: exact rational sums (sphere, shifted sphere,
    Rosenbrock) or an exact sum of fp64 terms (Rastrigin), one fp32 rounding."""
    D = len(x)
    X = [_q(v) for v in x]
    if problem == "sphere":
        return f32(sum(v * v for v in X))
    if problem == "shifted_sphere":
        return f32(sum((X[i] - _q(s[i])) ** 2 for i in range(D)))
    if problem == "rosenbrock":
        return f32(sum(100 * (X[i + 1] - X[i] ** 2) ** 2 + (1 - X[i]) ** 2 for i in range(D - 1)))
    if problem == "rastrigin":
        xs = [float(v) for v in x]
        terms = [a * D] + [xs[i] * xs[i] - a * math.cos(2.0 * math.pi * xs[i]) for i in range(D)]
        return f32(math.fsum(terms))
    raise ValueError(problem)


def ranks(f, maximize=False):
    """rank_j = #{k: key_k < key_j} + #{k < j: key_k == key_j}; NaN is worst."""
    def key(v):
        k = -v if maximize else v
        return math.inf if math.isnan(k) else k
    keys = [key(v) for v in f]
    N = len(f)
    return [sum(1 for k in range(N) if keys[k] < keys[j] or (keys[k] == keys[j] and k < j))
            for j in range(N)]


def centered(f, maximize=False):
    N = len(f)
    return [f32(Fraction(2 * r - (N - 1), 2 * (N - 1))) for r in ranks(f, maximize)]


def shaped_keys(f, pen, maximize, w_decay):
    """Minimisation keys with the weight-decay penalty added in fp32:
    k = f or -f, then fl32(k + fl32(w * pen)) for finite k; NaN is +inf."""
    out = []
    for j, v in enumerate(f):
        k = -v if maximize else v
        if math.isnan(k):
            out.append(math.inf)
        elif w_decay and math.isfinite(k):
            out.append(f32(_q(k) + _q(f32(_q(w_decay) * _q(pen[j])))))
        else:
            out.append(k)
    return out


def zscore(keys):
    """(k - mean) / (population sd + 1e-10) over the finite keys, from the exact
    rational mean and variance and a 60-digit square root, rounded once to fp32;
    non-finite keys give 0."""
    from decimal import Decimal, getcontext
    getcontext().prec = 60
    fin = [_q(k) for k in keys if math.isfinite(k)]
    n = len(fin)
    mu = sum(fin) / n if n else Fraction(0)
    var = sum((k - mu) ** 2 for k in fin) / n if n else Fraction(0)
    sd = (Decimal(var.numerator) / Decimal(var.denominator)).sqrt()
    den = sd + Decimal(1e-10)
    out = []
    for k in keys:
        if not math.isfinite(k):
            out.append(0.0)
            continue
        num = _q(k) - mu
        z = Decimal(num.numerator) / Decimal(num.denominator) / den
        out.append(f32(Fraction(z)))
    return out


class BruteES:
    """R=1 OpenAI-ES with antithetic pairs (+eps first half, -eps second half).
    sigma and lr follow the App. B schedules, max(x * decay, final) after each
    generation; shaping "centered", "raw" or "zscore", optional weight decay."""

    def __init__(self, problem, D, N, sigma, lr, seed, lo, hi, s=None, maximize=False,
                 beta1=0.9, beta2=0.999, eps=1e-8, a=10.0, shaping="centered",
                 sigma_decay=1.0, sigma_final=0.0, lr_decay=1.0, lr_final=0.0, w_decay=0.0):
        assert N % 2 == 0
        self.problem, self.D, self.N = problem, D, N
        self.sigma, self.lr = f32(sigma), f32(lr)
        self.sd, self.sf, self.ld, self.lf = f32(sigma_decay), f32(sigma_final), f32(lr_decay), f32(lr_final)
        self.w_decay = f32(w_decay)
        self.b1, self.b2, self.eps = f32(beta1), f32(beta2), f32(eps)
        self.seed, self.s, self.maximize, self.a, self.shaping = seed, s, maximize, a, shaping
        self.m = init_uniform(seed, D, lo, hi)
        self.m1 = [0.0] * D
        self.v = [0.0] * D
        self.t = 0

    def population(self):
        """E (N x D): row j = +eps_j for j < N/2, -eps_{j-N/2} otherwise; x = m + sigma E."""
        half = self.N // 2
        E = []
        for j in range(self.N):
            e = eps_vector(self.seed, 0, j % half, self.t, self.D)
            E.append(e if j < half else [-v for v in e])
        X = [[fma32(self.sigma, E[j][d], self.m[d]) for d in range(self.D)] for j in range(self.N)]
        return E, X

    def generation(self, fit=None):
        E, X = self.population()
        f = fit if fit is not None else [fitness(self.problem, x, self.s, self.a) for x in X]
        pen = [f32(sum(_q(v) ** 2 for v in x) / self.D) for x in X]
        keys = shaped_keys(f, pen, self.maximize, self.w_decay)
        if self.shaping == "centered":
            N = self.N
            rk = [sum(1 for k in range(N) if keys[k] < keys[j] or (keys[k] == keys[j] and k < j))
                  for j in range(N)]
            y = [f32(Fraction(2 * r - (N - 1), 2 * (N - 1))) for r in rk]
        elif self.shaping == "zscore":
            y = zscore(keys)
        else:
            y = keys
        Ns = Fraction(self.N) * _q(self.sigma)
        g = [f32(sum(_q(y[j]) * _q(E[j][d]) for j in range(self.N)) / Ns)
             for d in range(self.D)]
        tp = self.t + 1
        bc1 = f32(1.0 - math.pow(self.b1, tp))
        bc2 = f32(1.0 - math.pow(self.b2, tp))
        omb1 = f32(1 - _q(self.b1))
        omb2 = f32(1 - _q(self.b2))
        for d in range(self.D):
            a = f32(_q(omb1) * _q(g[d]))
            m1 = fma32(self.b1, self.m1[d], a)
            b = f32(_q(omb2) * _q(f32(_q(g[d]) ** 2)))
            v = fma32(self.b2, self.v[d], b)
            mhat = f32(_q(m1) / _q(bc1))
            vhat = f32(_q(v) / _q(bc2))
            den = f32(_q(f32(math.sqrt(vhat))) + _q(self.eps))
            q = f32(_q(mhat) / _q(den))
            self.m[d] = fma32(-self.lr, q, self.m[d])
            self.m1[d], self.v[d] = m1, v
        self.t += 1
        used = (self.sigma, self.lr)
        self.sigma = max(f32(_q(self.sigma) * _q(self.sd)), self.sf)
        self.lr = max(f32(_q(self.lr) * _q(self.ld)), self.lf)
        return {"E": E, "X": X, "fitness": f, "y": y, "g": g, "pen": pen, "sigma_lr": used}


def _dsqrt(q):
    """60-digit square root of an exact rational, as a Fraction."""
    from decimal import Decimal, getcontext
    getcontext().prec = 60
    q = _q(q)
    return Fraction((Decimal(q.numerator) / Decimal(q.denominator)).sqrt())


class BruteFamily:
    """R=1 PGPE / SNES / OpenAI-ES+ClipUp generation with per-dimension sigma,
    in exact rationals: the sums over pairs are exact, every fp32 result is
    rounded once (``f32``); square roots to 60 digits, exp in fp64."""

    def __init__(self, strategy, problem, D, N, sigma, lr, seed, lo, hi, sigma_lr=0.2, max_change=0.2,
                 optimizer="adam", max_speed=0.3, momentum=0.9, beta=12.0, b1=0.9, b2=0.999, eps=1e-8):
        self.strategy, self.problem, self.D, self.N = strategy, problem, D, N
        self.sig = [f32(sigma)] * D
        self.lr, self.seed = f32(lr), seed
        self.slr, self.mc = f32(sigma_lr), f32(max_change)
        self.opt, self.vmax, self.mom, self.beta = optimizer, f32(max_speed), f32(momentum), beta
        self.b1, self.b2, self.eps = f32(b1), f32(b2), f32(eps)
        self.m = init_uniform(seed, D, lo, hi)
        self.m1, self.v, self.vel = [0.0] * D, [0.0] * D, [0.0] * D
        self.t = 0

    def _adam(self, g):
        tp = self.t + 1
        bc1, bc2 = f32(1.0 - math.pow(self.b1, tp)), f32(1.0 - math.pow(self.b2, tp))
        omb1, omb2 = f32(1 - _q(self.b1)), f32(1 - _q(self.b2))
        for d in range(self.D):
            m1 = fma32(self.b1, self.m1[d], f32(_q(omb1) * _q(g[d])))
            v = fma32(self.b2, self.v[d], f32(_q(omb2) * _q(f32(_q(g[d]) ** 2))))
            den = f32(_q(f32(math.sqrt(f32(_q(v) / _q(bc2))))) + _q(self.eps))
            self.m[d] = fma32(-self.lr, f32(_q(f32(_q(m1) / _q(bc1))) / _q(den)), self.m[d])
            self.m1[d], self.v[d] = m1, v

    def _clipup(self, g):
        gg = sum(_q(x) ** 2 for x in g)
        inv = f32(1 / _dsqrt(gg)) if gg > 0 else 0.0
        vel = [fma32(self.lr, f32(_q(g[d]) * _q(inv)), f32(_q(self.mom) * _q(self.vel[d]))) for d in range(self.D)]
        nv = _dsqrt(sum(_q(x) ** 2 for x in vel))
        if nv > _q(self.vmax):
            sc = f32(_q(self.vmax) / nv)
            vel = [f32(_q(x) * _q(sc)) for x in vel]
        self.vel = vel
        self.m = [f32(_q(self.m[d]) - _q(vel[d])) for d in range(self.D)]

    def generation(self):
        P, D, N = self.N // 2, self.D, self.N
        Z = [eps_vector(self.seed, 0, p, self.t, D) for p in range(P)]
        X = [[fma32(self.sig[d] if j < P else -self.sig[d], Z[j % P][d], self.m[d]) for d in range(D)]
             for j in range(N)]
        f = [fitness(self.problem, x) for x in X]
        rk = ranks(f)
        if self.strategy == "snes":
            S = math.fsum(math.exp(self.beta * (k / N - 0.5)) for k in range(N))
            tab = [f32(math.exp(self.beta * (k / N - 0.5)) / S) for k in range(N)]
            w = [tab[N - 1 - r] for r in rk]
            a = [f32(_q(w[p]) - _q(w[p + P])) for p in range(P)]
            b = [f32(_q(w[p]) + _q(w[p + P])) for p in range(P)]
        else:
            y = [f32(Fraction(2 * r - (N - 1), 2 * (N - 1))) for r in rk]
            ybar = sum(_q(v) for v in y) / N
            a = [f32(_q(y[p]) - _q(y[p + P])) for p in range(P)]
            b = [f32(Fraction(1, 2) * (_q(y[p]) + _q(y[p + P])) - ybar) for p in range(P)]
        A = [sum(_q(a[p]) * _q(Z[p][d]) for p in range(P)) for d in range(D)]
        B = [sum(_q(b[p]) * (_q(Z[p][d]) ** 2 - 1) for p in range(P)) for d in range(D)]
        if self.strategy == "snes":
            h = f32(Fraction(1, 2) * _q(self.slr))
            for d in range(D):
                self.m[d] = fma32(f32(_q(self.lr) * _q(self.sig[d])), f32(A[d]), self.m[d])
                self.sig[d] = f32(_q(self.sig[d]) * _q(f32(math.exp(f32(_q(h) * _q(f32(B[d])))))))
            g = None
        else:
            if self.strategy == "pgpe":
                g = [f32(_q(self.sig[d]) * A[d] / N) for d in range(D)]
            else:  # OpenAI-ES: g = E^T y / (N sigma) over the unfolded population
                g = [f32(A[d] / (N * _q(self.sig[d]))) for d in range(D)]
            if self.opt == "clipup":
                self._clipup(g)
            else:
                self._adam(g)
            if self.strategy == "pgpe":
                for d in range(D):
                    sg = f32(_q(self.sig[d]) * B[d] / P)
                    dlt = -f32(_q(self.slr) * _q(sg))
                    lim = f32(_q(self.mc) * _q(self.sig[d]))
                    dlt = min(max(dlt, -lim), lim)
                    self.sig[d] = f32(_q(self.sig[d]) + _q(dlt))
        self.t += 1
        return {"X": X, "fitness": f, "g": g, "A": A, "B": B}


class BruteSepCMA:
    """R=1 Sep-CMA-ES generation (Ros & Hansen 2008) with independent members
    (row = member index): exact rational recombination sums, fp64 updates, one
    fp32 rounding per stored value.  Settings as the oracle's readings."""

    def __init__(self, problem, D, N, sigma, seed, lo, hi, elite_ratio=0.5):
        self.problem, self.D, self.N, self.seed = problem, D, N, seed
        self.mu = max(1, int(math.floor(elite_ratio * N)))
        wr = [math.log(self.mu + 0.5) - math.log(i + 1) for i in range(self.mu)]
        sw = math.fsum(wr)
        self.w = [v / sw for v in wr]
        self.sigma = f32(sigma)
        self.m = init_uniform(seed, D, lo, hi)
        self.C, self.ps, self.pc = [1.0] * D, [0.0] * D, [0.0] * D
        self.t = 0

    def generation(self):
        D, N, mu, w = self.D, self.N, self.mu, self.w
        mu_eff = 1.0 / math.fsum(v * v for v in w)
        c_s = (mu_eff + 2.0) / (D + mu_eff + 5.0)
        d_s = 1.0 + 2.0 * max(0.0, math.sqrt((mu_eff - 1.0) / (D + 1.0)) - 1.0) + c_s
        c_c = (4.0 + mu_eff / D) / (D + 4.0 + 2.0 * mu_eff / D)
        c1 = 2.0 / ((D + 1.3) ** 2 + mu_eff)
        cmu = min(1.0 - c1, 2.0 * (mu_eff - 2.0 + 1.0 / mu_eff) / ((D + 2.0) ** 2 + mu_eff))
        c1 = min(1.0, c1 * (D + 2.0) / 3.0)
        cmu = min(1.0 - c1, cmu * (D + 2.0) / 3.0)
        chi = math.sqrt(D) * (1.0 - 1.0 / (4.0 * D) + 1.0 / (21.0 * D * D))
        s = [f32(_q(self.sigma) * _q(f32(math.sqrt(self.C[d])))) for d in range(D)]
        Z = [eps_vector(self.seed, 0, j, self.t, D) for j in range(N)]
        X = [[fma32(s[d], Z[j][d], self.m[d]) for d in range(D)] for j in range(N)]
        f = [fitness(self.problem, x) for x in X]
        rk = ranks(f)
        elite = [0] * mu
        for j in range(N):
            if rk[j] < mu:
                elite[rk[j]] = j
        zw = [float(sum(_q(w[i]) * _q(Z[elite[i]][d]) for i in range(mu))) for d in range(D)]
        q = [float(sum(_q(w[i]) * _q(Z[elite[i]][d]) ** 2 for i in range(mu))) for d in range(D)]
        a_s = math.sqrt(c_s * (2.0 - c_s) * mu_eff)
        self.m = [f32(self.m[d] + s[d] * zw[d]) for d in range(D)]
        self.ps = [f32((1.0 - c_s) * self.ps[d] + a_s * zw[d]) for d in range(D)]
        nps = math.sqrt(math.fsum(v * v for v in self.ps))
        h = 1.0 if nps / math.sqrt(1.0 - (1.0 - c_s) ** (2.0 * (self.t + 1))) < (1.4 + 2.0 / (D + 1.0)) * chi else 0.0
        a_c = math.sqrt(c_c * (2.0 - c_c) * mu_eff)
        for d in range(D):
            Cd = self.C[d]
            self.pc[d] = f32((1.0 - c_c) * self.pc[d] + h * a_c * math.sqrt(Cd) * zw[d])
            self.C[d] = f32((1.0 - c1 - cmu) * Cd + c1 * (self.pc[d] ** 2 + (1.0 - h) * c_c * (2.0 - c_c) * Cd)
                            + cmu * Cd * q[d])
        self.sigma = f32(self.sigma * math.exp((c_s / d_s) * (nps / chi - 1.0)))
        self.t += 1
        return {"X": X, "fitness": f, "elite": elite, "h": h}
