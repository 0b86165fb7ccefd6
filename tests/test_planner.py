"""The planner of the system-planning phase (Section 4.3 "System Planning Phase", Algorithm 2):
the oracle's exhaustive search pinned by closed forms, the memory bound,
scaling and symmetry properties, and the library's vfl_plan against the
oracle on random profiles (host only, no GPU)."""
import math

import numpy as np
import pytest

from oracle import planner as OP


def _party(lam=1.0, gamma=1.0, phi=1.0, beta=1.0, top=(0.0, 0.0, 0.0, 0.0), cores=8.0,
           w=(1, 4), mem=(0.0, 0.0, 0.0)):
    return dict(lam=lam, gamma=gamma, phi=phi, beta=beta, lam_top=top[0], gamma_top=top[1],
                phi_top=top[2], beta_top=top[3], cores=cores, w_min=w[0], w_max=w[1],
                mem_base=mem[0], mem_coef=mem[1], mem_cap=mem[2])


LINK0 = dict(emb=0.0, grad=0.0, bandwidth=1.0, chi=1.0)
BATCHES = [16, 32, 64, 128, 256, 512, 1024]


def test_linear_profiles_closed_form():
    """Exponents 1, no exchange, no memory bound: every delay grows with w
    and B, so the minimum is at the smallest of each, and its value is the
    larger party's (sum of coefficients) * B * w / C."""
    a = _party(lam=2.0, phi=3.0, top=(1.0, 1.0, 0.5, 1.0), cores=16.0, w=(2, 6))
    p = _party(lam=1.5, phi=2.5, cores=8.0, w=(3, 5))
    arg, cost = OP.plan(a, p, LINK0, BATCHES)
    assert arg == (2, 3, 16)
    ta = (2.0 + 3.0 + 1.0 + 0.5) * 16 * 2 / 16.0      # 13
    tp = (1.5 + 2.5) * 16 * 3 / 8.0                   # 24
    assert cost == pytest.approx(max(ta, tp), rel=1e-15)


def test_exchange_term():
    """The exchange adds B (E + G) / B_b to every candidate: with equal
    compute it decides nothing, and its value is exact."""
    a, p = _party(w=(1, 1)), _party(w=(1, 1))
    link = dict(emb=512.0, grad=256.0, bandwidth=1e6, chi=1.0)
    arg, cost = OP.plan(a, p, link, [64])
    assert arg == (1, 1, 64)
    assert cost == pytest.approx(2.0 * 64 / 8.0 + 64 * 768 / 1e6, rel=1e-15)


def test_memory_bound_caps_the_batch():
    """Delays that fall with B (negative exponents) make the largest batch
    the best; the memory model's cap ((cap - base) / coef) ** (1 / chi)
    removes the larger candidates.  Here party B's cap, 300 ** 1 = 300,
    binds before party A's (1000 ** (1/1) over coef 2: 500)."""
    a = _party(gamma=-0.5, beta=-0.5, mem=(100.0, 2.0, 1100.0))
    p = _party(gamma=-0.5, beta=-0.5, mem=(50.0, 1.0, 350.0))
    link = dict(LINK0)
    assert OP.batch_cap(a, 1.0) == pytest.approx(500.0)
    assert OP.batch_cap(p, 1.0) == pytest.approx(300.0)
    arg, _ = OP.plan(a, p, link, BATCHES)
    assert arg[2] == 256
    # chi = 2: caps sqrt(500) = 22.4 and sqrt(300) = 17.3
    arg2, _ = OP.plan(a, p, dict(link, chi=2.0), BATCHES)
    assert arg2[2] == 16
    # nothing feasible
    assert OP.plan(a, _party(mem=(50.0, 1.0, 60.0)), dict(link, chi=1.0), BATCHES) is None


def test_more_cores_never_cost_more_and_swap_symmetry():
    rng = np.random.default_rng(5)
    for _ in range(50):
        a = _party(lam=rng.uniform(0.1, 3), gamma=rng.uniform(0.5, 1.5), phi=rng.uniform(0.1, 3),
                   beta=rng.uniform(0.5, 1.5), cores=rng.uniform(4, 32), w=(1, int(rng.integers(1, 6))))
        p = _party(lam=rng.uniform(0.1, 3), gamma=rng.uniform(0.5, 1.5), phi=rng.uniform(0.1, 3),
                   beta=rng.uniform(0.5, 1.5), cores=rng.uniform(4, 32), w=(1, int(rng.integers(1, 6))))
        link = dict(emb=rng.uniform(0, 100), grad=rng.uniform(0, 100), bandwidth=1e3, chi=1.0)
        _, c1 = OP.plan(a, p, link, BATCHES)
        _, c2 = OP.plan(dict(a, cores=2 * a["cores"]), dict(p, cores=2 * p["cores"]), link, BATCHES)
        assert c2 <= c1
        _, c3 = OP.plan(p, a, link, BATCHES)          # bottoms only: the parties swap
        assert c3 == pytest.approx(c1, rel=1e-14)


def _lib_party(V, q):
    s = V.vfl_plan_party()
    s.lambda_, s.gamma, s.phi, s.beta = q["lam"], q["gamma"], q["phi"], q["beta"]
    s.lambda_top, s.gamma_top, s.phi_top, s.beta_top = (q["lam_top"], q["gamma_top"], q["phi_top"],
                                                        q["beta_top"])
    s.cores, s.w_min, s.w_max = q["cores"], q["w_min"], q["w_max"]
    s.mem_base, s.mem_coef, s.mem_cap = q["mem_base"], q["mem_coef"], q["mem_cap"]
    return s


def test_library_equals_oracle():
    from paper_2510_12494_amd import vfl as V
    rng = np.random.default_rng(6)
    for _ in range(300):
        def rnd(top):
            return _party(lam=rng.uniform(0.01, 5), gamma=rng.uniform(-1, 2), phi=rng.uniform(0.01, 5),
                          beta=rng.uniform(-1, 2),
                          top=(rng.uniform(0, 2), rng.uniform(-1, 2), rng.uniform(0, 2), rng.uniform(-1, 2))
                          if top else (0.0, 0.0, 0.0, 0.0),
                          cores=rng.uniform(1, 64), w=(int(rng.integers(1, 4)), int(rng.integers(4, 12))),
                          mem=(rng.uniform(0, 10), rng.uniform(0, 0.2), rng.uniform(20, 200)))
        a, p = rnd(True), rnd(False)
        link = dict(emb=rng.uniform(0, 1e3), grad=rng.uniform(0, 1e3), bandwidth=rng.uniform(1e3, 1e6),
                    chi=rng.uniform(0.5, 2))
        batches = sorted(rng.choice(BATCHES, size=int(rng.integers(1, 7)), replace=False).tolist())
        ref = OP.plan(a, p, link, batches)
        lv = V.vfl_plan_link()
        lv.emb_bytes_per_row, lv.grad_bytes_per_row, lv.bandwidth, lv.chi = (link["emb"], link["grad"],
                                                                           link["bandwidth"], link["chi"])
        if ref is None:
            with pytest.raises(V.VflError):
                V.vfl_plan(_lib_party(V, a), _lib_party(V, p), lv, batches)
            continue
        arg, cost = V.vfl_plan(_lib_party(V, a), _lib_party(V, p), lv, batches)
        assert arg == tuple(int(x) for x in ref[0])
        assert cost == pytest.approx(ref[1], rel=1e-12)


# ---------------------------------------------------- delay-model fitting
def test_fit_recovers_exact_power_laws():
    """Times that follow coef * B**exp exactly (positive, zero and negative
    exponents, as in the Appendix's Table 7) give back coef and exp."""
    B = [16, 32, 64, 128, 256, 512, 1024]
    for coef, expo in [(0.018, -0.8015), (0.010, -1.0071), (3.5e-6, 1.0), (2.0e-4, 0.0),
                       (7.0e-9, 1.37)]:
        T = [coef * b ** expo for b in B]
        c, e = OP.fit_power_law(B, T)
        assert c == pytest.approx(coef, rel=1e-12) and e == pytest.approx(expo, abs=1e-12)


def test_fit_two_points_is_the_secant():
    """Two points: the exponent is the slope log(T2/T1) / log(B2/B1) and the
    line passes through both."""
    c, e = OP.fit_power_law([100.0, 400.0], [2.0, 5.0])
    assert e == pytest.approx(math.log(2.5) / math.log(4.0), rel=1e-14)
    assert c * 100.0 ** e == pytest.approx(2.0, rel=1e-13)


def test_fit_minimises_the_log_residuals():
    """Noisy times: the fitted line has zero mean log residual and residuals
    orthogonal to log B (the normal equations), and moving either constant
    raises the squared residual."""
    rng = np.random.default_rng(3)
    B = np.array([16, 32, 64, 128, 256, 512, 1024], float)
    T = 0.02 * B ** -0.7 * np.exp(rng.normal(0, 0.1, B.size))
    c, e = OP.fit_power_law(B, T)
    r = np.log(T) - np.log(c) - e * np.log(B)
    assert abs(r.sum()) < 1e-12 and abs((r * np.log(B)).sum()) < 1e-11
    sse = lambda cc, ee: float(((np.log(T) - np.log(cc) - ee * np.log(B)) ** 2).sum())
    for dc, de in [(1.01, 0), (0.99, 0), (1, 0.01), (1, -0.01)]:
        assert sse(c * dc, e + de) > sse(c, e)


def test_library_fit_equals_oracle():
    from paper_2510_12494_amd import vfl as V
    rng = np.random.default_rng(11)
    for _ in range(50):
        n = int(rng.integers(2, 12))
        B = np.sort(rng.choice(np.arange(1, 40000), n, replace=False)).astype(float)
        T = np.exp(rng.normal(-8, 2)) * B ** rng.normal(0, 1) * np.exp(rng.normal(0, 0.2, n))
        c1, e1 = OP.fit_power_law(B, T)
        c2, e2 = V.vfl_fit_delay(list(B), list(T))
        assert c2 == pytest.approx(c1, rel=1e-9) and e2 == pytest.approx(e1, rel=1e-9, abs=1e-12)
    for bad in ([1.0], [2.0, 2.0], [0.0, 3.0]):
        with pytest.raises(V.VflError):
            V.vfl_fit_delay(bad, [1.0] * len(bad))
