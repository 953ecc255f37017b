"""Pins of the oracle's regime controller (controller 2): the latency model of
Eq. latency-superlinear used as the TTFT stand-in, the EWMA of
Eq. saturation-signal, the regimes of Eq. saturation-state with k-sample
hysteresis, and the (tau, w_ov) of each regime inside an episode."""
import math

import numpy as np
import pytest

import brute
from paper_2606_17081_amd import workload as wl

RP = wl.REGIME_PARAMS


def test_latency_model_closed_form(orc):
    # f(n) = 0.005 n + 0.02 + 0.01 / max(64 - n, 1)^2, by hand
    assert orc.latency(0) == pytest.approx(0.02 + 0.01 / 4096, rel=1e-15)
    assert orc.latency(32) == pytest.approx(0.16 + 0.02 + 0.01 / 1024, rel=1e-15)
    assert orc.latency(63) == pytest.approx(0.315 + 0.02 + 0.01, rel=1e-15)
    assert orc.latency(64) == pytest.approx(0.32 + 0.02 + 0.01, rel=1e-15)       # pole guarded
    assert orc.latency(100) == pytest.approx(0.5 + 0.02 + 0.01, rel=1e-15)
    r3 = dict(RP, beta=3, d=2.0, n_sat=10)
    assert orc.latency(7, r3) == pytest.approx(0.035 + 0.02 + 2.0 / 27, rel=1e-15)
    v = [orc.latency(n) for n in range(0, 64)]
    assert all(b > a for a, b in zip(v, v[1:]))                                 # convex rise to the pole


def _run(orc, lats, regime=None):
    st = [0.0, 0, 0, 0]
    out = []
    for t, l in enumerate(lats):
        orc.regime_step(l, t, st, regime)
        out.append((st[0], st[1]))
    return out


def test_ewma_step_response(orc):
    a, th1, k = RP["alpha"], RP["theta1"], RP["k"]
    L1, L2 = 0.1, 0.5
    tr = _run(orc, [L1] + [L2] * 40)
    for m in range(1, 41):                      # ewma after m samples of L2
        assert tr[m][0] == pytest.approx(L2 + (L1 - L2) * (1 - a) ** m, rel=1e-12)
    # the first sample above theta1, then k of them in a row switch to Transition
    m0 = next(m for m in range(1, 41) if L2 + (L1 - L2) * (1 - a) ** m > th1)
    regimes = [r for _, r in tr]
    assert regimes.index(1) == m0 + k - 1
    assert max(regimes) == 1                    # theta2 = 2 s is never reached at 0.5 s


def test_saturated_and_back(orc):
    k, th2, eps = RP["k"], RP["theta2"], RP["eps"]
    tr = _run(orc, [0.5] * 10 + [5.0] * 20 + [0.05] * 60)
    regimes = [r for _, r in tr]
    assert 2 in regimes
    first_sat = regimes.index(2)
    # Saturated needs k consecutive samples with ewma >= theta2 while in Transition
    assert all(e >= th2 for e, _ in tr[first_sat - k + 1:first_sat + 1])
    # back down one regime at a time, each after k samples below the lower margin
    down = [i for i in range(1, len(regimes)) if regimes[i] < regimes[i - 1]]
    assert [regimes[i] for i in down] == [1, 0]
    assert all(e < th2 - eps for e, _ in tr[down[0] - k + 1:down[0] + 1])
    assert all(e < RP["theta1"] - eps for e, _ in tr[down[1] - k + 1:down[1] + 1])


def test_hysteresis_suppresses_chatter(orc):
    # 0 and L alternating: the ewma settles between 0.3 L / 0.51 and 0.7 times that, i.e.
    # around theta1 for L = 0.6; with k = 3 no switch, with k = 1 the regime chatters
    lats = [0.6 if i % 2 else 0.0 for i in range(80)]
    tr = _run(orc, lats)
    es = [e for e, _ in tr][40:]
    assert es[1::2] == pytest.approx([0.3 * 0.6 / 0.51] * len(es[1::2]), rel=1e-5)
    assert all(e > RP["theta1"] for e in es[1::2]) and all(e < RP["theta1"] for e in es[0::2])
    assert all(r == 0 for _, r in tr)
    tr1 = _run(orc, lats, dict(RP, k=1))
    assert any(r == 1 for _, r in tr1)


@pytest.mark.parametrize("seed", range(8))
def test_episode_regime_controller_matches_twin(orc, seed):
    from test_oracle_episode import _flat_chains, _random_case
    rng = np.random.default_rng(9100 + seed)
    W, cache, spec, turn_off, turn_blocks, chains = _random_case(rng, multiturn=seed % 2 == 1)
    # a latency model that saturates at a few requests, so the small episode visits every regime
    reg = dict(RP, a=0.2, b=0.0, d=0.5, n_sat=4, theta1=0.5, theta2=1.5, eps=0.1, k=2, tau=(0.0, 0.7, 3.0))
    spec.controller = 2
    n = int(turn_off[-1])
    rand = rng.integers(0, 1 << 32, size=2 * n, dtype=np.uint64).astype(np.uint32)
    flat, off = _flat_chains(chains)
    out = orc.simulate_episode(W, cache, spec, turn_off, turn_blocks, off, flat, rand=rand, regime=reg)
    state = [0.0, 0, 0, 0]

    def step(nf, t):
        orc.regime_step(orc.latency(nf, reg), t, state, reg)
        return state[1]

    fns = (lambda r: (reg["tau"][r], reg["w_ov"][r]), step,
           lambda costs, t, tau: orc.select(wl.POLICY_SOFTMAX, tau, np.array(costs, np.float32), t,
                                            int(rand[2 * t]), int(rand[2 * t + 1])))
    routes, _ = brute.episode(W, cache, spec.hold_steps, spec.routes_per_step, spec.w_ov, spec.w_act,
                              spec.w_sat, spec.cap, turn_off, turn_blocks, chains, 2, regime=fns)
    assert [r["worker"] for r in routes] == out["route_worker"].tolist()
    assert [r["regime"] for r in routes] == out["route_regime"].tolist()
    assert [r["cost"] for r in routes] == [list(c) for c in out["cost"]]
    assert out["totals"][3] == sum(r["regime"] > 0 for r in routes)
