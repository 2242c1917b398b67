"""Pins of the planner oracle (Sec. 3.2, Alg. 1, Eqs. 1 and 4-8) against closed
forms, hand-computed cases, an independent sort, and the C oracle's Eq. 1."""
import math

import numpy as np
import pytest

import oracle
from oracle import planner as P


def test_eq7_target_bytes():
    assert P.target_bytes(10, 8, 4096) == 0          # more free blocks than the threshold
    assert P.target_bytes(9, 8, 4096) == 0
    assert P.target_bytes(8, 8, 4096) == 4096        # threshold + 1 - free = 1 block
    assert P.target_bytes(0, 8, 1 << 21) == 9 << 21


def test_eq4_global_damage():
    assert P.global_damage(1.0, 3.5) == 2.5
    assert P.global_damage(2.0, 1.0) == 0.0          # never negative


def test_eq6_residual_scale():
    w, a, c = [0.5, -1.0, 2.0], 0.25, 0.8
    phi = [1.0, 0.5, 0.125]
    rho = 0.5 - 0.5 + 0.25 + 0.25                    # w . phi + a = 0.5
    assert P.residual_scale(w, a, c, phi, 0.0, -1, 1) == 1.0            # alpha = 0
    assert math.isclose(P.residual_scale(w, a, c, phi, 1.5, -1, 1), math.exp(1.5 * 0.8 * rho), rel_tol=1e-15)
    assert math.isclose(P.residual_scale(w, a, c, phi, 1.0, -1, 0.1), math.exp(0.8 * 0.1), rel_tol=1e-15)
    assert math.isclose(P.residual_scale(w, -9.0, c, phi, 1.0, -0.3, 1), math.exp(-0.8 * 0.3), rel_tol=1e-15)


def test_eq8_damage_floor():
    assert P.predicted_damage(2.0, 0.0, 5.0, 1e-6) == 1e-6
    assert P.predicted_damage(2.0, 3.0, 0.5, 1e-6) == 3.0


def test_routing_stats_hand_case_and_eq1():
    # 3 tokens, 2 experts, top-1: rows with norms 5, 1, 2
    rows = np.array([[3.0, 4.0], [1.0, 0.0], [0.0, 2.0]])
    ids = np.array([[0], [1], [0]], np.int32)
    w = np.array([[0.5], [1.0], [0.25]], np.float32)
    _, off, ss, _ = oracle.permute(ids, 2)
    st = P.routing_stats(rows, ss // 1, w, off, ss)
    np.testing.assert_array_equal(st[0], [0.75, 2, 0.5 * 5 + 0.25 * 2, 0.5 * 25 + 0.25 * 4, 5.0])
    np.testing.assert_array_equal(st[1], [1.0, 1, 1.0, 1.0, 1.0])
    m, phi = P.mass_and_features(st)
    np.testing.assert_allclose(m, [0.75 / 1.75, 1.0 / 1.75], rtol=1e-15)
    np.testing.assert_allclose(phi[0], [3.0 / 0.75, math.sqrt(13.5 / 0.75), 5.0], rtol=1e-15)


def test_routing_mass_matches_the_c_oracle():
    rng = np.random.default_rng(7)
    T, E, K = 50, 8, 2
    ids, w = oracle.route(rng.standard_normal((T, E)).astype(np.float32), K)
    _, off, ss, _ = oracle.permute(ids, E)
    rows = rng.standard_normal((T, 16))
    st = P.routing_stats(rows, ss // K, w, off, ss)
    m, _ = P.mass_and_features(st)
    np.testing.assert_allclose(m, oracle.routing_mass(ids, w.astype(np.float64), E), rtol=1e-12, atol=1e-15)
    assert abs(m.sum() - 1.0) < 1e-12
    assert st[:, 1].sum() == T * K


def test_buckets_by_mass():
    b = P.buckets(np.array([0.1, 0.4, 0.2, 0.3]), [0.25, 0.25, 0.5])
    np.testing.assert_array_equal(b, [2, 0, 2, 1])
    b = P.buckets(np.array([0.25, 0.25, 0.25, 0.25]), [0.5, 0.5])   # ties go to the lower index
    np.testing.assert_array_equal(b, [0, 0, 1, 1])


def _units(rng, n, E):
    us = []
    for i in range(n):
        m16 = int(rng.integers(4, 16)) * 4096
        s = np.sort(rng.uniform(0, 1, 3))           # s^16 <= s^8 <= s^4
        us.append(P.Unit(int(rng.integers(0, E)), int(rng.integers(0, 2)), (m16, m16 // 2 + 256, m16 // 4 + 256),
                         (float(s[0]), float(s[1]), float(s[2]))))
    return us


def test_greedy_one_level_is_the_sorted_prefix():
    """Units at 16 bits and floors at 8: each unit has one step, so the plan is
    the shortest prefix of the units sorted by damage per byte (independent
    numpy sort) that reaches the target."""
    rng = np.random.default_rng(3)
    E, n = 4, 40
    us = _units(rng, n, E)
    cfg = P.Config(bucket_frac=[0.5, 0.5], mult=[3.0, 1.0], floors=[[8, 8]], alpha=0.0)
    mass = np.array([0.4, 0.3, 0.2, 0.1])
    phi = np.zeros((E, 2, 3))
    bucket_of = P.buckets(mass, cfg.bucket_frac)
    delta = np.array([u.nbytes[0] - u.nbytes[1] for u in us], np.float64)
    dmg = np.array([max(cfg.eps, cfg.mult[bucket_of[u.expert]] * max(u.sens[1] - u.sens[0], 0)) for u in us])
    order = np.lexsort((np.arange(n), dmg / delta))
    D = int(delta.sum() * 0.4)
    D_, plans, best = P.plan_step(cfg, us, [16] * n, mass, phi, free_blocks=0, threshold=D // 4096 - 1,
                                   kv_block_bytes=4096)
    assert D_ == (D // 4096) * 4096
    D = D_
    take, tot = [], 0
    for i in order:
        if tot >= D:
            break
        take.append(int(i))
        tot += delta[i]
    assert [s[0] for s in best.steps] == take and best.nbytes == tot and best.nbytes >= D


def test_greedy_lowers_one_level_at_a_time():
    """A unit's 8 -> 4 step is only available once its 16 -> 8 step was taken."""
    us = [P.Unit(0, 0, (100000, 50256, 25256), (0.0, 10.0, 10.0)),   # 16->8 dear, 8->4 free
          P.Unit(1, 0, (100000, 50256, 25256), (0.0, 1.0, 5.0))]
    cfg = P.Config(bucket_frac=[1.0], mult=[1.0], floors=[[4]], alpha=0.0, eps=1e-12)
    _, _, best = P.plan_step(cfg, us, [16, 16], np.array([0.5, 0.5]), np.zeros((2, 2, 3)), 0, 0, 60000)
    assert best.steps[0] == (1, 16, 8)
    assert best.steps[1] == (1, 8, 4)             # cheaper than unit 0's first step
    assert best.nbytes >= 60000
    assert best.final() == {1: (16, 4)}


def test_infeasible_target_takes_every_legal_step():
    rng = np.random.default_rng(5)
    us = _units(rng, 12, 3)
    cfg = P.Config(bucket_frac=[1 / 3, 1 / 3, 1 / 3], mult=[4.0, 2.0, 1.0], floors=[[16, 8, 8], [8, 8, 4]])
    mass = np.array([0.5, 0.3, 0.2])
    D, plans, best = P.plan_step(cfg, us, [16] * 12, mass, np.zeros((3, 2, 3)), 0, 10 ** 6, 1 << 20)
    b = P.buckets(mass, cfg.bucket_frac)
    legal = sum(u.nbytes[0] - (u.nbytes[2] if cfg.floors[1][b[u.expert]] == 4 else u.nbytes[1])
                for u in us if cfg.floors[1][b[u.expert]] <= 8)
    assert best.stage == 1 and best.nbytes == legal < D
    assert all(s[0] not in [i for i, u in enumerate(us) if b[u.expert] == 0] or s[2] >= 8 for s in best.steps)


def test_depth_caps_relax_only_when_needed():
    us = [P.Unit(e, 0, (8192, 4352, 2304), (0.0, 1.0, 2.0)) for e in range(2)]
    cfg = P.Config(bucket_frac=[0.5, 0.5], mult=[1.0, 1.0], floors=[[8, 8], [4, 4]], alpha=0.0)
    mass = np.array([0.6, 0.4])
    _, _, small = P.plan_step(cfg, us, [16, 16], mass, np.zeros((2, 2, 3)), 0, 0, 3840)
    assert small.stage == 0
    _, plans, big = P.plan_step(cfg, us, [16, 16], mass, np.zeros((2, 2, 3)), 0, 1, 4096)  # 8192 bytes
    assert plans[0].nbytes == 2 * 3840 < 8192 and big.stage == 1 and big.nbytes >= 8192


def test_hot_experts_are_protected():
    us = [P.Unit(e, 0, (8192, 4352, 2304), (0.0, 1.0, 2.0)) for e in range(4)]
    cfg = P.Config(bucket_frac=[0.25, 0.75], mult=[100.0, 1.0], floors=[[4, 4]], alpha=0.0)
    mass = np.array([0.1, 0.2, 0.6, 0.1])     # expert 2 is hot
    _, _, best = P.plan_step(cfg, us, [16] * 4, mass, np.zeros((4, 2, 3)), 0, 0, 15000)   # others: 17664 B
    assert all(s[0] != 2 for s in best.steps)


def test_no_pressure_no_plan():
    us = [P.Unit(0, 0, (8192, 4352, 2304), (0.0, 1.0, 2.0))]
    cfg = P.Config(bucket_frac=[1.0], mult=[1.0], floors=[[4]])
    D, plans, best = P.plan_step(cfg, us, [16], np.array([1.0]), np.zeros((1, 2, 3)), 20, 8, 4096)
    assert D == 0 and best is None and plans[0].steps == []


def test_prompt_residual_reorders_steps():
    """Two otherwise equal units of different types: the head of the type with a
    positive predicted residual makes its step dearer."""
    us = [P.Unit(0, P.GATE_UP, (8192, 4352, 2304), (0.0, 1.0, 2.0)),
          P.Unit(0, P.DOWN_T, (8192, 4352, 2304), (0.0, 1.0, 2.0))]
    hw = np.zeros((2, 2, 3))
    hw[P.GATE_UP, 0] = [1.0, 0.0, 0.0]
    cfg = P.Config(bucket_frac=[1.0], mult=[1.0], floors=[[8]], alpha=1.0, head_w=hw)
    phi = np.zeros((1, 2, 3))
    phi[0, P.GATE_UP] = [0.5, 0.0, 0.0]
    _, _, best = P.plan_step(cfg, us, [16, 16], np.array([1.0]), phi, 0, 0, 3840)
    assert best.steps == [(1, 16, 8)]


def test_merge_requests_weights():
    m1, m2 = np.array([1.0, 0.0]), np.array([0.0, 1.0])
    p1, p2 = np.ones((2, 2, 3)), 3 * np.ones((2, 2, 3))
    m, p = P.merge_requests([m1, m2], [p1, p2], [3.0, 1.0])
    np.testing.assert_allclose(m, [0.75, 0.25])
    np.testing.assert_allclose(p, 1.5 * np.ones((2, 2, 3)))
    m, p = P.merge_requests([m1], [p1], [7.0])
    np.testing.assert_array_equal(m, m1)
