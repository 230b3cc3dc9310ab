"""The partition controller Phi (include/vla_suffix.h, vla_sched_*), on the CPU.

Pins: its predictions against the stream interval of Eq. (13) written out
here, its decisions against a brute-force search over the same candidate
set, and its fitted stage model against noiseless samples of a known line."""
import itertools
import random

import pytest

from paper_2608_14586_amd import binding as vb


def eq13(a, b, c, x, N, k, ug=0.0, uc=0.0):
    g = (a + b * k) / (1 - ug)
    cpu = c * (N - k) / (1 - uc)
    return g, cpu, max(g, (x if k < N else 0.0) + cpu)


def test_predict_is_eq13():
    s = vb.Sched(32, 8, 32, 16, 296.0, 7.0, 23.44, 0.41)
    for k, ug, uc in itertools.product(range(8, 33), (0.0, 0.3), (0.0, 0.6)):
        got = s.vla_sched_predict(k, ug, uc)
        want = eq13(296.0, 7.0, 23.44, 0.41, 32, k, ug, uc)
        assert all(abs(g - w) <= 1e-4 * max(1.0, abs(w)) for g, w in zip(got, want)), (k, got, want)


def test_decide_matches_brute_force():
    rng = random.Random(7)
    for trial in range(300):
        N = rng.randint(4, 40)
        k_lo = rng.randint(0, N)
        k_hi = rng.randint(k_lo, N)
        k0 = rng.randint(k_lo, k_hi)
        a, b, c, x = (rng.uniform(0, 50), rng.uniform(0, 10), rng.uniform(0, 50), rng.uniform(0, 2))
        bhi = rng.randint(1, 4)
        s = vb.Sched(N, k_lo, k_hi, k0, a, b, c, x, backlog_hi=bhi)
        k = k0
        for step in range(6):
            ug, uc = rng.choice((0.0, 0.5, 0.9)), rng.choice((0.0, 0.5))
            q = rng.randint(0, 4)
            budget = rng.choice((0.0, rng.uniform(1, 200)))
            got = s.vla_sched_decide(ug, uc, q, budget)
            lo = max(k_lo, k if q >= bhi else k - 1)
            hi = min(k_hi, k + 1)
            best = None
            for cand in range(lo, hi + 1):
                g, _, t = eq13(a, b, c, x, N, cand, ug, uc)
                fits = budget <= 0 or g <= budget
                key = (not fits, t if fits else g, cand)
                if best is None or key < best[0]:
                    best = (key, cand)
            # float32 inside the library: accept an exact tie broken either way
            if got != best[1]:
                tg = eq13(a, b, c, x, N, got, ug, uc)
                tb = eq13(a, b, c, x, N, best[1], ug, uc)
                assert abs(tg[2] - tb[2]) <= 1e-4 * max(1.0, tb[2]), (trial, step, got, best)
            k = got


def test_converges_to_all_gpu_on_this_machine():
    # the measured MI355X + EPYC stage model: 36 ms GPU stage at k = 32, 123 ms per host block
    s = vb.Sched(32, 24, 32, 28, 8.5, 0.86, 123.0, 0.31)
    ks = [s.vla_sched_decide() for _ in range(6)]
    assert ks == [29, 30, 31, 32, 32, 32]


def test_paper_stage_model_balances_the_stages():
    # Table III's L20 + Xeon numbers (a = 296 ms, b = 7 ms, c = 23.44 ms per block):
    # GPU and host stages cross between k = 14 and 15
    s = vb.Sched(32, 8, 24, 8, 296.0, 7.0, 23.44, 0.41)
    ks = [s.vla_sched_decide() for _ in range(10)]
    assert ks[-1] == 15 and ks[:7] == [9, 10, 11, 12, 13, 14, 15]
    # a GPU module taking half the GPU moves the balance towards the host
    ks = [s.vla_sched_decide(u_gpu=0.5) for _ in range(10)]
    g, c, t = s.vla_sched_predict(ks[-1], 0.5, 0.0)
    assert ks[-1] < 15 and all(s.vla_sched_predict(k, 0.5, 0.0)[2] >= t for k in range(8, 25))


def test_backlog_blocks_moves_towards_the_host():
    s = vb.Sched(32, 8, 24, 20, 296.0, 7.0, 23.44, 0.41, backlog_hi=2)
    assert s.vla_sched_decide(0.0, 0.0, 2) == 20      # would go to 19, but the queue is full
    assert s.vla_sched_decide(0.0, 0.0, 1) == 19


def test_gpu_budget_reserves_gpu_time():
    s = vb.Sched(32, 8, 24, 16, 296.0, 7.0, 23.44, 0.41)
    # a budget of 390 ms on the GPU stage forces k <= 13 (296 + 7 k <= 390)
    ks = [s.vla_sched_decide(gpu_budget_ms=390.0) for _ in range(5)]
    assert ks == [15, 14, 13, 13, 13]


def test_observe_recovers_a_known_model():
    s = vb.Sched(32, 0, 32, 16, 100.0, 1.0, 1.0, 1.0)
    for k in (16, 20, 16, 24, 18):
        s.vla_sched_observe(k, 9.0 + 0.86 * k, 0.3, 123.0 * (32 - k))
    a, b, c, x = s.vla_sched_model()
    assert abs(a - 9.0) < 1e-3 and abs(b - 0.86) < 1e-4 and abs(c - 123.0) < 1e-3 and abs(x - 0.3) < 1e-6


def test_observe_single_k_moves_only_the_intercept():
    s = vb.Sched(32, 0, 32, 16, 0.0, 1.0, 1.0, 0.0)
    for _ in range(3):
        s.vla_sched_observe(16, 50.0, 0.3, 160.0)
    a, b, c, x = s.vla_sched_model()
    assert abs(b - 1.0) < 1e-6 and abs(a - 34.0) < 1e-4 and abs(c - 10.0) < 1e-4


@pytest.mark.parametrize("args", [
    (0, 0, 0, 0, 1, 1, 1, 1, 1), (8, 4, 2, 3, 1, 1, 1, 1, 1), (8, 2, 4, 5, 1, 1, 1, 1, 1),
    (8, 2, 4, 3, -1, 1, 1, 1, 1), (8, 2, 4, 3, 1, 1, 1, 1, 0), (8, 2, 9, 3, 1, 1, 1, 1, 1)])
def test_create_rejects_bad_arguments(args):
    with pytest.raises(vb.VlaError) as e:
        vb.Sched(*args)
    assert e.value.name == "VLA_ERR_INVALID_ARG"


def test_decide_rejects_full_utilisation():
    s = vb.Sched(8, 2, 6, 4, 1, 1, 1, 1)
    with pytest.raises(vb.VlaError):
        s.vla_sched_decide(u_gpu=1.0)
