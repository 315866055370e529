"""Cold-start controller arithmetic (CPU): hand-computed worked examples of
the TTFT / TPOT predictions, a brute-force check of Algorithm 1's server
selection, and the bandwidth bookkeeping of the placement policy."""
import itertools
import math

import pytest

from paper_2502_15524_amd.controller import (History, Server, ServerBandwidth, allocate,
                                             enumerate_choices, predict_tpot, predict_ttft,
                                             predict_ttft_overlapped, prefill_factor)

H = History(t_c=2.0, t_n=0.01, t_p=0.5, t_d=0.03)
M = 13.5e9
NET, PCIE = 2e9, 25e9          # 16 Gbit/s network, PCIe as in the paper's testbeds


def srv(name, b=NET, p=PCIE, mem=80e9, workers=0):
    return Server(name, b, p, mem, workers)


def test_prefill_factor_closed_forms():
    assert prefill_factor(1, 1) == 1.0          # one full worker: the whole model once
    assert prefill_factor(4, 0) == 4.0          # four low-memory workers, each as slow as one
    assert prefill_factor(4, 4) == 1.0          # four full workers, a quarter each
    assert prefill_factor(2, 1) == 1.5
    with pytest.raises(ValueError):
        prefill_factor(2, 3)


def test_ttft_worked_examples():
    # s = 1, w = 1: 2 + 13.5e9 (1/2e9 + 1/25e9) + 0.5 + 0.01 = 2 + 7.29 + 0.51
    assert math.isclose(predict_ttft(H, M, 1, 1, [srv("a")]), 9.8, rel_tol=1e-12)
    # s = 4, w = 0: 2 + 3.375e9 * 0.54e-9 + 0.5 * 4 + 0.04 = 5.8625
    assert math.isclose(predict_ttft(H, M, 4, 0, [srv(c) for c in "abcd"]), 5.8625,
                        rel_tol=1e-12)
    # the slowest server decides: one server at 1 GB/s network
    slow = [srv("a"), srv("b", b=1e9)]
    # s = 2, w = 2: 2 + 6.75e9 (1e-9 + 0.04e-9) + 0.5 + 0.02 = 9.54
    assert math.isclose(predict_ttft(H, M, 2, 2, slow), 9.54, rel_tol=1e-12)


def test_tpot_worked_examples():
    assert math.isclose(predict_tpot(H, 1, 1), 0.04, rel_tol=1e-12)
    assert math.isclose(predict_tpot(H, 4, 0), 0.16, rel_tol=1e-12)
    assert math.isclose(predict_tpot(H, 3, 1), 0.03 * (2 + 1 / 3) + 0.03, rel_tol=1e-12)


def test_overlapped_ttft():
    h = History(t_c=0, t_n=0.01, t_p=0.5, t_d=0.03, t_cc=1.0, t_cu=0.5, t_l=3.0)
    # loading 13.5e9/25e9 = 0.54 s hides under library loading (3 s); fetching
    # 6.75 s over the network dominates: 6.75 + 0.5 + 0.01
    assert math.isclose(predict_ttft_overlapped(h, M, 1, 1, [srv("a")]), 7.26, rel_tol=1e-12)
    # s = 4: fetching 3.375e9 / 2e9 = 1.6875 s < 1 + 0.5 + 3 = 4.5 s
    assert math.isclose(predict_ttft_overlapped(h, M, 4, 4, [srv(c) for c in "abcd"]),
                        4.5 + 0.5 + 0.04, rel_tol=1e-12)


def _best_max_ratio(servers, s, w):
    """Brute force: the smallest max(1/b + 1/p) over all choices of w servers
    holding M and s - w further servers holding M / s."""
    best = None
    for group in itertools.permutations(servers, s):
        if all(x.free_mem >= M for x in group[:w]) and all(x.free_mem >= M / s for x in group[w:]):
            r = max(1 / x.b + 1 / x.p for x in group)
            best = r if best is None else min(best, r)
    return best


def test_server_selection_is_the_best_possible_for_every_s_and_w():
    cluster = [srv("a", b=4e9, mem=30e9), srv("b", b=1e9, mem=80e9), srv("c", b=3e9, mem=80e9),
               srv("d", b=2e9, p=10e9, mem=5e9), srv("e", b=6e9, mem=4e9),
               srv("f", b=2.5e9, mem=14e9)]
    seen = 0
    for c in enumerate_choices(H, M, cluster):
        r = _best_max_ratio(cluster, c.s, c.w)
        assert r is not None
        expected = H.t_c + M / c.s * r + H.t_p * ((c.s - c.w) + c.w / c.s) + H.t_n * c.s
        assert math.isclose(c.ttft, expected, rel_tol=1e-12), (c.s, c.w)
        seen += 1
    # every (s, w) for which brute force finds a placement is enumerated
    possible = sum(1 for s in range(1, 5) for w in range(s + 1)
                   if _best_max_ratio(cluster, s, w) is not None)
    assert seen == possible


def test_placement_takes_fewest_busy_gpus_at_the_best_bottleneck():
    """Brute force over random clusters: each (s, w) group reaches the
    smallest possible slowest fetch-and-load rate, and among the groups that
    reach it, places the fewest workers on busy GPUs."""
    import random
    rnd = random.Random(7)
    for trial in range(60):
        cluster = [srv(chr(97 + i), b=rnd.choice([1e9, 2e9, 4e9]), p=rnd.choice([10e9, 25e9]),
                       mem=rnd.choice([4e9, 8e9, 16e9, 80e9]), workers=rnd.choice([0, 0, 1, 2]))
                   for i in range(6)]
        for c in enumerate_choices(H, M, cluster):
            best_r, best_busy = None, None
            for group in itertools.permutations(cluster, c.s):
                if not (all(x.free_mem >= M for x in group[:c.w]) and
                        all(x.free_mem >= M / c.s for x in group[c.w:])):
                    continue
                r = max(x.ratio for x in group)
                busy = sum(x.workers > 0 for x in group)
                if best_r is None or r < best_r or (r == best_r and busy < best_busy):
                    best_r, best_busy = r, busy
            assert max(x.ratio for x in c.servers) == best_r, (trial, c.s, c.w)
            assert c.sharing == best_busy, (trial, c.s, c.w)
            assert len(set(x.name for x in c.servers)) == c.s


def test_allocation_meets_slos_with_least_memory_on_free_gpus():
    cluster = [srv(c) for c in "abcd"]
    c = allocate(H, M, cluster, slo_ttft=6.0, slo_tpot=0.2)
    # feasible with w = 0 at s = 3 (5.96 s) and s = 4 (5.8625 s), both reserving
    # one model's memory; the smaller group wins
    assert (c.s, c.w) == (3, 0)
    assert c.ttft <= 6.0 and c.tpot <= 0.2
    # a busy GPU is avoided when a free one is available
    busy = [srv("a", workers=2), srv("b"), srv("c"), srv("d")]
    c = allocate(H, M, busy, slo_ttft=6.0, slo_tpot=0.2)
    assert all(x.workers == 0 for x in c.servers)
    # nothing meets the SLO: one full worker on the best server
    c = allocate(H, M, [srv("a", b=1e9), srv("b")], slo_ttft=1.0, slo_tpot=0.2)
    assert (c.s, c.w) == (1, 1) and c.servers[0].name == "b"


def test_bandwidth_bookkeeping_worked_example():
    sb = ServerBandwidth(B=1e9)
    assert sb.add("A", T=0.0, size=4e9, deadline=10.0)     # 4e9 <= 1e9 * 10
    # at T = 2, A has fetched 2e9 alone; with B sharing: A 2e9 <= 0.5e9 * 8,
    # B 3e9 <= 0.5e9 * 8
    assert sb.add("B", T=2.0, size=3e9, deadline=10.0)
    assert math.isclose(sb.workers["A"][0], 2e9)
    # at T = 4 (two workers for 2 s): A 1e9, B 2e9 pending; a third worker
    # with 1e9 due at T = 6 would get 1e9/3 * 2 < 1e9: rejected, state kept
    assert not sb.add("C", T=4.0, size=1e9, deadline=6.0)
    assert math.isclose(sb.workers["A"][0], 1e9) and math.isclose(sb.workers["B"][0], 2e9)
    assert set(sb.workers) == {"A", "B"}
    # at T = 6 A has exactly nothing left and stays listed (only a negative
    # pending size removes a worker); by T = 6.5 it is gone
    sb.finish("nobody", T=6.0)
    assert set(sb.workers) == {"A", "B"} and sb.workers["A"][0] == 0.0
    sb.finish("nobody", T=6.5)
    assert set(sb.workers) == {"B"} and math.isclose(sb.workers["B"][0], 0.75e9)
