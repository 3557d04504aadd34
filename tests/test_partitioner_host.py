"""Model partitioner (HetPipe Sec. 4 model partitioning, Sec. 6 partitioning
algorithm) on the host: the dynamic program against brute-force enumeration
of every cut set (and GPU order) on random profiles, memory constraints,
heterogeneous speeds, and the stash counts of the pipeline schedule."""
import itertools
import math
import random

import pytest

from paper_2005_14038_amd import nets
from paper_2005_14038_amd import partitioner as pt
from paper_2005_14038_amd import pipeline as pl


def chain_layers():
    return nets.vgg19(H=32, W=32, classes=10, width=64).layers


def random_profile(layers, rng, dtype="fp32"):
    n = len(layers)
    return pt.LayerProfile(
        fwd_ms=[rng.uniform(0.0, 2.0) for _ in range(n)],
        bwd_ms=[rng.uniform(0.0, 4.0) for _ in range(n)],
        mem=[rng.randrange(0, 50_000_000) for _ in range(n)],
        shared=rng.randrange(0, 20_000_000),
        params=[rng.randrange(0, 2_000_000) for _ in range(n)],
        out_bytes=[rng.randrange(1, 30_000_000) for _ in range(n)],
        dtype=dtype)


def brute_force(layers, prof, gpus, n_m, link, orders):
    pts = pl.valid_cuts(layers)
    k = len(gpus)
    st = pl.stash_counts(k, n_m)
    best = math.inf
    for order in orders:
        for cuts in itertools.combinations(pts, k - 1):
            bounds = [-1] + list(cuts) + [len(layers) - 1]
            worst = 0.0
            for j in range(k):
                a, b = bounds[j] + 1, bounds[j + 1]
                if pt.partition_memory(prof, a, b, st[j], n_m) > order[j].mem_bytes:
                    worst = math.inf
                    break
                worst = max(worst, pt.partition_time(prof, a, b, order[j], link))
            best = min(best, worst)
    return best


@pytest.mark.parametrize("seed", range(6))
def test_dp_equals_brute_force(seed):
    rng = random.Random(seed)
    layers = chain_layers()
    prof = random_profile(layers, rng, "bf16" if seed % 2 else "fp32")
    k = 2 + seed % 2
    n_m = 1 + seed % 4
    gpus = [pt.GPUSpec(f"g{j}", speed=rng.choice([0.5, 1.0, 2.0]),
                       mem_bytes=rng.choice([math.inf, 4e8, 8e8])) for j in range(k)]
    link = None if seed % 3 == 0 else rng.uniform(5.0, 50.0)
    plan = pt.partition(layers, prof, gpus, n_m, link_GBps=link)
    ref = brute_force(layers, prof, gpus, n_m, link, [gpus])
    if ref == math.inf:
        assert plan is None
        return
    assert plan is not None
    assert plan.bottleneck_ms == pytest.approx(ref, rel=1e-12, abs=1e-12)
    # the plan's own partitions: contiguous, valid cuts, within memory, bottleneck attained
    assert all(c in pl.valid_cuts(layers) for c in plan.cuts)
    assert plan.parts[0][0] == 0 and plan.parts[-1][1] == len(layers) - 1
    for (a, b, name, ms, mem, nst), g in zip(plan.parts, gpus):
        assert mem <= g.mem_bytes
    assert max(p[3] for p in plan.parts) == pytest.approx(plan.bottleneck_ms)


@pytest.mark.parametrize("seed", range(3))
def test_order_search_equals_brute_force_over_orders(seed):
    rng = random.Random(100 + seed)
    layers = chain_layers()
    prof = random_profile(layers, rng)
    gpus = [pt.GPUSpec("fast", 3.0, 6e8), pt.GPUSpec("slow", 1.0, math.inf),
            pt.GPUSpec("slow", 1.0, math.inf)]
    plan = pt.partition(layers, prof, gpus, 3, search_order=True)
    orders = [list(p) for p in itertools.permutations(gpus)]
    ref = brute_force(layers, prof, gpus, 3, None, orders)
    assert plan.bottleneck_ms == pytest.approx(ref, rel=1e-12)


def test_infeasible_memory_returns_none():
    rng = random.Random(7)
    layers = chain_layers()
    prof = random_profile(layers, rng)
    assert pt.partition(layers, prof, [pt.GPUSpec("tiny", 1.0, 1e3)] * 2, 2) is None


def test_homogeneous_unbounded_matches_work_balanced_cuts():
    rng = random.Random(3)
    layers = chain_layers()
    prof = random_profile(layers, rng)
    cost = [f + b for f, b in zip(prof.fwd_ms, prof.bwd_ms)]
    for k in (2, 3, 4):
        plan = pt.partition(layers, prof, [pt.GPUSpec("g")] * k, 4)
        cuts = pl.balanced_cuts(layers, k, cost)
        bounds = [-1] + cuts + [len(layers) - 1]
        ref = max(sum(cost[bounds[j] + 1:bounds[j + 1] + 1]) for j in range(k))
        assert plan.bottleneck_ms == pytest.approx(ref)


def test_faster_gpu_takes_more_layers():
    layers = chain_layers()
    n = len(layers)
    prof = pt.LayerProfile(fwd_ms=[1.0] * n, bwd_ms=[2.0] * n, mem=[0] * n, shared=0,
                           params=[0] * n, out_bytes=[1] * n)
    plan = pt.partition(layers, prof, [pt.GPUSpec("fast", 3.0), pt.GPUSpec("slow", 1.0)], 1)
    (a0, b0, *_), (a1, b1, *_) = plan.parts
    n0, n1 = b0 - a0 + 1, b1 - a1 + 1
    # 3:1 split of equal layers, to within one layer
    assert abs(n0 - 3 * n1) <= 4 and n0 > n1
    assert plan.bottleneck_ms <= 3.0 * (n / 4 + 1)


def test_memory_cap_moves_the_cut():
    layers = chain_layers()
    n = len(layers)
    prof = pt.LayerProfile(fwd_ms=[1.0] * n, bwd_ms=[2.0] * n, mem=[10] * n, shared=0,
                           params=[0] * n, out_bytes=[0] * n)
    free = pt.partition(layers, prof, [pt.GPUSpec("a"), pt.GPUSpec("b")], 4)
    st = pl.stash_counts(2, 4)
    # the first GPU (4 stashes) may hold at most 5 layers
    capped = pt.partition(layers, prof, [pt.GPUSpec("a", 1.0, 10 * 5 * st[0]),
                                         pt.GPUSpec("b")], 4)
    assert free.parts[0][1] > 4
    assert capped.parts[0][1] <= 4
    assert capped.bottleneck_ms > free.bottleneck_ms


def test_link_time_counts_both_directions_at_inner_cuts():
    layers = chain_layers()
    n = len(layers)
    prof = pt.LayerProfile(fwd_ms=[0.0] * n, bwd_ms=[0.0] * n, mem=[0] * n, shared=0,
                           params=[0] * n, out_bytes=[10_000_000] * n)
    g = pt.GPUSpec("g")
    # 10 MB at 10 GB/s = 1 ms per crossing; a middle partition crosses twice
    assert pt.partition_time(prof, 0, 3, g, 10.0) == pytest.approx(1.0)
    assert pt.partition_time(prof, 4, 7, g, 10.0) == pytest.approx(2.0)
    assert pt.partition_time(prof, 8, n - 1, g, 10.0) == pytest.approx(1.0)


def test_stash_counts_hand_worked_and_invariants():
    # k = 2, N_m = 2 (forward 1, backward 2): partition 0 runs F1 F2, then B1
    # at t = 4 (after FB1 on partition 1), F3 when minibatch 1 completes; it
    # holds two minibatches; the last partition holds one
    assert pl.stash_counts(2, 2) == [2, 1]
    for k in (1, 2, 3, 5):
        for n_m in (1, 2, 4, 6):
            s = pl.stash_counts(k, n_m)
            assert len(s) == k and s[-1] == 1 and s[0] == (n_m if k > 1 else 1)
            assert all(1 <= v <= n_m for v in s)
            assert all(x >= y for x, y in zip(s, s[1:]))
