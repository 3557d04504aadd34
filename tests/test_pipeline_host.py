"""Host logic of the pipelined virtual worker (no GPU): cut points, partition
renumbering, balanced partitioning, and the task schedule of the partition
scheduling rules (HetPipe Sec. 4)."""
import itertools

import pytest

from paper_2005_14038_amd import nets
from paper_2005_14038_amd import pipeline as pl
from paper_2005_14038_amd.hetpipe import HP_ADD, HP_BN, HP_CONV, HP_RELU


@pytest.mark.parametrize("name", ["tiny", "vgg19", "resnet152"])
def test_valid_cuts_leave_one_tensor(name):
    layers = nets.by_name(name).layers
    cuts = pl.valid_cuts(layers)
    assert cuts
    for i in cuts:
        for j in range(i + 1, len(layers)):
            refs = [layers[j].get("in0", -1)]
            if layers[j]["kind"] == HP_ADD:
                refs.append(layers[j]["in1"])
            # nothing after the cut reads a tensor from before it, except layer i
            assert all(r >= i for r in refs), (i, j, refs)
    # every rejected index has some later layer reading across it, or
    # separates a conv from the batch norm that reads it
    for i in set(range(len(layers) - 1)) - set(cuts):
        crossing = any(min([layers[j].get("in0", -1)] +
                           ([layers[j]["in1"]] if layers[j]["kind"] == HP_ADD else [])) < i
                       for j in range(i + 1, len(layers)))
        conv_bn = layers[i]["kind"] == HP_CONV and any(
            d["kind"] == HP_BN and d.get("in0", -1) == i for d in layers[i + 1:])
        assert crossing or conv_bn or i == len(layers) - 2
    # no cut separates a conv from its batch norm
    for i in cuts:
        assert not (layers[i]["kind"] == HP_CONV and layers[i + 1]["kind"] == HP_BN
                    and layers[i + 1].get("in0", -1) == i)


def test_resnet_cuts_are_block_boundaries():
    b = nets.resnet152()
    cuts = set(pl.valid_cuts(b.layers))
    # the output of every bottleneck (a ReLU after the residual add) is a cut
    block_outs = [i for i, d in enumerate(b.layers)
                  if d["kind"] == HP_RELU and b.layers[d["in0"]]["kind"] == HP_ADD]
    assert len(block_outs) == 3 + 8 + 36 + 3
    assert set(block_outs[:-1]) <= cuts
    # and no cut falls inside a block (between its first conv and its add)
    adds = [i for i, d in enumerate(b.layers) if d["kind"] == HP_ADD]
    for a in adds:
        first = min(b.layers[a]["in0"], b.layers[a]["in1"])
        inside = [c for c in cuts if first < c < a]
        assert not inside, (a, inside)


@pytest.mark.parametrize("name,k", [("tiny", 3), ("vgg19", 4), ("resnet152", 4)])
def test_split_renumbers_and_slices_parameters(name, k):
    b = nets.by_name(name)
    H, W, C = b.input_shape
    cost = pl.layer_costs(b.layers, H, W, C, 32)
    cuts = pl.balanced_cuts(b.layers, k, cost)
    parts = pl.split(b.layers, cuts, H, W, C)
    assert len(parts) == k
    off = 0
    for p in parts:
        assert p.p_off == off
        off += p.p_cnt
        for j, d in enumerate(p.layers):
            assert -1 <= d.get("in0", -1) < j
            if d["kind"] == HP_ADD:
                assert -1 <= d["in1"] < j
        # the partition input is the previous partition's output
    assert off == b.param_count()
    for a, c in zip(parts[:-1], parts[1:]):
        assert a.out_shape == c.in_shape
        assert a.last + 1 == c.first


def test_balanced_cuts_is_optimal_on_tiny():
    b = nets.tiny()
    cost = pl.layer_costs(b.layers, 16, 16, 3, 4)
    valid = pl.valid_cuts(b.layers)
    for k in (2, 3):
        got = pl.balanced_cuts(b.layers, k, cost)

        def worst(cuts):
            bounds = [-1] + list(cuts) + [len(b.layers) - 1]
            return max(sum(cost[a + 1:c + 1]) for a, c in zip(bounds[:-1], bounds[1:]))
        brute = min(worst(c) for c in itertools.combinations(valid, k - 1))
        assert worst(got) == brute


def test_schedule_two_partitions_worked_example():
    # k = 2, N_m = 2, forward 1 and backward 2 time units per partition,
    # derived by hand from the three rules of Sec. 4 (forward in order,
    # backward in order, FIFO); the last partition's forward+backward is one task
    got = [(t.kind, t.m, t.q, t.start) for t in pl.schedule(2, 2, 4, [1, 1], [2, 2])]
    assert got == [("F", 1, 0, 0), ("F", 2, 0, 1), ("FB", 1, 1, 1), ("B", 1, 0, 4),
                   ("FB", 2, 1, 4), ("U", 1, -1, 6), ("F", 3, 0, 6), ("B", 2, 0, 7),
                   ("FB", 3, 1, 7), ("U", 2, -1, 9), ("F", 4, 0, 9), ("B", 3, 0, 10),
                   ("FB", 4, 1, 10), ("U", 3, -1, 12), ("B", 4, 0, 13), ("U", 4, -1, 15)]


@pytest.mark.parametrize("k,W,total", [(1, 4, 12), (2, 4, 12), (3, 4, 20), (4, 3, 15), (4, 6, 24)])
def test_schedule_rules(k, W, total):
    dF = [1.0 + 0.3 * q for q in range(k)]
    dB = [2.0 + 0.5 * q for q in range(k)]
    tasks = pl.schedule(k, W, total, dF, dB)
    work = [t for t in tasks if t.kind != "U"]
    ends = {(t.kind if t.kind != "FB" else "F", t.m, t.q): t.end for t in work}
    ends.update({("B", t.m, t.q): t.end for t in work if t.kind == "FB"})
    comp = {t.m: t.start for t in tasks if t.kind == "U"}
    assert sorted(comp) == list(range(1, total + 1))
    # completions in order
    assert [comp[m] for m in range(1, total + 1)] == sorted(comp.values())
    for q in range(k):
        mine = sorted((t for t in work if t.q == q), key=lambda t: t.start)
        # one task at a time
        for a, c in zip(mine, mine[1:]):
            assert a.end <= c.start
        # forward tasks and backward tasks each in minibatch order
        fw = [t.m for t in mine if t.kind in ("F", "FB")]
        bw = [t.m for t in mine if t.kind in ("B", "FB")]
        assert fw == sorted(fw) == list(range(1, total + 1))
        assert bw == sorted(bw) == list(range(1, total + 1))
    for t in work:
        if t.kind in ("F", "FB") and t.q > 0:
            assert t.start >= ends[("F", t.m, t.q - 1)]
        if t.kind == "B":
            assert t.start >= ends[("B", t.m, t.q + 1)]
        if t.kind in ("F", "FB") and t.q == 0 and t.m > W:
            # minibatch m enters when m - N_m completes
            assert t.start >= comp[t.m - W]
    # never more than N_m minibatches in flight
    for m in range(1, total + 1):
        entry = min(t.start for t in work if t.m == m)
        inflight = sum(1 for j in range(1, total + 1)
                       if min(t.start for t in work if t.m == j) <= entry < comp[j])
        assert inflight <= W
