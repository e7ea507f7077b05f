"""Pipeline loading plan across GPUs (host only, no GPU): the paper's worked
recovery example, the rotated start-up orders, and the balance / contiguity
properties for every failure pattern of up to eight GPUs."""
import itertools
import json
import os

import numpy as np
import pytest

from paper_2503_17707_amd import binding as pb

HERE = os.path.dirname(os.path.abspath(__file__))


def test_paper_recovery_example():
    ex = json.load(open(os.path.join(HERE, "golden", "recovery_example.json")))
    for phase in ("before", "after"):
        order, blocks = pb.plan_loading(ex["n_layers"], ex[phase]["alive"])
        for g, want in ex[phase]["order"].items():
            assert order[int(g)].tolist() == want, (phase, g)
        for g, want in ex[phase].get("blocks", {}).items():
            first, n = blocks[int(g)]
            assert list(range(first, first + n)) == want
    order, _ = pb.plan_loading(4, [1, 0, 0, 1])
    assert (order[1] == -1).all() and (order[2] == -1).all()


def test_two_way_startup_order_is_the_rotated_stage_order():
    # the OPT-13B workload's load order 20..39, 0..19 is GPU 1's of a 2-GPU split
    order, blocks = pb.plan_loading(40, [1, 1])
    assert order[0].tolist() == list(range(40))
    assert order[1].tolist() == list(range(20, 40)) + list(range(20))
    assert blocks == [(0, 20), (20, 20)]


@pytest.mark.parametrize("n_layers", [4, 7, 24, 64])
def test_balance_contiguity_and_permutations(n_layers):
    for G in range(1, 9):
        for alive in itertools.product([0, 1], repeat=G):
            if not any(alive):
                continue
            order, blocks = pb.plan_loading(n_layers, alive)
            live = [g for g in range(G) if alive[g]]
            sizes = [blocks[g][1] for g in live]
            assert max(sizes) - min(sizes) <= 1 and sum(sizes) == n_layers
            nxt = 0
            for g in live:  # consecutive blocks in GPU order, covering every layer once
                first, n = blocks[g]
                assert first == nxt
                nxt += n
                row = order[g].tolist()
                assert sorted(row) == list(range(n_layers))
                assert row[:n] == list(range(first, first + n))
                assert all((row[i + 1] - row[i]) % n_layers == 1 for i in range(n_layers - 1))
            for g in range(G):
                if not alive[g]:
                    assert (order[g] == -1).all() and blocks[g] == (-1, 0)


def test_invalid_arguments():
    with pytest.raises(pb.PbError) as e:
        pb.plan_loading(4, [0, 0])
    assert e.value.code == pb.PB_EINVAL
    with pytest.raises(pb.PbError):
        pb.plan_loading(0, [1])
