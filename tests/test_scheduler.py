"""The collective scheduler (Collective Scheduler section of the paper) on
described multi-node topologies, on the CPU: the forwarding expansion
against the paper's worked example, and the stage decomposition against the
paper's constraints (completeness, Eq. 7; per-stage RDMA degree bound,
Eq. 8; stage duration, Eq. 9-10; total, Eq. 11)."""
import itertools
import random

import pytest

import paper_2609_34334_amd as hc

# Worked example: 4 GPUs, nodes {g0, g1} and {g2, g3}, symmetric peers
# 0<->1 and 2<->3; the twelve flows f1..f12 are the off-diagonal entries of
# C in row-major order (C[0,1] = f1, C[0,2] = f2, ..., C[3,2] = f12).
NODE = [0, 0, 1, 1]
PEER = [1, 0, 3, 2]


def worked_example_C():
    f = {k: float(2 ** k) for k in range(1, 13)}   # distinct powers of two
    C = [[0.0] * 4 for _ in range(4)]
    k = 1
    for u in range(4):
        for v in range(4):
            if u != v:
                C[u][v] = f[k]
                k += 1
    return C, f


def test_expansion_reproduces_the_papers_F1():
    C, f = worked_example_C()
    T = hc.schedule(C, NODE, PEER, 400.0, 50.0)["T"]
    # printed in the paper: F1 = T[0,1] = f1 + f2' + f3' + f8'' + f11''
    # (forwarding copies carry the flow's bytes); with powers of two the sum
    # identifies exactly which flows contribute.
    assert T[0][1] == f[1] + f[2] + f[3] + f[8] + f[11]


def test_expansion_other_cells():
    C, f = worked_example_C()
    T = hc.schedule(C, NODE, PEER, 400.0, 50.0)["T"]
    # By the same rule for the other symmetric-peer edges:
    assert T[3][2] == f[12] + f[10] + f[11] + f[2] + f[5]
    assert T[1][0] == f[4] + f[5] + f[6] + f[7] + f[10]
    assert T[2][3] == f[9] + f[7] + f[8] + f[3] + f[6]
    # inter-node cells are the RDMA flows themselves
    for (u, v), k in {(0, 2): 2, (0, 3): 3, (1, 2): 5, (1, 3): 6, (2, 0): 7, (2, 1): 8,
                      (3, 0): 10, (3, 1): 11}.items():
        assert T[u][v] == f[k]
    for u in range(4):
        assert T[u][u] == 0


def check_schedule(C, node, peer, bwi, bwr):
    s = hc.schedule(C, node, peer, bwi, bwr)
    G = len(node)
    T, stages, tau = s["T"], s["stages"], s["tau"]
    # Eq. 7: completeness, element-wise
    for u in range(G):
        for v in range(G):
            tot = sum(S[u][v] for S in stages)
            assert abs(tot - T[u][v]) <= 1e-6 * max(1.0, T[u][v]), (u, v, tot, T[u][v])
    for k, S in enumerate(stages):
        # Eq. 8: at most one outgoing and one incoming RDMA flow per GPU
        for u in range(G):
            outs = [v for v in range(G) if node[v] != node[u] and S[u][v] > 1e-9]
            ins = [v for v in range(G) if node[v] != node[u] and S[v][u] > 1e-9]
            assert len(outs) <= 1 and len(ins) <= 1, (k, u, outs, ins)
        # Eq. 9-10: the stage lasts as long as its slowest domain
        lr = max([S[u][v] for u in range(G) for v in range(G) if node[u] != node[v]] + [0.0])
        ln = max([S[u][v] for u in range(G) for v in range(G) if node[u] == node[v]] + [0.0])
        assert abs(tau[k] - max(lr / bwr, ln / bwi)) <= 1e-9 * max(1.0, tau[k])
        assert any(S[u][v] > 0 for u in range(G) for v in range(G)), "empty stage"
    assert abs(s["total"] - sum(tau)) <= 1e-9 * max(1.0, s["total"])     # Eq. 11
    # a GPU sends one RDMA flow per stage, so the total cannot beat its
    # RDMA bytes at inter-node bandwidth
    for u in range(G):
        out_bytes = sum(C[u][v] for v in range(G) if node[v] != node[u])
        assert s["total"] >= out_bytes / bwr - 1e-9
    return s


def test_worked_example_decomposition():
    C, _ = worked_example_C()
    s = check_schedule(C, NODE, PEER, 400.0, 50.0)
    # every GPU sends to two GPUs of the other node: at least two stages
    assert len(s["stages"]) >= 2


def test_uniform_alltoall_two_nodes_needs_as_many_stages_as_remote_peers():
    G = 8
    node = [0] * 4 + [1] * 4
    peer = [1, 0, 3, 2, 5, 4, 7, 6]
    C = [[0.0 if u == v else 1e6 for v in range(G)] for u in range(G)]
    s = check_schedule(C, node, peer, 400.0, 50.0)
    rdma_stages = [S for S in s["stages"] if any(S[u][v] > 0 for u in range(G) for v in range(G)
                                                 if node[u] != node[v])]
    # 4 remote destinations per GPU, one RDMA flow per GPU per stage, equal
    # flows: exactly 4 stages carry RDMA traffic, each of 1e6 / 50
    assert len(rdma_stages) == 4
    for k, S in enumerate(s["stages"][:4]):
        assert s["tau"][k] == pytest.approx(1e6 / 50.0)


def test_single_node_has_no_forwarding_and_no_rdma():
    G = 4
    node = [0] * G
    peer = [-1] * G
    rng = random.Random(3)
    C = [[0.0 if u == v else float(rng.randint(1, 100)) for v in range(G)] for u in range(G)]
    s = check_schedule(C, node, peer, 100.0, 10.0)
    assert s["T"] == [[C[u][v] if u != v else 0.0 for v in range(G)] for u in range(G)]


@pytest.mark.parametrize("seed", range(8))
def test_random_topologies(seed):
    rng = random.Random(seed)
    nodes = rng.randint(2, 4)
    per = rng.choice([2, 4])
    G = nodes * per
    node = [g // per for g in range(G)]
    peer = [g ^ 1 for g in range(G)]
    C = [[0.0 if u == v or rng.random() < 0.2 else float(rng.randint(1, 1000))
          for v in range(G)] for u in range(G)]
    check_schedule(C, node, peer, rng.choice([100.0, 400.0]), rng.choice([25.0, 50.0]))


def test_interleave_is_proportional():
    sizes = [8e6, 2e6, 1e6, 5e6]
    order = hc.interleave(sizes, 1e6)
    totals = [8, 2, 1, 5]
    assert sorted(order) == sorted(sum(([i] * t for i, t in enumerate(totals)), []))
    done = [0] * 4
    for p, i in enumerate(order):
        done[i] += 1
        frac = [done[k] / totals[k] for k in range(4)]
        # every flow's completed fraction stays within one chunk of the others
        assert max(frac) - min(frac) <= max(1.0 / t for t in totals) + 1e-12, (p, frac)
    # all flows finish in the last len(sizes) chunks
    last = {i: p for p, i in enumerate(order)}
    assert min(last.values()) >= len(order) - len(sizes)


def test_interleave_equal_flows_is_round_robin():
    order = hc.interleave([4e6] * 3, 1e6)
    assert order == [0, 1, 2] * 4
