"""Mesh planner of adaptive tensor parallelism, written out plainly.

TEST INFRASTRUCTURE ONLY: the tests, smoke() and the bench's CPU baseline may
import this module; the library never does.

What it computes (Sec. 3.2 search space, Sec. 3.3 Eq. (tcomm), Sec. 3.4 the
hierarchical communication matrix, Sec. 3.5 Eq. (bwd) and Eq. (allreduce)):

* the candidate meshes for N devices are every (d1, d2) with d1 * d2 = N;
* a hierarchical communication matrix (HCM) is a list of layers, outermost
  first.  Layer j has R_j ranks (each rank of layer j holds the product of
  the inner layers' rank counts in devices), a per-rank group bandwidth and a
  R_j x R_j point-to-point (P2P) bandwidth matrix among the ranks that share
  a parent;
* device r of the mesh is (i1, i2) with r = i1 * d2 + i2; its digit at layer
  j is its rank index inside its parent at that layer (mixed radix, the
  innermost layer varying fastest);
* axis 1 all-reduces run inside each set of devices with equal i2 (d2 groups
  of d1 devices), axis 2 inside each set with equal i1 (d1 groups of d2);
* B1' and B2' (Eq. (bwd)): the bottleneck over the layers the axis's groups
  cross.  Reading used here: at a layer j where a group spans several ranks of
  one parent, each of those ranks offers the group min(group bandwidth, sum
  of its P2P bandwidth to the group's other ranks there) -- the P2P
  correction the paper applies to DeviceMesh(8, 2) -- divided by the number
  of the axis's groups that cross layer j through that same rank, which is
  the division by d2 of Eq. (bwd) when a node hosts d2 groups and no division
  when every rank is a single device (the fully connected and torus cases of
  Sec. 5.4, where both bandwidths equal the group bandwidth);
* B = d / (2 (d - 1)) * B' per axis (Eq. (allreduce), Rabenseifner's
  algorithm without the latency term); an axis of size 1 has no all-reduce,
  so its term of Eq. (tcomm) vanishes;
* T_comm = 2 L b s * (7 h / (d1 B2) + 2 h / (d2 B1)) (Eq. (tcomm)), counted
  here in bytes of `elem_bytes`-byte elements over bandwidths in GB/s, so in
  seconds;
* the plan is the mesh of least T_comm; ties go to the larger d1.
"""
from __future__ import annotations

import math


class Layer:
    """One HCM layer: `ranks` ranks per parent, `group_bw` GB/s per rank to
    the outside of the rank, `p2p[u][v]` GB/s between ranks u and v of one
    parent (None: every pair at `group_bw`, as behind a switch)."""

    def __init__(self, ranks, group_bw, p2p=None):
        self.ranks = int(ranks)
        self.group_bw = float(group_bw)
        if p2p is None:
            p2p = [[0.0 if u == v else self.group_bw for v in range(self.ranks)]
                   for u in range(self.ranks)]
        self.p2p = [[float(x) for x in row] for row in p2p]


def device_count(layers):
    n = 1
    for ly in layers:
        n *= ly.ranks
    return n


def meshes(n):
    """Every (d1, d2) with d1 * d2 = n, largest d1 first."""
    return [(d1, n // d1) for d1 in range(n, 0, -1) if n % d1 == 0]


def digits(r, layers):
    """Rank index of device r at each layer, outermost first."""
    out = []
    for j in range(len(layers) - 1, -1, -1):
        out.append(r % layers[j].ranks)
        r //= layers[j].ranks
    return out[::-1]


def axis_groups(d1, d2, axis):
    """Device sets that all-reduce together along mesh axis 1 or 2."""
    if axis == 1:
        return [[i1 * d2 + i2 for i1 in range(d1)] for i2 in range(d2)]
    return [[i1 * d2 + i2 for i2 in range(d2)] for i1 in range(d1)]


def layer_bandwidth(layers, j, groups):
    """Bandwidth one group of the axis gets through layer j, or None when no
    group crosses layer j."""
    ly = layers[j]
    # per group and parent (the digits above j): the layer-j ranks touched
    crossing = []     # (parent, set of ranks) for spans of more than one rank
    for g in groups:
        spans = {}
        for r in g:
            dg = digits(r, layers)
            spans.setdefault(tuple(dg[:j]), set()).add(dg[j])
        for parent, units in spans.items():
            if len(units) > 1:
                crossing.append((parent, units))
    if not crossing:
        return None
    # how many crossing groups pass through each (parent, rank)
    share = {}
    for parent, units in crossing:
        for u in units:
            share[(parent, u)] = share.get((parent, u), 0) + 1
    best = math.inf
    for parent, units in crossing:
        for u in units:
            p2p_sum = sum(ly.p2p[u][v] for v in units if v != u)
            bw = min(ly.group_bw, p2p_sum) / share[(parent, u)]
            best = min(best, bw)
    return best


def effective_bandwidth(layers, d1, d2, axis):
    """B1' (axis 1) or B2' (axis 2) of Eq. (bwd); None for an axis of size 1."""
    if (d1 if axis == 1 else d2) == 1:
        return None
    groups = axis_groups(d1, d2, axis)
    vals = [layer_bandwidth(layers, j, groups) for j in range(len(layers))]
    vals = [v for v in vals if v is not None]
    return min(vals)


def algorithm_bandwidth(d, b_eff):
    """Eq. (allreduce): B = d / (2 (d - 1)) B'; infinite for d = 1."""
    if d == 1:
        return math.inf
    return d / (2.0 * (d - 1)) * b_eff


def t_comm(L, b, s, h, d1, d2, B1, B2, elem_bytes=2):
    """Eq. (tcomm) in seconds for bandwidths in GB/s."""
    def term(num, d, B):
        if math.isinf(B):
            return 0.0
        if B <= 0.0:
            return math.inf
        return num / (d * B * 1e9)
    return 2.0 * L * b * s * elem_bytes * (term(7.0 * h, d1, B2) + term(2.0 * h, d2, B1))


def mesh_cost(layers, d1, d2, L, b, s, h, elem_bytes=2):
    """B1', B2', B1, B2 and T_comm of DeviceMesh(d1, d2) on the HCM."""
    if d1 * d2 != device_count(layers):
        raise ValueError("mesh does not cover the HCM's devices")
    e1 = effective_bandwidth(layers, d1, d2, 1)
    e2 = effective_bandwidth(layers, d1, d2, 2)
    B1 = algorithm_bandwidth(d1, e1) if e1 is not None else math.inf
    B2 = algorithm_bandwidth(d2, e2) if e2 is not None else math.inf
    return dict(d1=d1, d2=d2, b1_eff=e1, b2_eff=e2, b1=B1, b2=B2,
                t_comm=t_comm(L, b, s, h, d1, d2, B1, B2, elem_bytes))


def plan(layers, L, b, s, h, elem_bytes=2):
    """(best mesh, costs of every mesh in search order)."""
    costs = [mesh_cost(layers, d1, d2, L, b, s, h, elem_bytes)
             for d1, d2 in meshes(device_count(layers))]
    best = costs[0]
    for c in costs[1:]:
        if c["t_comm"] < best["t_comm"]:
            best = c
    return (best["d1"], best["d2"]), costs
