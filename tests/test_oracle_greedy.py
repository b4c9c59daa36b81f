"""Pins for the greedy mask-construction oracle (Sec. "Dependency-Closed Masks and
Cache-Consistent Routing"; costs from Eqs. flop-attn and flop-mlp).

Pinned against what does not depend on the greedy code: brute-force optima on tiny inputs (the
greedy never beats them and equals them when every candidate costs the same), a hand-derived
scan, the paper's printed 70B candidate count, and closure / budget invariants."""
import itertools
import json
import os

import numpy as np
import pytest

import synth
from oracle import greedy as G
from oracle import reference as ref

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _closed_subset_cost_value(sh, granule, hs, cs, pick_heads, pick_groups):
    q = np.zeros((sh.n_layers, sh.n_q_heads), np.uint8)
    f = np.zeros((sh.n_layers, sh.d_ffn), np.uint8)
    for (l, h) in pick_heads:
        q[l, h] = 1
    for (l, g) in pick_groups:
        f[l, g * granule:(g + 1) * granule] = 1
    qc, kvc, fc = ref.close_mask(q, None, f, sh.group_size)
    cost = G.mask_cost(sh, granule, qc.astype(np.uint8), kvc.astype(np.uint8), fc.astype(np.uint8))
    return cost, G.mask_value(sh, hs, cs, granule, qc, fc)


def _brute_force_optimum(sh, granule, hs, cs, B):
    heads = [(l, h) for l in range(sh.n_layers) for h in range(sh.n_q_heads)]
    groups = [(l, g) for l in range(sh.n_layers) for g in range(sh.d_ffn // granule)]
    best = -np.inf
    for mh in itertools.product((0, 1), repeat=len(heads)):
        ph = [x for x, m in zip(heads, mh) if m]
        for mg in itertools.product((0, 1), repeat=len(groups)):
            pg = [x for x, m in zip(groups, mg) if m]
            cost, val = _closed_subset_cost_value(sh, granule, hs, cs, ph, pg)
            if cost <= B:
                best = max(best, val)
    return best


def test_hand_derived_scan():
    """d = d_h = 1, 4 heads in 2 groups of r = 2, 4 single channels: head 4 FLOPs, group 4,
    channel 6; a head ranks at 4 + 4/2 = 6. Full width 48, target 0.5 -> budget 24. Keys,
    descending with index ties: ch1 2.0, head0 1.33, ch0 1.0, head2 0.67, head3 0.67, ch3 0.5,
    head1 0.17, ch2 0.1. The scan takes ch1 (6), head0 (+group 0: 8), ch0 (6) = 20; head2 and head3
    would open group 1 (8) and ch3 (6) no longer fits; head1 joins the open group 0 (4) = 24."""
    sh = synth.tiny_shape(d=1, hq=4, hkv=2, dh=1, f=4)
    assert G.full_flops(sh) == 48 and G.budget(sh, 0.5) == 24
    hs = np.array([[8.0, 1.0, 4.0, 4.0]])
    cs = np.array([[6.0, 12.0, 0.6, 3.0]])
    q, kv, f, spent, acc = G.greedy_mask(sh, hs, cs, 1, 0.5)
    assert q.tolist() == [[1, 1, 0, 0]] and kv.tolist() == [[1, 0]] and f.tolist() == [[1, 1, 0, 0]]
    assert spent == 24 and acc == [5, 0, 4, 1]
    assert G.mask_value(sh, hs, cs, 1, q, f) == _brute_force_optimum(sh, 1, hs, cs, 24) == 27


@pytest.mark.parametrize("seed", range(12))
def test_never_beats_brute_force_and_respects_budget(seed):
    sh = synth.tiny_shape(d=2, hq=4, hkv=2, dh=1, f=6)
    rng = np.random.default_rng(seed)
    hs, cs = rng.uniform(0, 1, (1, 4)), rng.uniform(0, 1, (1, 3))
    target = rng.uniform(0.2, 0.9)
    q, kv, f, spent, _ = G.greedy_mask(sh, hs, cs, 2, target)
    B = G.budget(sh, target)
    assert spent <= B and spent == G.mask_cost(sh, 2, q, kv, f)
    qc, kvc, fc = ref.close_mask(q, kv, f, sh.group_size)      # already closed
    assert np.array_equal(qc, q.astype(bool)) and np.array_equal(kvc, kv.astype(bool))
    assert G.mask_value(sh, hs, cs, 2, q, f) <= _brute_force_optimum(sh, 2, hs, cs, B) + 1e-12


@pytest.mark.parametrize("seed", range(8))
def test_equal_costs_reach_the_knapsack_optimum(seed):
    """One head per group (head + its group = 8 d d_h, also its ranking cost) and channel groups
    of G with 6 d G equal to it (d_h = 3, G = 4): every candidate costs the same, so the optimum is
    the k best scores and the greedy must reach it."""
    sh = synth.tiny_shape(d=1, hq=3, hkv=3, dh=3, f=12)
    hc, gc, cc = G.candidate_costs(sh, 4)
    assert hc + gc == cc
    rng = np.random.default_rng(100 + seed)
    hs, cs = rng.uniform(0, 1, (1, 3)), rng.uniform(0, 1, (1, 3))
    target = rng.uniform(0.1, 0.95)
    q, kv, f, spent, _ = G.greedy_mask(sh, hs, cs, 4, target)
    B = G.budget(sh, target)
    k = B // cc
    top = np.sort(np.concatenate([hs[0], cs[0]]))[::-1][:k].sum()
    assert G.mask_value(sh, hs, cs, 4, q, f) == pytest.approx(top, abs=1e-12)
    assert G.mask_value(sh, hs, cs, 4, q, f) == pytest.approx(_brute_force_optimum(sh, 4, hs, cs, B), abs=1e-12)


def test_extreme_budgets():
    sh = synth.tiny_shape(d=4, hq=4, hkv=2, dh=2, f=8, layers=2)
    rng = np.random.default_rng(3)
    hs, cs = rng.uniform(0, 1, (2, 4)), rng.uniform(0, 1, (2, 4))
    q, kv, f, spent, _ = G.greedy_mask(sh, hs, cs, 2, 1.0)
    assert q.all() and kv.all() and f.all() and spent == G.full_flops(sh)
    q, kv, f, spent, _ = G.greedy_mask(sh, hs, cs, 2, 0.0)
    assert not q.any() and not kv.any() and not f.any() and spent == 0


def test_paper_70b_candidate_partition():
    g = json.load(open(os.path.join(GOLDEN, "paper_70b_ledger.json")))
    sh = synth.Shape(**g["shape"])
    cands = G.candidate_list(sh, g["swiglu_group_channels"])
    assert len(cands) == g["total_candidates"]
    # the costs partition the full-width FLOPs exactly: all heads + all groups + all channels
    hc, gc, cc = G.candidate_costs(sh, g["swiglu_group_channels"])
    assert sh.n_layers * (sh.n_q_heads * hc + sh.n_kv_heads * gc + g["swiglu_groups_per_layer"] * cc) \
        == G.full_flops(sh)


def test_budget_is_the_active_flop_ratio():
    """The spent FLOPs over full width is the ledger's active-FLOP ratio of the mask, and stays
    within one candidate's cost below the target at the 8B shape."""
    sh = synth.LLAMA3_8B.with_layers(4, vocab=0)
    rng = np.random.default_rng(5)
    hs, cs = rng.uniform(0, 1, (4, 32)), rng.uniform(0, 1, (4, 14))
    q, kv, f, spent, _ = G.greedy_mask(sh, hs, cs, 1024, 0.57)
    counts = synth.mask_counts(q.astype(bool), kv.astype(bool), f.astype(bool))
    assert ref.active_flop_ratio(sh, counts) == pytest.approx(spent / G.full_flops(sh), rel=1e-12)
    hc, gc, cc = G.candidate_costs(sh, 1024)
    assert 0.57 * G.full_flops(sh) - spent < hc + gc + cc
