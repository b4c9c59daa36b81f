"""Pins for the oracle's mask closure, index lists and FLOP/byte ledgers.

Closure (Sec. "Dependency-Closed Masks and Cache-Consistent Routing"): a KV group is needed
exactly when one of its own query heads survives, heads keep their group, and a SwiGLU channel is
one unit (gate row, up row, down column). The closure is checked exhaustively on a tiny layer
against properties that any correct closure has, and on hand-derived cases.
"""
import itertools
import json
import os

import numpy as np
import pytest

import synth
from oracle import compact, reference as ref

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _bits(v, n):
    return np.array([(v >> i) & 1 for i in range(n)], dtype=np.uint8)


def test_closure_exhaustive_properties():
    Hq, Hkv, F, r = 4, 2, 8, 2
    for qv, kvv in itertools.product(range(2 ** Hq), range(2 ** Hkv)):
        q, kv = _bits(qv, Hq)[None], _bits(kvv, Hkv)[None]
        for fv in (0, 0b10110101, 255):
            f = _bits(fv, F)[None]
            qc, kvc, fc = ref.close_mask(q, kv, f, r)
            g = np.arange(Hq) // r
            # a head survives iff it was kept and its group was not dropped (never moved)
            assert np.array_equal(qc[0], q[0].astype(bool) & kv[0, g].astype(bool))
            # a group is active iff at least one of its query heads survives
            for gg in range(Hkv):
                assert kvc[0, gg] == qc[0, g == gg].any()
            assert not (kvc & ~kv.astype(bool)).any()          # never activates a dropped group
            assert np.array_equal(fc, f.astype(bool))
            # idempotent: closing a closed mask changes nothing
            again = ref.close_mask(qc, kvc, fc, r)
            assert all(np.array_equal(a, b) for a, b in zip(again, (qc, kvc, fc)))
            qi, kvi, slot, fi = ref.index_lists(qc[0], kvc[0], fc[0], r)
            assert np.all(np.diff(qi) > 0) and np.all(np.diff(kvi) > 0) and np.all(np.diff(fi) > 0)
            assert np.array_equal(kvi[slot], qi // r)           # slot points at the head's own group


def test_closure_hand_cases():
    r = 4
    # Hq = 8, Hkv = 2.  Dropping group 0 removes heads 0-3 even if they were kept.
    q = np.array([[1, 1, 1, 1, 0, 1, 0, 0]])
    qc, kvc, _ = ref.close_mask(q, np.array([[0, 1]]), np.ones((1, 4)), r)
    assert qc[0].tolist() == [False] * 5 + [True, False, False] and kvc[0].tolist() == [False, True]
    # a kept group whose heads are all dropped is inactive (charged per active group)
    qc, kvc, _ = ref.close_mask(np.array([[0, 0, 0, 0, 1, 0, 0, 0]]), None, np.ones((1, 4)), r)
    assert kvc[0].tolist() == [False, True]
    qi, kvi, slot, _ = ref.index_lists(qc[0], kvc[0], np.ones(4, bool), r)
    assert qi.tolist() == [4] and kvi.tolist() == [1] and slot.tolist() == [0]
    # ragged groups: slots follow the retained-group ranks
    qc, kvc, _ = ref.close_mask(np.array([[0, 1, 0, 0, 1, 1, 0, 1]]), None, np.ones((1, 4)), r)
    qi, kvi, slot, _ = ref.index_lists(qc[0], kvc[0], np.ones(4, bool), r)
    assert qi.tolist() == [1, 4, 5, 7] and kvi.tolist() == [0, 1] and slot.tolist() == [0, 1, 1, 1]


def test_flop_ledger_equals_twice_panel_sizes():
    """The analytical ledger (Eqs. flop-attn, flop-mlp) against the dimensions actually packed:
    every retained weight is one multiply-add per token."""
    sh = synth.tiny_shape(d=24, hq=8, hkv=2, dh=4, f=12)
    layer = synth.layer_weights(sh, 0)
    for seed in range(20):
        q, kv, f = synth.raw_mask(sh, seed)
        qc, kvc, fc = ref.close_mask(q, kv, f, sh.group_size)
        pn = compact.compact_panels(layer, qc[0], kvc[0], fc[0], sh)
        n_weights = sum(pn[k].size for k in ("qkv", "o", "gate", "up", "down"))
        m = synth.mask_counts(qc, kvc, fc)
        assert ref.layer_flops(sh, int(m[0][0]), int(m[1][0]), int(m[2][0])) == 2 * n_weights
        b = ref.decode_bytes(sh, m, batch=1, pos=7)
        assert b["weights"] == n_weights
        n_rows = pn["qkv"].shape[0] + pn["o"].shape[0] + 2 * pn["gate"].shape[0] + pn["down"].shape[0]
        assert b["scales"] == 4 * n_rows
        assert b["kv"] == 2 * 2 * int(m[1][0]) * 8 * sh.head_dim


def test_ledger_reproduces_paper_70b_figures():
    g = json.load(open(os.path.join(GOLDEN, "paper_70b_ledger.json")))
    sh = synth.Shape(**g["shape"])
    assert g["query_head_candidates_per_layer"] == sh.n_q_heads
    assert g["swiglu_groups_per_layer"] * g["swiglu_group_channels"] == sh.d_ffn
    assert sh.n_layers * (sh.n_q_heads + sh.d_ffn // g["swiglu_group_channels"]) == g["total_candidates"]
    dense = [np.full(sh.n_layers, v) for v in (sh.n_q_heads, sh.n_kv_heads, sh.d_ffn)]
    layer_w = ref.decode_bytes(sh, dense, batch=1, pos=0)["weights"]
    # the packed store holds every decoder projection plus the INT8 embedding and LM head
    store = layer_w + 2 * sh.vocab * sh.d_model
    assert abs(store / 1e9 - g["int8_weights_GB"]) / g["int8_weights_GB"] < g["store_rel_tol"]
    scales = store / g["scale_group"] * g["scale_bytes"]
    assert abs(scales / 1e9 - g["scales_GB"]) / g["scales_GB"] < g["scales_rel_tol"]
    assert ref.active_flop_ratio(sh, dense) == 1.0


def test_active_ratio_examples():
    sh = synth.LLAMA3_8B.with_layers(2)
    # dropping all FFN channels of one layer of two removes exactly half the FFN FLOPs
    full = ref.layer_flops(sh, 32, 8, 14336)
    ffn = 6 * sh.d_model * sh.d_ffn
    counts = (np.array([32, 32]), np.array([8, 8]), np.array([14336, 0]))
    assert ref.active_flop_ratio(sh, counts) == pytest.approx((2 * full - ffn) / (2 * full), rel=1e-15)
    # a KV group with 1 retained head costs the same as a head plus a group
    unit = 4 * sh.d_model * sh.head_dim
    assert ref.layer_flops(sh, 1, 1, 0) == 2 * unit
