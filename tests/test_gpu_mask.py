"""GPU parity of greedy dependency-closed mask construction against the oracle: the masks and
the FLOPs spent are integer results and must match bit for bit."""
import numpy as np
import pytest
import torch

import synth
from oracle import greedy as G
from oracle import reference as ref
from paper_2609_29499_amd import binding as B
from paper_2609_29499_amd import session as S

pytestmark = pytest.mark.gpu


def _flush(msg):
    print(msg, flush=True)


def _scores(sh, granule, seed, kind="uniform"):
    rng = np.random.default_rng(seed)
    nG = sh.d_ffn // granule
    if kind == "uniform":
        hs = rng.uniform(0, 1, (sh.n_layers, sh.n_q_heads))
        cs = rng.uniform(0, 1, (sh.n_layers, nG))
    elif kind == "ties":                                  # few distinct values: index tie-breaks
        hs = rng.integers(0, 4, (sh.n_layers, sh.n_q_heads)) * 0.25
        cs = rng.integers(0, 4, (sh.n_layers, nG)) * 0.25
    else:                                                 # signed, with zeros
        hs = rng.normal(0, 1, (sh.n_layers, sh.n_q_heads))
        cs = rng.normal(0, 1, (sh.n_layers, nG))
        hs[rng.uniform(size=hs.shape) < 0.2] = 0.0
        cs[rng.uniform(size=cs.shape) < 0.2] = -0.0
    return hs.astype(np.float32), cs.astype(np.float32)


def _gpu(sh, hs, cs, granule, target):
    desc = S.desc_from_shape(sh)
    q, kv, f, spent = S.build_mask(desc, torch.from_numpy(hs).cuda(), torch.from_numpy(cs).cuda(),
                                   granule, target)
    torch.cuda.synchronize()
    return q.cpu().numpy(), kv.cpu().numpy(), f.cpu().numpy(), spent


def _check(sh, granule, target, seed, kind):
    hs, cs = _scores(sh, granule, seed, kind)
    q, kv, f, spent = _gpu(sh, hs, cs, granule, target)
    wq, wkv, wf, wspent, _ = G.greedy_mask(sh, hs, cs, granule, target)
    assert spent == wspent
    assert np.array_equal(q, wq) and np.array_equal(kv, wkv) and np.array_equal(f, wf)
    return q, kv, f


@pytest.mark.parametrize("kind", ["uniform", "ties", "signed"])
@pytest.mark.parametrize("target", [0.0, 0.3, 0.57, 1.0])
def test_tiny(kind, target):
    _flush(f"case mask tiny {kind} {target}")
    sh = synth.tiny_shape(d=16, hq=8, hkv=2, dh=64, f=48, layers=3)
    _check(sh, 4, target, 7, kind)


@pytest.mark.parametrize("granule", [1024, 128])
def test_llama3_8b(granule):
    _flush(f"case mask 8b granule={granule}")
    sh = synth.LLAMA3_8B
    q, kv, f = _check(sh, granule, 0.57, 1, "uniform")
    m = synth.mask_counts(q.astype(bool), kv.astype(bool), f.astype(bool))
    assert ref.active_flop_ratio(sh, m) <= 0.57


@pytest.mark.parametrize("granule,kind", [(1024, "uniform"), (128, "ties")])
def test_llama3_70b(granule, kind):
    """The paper's 70B candidate partition (64 heads + 28 groups of 1024 per layer, 7360 in all)
    and a finer one (224 groups of 128 per layer, 23040 candidates)."""
    _flush(f"case mask 70b granule={granule} {kind}")
    _check(synth.LLAMA3_70B, granule, 0.57, 2, kind)


def test_mask_compiles_into_a_plan():
    """The constructed mask feeds tasp_compile_plan unchanged (already closed)."""
    _flush("case mask -> plan")
    sh = synth.tiny_shape(d=64, hq=8, hkv=2, dh=64, f=128, layers=2)
    hs, cs = _scores(sh, 16, 3)
    q, kv, f, _ = _gpu(sh, hs, cs, 16, 0.5)
    store = S.DeviceStore([synth.layer_weights(sh, l) for l in range(2)])
    plan = S.Plan(S.desc_from_shape(sh), store, (q, kv, f))
    for l in range(2):
        assert plan.counts(l) == (int(q[l].sum()), int(kv[l].sum()), int(f[l].sum()))


def test_non_finite_score_rejected():
    _flush("case mask nan")
    sh = synth.tiny_shape(d=16, hq=4, hkv=2, dh=64, f=16)
    hs, cs = _scores(sh, 4, 1)
    hs[0, 1] = np.nan
    with pytest.raises(B.TaspError) as e:
        _gpu(sh, hs, cs, 4, 0.5)
    assert e.value.status == -1
