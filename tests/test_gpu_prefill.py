"""GPU parity of the prefill path (projections and causal attention on the matrix cores)
against the oracle's matrix-form prefill, plus cache contents and the prefill -> decode handoff."""
import numpy as np
import pytest
import torch

import synth
from oracle import reference as ref
from paper_2609_29499_amd import binding as B
from paper_2609_29499_amd import session as S
from tests.gpu_case import Case, PrefillCase
from tests.helpers import assert_parity

pytestmark = pytest.mark.gpu

SMALL = synth.tiny_shape(d=256, hq=8, hkv=2, dh=64, f=640, theta=500000.0)
SMALL128 = synth.tiny_shape(d=512, hq=16, hkv=4, dh=128, f=1024, theta=500000.0)


def _flush(msg):
    print(msg, flush=True)


def _check_cache(case):
    """Rows pos0..pos0+T-1 of retained groups hold the oracle's BF16 k / v (to the tolerance:
    the two sides round k, v from slightly different float values); prior rows are untouched."""
    sh, p0, T = case.sh, case.pos0, case.T
    for l in range(sh.n_layers):
        kv = case.closed[1][l]
        for which, bits, want in (("k", case.priors[l][0], case.oracle_caches[l][0]),
                                  ("v", case.priors[l][1], case.oracle_caches[l][1])):
            got = synth.bf16_bits_to_f32(case.cache.bits(which, l)[0]).astype(np.float64)
            assert np.array_equal(case.cache.bits(which, l)[0][:, :p0][kv], bits[0][:, :p0][kv])
            new, ref_new = got[kv][:, p0:p0 + T], want[kv][:, p0:p0 + T]
            if new.size:
                assert_parity(new, ref_new, what=f"prefill cache {which} layer {l}")


@pytest.mark.parametrize("masked", [True, False], ids=["tiny_mask", "dense"])
def test_tiny_layer_prefill(masked):
    _flush(f"case prefill tiny masked={masked}")
    sh = synth.TINY
    case = PrefillCase(sh, synth.tiny_mask(sh) if masked else None, 128, 0)
    got, want = case.run(), case.oracle()
    m, s = assert_parity(got, want, what="prefill tiny")
    _flush(f"  max_rel={m:.2e} sum_rel={s:.2e}")
    _check_cache(case)


def test_prefill_70b_width_split_k():
    """Llama-3-70B width (8192, 64 / 8 heads, d_h 128) with a narrow FFN, 256 tokens after 64
    prior positions: the 8192-row O and down panels and the QKV panel run as 256 tiles of 64
    tokens with K split 4 ways (down: 1024 / 32 = 32 k chunks)."""
    _flush("case prefill 70b width split k")
    sh = synth.tiny_shape(d=8192, hq=64, hkv=8, dh=128, f=1024, theta=500000.0)
    case = PrefillCase(sh, synth.raw_mask(sh, 12, p_q=0.7, p_kv=0.9), 256, 64)
    got, want = case.run(), case.oracle()
    m, s = assert_parity(got, want, what="prefill 70b width")
    _flush(f"  max_rel={m:.2e} sum_rel={s:.2e}")
    _check_cache(case)


@pytest.mark.parametrize("T,pos0", [(128, 0), (330, 100)])
def test_prefill_repeat_bit_exact(T, pos0):
    """The QKV, O and down GEMMs of these prefills split K (2 to 4 splits per tile, summed in split
    order by the reduction), and at 330 tokens after 100 prior positions the attention splits its
    longest query blocks over two workgroups (the second to finish combines the records, in an
    order-independent way): repeated prefills give the same bits."""
    _flush(f"case prefill repeat T={T} pos0={pos0}")
    sh = synth.TINY
    case = PrefillCase(sh, synth.tiny_mask(sh), T, pos0)
    first = case.run()
    for _ in range(3):
        assert np.array_equal(case.run(), first)
    assert_parity(first, case.oracle(), what="prefill repeat")


@pytest.mark.parametrize("T,pos0", [(1, 0), (77, 0), (77, 128), (130, 5), (200, 300)])
def test_prefill_ragged_and_offset(T, pos0):
    """Token counts that are not tile multiples, and prompts continuing a prior cache."""
    _flush(f"case prefill T={T} pos0={pos0}")
    sh = SMALL.with_layers(2)
    case = PrefillCase(sh, synth.raw_mask(sh, 11, p_q=0.6, p_kv=0.8), T, pos0, max_prefill=256)
    got, want = case.run(), case.oracle()
    assert_parity(got, want, what=f"prefill T={T} pos0={pos0}")
    _check_cache(case)


def test_prefill_group_of_eight_dh128():
    """Eight query heads per KV group (two heads per wave) with head_dim 128 and ragged groups."""
    _flush("case prefill group of eight")
    sh = synth.tiny_shape(d=512, hq=16, hkv=2, dh=128, f=768, theta=500000.0)
    q, kv, f = synth.all_kept_mask(sh)
    q[0, [2, 9, 10]] = 0
    f[0, ::3] = 0
    case = PrefillCase(sh, (q, kv, f), 96, 40)
    got, want = case.run(), case.oracle()
    assert_parity(got, want, what="prefill group of eight")
    _check_cache(case)


@pytest.mark.parametrize("what", ["no_heads", "no_ffn"])
def test_prefill_empty_modules(what):
    _flush(f"case prefill empty {what}")
    sh = SMALL.with_layers(2)
    q, kv, f = synth.all_kept_mask(sh)
    if what == "no_heads":
        q[0] = 0
    else:
        f[1] = 0
    case = PrefillCase(sh, (q, kv, f), 50, 0)
    got, want = case.run(), case.oracle()
    assert_parity(got, want, what=f"prefill {what}")


def test_prefill_stack_with_lm_head():
    _flush("case prefill stack + lm head")
    sh = synth.tiny_shape(d=256, hq=8, hkv=2, dh=64, f=512, layers=3, vocab=3000)
    case = PrefillCase(sh, synth.raw_mask(sh, 6), 40, 0)
    got, want = case.run(), case.oracle()
    assert_parity(got, want, what="prefill logits")
    assert (got.argmax(axis=1) == want.argmax(axis=1)).all()


def test_prefill_last_logits():
    """tasp_prefill_last: the last token's logits (the decode LM head over its final residual) at
    parity with the full prefill's last row and the oracle's, with the same cache rows, bit for
    bit; refused for a plan without an LM head."""
    _flush("case prefill last logits")
    sh = synth.tiny_shape(d=256, hq=8, hkv=2, dh=64, f=512, layers=3, vocab=3000)
    for T, pos0 in ((40, 0), (130, 20)):
        case = PrefillCase(sh, synth.raw_mask(sh, 6), T, pos0, max_seq=pos0 + T)
        init = [(case.cache.bits("k", l).copy(), case.cache.bits("v", l).copy())
                for l in range(sh.n_layers)]
        full = case.run()
        full_k = [case.cache.bits("k", l).copy() for l in range(sh.n_layers)]
        full_v = [case.cache.bits("v", l).copy() for l in range(sh.n_layers)]
        for l, (k0, v0) in enumerate(init):             # the cache as it was before the prefill
            case.cache.load_layer(l, k0, v0)
        last = torch.full((sh.vocab,), float("nan"), device="cuda")
        case.plan.prefill_last(case.xd, T, case.cache, pos0, last)
        torch.cuda.synchronize()
        got = last.cpu().numpy().astype(np.float64)
        for l in range(sh.n_layers):
            assert np.array_equal(case.cache.bits("k", l), full_k[l])
            assert np.array_equal(case.cache.bits("v", l), full_v[l])
        want = case.oracle()[T - 1]
        assert_parity(got, want, what=f"prefill last logits T={T}")
        assert_parity(got, full[T - 1], what=f"prefill last vs full T={T}")
        assert int(got.argmax()) == int(want.argmax())
    nolm = PrefillCase(synth.tiny_shape(d=256, hq=8, hkv=2, dh=64, f=512, layers=1), None, 8, 0)
    with pytest.raises(B.TaspError) as e:
        nolm.plan.prefill_last(nolm.xd, 8, nolm.cache, 0, torch.empty(256, device="cuda"))
    assert B.STATUS[e.value.status] == "TASP_ERR_UNSUPPORTED"


def test_prefill_then_decode():
    """The cache a GPU prefill leaves is the one the decode path continues from: prefill 100
    tokens, then decode token 100 on the GPU; compare with the oracle doing the same."""
    _flush("case prefill -> decode")
    sh = SMALL128.with_layers(2)
    mask = synth.raw_mask(sh, 12, p_q=0.7, p_kv=0.9)
    case = PrefillCase(sh, mask, 100, 0, max_seq=128)
    case.run()
    want_pf = case.oracle()
    x1 = synth.activations(1, sh.d_model, 9)
    out = torch.full((1, sh.d_model), float("nan"), device="cuda")
    case.plan.decode(torch.from_numpy(x1).cuda(), case.cache, 100, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    r = np.asarray(x1, np.float64)
    for l in range(sh.n_layers):
        W = ref.masked_layer(case.store[l], case.closed[0][l], case.closed[1][l], case.closed[2][l],
                             sh.head_dim)
        K, V = case.oracle_caches[l]
        r = ref.decode_layer(W, r, K[None], V[None], 100, sh)
    assert_parity(got, r, what="decode after prefill")
    assert np.isfinite(want_pf).all()


def test_prefill_token_matches_decode():
    """One prompt token at pos0 through prefill equals a decode step at pos = pos0 (different
    arithmetic on the two sides: compared to the tolerance)."""
    _flush("case prefill T=1 vs decode")
    sh = SMALL.with_layers(2)
    mask = synth.raw_mask(sh, 13)
    pf = PrefillCase(sh, mask, 1, 60, max_seq=64)
    got_pf = pf.run()
    dc = Case(sh, mask, 1, 60, max_seq=64, seed_x=3)
    got_dc = dc.run()
    assert_parity(got_pf, got_dc, what="prefill vs decode")


@pytest.mark.timeout(600)
def test_llama3_8b_prefill512_full_size():
    """One Llama-3-8B-shaped layer under the seed-1 budget mask: a 512-token prompt from an empty
    cache (the prefill benchmark workload)."""
    _flush("case 8b prefill 512")
    sh = synth.LLAMA3_8B.with_layers(1, vocab=0)
    case = PrefillCase(sh, synth.budget_mask(sh, 1), 512, 0)
    got, want = case.run(), case.oracle()
    m, s = assert_parity(got, want, what="8b prefill")
    _flush(f"  max_rel={m:.2e} sum_rel={s:.2e}")
    _check_cache(case)


@pytest.mark.timeout(600)
def test_llama3_8b_prefill2048_full_size():
    """One Llama-3-8B-shaped layer under the seed-1 budget mask: a 2048-token prompt from an empty
    cache, the prompt length of the timed request (Table "configuration")."""
    _flush("case 8b prefill 2048")
    sh = synth.LLAMA3_8B.with_layers(1, vocab=0)
    case = PrefillCase(sh, synth.budget_mask(sh, 1), 2048, 0)
    got, want = case.run(), case.oracle()
    m, s = assert_parity(got, want, what="prefill 8b 2048")
    _flush(f"  max_rel={m:.2e} sum_rel={s:.2e}")
    _check_cache(case)


@pytest.mark.timeout(600)
def test_llama3_8b_prefill_ragged_wide_tiles():
    """8B layer, seed-1 mask, 700 tokens after 48 prior positions: every projection's last
    128-token tile holds 60 tokens, at the full width of the layer."""
    _flush("case 8b prefill 700 at pos0 48")
    sh = synth.LLAMA3_8B.with_layers(1, vocab=0)
    case = PrefillCase(sh, synth.budget_mask(sh, 1), 700, 48)
    got, want = case.run(), case.oracle()
    m, s = assert_parity(got, want, what="prefill 8b 700")
    _flush(f"  max_rel={m:.2e} sum_rel={s:.2e}")
    _check_cache(case)


def test_prefill_errors():
    _flush("case prefill errors")
    sh = SMALL
    case = PrefillCase(sh, synth.raw_mask(sh, 1), 8, 0, max_seq=32, max_prefill=16)
    with pytest.raises(B.TaspError) as e:                 # T beyond max_prefill
        case.plan.prefill(case.xd, 17, case.cache, 0, case.out)
    assert e.value.status == -2
    with pytest.raises(B.TaspError) as e:                 # past the cache end
        case.plan.prefill(case.xd, 8, case.cache, 25, case.out)
    assert e.value.status == -5
    other = S.Plan(case.desc, case.dstore, synth.raw_mask(sh, 2))
    case.run()                                            # binds the cache to case.plan
    with pytest.raises(B.TaspError) as e:                 # continuing with another plan
        other.prefill(case.xd, 8, case.cache, 8, case.out)
    assert e.value.status == -6
    d0 = S.desc_from_shape(sh, max_batch=1, max_seq=32, max_prefill=0)
    p0 = S.Plan(d0, case.dstore, None)
    with pytest.raises(B.TaspError) as e:
        p0.prefill(case.xd, 8, case.cache, 0, case.out)
    assert e.value.status == -8
    d2 = S.desc_from_shape(sh, max_batch=2, max_seq=32, max_prefill=16)
    p2 = S.Plan(d2, case.dstore, None)
    c2 = S.KVCache(d2, 2, 32)
    with pytest.raises(B.TaspError) as e:
        p2.prefill(case.xd, 8, c2, 0, case.out)
    assert e.value.status == -2
