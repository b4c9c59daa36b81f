"""GPU parity of the compiled decode path against the CPU oracle, through the C ABI.

Integer work (closure, index lists, panels) must be bit-exact; floating-point outputs must meet
max|err| <= 1e-2 max|ref| and sum|err| / sum|ref| <= 2e-3 (tests.helpers.assert_parity)."""
import numpy as np
import pytest
import torch

import synth
from oracle import compact, reference as ref
from paper_2609_29499_amd import binding as B
from paper_2609_29499_amd import session as S
from tests.gpu_case import Case, PrefillCase
from tests.helpers import assert_parity, check_greedy_ids, rel_errors

pytestmark = pytest.mark.gpu

SMALL = synth.tiny_shape(d=256, hq=8, hkv=2, dh=64, f=640, theta=500000.0)
SMALL128 = synth.tiny_shape(d=512, hq=16, hkv=4, dh=128, f=1024, theta=500000.0)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.load()


def _flush(msg):
    print(msg, flush=True)


def _check_indices(case):
    sh = case.sh
    qc, kvc, fc = case.closed
    for l in range(sh.n_layers):
        qi, kvi, slot, fi = ref.index_lists(qc[l], kvc[l], fc[l], sh.group_size)
        assert case.plan.indices(l, B.IDX_Q) == qi.tolist()
        assert case.plan.indices(l, B.IDX_KV) == kvi.tolist()
        assert case.plan.indices(l, B.IDX_QKVSLOT) == slot.tolist()
        assert case.plan.indices(l, B.IDX_FFN) == fi.tolist()
        assert case.plan.counts(l) == (len(qi), len(kvi), len(fi))


@pytest.mark.parametrize("which", ["tiny_mask", "dense", "raw1", "raw2"])
def test_closure_indices_and_ledger_bit_exact(which):
    _flush(f"case closure {which}")
    sh = synth.TINY.with_layers(3)
    mask = {"tiny_mask": synth.tiny_mask(sh), "dense": None, "raw1": synth.raw_mask(sh, 1),
            "raw2": synth.raw_mask(sh, 2, p_q=0.3, p_kv=0.5)}[which]
    case = Case(sh, mask, batch=1, pos=4)
    _check_indices(case)
    counts = synth.mask_counts(*case.closed)
    led = case.plan.ledger()
    assert led["active_flop_ratio"] == pytest.approx(ref.active_flop_ratio(sh, counts), rel=1e-14)
    nb = ref.decode_bytes(sh, counts, batch=1, pos=0)
    assert led["weight_bytes"] == nb["weights"] and led["scale_bytes"] == nb["scales"]


def test_budget_masks_8b_indices():
    sh = synth.LLAMA3_8B.with_layers(32, vocab=0)
    for seed in (1, 2):
        q, kv, f = synth.budget_mask(sh, seed)
        desc = S.desc_from_shape(sh, max_seq=16)
        # closure/index lists on a store of one shared layer repeated: only indices are checked
        lay = synth.layer_weights(sh.with_layers(1), 0)
        dev = {k: tuple(torch.from_numpy(a).cuda() for a in v) if isinstance(v, tuple)
               else torch.from_numpy(v).cuda() for k, v in lay.items()}
        store = S.DeviceStore([dev] * sh.n_layers)
        plan = S.Plan(desc, store, (q, kv, f))
        closed = ref.close_mask(q, kv, f, sh.group_size)
        for l in range(0, 32, 7):
            qi, kvi, slot, fi = ref.index_lists(closed[0][l], closed[1][l], closed[2][l], sh.group_size)
            assert plan.indices(l, B.IDX_Q) == qi.tolist()
            assert plan.indices(l, B.IDX_KV) == kvi.tolist()
            assert plan.indices(l, B.IDX_QKVSLOT) == slot.tolist()
            assert plan.indices(l, B.IDX_FFN) == fi.tolist()
        del plan, store
        torch.cuda.empty_cache()


@pytest.mark.parametrize("sh", [synth.TINY, SMALL128], ids=["tiny", "dh128"])
def test_panels_byte_exact(sh):
    _flush(f"case panels {sh.d_model}")
    mask = synth.tiny_mask(sh) if sh is synth.TINY else synth.raw_mask(sh, 3)
    case = Case(sh, mask, batch=1, pos=2)
    qc, kvc, fc = case.closed
    pn = compact.compact_panels(case.store[0], qc[0], kvc[0], fc[0], sh)
    for which, key in ((B.PANEL_QKV, "qkv"), (B.PANEL_O, "o"), (B.PANEL_GATE, "gate"),
                       (B.PANEL_UP, "up"), (B.PANEL_DOWN, "down")):
        w, s, cols = case.plan.panel(0, which)
        w = w.cpu().numpy()
        s = s.cpu().numpy()
        assert cols == pn[key].shape[1]
        assert np.array_equal(w[:, :cols], pn[key]), key
        assert not w[:, cols:].any(), key                     # padding columns are zero
        assert np.array_equal(s, pn[key + "_scale"]), key


def _decode_case(sh, mask, batch, pos, max_seq=None, **kw):
    case = Case(sh, mask, batch, pos, max_seq=max_seq, **kw)
    got = case.run()
    want = case.oracle()
    return case, got, want


def _check_cache_rows(case):
    """Row pos of retained groups holds the BF16 new k / v; all other rows are untouched."""
    sh, pos = case.sh, case.pos
    for l in range(sh.n_layers):
        kvc = case.closed[1][l]
        for which, idx in (("k", 0), ("v", 1)):
            dev = case.cache.bits(which, l)
            prior = case.priors[l][idx]
            # rows below pos unchanged (bit-exact), other groups and rows above pos still NaN
            assert np.array_equal(dev[:, kvc, :pos], prior[:, kvc, :pos])
            assert (dev[:, ~kvc] == 0x7FC0).all()
            assert (dev[:, :, pos + 1:] == 0x7FC0).all()
            new = synth.bf16_bits_to_f32(dev[:, kvc, pos]).astype(np.float64)
            want = case.oracle_caches[l][idx][:, kvc, pos]
            if new.size:
                assert_parity(new, want, what=f"cache {which} layer {l}")


@pytest.mark.parametrize("masked", [True, False], ids=["tiny_mask", "dense"])
def test_tiny_layer_decode(masked):
    """The tiny single layer: 6/8 heads, 1024/1536 channels, 128 prior positions; plus dense."""
    _flush(f"case tiny decode masked={masked}")
    sh = synth.TINY
    case, got, want = _decode_case(sh, synth.tiny_mask(sh) if masked else None, 1, 128)
    m, s = assert_parity(got, want, what="tiny layer")
    _flush(f"  max_rel={m:.2e} sum_rel={s:.2e}")
    _check_cache_rows(case)


@pytest.mark.parametrize("seed,batch", [(1, 1), (2, 3), (5, 2)])
def test_raw_masks_and_batches(seed, batch):
    _flush(f"case raw mask seed={seed} batch={batch}")
    sh = SMALL.with_layers(2)
    case, got, want = _decode_case(sh, synth.raw_mask(sh, seed, p_q=0.5, p_kv=0.7), batch, 77,
                                   max_seq=100)
    assert_parity(got, want, what="raw mask")
    _check_cache_rows(case)


def test_head_dim_128_ragged_groups():
    _flush("case dh128 ragged")
    sh = SMALL128.with_layers(2)
    q, kv, f = synth.all_kept_mask(sh)
    q[0, [1, 2, 3, 5, 10, 11]] = 0               # groups keep 1, 3, 2 and 4 heads
    kv[1, 2] = 0
    q[1, :3] = 0
    f[0, 100:777] = 0
    case, got, want = _decode_case(sh, (q, kv, f), 2, 300, max_seq=333)
    assert_parity(got, want, what="dh128")
    _check_cache_rows(case)


@pytest.mark.parametrize("batch", [1, 3])
@pytest.mark.parametrize("what", ["no_heads", "no_ffn", "nothing"])
def test_empty_modules(what, batch):
    _flush(f"case empty {what} batch={batch}")
    sh = SMALL.with_layers(2)
    q, kv, f = synth.all_kept_mask(sh)
    if what in ("no_heads", "nothing"):
        q[0] = 0
    if what in ("no_ffn", "nothing"):
        f[1] = 0
    case, got, want = _decode_case(sh, (q, kv, f), batch, 9, max_seq=16)
    assert_parity(got, want, what=what)


@pytest.mark.parametrize("pos", [0, 1, 63, 64, 65, 511])
def test_positions_and_split_boundaries(pos):
    _flush(f"case pos={pos}")
    sh = SMALL
    case, got, want = _decode_case(sh, synth.raw_mask(sh, 4), 1, pos, max_seq=512)
    assert_parity(got, want, what=f"pos {pos}")
    _check_cache_rows(case)


@pytest.mark.parametrize("pos", [1087, 1088, 1500, 2047, 2175, 3000, 4095, 4097])
def test_long_context_splits(pos):
    """From 256 rows on the batch-1 attention takes splits of at least 128 rows (multiples of 64,
    at most 32 splits), the remainder in the last split: ragged last splits, 17 to 32 splits, two
    to four tiles per wave, head_dim 64 and 128. The new token's row is folded into the last split after its tiles,
    whether the cached rows fill those tiles (4095: 127 rows) or spill into one more (4097)."""
    _flush(f"case long context pos={pos}")
    for sh in (SMALL, synth.tiny_shape(d=512, hq=8, hkv=2, dh=128, f=1024, layers=1)):
        case, got, want = _decode_case(sh, synth.raw_mask(sh, 4), 1, pos, max_seq=pos + 1)
        assert_parity(got, want, what=f"pos {pos} dh {sh.head_dim}")
        _check_cache_rows(case)


@pytest.mark.parametrize("batch", [1, 2, 7])
def test_stack_with_lm_head_logits(batch):
    _flush(f"case stack + lm head batch={batch}")
    sh = synth.tiny_shape(d=256, hq=8, hkv=2, dh=64, f=512, layers=3, vocab=3000)
    case, got, want = _decode_case(sh, synth.raw_mask(sh, 6), batch, 40, max_seq=48)
    m, s = assert_parity(got, want, what="logits")
    assert (got.argmax(axis=1) == want.argmax(axis=1)).all()
    assert np.abs(got - want).max() < 2e-3 * max(1.0, np.abs(want).max())


@pytest.mark.parametrize("batch", [2, 5, 8])
def test_batched_tiny_layer(batch):
    """Batches of 2..8 run every projection on the matrix cores over hi/lo BF16 operands."""
    _flush(f"case batched tiny batch={batch}")
    sh = synth.TINY
    case, got, want = _decode_case(sh, synth.tiny_mask(sh), batch, 128)
    m, s = assert_parity(got, want, what="batched tiny")
    _flush(f"  max_rel={m:.2e} sum_rel={s:.2e}")
    _check_cache_rows(case)


@pytest.mark.parametrize("batch,pos", [(2, 255), (2, 256), (3, 1000), (5, 2049), (7, 3001), (2, 4096)])
def test_batched_attention_splits(batch, pos):
    """Batched attention splits the cache rows over about one workgroup per CU: split lengths of
    64-row multiples with a short last split (or none besides the new row), from one split to
    32, head_dim 64 and 128."""
    for sh in (SMALL, SMALL128):
        _flush(f"case batched splits batch={batch} pos={pos} dh={sh.head_dim}")
        case, got, want = _decode_case(sh, synth.raw_mask(sh, 12, p_q=0.7, p_kv=0.9), batch, pos,
                                       max_seq=pos + 1)
        assert_parity(got, want, what=f"batched splits {batch} x {pos} dh {sh.head_dim}")
        _check_cache_rows(case)


@pytest.mark.parametrize("pos", [0, 1, 129, 511])
def test_batched_positions(pos):
    _flush(f"case batched pos={pos}")
    sh = SMALL.with_layers(2)
    case, got, want = _decode_case(sh, synth.raw_mask(sh, 9, p_q=0.6, p_kv=0.8), 8, pos,
                                   max_seq=512)
    assert_parity(got, want, what=f"batched pos {pos}")
    _check_cache_rows(case)


def test_batched_tall_panels():
    """Hidden 8192 with 64 query heads: the QKV, O and down panels are tall enough for the
    two-row-tile batched kernels (RMS partials, residual and next-operand epilogues)."""
    _flush("case batched tall panels")
    sh = synth.tiny_shape(d=8192, hq=64, hkv=8, dh=128, f=1024, theta=500000.0)
    q, kv, f = synth.all_kept_mask(sh)
    q[0, 5:9] = 0
    f[0, 3::5] = 0
    case, got, want = _decode_case(sh, (q, kv, f), 3, 100, max_seq=128)
    m, s = assert_parity(got, want, what="tall panels")
    _flush(f"  max_rel={m:.2e} sum_rel={s:.2e}")
    _check_cache_rows(case)


@pytest.mark.parametrize("pos", [511, 512, 640])
def test_attention_splits_sized_to_residency(pos):
    """Eight sequences over eight groups of eight heads (head dimension 128): 64 (sequence, group)
    units, so the batched split rule takes four splits (about one workgroup per CU). 511 cache
    rows make four 128-row splits, the last one short; 512 fill them exactly (the new row folded
    into the last); 640 take three 192-row splits and a 64-row one."""
    _flush(f"case attention splits pos={pos}")
    sh = synth.tiny_shape(d=8192, hq=64, hkv=8, dh=128, f=512, theta=500000.0)
    q, kv, f = synth.all_kept_mask(sh)
    f[0, 1::3] = 0
    case, got, want = _decode_case(sh, (q, kv, f), 8, pos, max_seq=pos + 1)
    assert_parity(got, want, what=f"splits pos {pos}")
    _check_cache_rows(case)


@pytest.mark.timeout(600)
def test_llama3_8b_batch8_full_size():
    """One Llama-3-8B-shaped layer under the seed-1 budget mask, 8 sequences at 8192 prior
    positions each (batched decode)."""
    _flush("case 8b layer batch 8 pos 8192")
    sh = synth.LLAMA3_8B.with_layers(1, vocab=0)
    case, got, want = _decode_case(sh, synth.budget_mask(sh, 1), 8, 8192)
    m, s = assert_parity(got, want, what="8b batch 8")
    _flush(f"  max_rel={m:.2e} sum_rel={s:.2e}")
    _check_cache_rows(case)


def test_llama3_8b_layer_full_size():
    """One Llama-3-8B-shaped layer at 2048 prior positions: seed-1 budget mask and dense."""
    sh = synth.LLAMA3_8B.with_layers(1, vocab=0)
    store = [synth.layer_weights(sh, 0)]
    for mask in (synth.budget_mask(sh, 1), None):
        _flush(f"case 8b layer masked={mask is not None}")
        case, got, want = _decode_case(sh, mask, 1, 2048, store=store)
        m, s = assert_parity(got, want, what="8b layer")
        _flush(f"  max_rel={m:.2e} sum_rel={s:.2e}")
        _check_cache_rows(case)
        del case
        torch.cuda.empty_cache()


@pytest.mark.parametrize("batch", [1, 4])
def test_mask_as_zero_control(batch):
    """The mask-as-zero control at the Llama-3-8B layer shape (seed-1 budget mask, 512 prior
    positions): a dense plan over the store whose dropped modules' INT8 weights are zeroed runs
    the dense launch shapes yet computes the masked layer, so it meets the oracle's tolerance and
    agrees with the compiled sparse plan to float32 rounding."""
    _flush(f"case mask-as-zero control batch {batch}")
    sh = synth.LLAMA3_8B.with_layers(1, vocab=0)
    layer = synth.layer_weights(sh, 0)
    sp, got_sp, want = _decode_case(sh, synth.budget_mask(sh, 1), batch, 512, store=[layer])
    assert_parity(got_sp, want, what="compiled sparse")
    qc, kvc, fc = sp.closed
    del sp
    torch.cuda.empty_cache()
    zc = Case(sh, None, batch, 512, store=[synth.zero_dropped(layer, sh, qc[0], kvc[0], fc[0])])
    assert zc.plan.counts(0) == (sh.n_q_heads, sh.n_kv_heads, sh.d_ffn)
    got_z = zc.run()
    m, s = assert_parity(got_z, want, what="mask as zero")
    _flush(f"  max_rel={m:.2e} sum_rel={s:.2e}")
    assert np.abs(got_z - got_sp).max() <= 1e-4 * np.abs(got_sp).max()


@pytest.mark.parametrize("batch,f", [(1, 24576), (2, 12288)])
def test_wide_ffn_group_of_eight(batch, f):
    """Eight query heads per KV group and a down-projection input wider than 64 KiB of LDS
    (24576 channels at batch 1, 2 x 12288 at batch 2) on a narrow model."""
    _flush(f"case wide ffn batch={batch} f={f}")
    sh = synth.tiny_shape(d=256, hq=16, hkv=2, dh=128, f=f, theta=500000.0)
    q, kv, ff = synth.all_kept_mask(sh)
    q[0, 3] = 0
    ff[0, ::7] = 0
    case, got, want = _decode_case(sh, (q, kv, ff), batch, 70, max_seq=80)
    assert_parity(got, want, what="wide ffn")
    _check_cache_rows(case)


@pytest.mark.timeout(600)
def test_llama3_70b_layer_full_size():
    """One Llama-3-70B-shaped layer (8192, 64/8 heads, 28672): 8 query heads per KV group and a
    112 KiB down-projection input in LDS; seed-1 budget mask, 4096 prior positions."""
    _flush("case 70b layer")
    sh = synth.LLAMA3_70B.with_layers(1, vocab=0)
    case, got, want = _decode_case(sh, synth.budget_mask(sh, 1), 1, 4096)
    m, s = assert_parity(got, want, what="70b layer")
    _flush(f"  max_rel={m:.2e} sum_rel={s:.2e}")
    _check_cache_rows(case)


def test_llama3_8b_two_layer_stack_with_lm_head():
    """Full Llama-3-8B width: two layers under seed-2 budget masks, the dense BF16 LM head over
    the 128256-token vocabulary, 512 prior positions, batch 2; logits and greedy tokens."""
    _flush("case 8b 2-layer stack + lm head")
    sh = synth.LLAMA3_8B.with_layers(2)
    case, got, want = _decode_case(sh, synth.budget_mask(sh, 2), 2, 512)
    m, s = assert_parity(got, want, what="8b stack logits")
    _flush(f"  max_rel={m:.2e} sum_rel={s:.2e}")
    check_greedy_ids(got.argmax(axis=1), want, "8b stack")
    assert np.abs(got - want).max() < 2e-3 * max(1.0, np.abs(want).max())


@pytest.mark.timeout(900)
def test_llama3_70b_two_layer_stack_with_lm_head():
    """Full Llama-3-70B width (8192, 64 / 8 heads, 28672) with the dense 128256 x 8192 BF16 LM
    head (2,101,346,304 bytes: the largest panel one buffer resource addresses): two layers under
    the seed-1 budget mask, 256 prior positions, batch 1 (the VALU head) and batch 2 (the
    matrix-core head); then a 5-token prefill through the same stack, whose LM head runs as a
    GEMM. Logits at parity, every greedy token admissible."""
    sh = synth.LLAMA3_70B.with_layers(2)
    _flush("case 70b 2-layer stack + lm head: drawing the store")
    store = [synth.layer_weights(sh, l) for l in range(sh.n_layers)]
    lm = (synth.final_norm(sh), synth.lm_head(sh))
    mask = synth.budget_mask(sh, 1)
    for batch in (1, 2):
        _flush(f"case 70b 2-layer stack + lm head batch {batch}")
        case, got, want = _decode_case(sh, mask, batch, 256, store=store, lm=lm)
        m, s = assert_parity(got, want, what=f"70b stack logits batch {batch}")
        _flush(f"  max_rel={m:.2e} sum_rel={s:.2e}")
        check_greedy_ids(got.argmax(axis=1), want, f"70b stack batch {batch}")
        del case
        torch.cuda.empty_cache()
    _flush("case 70b 2-layer stack + lm head prefill T=5")
    pc = PrefillCase(sh, mask, 5, 0, store=store, lm=lm)
    got, want = pc.run(), pc.oracle()
    m, s = assert_parity(got, want, what="70b stack prefill logits")
    _flush(f"  max_rel={m:.2e} sum_rel={s:.2e}")
    check_greedy_ids(got.argmax(axis=1), want, "70b stack prefill")


@pytest.mark.parametrize("batch", [1, 4])
def test_repeat_and_graph_replay_are_stable(batch):
    """Repeated decode and HIP-graph replays give the eager result bit for bit."""
    _flush(f"case repeat + graph batch={batch}")
    sh = SMALL
    case = Case(sh, synth.raw_mask(sh, 7), batch, 200, max_seq=256)
    first = case.run()
    for _ in range(3):
        assert np.array_equal(case.run(), first)
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        case.plan.decode(case.xd, case.cache, case.pos, case.out, stream=S.current_stream())
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        case.plan.decode(case.xd, case.cache, case.pos, case.out, stream=S.current_stream())
    for _ in range(3):
        case.out.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(case.out.cpu().numpy().astype(np.float64), first)


@pytest.mark.parametrize("batch", [1, 3])
def test_profile_stage(batch):
    """The stage profiler times attention, gate/up and down over plan copies; it leaves the
    decode result unchanged and rejects a cache of another plan."""
    _flush(f"case profile stage batch={batch}")
    sh = SMALL
    case = Case(sh, synth.raw_mask(sh, 3), batch, 150, max_seq=160)
    first = case.run()
    for kind in (1, 3, 4):
        ms = B.tasp_profile_stage([case.plan.handle], [case.cache.struct], 0, kind, case.pos, 3,
                                  S.current_stream())
        assert ms > 0.0
    assert np.array_equal(case.run(), first)
    other = S.Plan(case.desc, case.dstore, synth.raw_mask(sh, 4))
    with pytest.raises(B.TaspError) as e:
        B.tasp_profile_stage([other.handle], [case.cache.struct], 0, 3, case.pos, 1,
                             S.current_stream())
    assert e.value.status == -6
    with pytest.raises(B.TaspError):
        B.tasp_profile_stage([case.plan.handle], [case.cache.struct], 0, 2, case.pos, 1,
                             S.current_stream())


def test_cache_plan_binding_errors():
    _flush("case errors")
    sh = SMALL
    a = Case(sh, synth.raw_mask(sh, 1), 1, 5, max_seq=8)
    b_mask = synth.raw_mask(sh, 2)
    plan_b = S.Plan(a.desc, a.dstore, b_mask)
    with pytest.raises(B.TaspError) as e:
        plan_b.decode(a.xd, a.cache, a.pos, a.out)
    assert e.value.status == -6
    same = S.Plan(a.desc, a.dstore, a.mask)
    assert same.ledger()["signature"] == a.plan.ledger()["signature"]
    assert plan_b.ledger()["signature"] != a.plan.ledger()["signature"]
    # the signature also names the store and the numerics: the same mask over a second copy of
    # the weights, or under another RMSNorm epsilon or RoPE base, gets a cache of its own
    sig = a.plan.ledger()["signature"]
    assert S.Plan(a.desc, S.DeviceStore(a.store), a.mask).ledger()["signature"] != sig
    d_eps = S.model_desc(sh.n_layers, sh.d_model, sh.n_q_heads, sh.n_kv_heads, sh.head_dim,
                         sh.d_ffn, sh.vocab, 1, 8, 0, 1e-6, sh.rope_theta)
    d_theta = S.model_desc(sh.n_layers, sh.d_model, sh.n_q_heads, sh.n_kv_heads, sh.head_dim,
                           sh.d_ffn, sh.vocab, 1, 8, 0, sh.rms_eps, 10000.0)
    for d in (d_eps, d_theta):
        other = S.Plan(d, a.dstore, a.mask)
        assert other.ledger()["signature"] != sig
        with pytest.raises(B.TaspError) as e:
            other.decode(a.xd, a.cache, a.pos, a.out)
        assert e.value.status == -6
    with pytest.raises(B.TaspError) as e:
        a.plan.decode(a.xd, a.cache, 8, a.out)
    assert e.value.status == -5
    with pytest.raises(B.TaspError) as e:
        a.plan.decode(a.xd, a.cache, 2, a.xd)
    assert e.value.status == -1
