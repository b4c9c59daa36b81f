"""GPU parity of shared-store plans (groupwise INT8 with BF16 scales per 128 inputs; plans are
maps into one store and copy no weights) against the oracle, and the one-store validation: a
shared-store plan against a separately materialised plan at identical quantisation scales (max
absolute logit difference below 2e-3 and at least 99.98% greedy-token agreement, the targets
the paper states for its one-store check)."""
import numpy as np
import pytest
import torch

import synth
from paper_2609_29499_amd import binding as B
from paper_2609_29499_amd import session as S
from oracle import reference as ref
from tests.gpu_case import Case, PrefillCase
from tests.helpers import assert_parity, check_greedy_ids, teacher_forced_rows

pytestmark = pytest.mark.gpu


def _flush(msg):
    print(msg, flush=True)


def _check(case):
    got = case.run()
    want = case.oracle()
    return assert_parity(got, want, what="shared decode")


TINY = dict(d=256, hq=8, hkv=2, dh=64, f=512)


@pytest.mark.parametrize("seed,pos", [(1, 0), (2, 1), (3, 77), (4, 300)])
def test_tiny_layer_block_masks(seed, pos):
    _flush(f"case shared tiny seed={seed} pos={pos}")
    sh = synth.tiny_shape(layers=1, **TINY)
    _check(Case(sh, synth.raw_mask(sh, seed, block=16), 1, pos, shared=True))


def test_tiny_layer_dense_and_head_dim_128():
    _flush("case shared dense / dh128")
    sh = synth.tiny_shape(layers=1, **TINY)
    _check(Case(sh, None, 1, 64, shared=True))
    sh = synth.tiny_shape(d=512, hq=8, hkv=2, dh=128, f=1024, layers=1)
    _check(Case(sh, synth.raw_mask(sh, 5, block=16), 1, 129, shared=True))


def test_empty_modules():
    """A layer with no retained head and no channel: both branches add zero."""
    _flush("case shared empty modules")
    sh = synth.tiny_shape(layers=2, **TINY)
    q, kv, f = synth.all_kept_mask(sh)
    q[0, :] = 0
    f[1, :] = 0
    f[0, 64:128] = 0
    _check(Case(sh, (q, kv, f), 1, 33, shared=True))


def test_stack_with_lm_head():
    _flush("case shared stack + LM head")
    sh = synth.tiny_shape(layers=3, vocab=3000, **TINY)
    case = Case(sh, synth.raw_mask(sh, 6, block=16), 1, 40, shared=True)
    got = case.run()
    want = case.oracle()
    assert_parity(got, want, what="logits")
    margin = np.sort(want[0])[-2:]
    if margin[1] - margin[0] > 1e-2 * np.abs(want).max():
        assert int(np.argmax(got[0])) == int(np.argmax(want[0]))


def test_llama3_8b_layer_budget_mask():
    """Full Llama-3-8B layer, seed-1 budget mask (128-channel granules), 2048 prior positions."""
    _flush("case shared 8B layer")
    sh = synth.LLAMA3_8B.with_layers(1, vocab=0)
    _check(Case(sh, synth.budget_mask(sh, 1), 1, 2048, shared=True))


def test_wide_inputs_staged_in_several_batches():
    """Inputs wider than one batch of staging loads: a gain-applying projection with K = 8320
    (more than 8 float4 loads per thread) and a down projection with 12416 retained channels (more
    than 12), dense and under a block mask, plus the dense 8B layer (down K = 14336)."""
    sh = synth.tiny_shape(d=8320, hq=8, hkv=2, dh=128, f=12416, layers=1)
    _flush("case shared wide inputs dense")
    _check(Case(sh, None, 1, 37, shared=True))
    _flush("case shared wide inputs block mask")
    _check(Case(sh, synth.raw_mask(sh, 11, block=16), 1, 37, shared=True))
    _flush("case shared 8B layer dense")
    _check(Case(synth.LLAMA3_8B.with_layers(1, vocab=0), None, 1, 40, shared=True))


def test_graph_replay_and_timed_kernels():
    _flush("case shared graph replay")
    sh = synth.tiny_shape(layers=2, **TINY)
    case = Case(sh, synth.raw_mask(sh, 7, block=16), 1, 50, shared=True)
    eager = case.run().copy()
    g = torch.cuda.CUDAGraph()
    st = torch.cuda.Stream()
    st.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(st):
        case.plan.decode(case.xd, case.cache, case.pos, case.out, stream=S.current_stream())
    torch.cuda.current_stream().wait_stream(st)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        case.plan.decode(case.xd, case.cache, case.pos, case.out, stream=S.current_stream())
    for rep in range(3):
        case.out.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(case.out.cpu().numpy().astype(np.float64), eager), rep
    kinds = [k for k, _ in case.plan.decode_timed(case.xd, case.cache, case.pos, case.out)]
    assert kinds == ["qkv_gemv", "attention", "o_gemv", "gateup_gemv", "down_gemv"] * 2


def test_shared_plans_own_no_weights():
    """Five masks over one store, prefill and batches enabled: every plan's workspace has the
    same small size (metadata), all five share one scratch arena, no weights are copied, and
    the device allocation grows by the workspaces and the arena only. Requests then alternate
    over the five plans on the shared arena at parity with the oracle."""
    _flush("case shared memory ledger")
    sh = synth.tiny_shape(layers=2, vocab=1000, **TINY)
    layers = [synth.layer_weights(sh, l, quant="group") for l in range(sh.n_layers)]
    desc = S.desc_from_shape(sh, max_batch=4, max_seq=256, max_prefill=64)
    store = S.GroupStore(layers, synth.final_norm(sh), synth.lm_head(sh))
    torch.cuda.synchronize()
    before = torch.cuda.memory_allocated()
    arena = S.SharedScratch(desc)
    masks = [synth.raw_mask(sh, 10 + i, block=16) for i in range(5)]
    plans = [S.Plan.shared(desc, store, m, scratch=arena) for m in masks]
    torch.cuda.synchronize()
    grown = torch.cuda.memory_allocated() - before
    ws = {p.ws_bytes for p in plans}
    assert len(ws) == 1
    assert grown <= 5 * (ws.pop() + 1024) + arena.bytes + 1024
    # prefill then decode on each plan in turn, all on the one arena
    table, scales = synth.embedding(sh)
    fn, lm = synth.final_norm(sh), synth.lm_head(sh)
    T = 12
    for i in (0, 3, 1, 4, 2, 0):
        prompt = synth.prompt_ids(T + 1, sh.vocab, seed=40 + i)
        x = ref.embed_rows(table, scales, prompt).astype(np.float32).astype(np.float64)
        cache = S.KVCache(desc, 1, 64)
        out = torch.empty((T, sh.vocab), device="cuda")
        plans[i].prefill(torch.from_numpy(x[:T].astype(np.float32)).cuda(), T, cache, 0, out)
        o1 = torch.empty((1, sh.vocab), device="cuda")
        plans[i].decode(torch.from_numpy(x[T:].astype(np.float32)).cuda(), cache, T, o1)
        torch.cuda.synchronize()
        closed = ref.close_mask(*masks[i], sh.group_size)
        caches = [(np.zeros((sh.n_kv_heads, T + 1, sh.head_dim)), np.zeros((sh.n_kv_heads, T + 1, sh.head_dim)))
                  for _ in range(sh.n_layers)]
        want = ref.prefill_stack(lambda l: layers[l], closed, x, caches, 0, sh, fn, lm)
        got = np.concatenate([out.cpu().numpy(), o1.cpu().numpy()]).astype(np.float64)
        assert_parity(got, want, what=f"plan {i} on the shared arena")
    # a materialised plan of the same mask holds its panels
    mat = S.Plan(S.desc_from_shape(sh, max_batch=1, max_seq=256),
                 S.DeviceStore([synth.layer_weights(sh, l) for l in range(2)], synth.final_norm(sh),
                               synth.lm_head(sh)), synth.raw_mask(sh, 10, block=16))
    assert mat.ws_bytes > plans[0].ws_bytes + plans[0].ledger()["weight_bytes"]
    # equal masks: equal signatures within a format, different across formats
    again = S.Plan.shared(desc, store, synth.raw_mask(sh, 10, block=16))
    assert again.ledger()["signature"] == plans[0].ledger()["signature"]
    assert mat.ledger()["signature"] != plans[0].ledger()["signature"]


def test_shared_plan_rejections():
    _flush("case shared rejections")
    sh = synth.tiny_shape(layers=1, **TINY)
    layers = [synth.layer_weights(sh, 0, quant="group")]
    store = S.GroupStore(layers)
    desc = S.desc_from_shape(sh, max_batch=1, max_seq=64)
    with pytest.raises(B.TaspError, match="UNSUPPORTED"):
        S.Plan.shared(desc, store, synth.raw_mask(sh, 1))          # per-channel FFN bits
    plan = S.Plan.shared(desc, store, synth.raw_mask(sh, 1, block=16))
    with pytest.raises(B.TaspError, match="UNSUPPORTED"):
        plan.panel(0, B.PANEL_QKV)
    cache = S.KVCache(desc, 1, 64)
    # a cache filled under the per-row plan of the same mask is refused
    mat = S.Plan(desc, S.DeviceStore([synth.layer_weights(sh, 0)]), synth.raw_mask(sh, 1, block=16))
    mat.bind(cache)
    with pytest.raises(B.TaspError, match="CACHE_PLAN_MISMATCH"):
        plan.decode(torch.zeros((1, sh.d_model), device="cuda"), cache, 3,
                    torch.empty((1, sh.d_model), device="cuda"))


def _equal_scale_stores(sh):
    """The same INT8 bytes as a per-row store (BF16-valued float32 scales) and as a groupwise
    store whose group scales all equal the row's: identical quantisation in the two formats."""
    rows, groups = [], []
    for l in range(sh.n_layers):
        lw = synth.layer_weights(sh, l, quant="row_bf16")
        gw = dict(lw)
        for n in synth.WEIGHT_NAMES:
            q, s = lw[n]
            gw[n] = (q, np.repeat(synth.to_bf16_bits(s)[:, None], q.shape[1] // 128, axis=1))
        rows.append(lw)
        groups.append(gw)
    return rows, groups


def test_one_store_validation_greedy_decode():
    """Shared-store vs materialised plans of three masks, 48 greedy steps each from the same
    start: max |logit difference| < 2e-3 and >= 99.98% token agreement (teacher-forced on the
    materialised plan's tokens so every step compares the same history)."""
    _flush("case one-store validation")
    sh = synth.tiny_shape(layers=4, vocab=4000, **TINY)
    rows, groups = _equal_scale_stores(sh)
    fn, lm = synth.final_norm(sh), synth.lm_head(sh)
    table, scales = synth.embedding(sh)
    steps = 48
    desc = S.desc_from_shape(sh, max_batch=1, max_seq=steps + 1)
    mstore = S.DeviceStore(rows, fn, lm)
    gstore = S.GroupStore(groups, fn, lm)
    worst, agree, total = 0.0, 0, 0
    for seed in (21, 22, 23):
        mask = synth.raw_mask(sh, seed, block=16)
        pm, ps = S.Plan(desc, mstore, mask), S.Plan.shared(desc, gstore, mask)
        cm, cs = S.KVCache(desc, 1, steps + 1), S.KVCache(desc, 1, steps + 1)
        pm.bind(cm)
        ps.bind(cs)
        tok = 7
        lm_out = torch.empty((1, sh.vocab), device="cuda")
        ls_out = torch.empty((1, sh.vocab), device="cuda")
        for pos in range(steps):
            x = torch.from_numpy((table[tok].astype(np.float32) * scales[tok])[None, :]).cuda()
            pm.decode(x, cm, pos, lm_out)
            ps.decode(x, cs, pos, ls_out)
            torch.cuda.synchronize()
            a, b = lm_out.cpu().numpy()[0], ls_out.cpu().numpy()[0]
            assert np.all(np.isfinite(b))
            worst = max(worst, float(np.abs(a - b).max()))
            agree += int(np.argmax(a) == np.argmax(b))
            total += 1
            tok = int(np.argmax(a))
    assert worst < 2e-3, worst
    assert agree / total >= 0.9998, (agree, total)


# ---- prefill and batched decode from the shared store (matrix cores: each weight times its
# group scale split exactly into BF16 hi and lo parts)


@pytest.mark.parametrize("batch,pos", [(2, 0), (5, 77), (8, 130)])
def test_batched_decode(batch, pos):
    _flush(f"case shared batched decode B={batch} pos={pos}")
    sh = synth.tiny_shape(layers=2, **TINY)
    _check(Case(sh, synth.raw_mask(sh, 40 + batch, block=16), batch, pos, shared=True))


def test_batched_decode_head_dim_128_and_empty_modules():
    _flush("case shared batched decode dh128 / empty modules")
    sh = synth.tiny_shape(d=512, hq=8, hkv=2, dh=128, f=1024, layers=1)
    _check(Case(sh, synth.raw_mask(sh, 5, block=16), 3, 129, shared=True))
    sh = synth.tiny_shape(layers=2, **TINY)
    q, kv, f = synth.all_kept_mask(sh)
    q[0, :] = 0
    f[1, :] = 0
    _check(Case(sh, (q, kv, f), 4, 33, shared=True))


@pytest.mark.parametrize("T,pos0", [(77, 0), (40, 33), (1, 5)])
def test_prefill(T, pos0):
    _flush(f"case shared prefill T={T} pos0={pos0}")
    sh = synth.tiny_shape(layers=2, **TINY)
    case = PrefillCase(sh, synth.raw_mask(sh, 50 + T, block=16), T, pos0, shared=True)
    got, want = case.run(), case.oracle()
    m, s_ = assert_parity(got, want, what="shared prefill")
    _flush(f"  max_rel={m:.2e} sum_rel={s_:.2e}")


def test_prefill_head_dim_128_empty_modules_and_lm_head():
    _flush("case shared prefill dh128 / empty / lm head")
    sh = synth.tiny_shape(d=512, hq=8, hkv=2, dh=128, f=1024, layers=1)
    case = PrefillCase(sh, synth.raw_mask(sh, 7, block=16), 130, 0, shared=True)
    assert_parity(case.run(), case.oracle(), what="shared prefill dh128")
    sh = synth.tiny_shape(layers=2, **TINY)
    q, kv, f = synth.all_kept_mask(sh)
    q[1, :] = 0
    f[0, :] = 0
    case = PrefillCase(sh, (q, kv, f), 20, 0, shared=True)
    assert_parity(case.run(), case.oracle(), what="shared prefill empty modules")
    sh = synth.tiny_shape(layers=3, vocab=3000, **TINY)
    case = PrefillCase(sh, synth.raw_mask(sh, 8, block=16), 9, 0, shared=True)
    got, want = case.run(), case.oracle()
    assert_parity(got, want, what="shared prefill logits")
    check_greedy_ids(got.argmax(axis=1), want, "shared prefill")


@pytest.mark.timeout(600)
def test_llama3_8b_layer_prefill_and_batch8():
    """Full Llama-3-8B layer from the groupwise store under the seed-1 budget mask: a 512-token
    prefill, and decode of 8 sequences at 2048 prior positions."""
    sh = synth.LLAMA3_8B.with_layers(1, vocab=0)
    store = [synth.layer_weights(sh, 0, quant="group")]
    mask = synth.budget_mask(sh, 1)
    _flush("case shared 8B prefill 512")
    case = PrefillCase(sh, mask, 512, 0, store=store, shared=True)
    m, s_ = assert_parity(case.run(), case.oracle(), what="shared 8B prefill")
    _flush(f"  max_rel={m:.2e} sum_rel={s_:.2e}")
    del case
    torch.cuda.empty_cache()
    _flush("case shared 8B batch 8")
    m, s_ = _check(Case(sh, mask, 8, 2048, store=store, shared=True))
    _flush(f"  max_rel={m:.2e} sum_rel={s_:.2e}")


def test_generate_on_shared_plan():
    """tasp_generate on a shared-store plan (prefill + greedy decode from the one store),
    teacher-forced against the oracle."""
    _flush("case shared generate")
    sh = synth.tiny_shape(layers=3, vocab=3000, **TINY)
    layers = [synth.layer_weights(sh, l, quant="group") for l in range(sh.n_layers)]
    fn, lm = synth.final_norm(sh), synth.lm_head(sh)
    table, scales = synth.embedding(sh)
    T, n_new = 24, 10
    prompt = synth.prompt_ids(T, sh.vocab, seed=12)
    mask = synth.raw_mask(sh, 9, block=16)
    desc = S.desc_from_shape(sh, max_batch=1, max_seq=T + n_new, max_prefill=T)
    plan = S.Plan.shared(desc, S.GroupStore(layers, fn, lm), mask)
    cache = S.KVCache(desc, 1, T + n_new)
    scratch = (torch.empty((T, sh.d_model), device="cuda"), torch.empty((T, sh.vocab), device="cuda"))
    ids = plan.generate(torch.from_numpy(table).cuda(), torch.from_numpy(scales).cuda(),
                        torch.from_numpy(prompt).cuda(), n_new, cache, scratch=scratch)
    torch.cuda.synchronize()
    got = ids.cpu().numpy()
    last = scratch[1][0].cpu().numpy().astype(np.float64)
    closed = ref.close_mask(*mask, sh.group_size)
    rows = teacher_forced_rows(lambda l: layers[l], closed, table, scales, prompt, got, sh, fn, lm)
    check_greedy_ids(got, rows, "shared generate")
    assert_parity(last, rows[-1], what="shared generate last logits")


def test_one_store_validation_prefill_and_batches():
    """The one-store validation with prefill and batched decode: shared-store vs materialised
    plans (identical quantisation) over a 32-token prefill (logits of every position) and 16
    teacher-forced decode steps of 4 sequences: max |logit difference| < 2e-3 and >= 99.98 %
    greedy agreement."""
    _flush("case one-store validation prefill + batches")
    sh = synth.tiny_shape(layers=3, vocab=4000, **TINY)
    rows, groups = _equal_scale_stores(sh)
    fn, lm = synth.final_norm(sh), synth.lm_head(sh)
    table, scales = synth.embedding(sh)
    T, steps, Bt = 32, 16, 4
    desc = S.desc_from_shape(sh, max_batch=Bt, max_seq=T + steps, max_prefill=T)
    mstore, gstore = S.DeviceStore(rows, fn, lm), S.GroupStore(groups, fn, lm)
    emb = lambda ids: torch.from_numpy(  # noqa: E731
        (table[np.asarray(ids)].astype(np.float32) * scales[np.asarray(ids), None]).astype(np.float32)).cuda()
    worst, agree, total = 0.0, 0, 0
    arena = S.SharedScratch(desc)                 # one scratch arena for both shared plans
    for seed in (31, 32):
        mask = synth.raw_mask(sh, seed, block=16)
        pm, ps = S.Plan(desc, mstore, mask), S.Plan.shared(desc, gstore, mask, scratch=arena)
        # prefill of one sequence
        prompt = synth.prompt_ids(T, sh.vocab, seed=seed)
        outs = []
        for plan in (pm, ps):
            c1 = S.KVCache(desc, 1, T + steps)
            o = torch.empty((T, sh.vocab), device="cuda")
            plan.prefill(emb(prompt), T, c1, 0, o)
            outs.append(o.cpu().numpy())
        worst = max(worst, float(np.abs(outs[0] - outs[1]).max()))
        agree += int((outs[0].argmax(1) == outs[1].argmax(1)).sum())
        total += T
        # batched decode of Bt sequences from position 0, teacher-forced on the materialised ids
        cm, cs = S.KVCache(desc, Bt, T + steps), S.KVCache(desc, Bt, T + steps)
        pm.bind(cm)
        ps.bind(cs)
        toks = [7, 11, 13, 17]
        om = torch.empty((Bt, sh.vocab), device="cuda")
        os_ = torch.empty((Bt, sh.vocab), device="cuda")
        for pos in range(steps):
            x = emb(toks)
            pm.decode(x, cm, pos, om)
            ps.decode(x, cs, pos, os_)
            torch.cuda.synchronize()
            a, b = om.cpu().numpy(), os_.cpu().numpy()
            assert np.all(np.isfinite(b))
            worst = max(worst, float(np.abs(a - b).max()))
            agree += int((a.argmax(1) == b.argmax(1)).sum())
            total += Bt
            toks = [int(v) for v in a.argmax(1)]
    assert worst < 2e-3, worst
    assert agree / total >= 0.9998, (agree, total)
