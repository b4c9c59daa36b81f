"""GPU parity of the request loop (tasp_generate: embedding, prefill, device-side greedy ids,
decode steps) against the oracle, teacher-forced on the GPU's own ids.

Greedy ids are integers decided by floating point, so near ties can legitimately go either way.
The check therefore never stops at a near tie: the oracle is run along the GPU's sequence, every
step's id must be one whose oracle logit is within the parity tolerance of the oracle maximum,
and every step's logits (from the same kernels, stepped from the host) are compared with the
oracle's at the parity bar. The device-side loop must pick exactly the argmax of those logits."""
import numpy as np
import pytest
import torch

import synth
from oracle import reference as ref
from paper_2609_29499_amd import binding as B
from paper_2609_29499_amd import session as S
from tests.helpers import assert_parity, check_greedy_ids, teacher_forced_rows

pytestmark = pytest.mark.gpu


def _flush(msg):
    print(msg, flush=True)


def _embed(table, scales, ids):
    # float32 product of the INT8 row and its float32 scale, as the embedding kernel forms it
    ids = np.asarray(ids, np.int64)
    return (table[ids].astype(np.float32) * scales[ids, None]).astype(np.float32)


def _stepped_logits(plan, desc, table, scales, prompt, ids, S_):
    """The plan's logits at every step of the request, stepped from the host: prefill of the
    prompt (last token's logits only, as the device loop), then one decode step per generated id
    (the device loop's kernels on the same inputs)."""
    T, V = len(prompt), desc.vocab
    cache = S.KVCache(desc, 1, S_)
    out = torch.empty((V,), device="cuda")
    plan.prefill_last(torch.from_numpy(_embed(table, scales, prompt)).cuda(), T, cache, 0, out)
    rows = [out.clone()]
    o1 = torch.empty((1, V), device="cuda")
    for s_, i in enumerate(ids[:-1]):
        plan.decode(torch.from_numpy(_embed(table, scales, [i])).cuda(), cache, T + s_, o1)
        rows.append(o1[0].clone())
    torch.cuda.synchronize()
    return np.stack([r.cpu().numpy() for r in rows]).astype(np.float64)


def _run(sh, mask, T, n_new, max_seq=None, store=None):
    layers = store if store is not None else [synth.layer_weights(sh, l) for l in range(sh.n_layers)]
    fn, lm = synth.final_norm(sh), synth.lm_head(sh)
    table, scales = synth.embedding(sh)
    prompt = synth.prompt_ids(T, sh.vocab)
    S_ = max_seq or T + n_new
    desc = S.desc_from_shape(sh, max_batch=1, max_seq=S_, max_prefill=T)
    dstore = S.DeviceStore(layers, fn, lm)
    plan = S.Plan(desc, dstore, mask)
    cache = S.KVCache(desc, 1, S_)
    emb, sc = torch.from_numpy(table).cuda(), torch.from_numpy(scales).cuda()
    scratch = (torch.empty((T, sh.d_model), device="cuda"), torch.empty((T, sh.vocab), device="cuda"))
    ids = plan.generate(emb, sc, torch.from_numpy(prompt).cuda(), n_new, cache, scratch=scratch)
    torch.cuda.synchronize()
    got_ids = ids.cpu().numpy()
    last_logits = scratch[1][0 if n_new else T - 1].cpu().numpy().astype(np.float64)
    gpu_rows = _stepped_logits(plan, desc, table, scales, prompt, got_ids, S_)
    closed = ref.close_mask(*(mask if mask is not None else synth.all_kept_mask(sh)), sh.group_size)
    want_rows = teacher_forced_rows(lambda l: layers[l], closed, table, scales, prompt, got_ids, sh,
                                    fn, lm)
    return got_ids, gpu_rows, want_rows, last_logits


def _compare(got, gpu_rows, want_rows, last_logits):
    """Every step: the device loop's id is the argmax of the plan's logits (lowest id on ties),
    those logits are at parity with the oracle's along the same sequence, and the id is one the
    oracle admits within the tolerance. Returns the number of clear (non-tie) decisions."""
    assert len(got) == len(gpu_rows) == len(want_rows)
    np.testing.assert_array_equal(gpu_rows[-1], last_logits)
    for s in range(len(got)):
        assert got[s] == int(np.argmax(gpu_rows[s])), f"step {s}: device id {got[s]}"
        assert_parity(gpu_rows[s], want_rows[s], what=f"step {s} logits")
    return check_greedy_ids(got, want_rows, "request")


@pytest.mark.parametrize("masked", [True, False])
def test_tiny_stack_request(masked):
    _flush(f"case generate tiny masked={masked}")
    sh = synth.tiny_shape(d=256, hq=8, hkv=2, dh=64, f=512, layers=3, vocab=3000)
    got, gpu_rows, want_rows, last = _run(sh, synth.raw_mask(sh, 6) if masked else None, 20, 12)
    assert len(got) == 13
    _compare(got, gpu_rows, want_rows, last)


def test_prompt_only():
    _flush("case generate prompt only")
    sh = synth.tiny_shape(d=128, hq=4, hkv=2, dh=64, f=256, layers=2, vocab=500)
    got, gpu_rows, want_rows, last = _run(sh, None, 33, 0)
    assert len(got) == 1
    _compare(got, gpu_rows, want_rows, last)


def test_llama3_8b_width_two_layer_request():
    """Full 8B width, two layers, the 128256-row LM head and INT8 embedding: 64-token prompt and
    4 decode steps under the seed-2 budget mask."""
    _flush("case generate 8b width")
    sh = synth.LLAMA3_8B.with_layers(2)
    got, gpu_rows, want_rows, last = _run(sh, synth.budget_mask(sh, 2), 64, 4)
    assert len(got) == 5
    _compare(got, gpu_rows, want_rows, last)


def test_generate_errors():
    _flush("case generate errors")
    sh = synth.tiny_shape(d=128, hq=4, hkv=2, dh=64, f=256, layers=1, vocab=100)
    layers = [synth.layer_weights(sh, 0)]
    desc = S.desc_from_shape(sh, max_batch=1, max_seq=16, max_prefill=8)
    plan = S.Plan(desc, S.DeviceStore(layers, synth.final_norm(sh), synth.lm_head(sh)), None)
    cache = S.KVCache(desc, 1, 16)
    table, scales = synth.embedding(sh)
    emb, sc = torch.from_numpy(table).cuda(), torch.from_numpy(scales).cuda()
    prompt = torch.from_numpy(synth.prompt_ids(8, sh.vocab)).cuda()
    with pytest.raises(B.TaspError) as e:                 # 8 + 9 > 16 positions
        plan.generate(emb, sc, prompt, 9, cache)
    assert e.value.status == -5
    sh0 = synth.tiny_shape(d=128, hq=4, hkv=2, dh=64, f=256, layers=1, vocab=0)
    d0 = S.desc_from_shape(sh0, max_batch=1, max_seq=16, max_prefill=8)
    p0 = S.Plan(d0, S.DeviceStore(layers), None)
    with pytest.raises(B.TaspError) as e:                 # no LM head
        p0.generate(emb, sc, prompt, 2, S.KVCache(d0, 1, 16))
    assert e.value.status == -8
