"""GPU parity of the request loop (tasp_generate: embedding, prefill, device-side greedy ids,
decode steps) against the oracle's loop. Greedy ids are integers decided by floating point: they
are compared while the oracle's top-two margin clears the parity tolerance, after which a
different id would be a legitimate near-tie outcome."""
import numpy as np
import pytest
import torch

import synth
from oracle import reference as ref
from paper_2609_29499_amd import binding as B
from paper_2609_29499_amd import session as S
from tests.helpers import assert_parity

pytestmark = pytest.mark.gpu


def _flush(msg):
    print(msg, flush=True)


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
    closed = ref.close_mask(*(mask if mask is not None else synth.all_kept_mask(sh)), sh.group_size)
    caches = [(np.zeros((sh.n_kv_heads, S_, sh.head_dim)), np.zeros((sh.n_kv_heads, S_, sh.head_dim)))
              for _ in range(sh.n_layers)]
    want_ids, rows = ref.generate(lambda l: layers[l], closed, table, scales, prompt, n_new, caches, sh,
                                  fn, lm)
    return got_ids, want_ids, rows, last_logits


def _compare(got, want, rows, last_logits):
    """Ids equal while the oracle's decision is clear of the tolerance; the final logits at
    parity when the whole sequence was clear."""
    clear = 0
    for s in range(len(want)):
        top2 = np.sort(rows[s])[-2:]
        if top2[1] - top2[0] <= 1e-2 * np.abs(rows[s]).max():
            break
        assert got[s] == want[s], f"id {s}: {got[s]} vs {want[s]}"
        clear += 1
    if clear == len(want):
        assert_parity(last_logits, rows[-1], what="last logits")
    return clear


@pytest.mark.parametrize("masked", [True, False])
def test_tiny_stack_request(masked):
    _flush(f"case generate tiny masked={masked}")
    sh = synth.tiny_shape(d=256, hq=8, hkv=2, dh=64, f=512, layers=3, vocab=3000)
    got, want, rows, last = _run(sh, synth.raw_mask(sh, 6) if masked else None, 20, 12)
    assert len(got) == 13
    assert _compare(got, want, rows, last) >= 4


def test_prompt_only():
    _flush("case generate prompt only")
    sh = synth.tiny_shape(d=128, hq=4, hkv=2, dh=64, f=256, layers=2, vocab=500)
    got, want, rows, last = _run(sh, None, 33, 0)
    assert len(got) == 1
    _compare(got, want, rows, last)


def test_llama3_8b_width_two_layer_request():
    """Full 8B width, two layers, the 128256-row LM head and INT8 embedding: 64-token prompt and
    4 decode steps under the seed-2 budget mask."""
    _flush("case generate 8b width")
    sh = synth.LLAMA3_8B.with_layers(2)
    got, want, rows, last = _run(sh, synth.budget_mask(sh, 2), 64, 4)
    assert _compare(got, want, rows, last) >= 1


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
