"""Builds one decode case for the GPU parity tests: the synthetic store on the host and device,
a compiled plan, a NaN-poisoned device KV cache, and the oracle's result on the same inputs.

The device cache holds the synthetic prior rows 0..pos-1 of retained KV groups only; every other
row (later positions, dropped groups) is NaN, so any read of a row the path must not touch
shows up as a non-finite output. The oracle receives the same prior rows and finite zeros
elsewhere (its zero-masked dropped heads do read their group's rows, with no effect)."""
from __future__ import annotations

import numpy as np
import torch

import synth
from oracle import reference as ref
from paper_2609_29499_amd import session as S

NAN_BF16 = np.uint16(0x7FC0)


class Case:
    def __init__(self, sh, mask, batch, pos, max_seq=None, seed_w=0, seed_x=1, seed_kv=2,
                 with_lm_head=None, store=None, device="cuda", shared=False, lm=None):
        """shared: a groupwise store (BF16 scales per 128 inputs) and a shared-store plan;
        lm: a pre-drawn (final norm, LM head) pair for this shape (large heads are drawn once)."""
        self.sh, self.batch, self.pos = sh, batch, pos
        self.max_seq = max_seq or pos + 1
        self.mask = mask
        quant = "group" if shared else "row"
        self.store = store if store is not None else [synth.layer_weights(sh, l, seed_w, quant=quant)
                                                      for l in range(sh.n_layers)]
        pre = lm
        lm = sh.vocab > 0 if with_lm_head is None else with_lm_head
        self.final_norm, self.lm_head = (pre if pre is not None else
                                         (synth.final_norm(sh, seed_w), synth.lm_head(sh, seed_w))
                                         ) if lm else (None, None)
        self.closed = ref.close_mask(*(mask if mask is not None else synth.all_kept_mask(sh)),
                                     sh.group_size)
        self.x = synth.activations(batch, sh.d_model, seed_x)
        self.desc = S.desc_from_shape(sh, max_batch=batch, max_seq=self.max_seq)
        if shared:
            self.dstore = S.GroupStore(self.store, self.final_norm, self.lm_head, device)
            self.plan = S.Plan.shared(self.desc, self.dstore, mask)
        else:
            self.dstore = S.DeviceStore(self.store, self.final_norm, self.lm_head, device)
            self.plan = S.Plan(self.desc, self.dstore, mask)
        torch.cuda.synchronize()
        self.priors = [synth.kv_prior(sh, l, batch, pos, self.max_seq, seed_kv)
                       for l in range(sh.n_layers)]
        self.cache = S.KVCache(self.desc, batch, self.max_seq, device)
        for l, (k, v) in enumerate(self.priors):
            self.cache.load_layer(l, self._poison(k, l), self._poison(v, l))
        self.plan.bind(self.cache)
        self.xd = torch.from_numpy(self.x).to(device)
        n_out = sh.vocab if lm else sh.d_model
        self.out = torch.full((batch, n_out), float("nan"), device=device)

    def _poison(self, bits, layer):
        b = bits.copy()
        b[:, :, self.pos:] = NAN_BF16
        b[:, ~self.closed[1][layer]] = NAN_BF16
        return b

    def run(self):
        self.plan.decode(self.xd, self.cache, self.pos, self.out)
        torch.cuda.synchronize()
        return self.out.cpu().numpy().astype(np.float64)

    def oracle(self):
        caches = [(synth.bf16_bits_to_f32(k).astype(np.float64),
                   synth.bf16_bits_to_f32(v).astype(np.float64)) for k, v in self.priors]
        res = ref.decode_stack(lambda l: self.store[l], self.closed, self.x, caches, self.pos,
                               self.sh, self.final_norm, self.lm_head)
        self.oracle_caches = caches
        return res


class PrefillCase:
    """A prefill of T tokens of one sequence at pos0 (prior rows 0..pos0-1 from the synthetic
    cache, everything else NaN until the prefill writes it), with the oracle's result."""

    def __init__(self, sh, mask, T, pos0, max_seq=None, max_prefill=None, seed_w=0, seed_x=3,
                 seed_kv=2, store=None, device="cuda", lm=None, shared=False):
        """shared: a groupwise store (BF16 scales per 128 inputs) and a shared-store plan."""
        self.sh, self.T, self.pos0 = sh, T, pos0
        self.max_seq = max_seq or pos0 + T
        self.mask = mask
        quant = "group" if shared else "row"
        self.store = store if store is not None else [synth.layer_weights(sh, l, seed_w, quant=quant)
                                                      for l in range(sh.n_layers)]
        pre = lm
        lm = sh.vocab > 0
        self.final_norm, self.lm_head = (pre if pre is not None else
                                         (synth.final_norm(sh, seed_w), synth.lm_head(sh, seed_w))
                                         ) if lm else (None, None)
        self.closed = ref.close_mask(*(mask if mask is not None else synth.all_kept_mask(sh)),
                                     sh.group_size)
        self.x = synth.activations(T, sh.d_model, seed_x)
        self.desc = S.desc_from_shape(sh, max_batch=1, max_seq=self.max_seq,
                                      max_prefill=max_prefill or T)
        if shared:
            self.dstore = S.GroupStore(self.store, self.final_norm, self.lm_head, device)
            self.plan = S.Plan.shared(self.desc, self.dstore, mask)
        else:
            self.dstore = S.DeviceStore(self.store, self.final_norm, self.lm_head, device)
            self.plan = S.Plan(self.desc, self.dstore, mask)
        torch.cuda.synchronize()
        self.priors = [synth.kv_prior(sh, l, 1, pos0, self.max_seq, seed_kv)
                       for l in range(sh.n_layers)]
        self.cache = S.KVCache(self.desc, 1, self.max_seq, device)
        for l, (k, v) in enumerate(self.priors):
            b = k.copy(), v.copy()
            for a in b:
                a[:, :, pos0:] = NAN_BF16
                a[:, ~self.closed[1][l]] = NAN_BF16
            self.cache.load_layer(l, *b)
        if pos0 > 0:
            self.plan.bind(self.cache)
        self.xd = torch.from_numpy(self.x).to(device)
        self.out = torch.full((T, sh.vocab if lm else sh.d_model), float("nan"), device=device)

    def run(self):
        self.plan.prefill(self.xd, self.T, self.cache, self.pos0, self.out)
        torch.cuda.synchronize()
        return self.out.cpu().numpy().astype(np.float64)

    def oracle(self):
        caches = [(synth.bf16_bits_to_f32(k[0]).astype(np.float64),
                   synth.bf16_bits_to_f32(v[0]).astype(np.float64)) for k, v in self.priors]
        res = ref.prefill_stack(lambda l: self.store[l], self.closed, self.x, caches, self.pos0,
                                self.sh, self.final_norm, self.lm_head)
        self.oracle_caches = caches
        return res
