"""Device-memory plumbing around the C ABI: PyTorch tensors own the INT8 store, the plan
workspace, activations and the KV cache; this module only builds the ABI structs from them and
forwards calls. No arithmetic of the decode path happens here.
"""
from __future__ import annotations

import ctypes as C

import numpy as np
import torch

from . import binding as B  # noqa: F401  (re-exported for callers)

WEIGHT_NAMES = ("wq", "wk", "wv", "wo", "wg", "wu", "wd")


def model_desc(n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ffn, vocab=0, max_batch=1,
               max_seq=4096, max_prefill=0, rms_eps=1e-5, rope_theta=500000.0):
    return B.tasp_model_desc(n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ffn, vocab,
                             max_batch, max_seq, max_prefill, rms_eps, 0.0, rope_theta)


def desc_from_shape(sh, max_batch=1, max_seq=4096, max_prefill=0):
    """``sh`` is any object with the Shape fields (n_layers, d_model, ...)."""
    return model_desc(sh.n_layers, sh.d_model, sh.n_q_heads, sh.n_kv_heads, sh.head_dim, sh.d_ffn,
                      sh.vocab, max_batch, max_seq, max_prefill, sh.rms_eps, sh.rope_theta)


def current_stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev(a, device):
    t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(device)


class DeviceStore:
    """The INT8 store on the device. ``layers`` is a list of dicts ``name: (int8 [out][in],
    float32 [out])`` plus ``attn_norm`` / ``ffn_norm`` BF16 bits (uint16 [d]); a layer may also be
    given directly as device tensors with the same keys."""

    def __init__(self, layers, final_norm=None, lm_head=None, device="cuda"):
        self.tensors = []
        arr = (B.tasp_layer * len(layers))()
        for i, lay in enumerate(layers):
            keep = {}
            for n in WEIGHT_NAMES:
                w, s = lay[n]
                w = w if torch.is_tensor(w) else _dev(w, device)
                s = s if torch.is_tensor(s) else _dev(s, device)
                keep[n] = (w, s)
                setattr(arr[i], n, B.tasp_qmat(w.data_ptr(), s.data_ptr()))
            for n in ("attn_norm", "ffn_norm"):
                g = lay[n] if torch.is_tensor(lay[n]) else _dev(lay[n], device)
                keep[n] = g
                setattr(arr[i], n, g.data_ptr())
            self.tensors.append(keep)
        self.final_norm = None if final_norm is None else (
            final_norm if torch.is_tensor(final_norm) else _dev(final_norm, device))
        self.lm_head = None if lm_head is None else (
            lm_head if torch.is_tensor(lm_head) else _dev(lm_head, device))
        self._layers = arr
        self.struct = B.tasp_store(arr, self.final_norm.data_ptr() if self.final_norm is not None else None,
                                   self.lm_head.data_ptr() if self.lm_head is not None else None)


class GroupStore:
    """The packed groupwise store on the device. ``layers`` is a list of dicts ``name: (int8
    [out][in], BF16 scale bits uint16 [out][in / 128])`` for wq, wk, wv, wo, wg, wu, wd plus the
    two gains; wq, wk and wv are stacked into the store's QKV matrix (layout only). A layer may
    also be given as device tensors with the same keys (scale bits as int16)."""

    def __init__(self, layers, final_norm=None, lm_head=None, device="cuda"):
        self.tensors = []
        arr = (B.tasp_glayer * len(layers))()
        for i, lay in enumerate(layers):
            keep = {}
            on_dev = torch.is_tensor(lay["wq"][0])
            cat = torch.cat if on_dev else np.concatenate
            qkv = (cat([lay["wq"][0], lay["wk"][0], lay["wv"][0]]),
                   cat([lay["wq"][1], lay["wk"][1], lay["wv"][1]]))
            for n, (w, sc) in (("wqkv", qkv), ("wo", lay["wo"]), ("wg", lay["wg"]),
                               ("wu", lay["wu"]), ("wd", lay["wd"])):
                if on_dev:
                    w, sc = w.contiguous(), sc.contiguous().view(torch.int16)
                else:
                    w, sc = _dev(w, device), _dev(np.ascontiguousarray(sc, np.uint16).view(np.int16), device)
                keep[n] = (w, sc)
                setattr(arr[i], n, B.tasp_gqmat(w.data_ptr(), sc.data_ptr()))
            for n in ("attn_norm", "ffn_norm"):
                g = lay[n] if torch.is_tensor(lay[n]) else _dev(lay[n], device)
                keep[n] = g
                setattr(arr[i], n, g.data_ptr())
            self.tensors.append(keep)
        self.final_norm = None if final_norm is None else (
            final_norm if torch.is_tensor(final_norm) else _dev(final_norm, device))
        self.lm_head = None if lm_head is None else (
            lm_head if torch.is_tensor(lm_head) else _dev(lm_head, device))
        self._layers = arr
        self.struct = B.tasp_gstore(arr, self.final_norm.data_ptr() if self.final_norm is not None else None,
                                    self.lm_head.data_ptr() if self.lm_head is not None else None)

    def nbytes(self):
        n = sum(t.numel() * t.element_size() for lay in self.tensors for v in lay.values()
                for t in (v if isinstance(v, tuple) else (v,)))
        for t in (self.final_norm, self.lm_head):
            if t is not None:
                n += t.numel() * t.element_size()
        return n


def mask_struct(mask):
    """(q_keep, kv_keep or None, ffn_keep) uint8 numpy arrays -> (tasp_mask, keepalive)."""
    if mask is None:
        return None, None
    q, kv, f = (None if a is None else np.ascontiguousarray(a, dtype=np.uint8) for a in mask)
    m = B.tasp_mask(q.ctypes.data, None if kv is None else kv.ctypes.data, f.ctypes.data)
    return C.pointer(m), (q, kv, f, m)


class KVCache:
    """BF16 K and V ``[L][B][Hkv][S][dh]`` owned by torch."""

    def __init__(self, desc, batch, max_seq, device="cuda", fill=0.0):
        shp = (desc.n_layers, batch, desc.n_kv_heads, max_seq, desc.head_dim)
        self.k = torch.full(shp, fill, dtype=torch.bfloat16, device=device)
        self.v = torch.full(shp, fill, dtype=torch.bfloat16, device=device)
        self.struct = B.tasp_kv_cache(self.k.data_ptr(), self.v.data_ptr(), batch, max_seq, 0)

    def load_layer(self, layer, k_bits, v_bits):
        """Copy BF16 bit patterns ``uint16 [B][Hkv][S][dh]`` into one layer."""
        self.k[layer].copy_(torch.from_numpy(np.ascontiguousarray(k_bits)).view(torch.bfloat16))
        self.v[layer].copy_(torch.from_numpy(np.ascontiguousarray(v_bits)).view(torch.bfloat16))

    def bits(self, which, layer):
        t = self.k if which == "k" else self.v
        return t[layer].view(torch.int16).cpu().numpy().view(np.uint16)


class SharedScratch:
    """Decode / prefill scratch arena that several shared-store plans of one desc may share
    (their calls must then run in order, e.g. on one stream)."""

    def __init__(self, desc, device="cuda"):
        self.bytes = B.tasp_shared_plan_workspace_bytes(desc)[1]
        self.buf = torch.empty(self.bytes + 256, dtype=torch.uint8, device=device)
        self.base = self.buf.data_ptr() + (-self.buf.data_ptr()) % 256


class Plan:
    """A compiled plan with its torch-owned workspace."""

    def __init__(self, desc, store, mask=None, stream=None, device="cuda"):
        self.desc = desc
        self.store = store
        mptr, self._mask_keep = mask_struct(mask)
        self.ws_bytes = B.tasp_plan_workspace_bytes(desc, mptr)
        self.ws = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=device)
        off = (-self.ws.data_ptr()) % 256
        self.ws_base = self.ws.data_ptr() + off
        self.ws_off = off
        self.handle = B.tasp_compile_plan(desc, store.struct, mptr, self.ws_base, self.ws_bytes,
                                          stream if stream is not None else current_stream())

    def __del__(self):
        h = getattr(self, "handle", None)
        if h:
            try:
                B.tasp_plan_destroy(h)
            except Exception:
                pass
            self.handle = None

    @classmethod
    def shared(cls, desc, gstore, mask=None, stream=None, device="cuda", scratch=None):
        """A plan over the shared groupwise store (no weight copies). ``scratch``: a
        SharedScratch to share with other plans (else the plan gets its own)."""
        self = cls.__new__(cls)
        self.desc = desc
        self.store = gstore
        mptr, self._mask_keep = mask_struct(mask)
        self.ws_bytes = B.tasp_shared_plan_workspace_bytes(desc)[0]
        self.ws = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=device)
        off = (-self.ws.data_ptr()) % 256
        self.ws_base = self.ws.data_ptr() + off
        self.ws_off = off
        self.scratch = scratch if scratch is not None else SharedScratch(desc, device)
        self.handle = B.tasp_compile_shared_plan(desc, gstore.struct, mptr, self.ws_base,
                                                 self.ws_bytes, self.scratch.base, self.scratch.bytes,
                                                 stream if stream is not None else current_stream())
        return self

    def counts(self, layer):
        return B.tasp_plan_counts(self.handle, layer)

    def indices(self, layer, which):
        return B.tasp_plan_indices(self.handle, layer, which)

    def ledger(self):
        ratio, wb, sb, sig = B.tasp_plan_ledger(self.handle)
        return {"active_flop_ratio": ratio, "weight_bytes": wb, "scale_bytes": sb, "signature": sig}

    def _view(self, ptr, nbytes, dtype):
        start = ptr - self.ws.data_ptr()
        return self.ws[start:start + nbytes].view(dtype)

    def panel(self, layer, which):
        """(int8 rows [rows][ld], float32 scales [rows]) as views into the workspace."""
        w, s, rows, cols, ld = B.tasp_plan_panel(self.handle, layer, which)
        if rows * ld == 0:
            return torch.empty((rows, ld), dtype=torch.int8), torch.empty(rows), cols
        wt = self._view(w, rows * ld, torch.int8).view(rows, ld)
        st = self._view(s, rows * 4, torch.float32)
        return wt, st, cols

    def bind(self, cache):
        B.tasp_kv_bind(self.handle, cache.struct)

    def decode(self, x, cache, pos, out, stream=None):
        B.tasp_decode_step(self.handle, x.data_ptr(), cache.struct, pos, out.data_ptr(),
                           stream if stream is not None else current_stream())

    def decode_timed(self, x, cache, pos, out, stream=None):
        return B.tasp_decode_step_timed(self.handle, x.data_ptr(), cache.struct, pos, out.data_ptr(),
                                        stream if stream is not None else current_stream())

    def prefill(self, x, T, cache, pos0, out, stream=None):
        B.tasp_prefill(self.handle, x.data_ptr(), T, cache.struct, pos0, out.data_ptr(),
                       stream if stream is not None else current_stream())

    def prefill_last(self, x, T, cache, pos0, out, stream=None):
        """The prefill with the last token's logits only: out is float32 [vocab]."""
        B.tasp_prefill_last(self.handle, x.data_ptr(), T, cache.struct, pos0, out.data_ptr(),
                            stream if stream is not None else current_stream())

    def generate(self, embed, embed_scale, prompt, n_new, cache, stream=None, scratch=None):
        """Prompt ids (device int32 [T]) -> n_new + 1 greedy ids (device int32). ``scratch`` may
        pass (x [T][d], logits [T][vocab]) float32 device tensors to reuse."""
        T = int(prompt.numel())
        dev = prompt.device
        if scratch is None:
            scratch = (torch.empty((T, self.desc.d_model), device=dev),
                       torch.empty((T, self.desc.vocab), device=dev))
        out = torch.empty(n_new + 1, dtype=torch.int32, device=dev)
        B.tasp_generate(self.handle, embed.data_ptr(), embed_scale.data_ptr(), prompt.data_ptr(), T,
                        n_new, cache.struct, out.data_ptr(), scratch[0].data_ptr(),
                        scratch[1].data_ptr(), stream if stream is not None else current_stream())
        return out

    def prefill_timed(self, x, T, cache, pos0, out, stream=None):
        return B.tasp_prefill_timed(self.handle, x.data_ptr(), T, cache.struct, pos0, out.data_ptr(),
                                    stream if stream is not None else current_stream())


def build_mask(desc, head_scores, chan_scores, granule, target, stream=None):
    """Greedy dependency-closed mask from device float32 scores ([L][Hq], [L][d_ffn/granule]).
    Returns (q_keep, kv_keep, ffn_keep) as device uint8 tensors and the FLOPs spent."""
    dev = head_scores.device
    n = B.tasp_mask_workspace_bytes(desc, granule)
    ws = torch.empty(n + 256, dtype=torch.uint8, device=dev)
    base = ws.data_ptr() + (-ws.data_ptr()) % 256
    q = torch.empty((desc.n_layers, desc.n_q_heads), dtype=torch.uint8, device=dev)
    kv = torch.empty((desc.n_layers, desc.n_kv_heads), dtype=torch.uint8, device=dev)
    f = torch.empty((desc.n_layers, desc.d_ffn), dtype=torch.uint8, device=dev)
    spent = B.tasp_build_mask(desc, head_scores.data_ptr(), chan_scores.data_ptr(), granule, target,
                              base, n, q.data_ptr(), kv.data_ptr(), f.data_ptr(),
                              stream if stream is not None else current_stream())
    return q, kv, f, spent


class Router:
    """Router weights on the device (float32 tensors keyed proj, w1, b1, w2, b2, w3, b3, row-major
    [out][in]) and the ABI struct over them."""

    def __init__(self, weights, temperature=1.0, tau=0.85, device="cuda"):
        self.t = {k: torch.as_tensor(np.ascontiguousarray(v, np.float32)).to(device)
                  for k, v in weights.items()}
        proj_dim, n_bins = self.t["proj"].shape
        self.struct = B.tasp_router(int(n_bins), int(proj_dim), int(self.t["w1"].shape[0]),
                                    int(self.t["w2"].shape[0]), int(self.t["w3"].shape[0]),
                                    float(temperature), float(tau),
                                    *[self.t[k].data_ptr() for k in ("proj", "w1", "b1", "w2",
                                                                      "b2", "w3", "b3")])
        self.feat_dim = int(proj_dim) + B.ROUTER_SCALARS
        self.n_tasks = int(self.t["w3"].shape[0])
        self._ws = {}

    def workspace(self, n, device):
        """A 256-byte aligned workspace for n prompts: (tensor, base pointer, bytes)."""
        if n not in self._ws:
            nb = B.tasp_router_workspace_bytes(self.struct, n)
            t = torch.empty(nb + 256, dtype=torch.uint8, device=device)
            self._ws[n] = (t, t.data_ptr() + (-t.data_ptr()) % 256, nb)
        return self._ws[n]

    def route(self, text, offsets, logprob, stream=None, features=True):
        """text: device uint8 [n_text]; offsets: device int32 [n + 1] (None: one prompt);
        logprob: device float32 [n]. Returns (features or None, probs, choice) device tensors."""
        n = int(logprob.numel())
        dev = logprob.device
        _, base, nb = self.workspace(n, dev)
        feats = torch.empty((n, self.feat_dim), device=dev) if features else None
        probs = torch.empty((n, self.n_tasks), device=dev)
        choice = torch.empty(n, dtype=torch.int32, device=dev)
        B.tasp_route(self.struct, text.data_ptr() if text.numel() else None, int(text.numel()),
                     offsets.data_ptr() if offsets is not None else None, n, logprob.data_ptr(),
                     base, nb, feats.data_ptr() if feats is not None else None, probs.data_ptr(),
                     choice.data_ptr(), stream if stream is not None else current_stream())
        return feats, probs, choice

    def serve_turn(self, task_plans, dense_plan, text, logprob, embed, embed_scale, prompt,
                   n_cached, n_new, cache, stream=None, scratch=None):
        """One routed turn. Returns (choice, reused, out ids device int32 [n_new + 1])."""
        T = int(prompt.numel())
        dev = prompt.device
        d = dense_plan.desc
        if scratch is None:
            scratch = (torch.empty((T, d.d_model), device=dev), torch.empty((T, d.vocab), device=dev))
        out = torch.empty(n_new + 1, dtype=torch.int32, device=dev)
        _, base, nb = self.workspace(1, dev)
        c, reused = B.tasp_serve_turn(
            self.struct, [p.handle for p in task_plans], dense_plan.handle,
            text.data_ptr() if text.numel() else None, int(text.numel()), logprob.data_ptr(),
            embed.data_ptr(), embed_scale.data_ptr(), prompt.data_ptr(), T, n_cached, n_new,
            cache.struct, out.data_ptr(), scratch[0].data_ptr(), scratch[1].data_ptr(), base, nb,
            stream if stream is not None else current_stream())
        return c, reused, out
