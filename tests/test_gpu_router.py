"""GPU parity of router inference (tasp_route) and routed turns (tasp_serve_turn).

Features: the trigram histogram is checked bit-exactly through an identity projection (each
output then is one term frequency, count / (bytes - 2) in float32, which the oracle's float64
quotient rounds to identically); descriptors and counts exactly; the float32 arithmetic after
them within bounds derived from float32 rounding. Decisions are integers decided by floating
point: the kernel's choice must follow from the probabilities it wrote, and must equal the
oracle's wherever the oracle's top-two gap and its distance to tau clear the tolerance."""
import numpy as np
import pytest
import torch

import synth
from oracle import reference as ref
from oracle import router as R
from paper_2609_29499_amd import binding as B
from paper_2609_29499_amd import session as S
from synth import text as T
from tests.helpers import assert_parity, check_greedy_ids, teacher_forced_rows

pytestmark = pytest.mark.gpu

# probabilities: float32 rounding through three layers leaves the logits within ~1e-6 relative
# (magnitudes <= ~10), i.e. |du| <= ~4e-5 after a temperature of 0.25, and |dp| <= |du| / 2
P_TOL = 1e-4


def _flush(msg):
    print(msg, flush=True)


def _dev_text(texts):
    buf, offs = T.pack(texts)
    tb = torch.from_numpy(buf).cuda() if len(buf) else torch.zeros(1, dtype=torch.uint8, device="cuda")[:0]
    return tb, torch.from_numpy(offs).cuda()


def _route(router, texts, lps):
    tb, to = _dev_text(texts)
    f, p, c = router.route(tb, to, torch.from_numpy(np.asarray(lps, np.float32)).cuda())
    torch.cuda.synchronize()
    return f.cpu().numpy(), p.cpu().numpy(), c.cpu().numpy()


def _filler(n, seed):
    # bytes that form no descriptor pattern, digit or operator
    return bytes(np.random.default_rng(seed).choice(np.frombuffer(b"xyz qv", np.uint8), n))


def _boundary_prompts():
    """Prompts whose patterns straddle the kernel's 8,192-byte staging chunks."""
    out = []
    for k, (pat, at) in enumerate([(b"translat", 8188), (b"```", 16383), (b"\n1. go", 8191),
                                   (b"\nA. x\nB. y", 16380), (b" who ", 8191), (b" Which", 8190),
                                   (b"?12+3", 8190)]):
        s = bytearray(_filler(20000, k))
        s[at:at + len(pat)] = pat
        out.append(bytes(s))
    return out


def _edge_prompts():
    return [b"", b"a", b"ab", b"abc", b"Who", "Übersetze: translate ä€ ```".encode(),
            b"A. x\r\nB. y", b"a\x00b\x00who\x00", b"1. x\n2) y", b"\n\n(A) p\n(B) q\n"]


def _oracle_features(texts, lps, w):
    return np.stack([R.features(t, lp, w["proj"], w["proj"].shape[1]) for t, lp in zip(texts, lps)])


def test_features_histogram_exact_and_scalars():
    """Identity projection: every term frequency and scalar feature against the oracle."""
    nb = 2048
    texts = T.prompts(30, seed=21) + _edge_prompts() + _boundary_prompts()
    _flush(f"case router features identity n={len(texts)} max_len={max(map(len, texts))}")
    w = T.router_weights(seed=1, n_bins=nb, proj_dim=nb)
    w["proj"] = np.eye(nb, dtype=np.float32)
    lps = T.proxy_logprobs(len(texts), seed=3)
    got, _, _ = _route(S.Router(w), texts, lps)
    for i, t in enumerate(texts):
        tf = (R.trigram_counts(t, nb) / max(1, len(t) - 2)).astype(np.float32)
        assert np.array_equal(got[i, :nb], tf), f"prompt {i}: histogram"
        want = R.features(t, float(lps[i]), np.zeros((0, nb)), nb)
        assert got[i, nb + 1] == lps[i]
        np.testing.assert_allclose(got[i, nb:nb + 6], want[:6], rtol=1e-6, atol=0, err_msg=f"prompt {i}")
        assert np.array_equal(got[i, nb + 6:], want[6:]), f"prompt {i}: descriptors"


def test_boundary_prompts_raise_their_descriptor():
    # the fixtures above are meaningful only if each raises a descriptor or count in the oracle
    for t in _boundary_prompts():
        d = R.descriptors(t)
        assert sum(d) >= 1 or R.char_counts(t)[0] > 0


@pytest.mark.parametrize("temperature", [1.0, 0.25])
def test_route_parity_paper_shape(temperature):
    """The paper's router (2,048 bins -> 256, 512, 256, 5 tasks) on 64 prompts of the five
    families, including 2,048-token-sized ones."""
    texts = T.prompts(56, seed=22) + T.prompts(8, seed=23, n_sent=130)
    _flush(f"case router paper shape T={temperature} n={len(texts)}")
    w = T.router_weights(seed=2)
    lps = T.proxy_logprobs(len(texts), seed=4)
    tau = 0.85
    f, p, c = _route(S.Router(w, temperature=temperature, tau=tau), texts, lps)
    fo = _oracle_features(texts, lps, w)
    scale = np.abs(w["proj"]).max() * 1.0
    np.testing.assert_allclose(f[:, :256], fo[:, :256], rtol=0, atol=1e-5 * scale)
    np.testing.assert_allclose(f[:, 256:], fo[:, 256:], rtol=1e-6, atol=1e-7)
    po = np.stack([R.probabilities(R.mlp_logits(fo[i], w["w1"], w["b1"], w["w2"], w["b2"], w["w3"],
                                                w["b3"]), temperature) for i in range(len(texts))])
    assert np.abs(p - po).max() <= P_TOL
    clear = 0
    for i in range(len(texts)):
        task = int(np.argmax(p[i]))
        assert c[i] == (task if p[i, task] >= np.float32(tau) else -1), f"prompt {i}: self"
        s = np.sort(po[i])
        if s[-1] - s[-2] > 2 * P_TOL and abs(s[-1] - tau) > 2 * P_TOL:
            assert c[i] == R.decide(po[i], tau), f"prompt {i}"
            clear += 1
    assert clear >= len(texts) - 4
    if temperature < 1.0:
        assert (c >= 0).any() and (c == -1).any()     # both branches exercised


def test_route_batch_equals_single_and_graph_replay():
    texts = T.prompts(9, seed=24)
    _flush("case router batch vs single, graph replay")
    w = T.router_weights(seed=5)
    router = S.Router(w, temperature=0.5)
    lps = T.proxy_logprobs(9, seed=6)
    f, p, c = _route(router, texts, lps)
    for i in (0, 4, 8):
        f1, p1, c1 = _route(router, [texts[i]], lps[i:i + 1])
        assert np.array_equal(f1[0], f[i]) and np.array_equal(p1[0], p[i]) and c1[0] == c[i]
    # capture into a graph and replay with eager work in between
    tb, to = _dev_text(texts)
    lp = torch.from_numpy(lps).cuda()
    router.route(tb, to, lp)                 # warm-up outside capture (workspace allocation)
    feats = torch.empty((9, router.feat_dim), device="cuda")
    probs = torch.empty((9, 5), device="cuda")
    choice = torch.empty(9, dtype=torch.int32, device="cuda")
    _, base, nb = router.workspace(9, torch.device("cuda"))
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            B.tasp_route(router.struct, tb.data_ptr(), tb.numel(), to.data_ptr(), 9, lp.data_ptr(),
                         base, nb, feats.data_ptr(), probs.data_ptr(), choice.data_ptr(),
                         C_stream(s))
    torch.cuda.current_stream().wait_stream(s)
    for rep in range(3):
        feats.fill_(-7.0)
        probs.fill_(-7.0)
        choice.fill_(99)
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(feats.cpu().numpy(), f), f"replay {rep}"
        assert np.array_equal(probs.cpu().numpy(), p) and np.array_equal(choice.cpu().numpy(), c)


def C_stream(s):
    import ctypes
    return ctypes.c_void_p(s.cuda_stream)


def test_route_small_shapes_and_offsets():
    """One task, sixteen tasks, odd widths, clamped offsets."""
    _flush("case router small shapes")
    texts = [b"who is it?", b"translate ```x```", b"", b"1. a\n2. b"]
    w = T.router_weights(seed=7, n_bins=100, proj_dim=3, hidden1=5, hidden2=7, n_tasks=1)
    f, p, c = _route(S.Router(w, tau=0.5), texts, [0.0] * 4)
    assert np.all(p == 1.0) and np.all(c == 0)
    w = T.router_weights(seed=8, n_bins=997, proj_dim=33, hidden1=65, hidden2=129, n_tasks=16)
    lps = [-1.0, -2.0, -3.0, -4.0]
    f, p, c = _route(S.Router(w, temperature=0.1, tau=0.3), texts, lps)
    fo = _oracle_features(texts, lps, w)
    np.testing.assert_allclose(f, fo, rtol=1e-5, atol=1e-5 * np.abs(w["proj"]).max())
    po = np.stack([R.probabilities(R.mlp_logits(fo[i], w["w1"], w["b1"], w["w2"], w["b2"], w["w3"],
                                                w["b3"]), 0.1) for i in range(4)])
    assert np.abs(p - po).max() <= P_TOL
    # offsets beyond the text and a decreasing pair are clamped on the device
    buf, _ = T.pack(texts)
    tb = torch.from_numpy(buf).cuda()
    n = len(buf)
    offs = torch.tensor([-5, 10, 4, n + 100], dtype=torch.int32, device="cuda")
    router = S.Router(w, temperature=0.1, tau=0.3)
    f2, _, _ = router.route(tb, offs, torch.tensor([0.0, 0.0, 0.0], device="cuda"))
    torch.cuda.synchronize()
    raw = bytes(buf)
    clamped = [raw[0:10], b"", raw[4:n]]
    fo2 = _oracle_features(clamped, [0.0] * 3, w)
    np.testing.assert_allclose(f2.cpu().numpy(), fo2, rtol=1e-5, atol=1e-5 * np.abs(w["proj"]).max())


def test_route_argument_errors():
    w = T.router_weights(seed=9, n_bins=64, proj_dim=4, hidden1=8, hidden2=8)
    router = S.Router(w)
    tb, to = _dev_text([b"abc"])
    lp = torch.zeros(1, device="cuda")
    _, base, nb = router.workspace(1, torch.device("cuda"))
    out = torch.empty(8, device="cuda")
    ch = torch.empty(1, dtype=torch.int32, device="cuda")
    st = S.current_stream()
    with pytest.raises(B.TaspError, match="WORKSPACE"):
        B.tasp_route(router.struct, tb.data_ptr(), 3, to.data_ptr(), 1, lp.data_ptr(), base, nb - 1,
                     None, out.data_ptr(), ch.data_ptr(), st)
    with pytest.raises(B.TaspError, match="INVALID_ARG"):
        B.tasp_route(router.struct, tb.data_ptr(), 3, None, 2, lp.data_ptr(), base, nb, None,
                     out.data_ptr(), ch.data_ptr(), st)


# ---- routed turns


class _Deployment:
    """A tiny model with an LM head, five task plans (different masks) and the dense plan."""

    def __init__(self, max_seq=96, max_prefill=64):
        self.sh = synth.tiny_shape(d=256, hq=8, hkv=2, dh=64, f=512, layers=2, vocab=1500)
        sh = self.sh
        self.layers = [synth.layer_weights(sh, l) for l in range(sh.n_layers)]
        self.fn, self.lm = synth.final_norm(sh), synth.lm_head(sh)
        self.table, self.scales = synth.embedding(sh)
        self.desc = S.desc_from_shape(sh, max_batch=1, max_seq=max_seq, max_prefill=max_prefill)
        self.store = S.DeviceStore(self.layers, self.fn, self.lm)
        self.masks = [synth.raw_mask(sh, 30 + t) for t in range(5)]
        self.plans = [S.Plan(self.desc, self.store, m) for m in self.masks]
        self.dense = S.Plan(self.desc, self.store, None)
        self.emb = torch.from_numpy(self.table).cuda()
        self.sc = torch.from_numpy(self.scales).cuda()
        self.max_seq = max_seq

    def router(self, task):
        """Router weights that pick `task` for every prompt (-1: uniform, the dense fallback)."""
        w = T.router_weights(seed=10)
        w["w3"] = np.zeros_like(w["w3"])
        w["b3"] = np.zeros(5, np.float32)
        if task >= 0:
            w["b3"][task] = 12.0
        return S.Router(w)

    def cache(self):
        return S.KVCache(self.desc, 1, self.max_seq)

    def oracle_rows(self, mask, prompt, ids):
        """The oracle's logits along prompt + ids (teacher-forced on the turn's own ids)."""
        sh = self.sh
        closed = ref.close_mask(*(mask if mask is not None else synth.all_kept_mask(sh)), sh.group_size)
        return teacher_forced_rows(lambda l: self.layers[l], closed, self.table, self.scales, prompt,
                                   ids, sh, self.fn, self.lm)


def _turn(dep, router, text, prompt, n_cached, n_new, cache, with_logits=False):
    tb = torch.from_numpy(np.frombuffer(text, np.uint8).copy()).cuda()
    lp = torch.tensor([-2.0], device="cuda")
    T = len(prompt)
    scratch = (torch.empty((T, dep.sh.d_model), device="cuda"),
               torch.empty((T, dep.sh.vocab), device="cuda"))
    c, reused, ids = router.serve_turn(dep.plans, dep.dense, tb, lp, dep.emb, dep.sc,
                                       torch.from_numpy(prompt).cuda(), n_cached, n_new, cache,
                                       scratch=scratch)
    torch.cuda.synchronize()
    if with_logits:   # the last step's logits (row 0 after a decode step, T - 1 without one)
        last = scratch[1][0 if n_new else T - 1].cpu().numpy().astype(np.float64)
        return c, reused, ids.cpu().numpy(), last
    return c, reused, ids.cpu().numpy()


def _fresh_generate(plan, dep, prompt, n_new):
    cache = dep.cache()
    ids = plan.generate(dep.emb, dep.sc, torch.from_numpy(prompt).cuda(), n_new, cache)
    torch.cuda.synchronize()
    return ids.cpu().numpy()


@pytest.fixture(scope="module")
def dep():
    return _Deployment()


@pytest.mark.parametrize("task", [0, 3, -1])
def test_serve_turn_dispatches_the_chosen_plan(dep, task):
    _flush(f"case serve_turn task={task}")
    prompt = synth.prompt_ids(24, dep.sh.vocab, seed=5)
    c, reused, ids = _turn(dep, dep.router(task), b"Who wrote it? 1. a", prompt, 0, 6, dep.cache())
    assert c == task and reused == 0
    plan = dep.plans[task] if task >= 0 else dep.dense
    assert np.array_equal(ids, _fresh_generate(plan, dep, prompt, 6))


def test_serve_turn_conversation_reuse_and_switch(dep):
    """Turn 1 and turn 2 on plan 2 (the cache is kept: only the new ids are prefilled), turn 3
    routed to plan 4 (the cache is invalidated and the whole conversation prefilled)."""
    _flush("case serve_turn conversation")
    cache = dep.cache()
    r2, r4 = dep.router(2), dep.router(4)
    p1 = synth.prompt_ids(20, dep.sh.vocab, seed=6)
    c, reused, ids1 = _turn(dep, r2, b"first turn", p1, 0, 5, cache)
    assert (c, reused) == (2, 0)
    check_greedy_ids(ids1, dep.oracle_rows(dep.masks[2], p1, ids1), "first turn")
    conv2 = np.concatenate([p1, ids1[:5], synth.prompt_ids(9, dep.sh.vocab, seed=7)]).astype(np.int32)
    c, reused, ids2, last2 = _turn(dep, r2, b"second turn", conv2, len(p1) + 5, 6, cache,
                                   with_logits=True)
    assert (c, reused) == (2, 1)
    # the continued turn against the oracle's one-shot pass over the whole conversation, along
    # the turn's own ids: every id admissible, the last step's logits at parity
    rows = dep.oracle_rows(dep.masks[2], conv2, ids2)
    check_greedy_ids(ids2, rows, "continued turn")
    assert_parity(last2, rows[-1], what="continued turn last logits")
    conv3 = np.concatenate([conv2, ids2[:6], synth.prompt_ids(7, dep.sh.vocab, seed=8)]).astype(np.int32)
    c, reused, ids3 = _turn(dep, r4, b"third turn", conv3, len(conv2) + 6, 4, cache)
    assert (c, reused) == (4, 0)
    assert np.array_equal(ids3, _fresh_generate(dep.plans[4], dep, conv3, 4))
    # a cache bound to another plan is never continued, even when n_cached is given
    c, reused, _ = _turn(dep, r2, b"fourth", conv3, len(conv3) - 1, 1, cache)
    assert (c, reused) == (2, 0)


def test_serve_turn_errors(dep):
    _flush("case serve_turn errors")
    router = dep.router(1)
    prompt = synth.prompt_ids(8, dep.sh.vocab, seed=9)
    with pytest.raises(B.TaspError, match="INVALID_ARG"):
        _turn(dep, router, b"x", prompt, -1, 2, dep.cache())
    other = synth.tiny_shape(d=128, hq=4, hkv=2, dh=64, f=256, layers=2, vocab=1500)
    od = S.desc_from_shape(other, max_batch=1, max_seq=96, max_prefill=64)
    oplan = S.Plan(od, S.DeviceStore([synth.layer_weights(other, l) for l in range(2)],
                                     synth.final_norm(other), synth.lm_head(other)), None)
    plans = list(dep.plans)
    plans[3] = oplan
    tb = torch.from_numpy(np.frombuffer(b"x", np.uint8).copy()).cuda()
    with pytest.raises(B.TaspError, match="SHAPE"):
        router.serve_turn(plans, dep.dense, tb, torch.zeros(1, device="cuda"), dep.emb, dep.sc,
                          torch.from_numpy(prompt).cuda(), 0, 2, dep.cache())
