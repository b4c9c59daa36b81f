"""The C-ABI library loads, exports every entry point that include/tasp.h declares, and rejects
bad arguments on the host before enqueuing any GPU work (no GPU needed)."""
import ctypes as C
import os
import re
import shutil
import subprocess

import numpy as np
import pytest

from paper_2609_29499_amd import binding as B
from paper_2609_29499_amd import session as S

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _lib():
    if not os.path.exists(B.LIB_PATH):
        pytest.fail("libtasp.so is not built (run __graft_entry__.build())")
    return B.load()


def test_every_declared_symbol_is_exported():
    lib = _lib()
    header = open(os.path.join(ROOT, "include", "tasp.h")).read()
    declared = set(re.findall(r"^\s*(?:tasp_status|const char\*)\s+(tasp_\w+)\s*\(", header, re.M))
    assert declared == set(B.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name
    # and nothing else: internal helpers keep internal linkage
    nm = shutil.which("nm")
    if nm:
        out = subprocess.run([nm, "-D", "--defined-only", B.LIB_PATH], capture_output=True,
                             text=True, check=True).stdout
        c_names = {l.split()[-1] for l in out.splitlines()
                   if l.split()[1:2] == ["T"] and not l.split()[-1].startswith("_Z")}
        assert c_names == declared, c_names ^ declared
        # every kernel the library launches is defined in it (a missing host stub is an
        # undefined symbol that only shows when the library is loaded on a GPU host)
        undef = subprocess.run([nm, "-D", "--undefined-only", B.LIB_PATH], capture_output=True,
                               text=True, check=True).stdout
        assert not [l for l in undef.splitlines() if "tasp" in l], undef


def _desc(**kw):
    base = dict(n_layers=1, d_model=512, n_q_heads=8, n_kv_heads=2, head_dim=64, d_ffn=1536,
                max_seq=256)
    base.update(kw)
    return S.model_desc(**base)


def test_workspace_bytes_scales_with_mask():
    _lib()
    d = _desc()
    dense = B.tasp_plan_workspace_bytes(d, None)
    q = np.ones((1, 8), np.uint8)
    q[0, :4] = 0                                           # group 0 dropped entirely
    f = np.zeros((1, 1536), np.uint8)
    f[0, :512] = 1
    m, keep = S.mask_struct((q, None, f))
    sparse = B.tasp_plan_workspace_bytes(d, m)
    assert sparse < dense
    # retained bytes shrink by at least the dropped panels: 2/3 of FFN rows, 4 q heads + 1 group
    dropped = 3 * 512 * 1024 + (4 * 64 + 2 * 64) * 512 + 512 * 4 * 64
    assert dense - sparse >= dropped


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=96), "TASP_ERR_SHAPE"),
    (dict(n_q_heads=6, n_kv_heads=4), "TASP_ERR_SHAPE"),
    (dict(n_q_heads=32, n_kv_heads=2), "TASP_ERR_SHAPE"),      # 16 heads per group
    (dict(d_model=520), "TASP_ERR_SHAPE"),
    (dict(max_batch=9), "TASP_ERR_SHAPE"),
    (dict(n_layers=0), "TASP_ERR_SHAPE"),
    (dict(d_model=16400, n_q_heads=8, n_kv_heads=2), "TASP_ERR_SHAPE"),
    (dict(d_ffn=49152), "TASP_ERR_UNSUPPORTED"),             # batch-1 input beyond LDS
])
def test_bad_desc_rejected(kw, status):
    _lib()
    with pytest.raises(B.TaspError) as e:
        B.tasp_plan_workspace_bytes(_desc(**kw), None)
    assert B.STATUS[e.value.status] == status


def test_batched_desc_accepted():
    """Batches of 2..8 do not stage inputs in LDS: a wide FFN at batch 8 is a valid desc, and the
    batched operands add workspace."""
    _lib()
    one = B.tasp_plan_workspace_bytes(_desc(d_ffn=14336), None)
    eight = B.tasp_plan_workspace_bytes(_desc(d_ffn=14336, max_batch=8), None)
    assert eight > one


def test_bad_mask_byte_rejected():
    _lib()
    q = np.ones((1, 8), np.uint8)
    q[0, 3] = 2
    m, keep = S.mask_struct((q, None, np.ones((1, 1536), np.uint8)))
    with pytest.raises(B.TaspError) as e:
        B.tasp_plan_workspace_bytes(_desc(), m)
    assert e.value.status == -3 and "q_keep[3]" in str(e.value)


def test_compile_rejects_null_and_small_workspace():
    lib = _lib()
    d = _desc()
    store = B.tasp_store(None, None, None)
    plan = C.c_void_p()
    st = lib.tasp_compile_plan(C.byref(d), C.byref(store), None, C.c_void_p(256), 1 << 30, None,
                               C.byref(plan))
    assert st == -1
    layers = (B.tasp_layer * 1)()
    for n in S.WEIGHT_NAMES:
        setattr(layers[0], n, B.tasp_qmat(4096, 4096))
    layers[0].attn_norm = layers[0].ffn_norm = 4096
    store = B.tasp_store(layers, None, None)
    st = lib.tasp_compile_plan(C.byref(d), C.byref(store), None, C.c_void_p(256), 1024, None,
                               C.byref(plan))
    assert st == -4 and b"workspace" in lib.tasp_last_error()
    st = lib.tasp_compile_plan(C.byref(d), C.byref(store), None, C.c_void_p(100), 1 << 40, None,
                               C.byref(plan))
    assert st == -4 and b"aligned" in lib.tasp_last_error()


def test_calls_on_null_plan_fail_cleanly():
    lib = _lib()
    cache = B.tasp_kv_cache(None, None, 1, 16, 0)
    assert lib.tasp_decode_step(None, None, C.byref(cache), 0, None, None) == -1
    assert lib.tasp_prefill(None, None, 1, C.byref(cache), 0, None, None) == -1
    assert lib.tasp_kv_bind(None, C.byref(cache)) == -1
    assert lib.tasp_plan_ledger(None, None, None, None, None) == -1
    assert lib.tasp_copy_probe(None, None, 16, None) == -1
    assert lib.tasp_status_string(-6) == b"KV cache belongs to another plan"


def test_mask_workspace_and_granule_checks():
    _lib()
    d = _desc(n_layers=3, d_ffn=2048)
    small = B.tasp_mask_workspace_bytes(d, 1024)
    big = B.tasp_mask_workspace_bytes(d, 128)
    assert big > small > 0                                   # more candidates, more workspace
    with pytest.raises(B.TaspError) as e:
        B.tasp_mask_workspace_bytes(d, 1000)                 # does not divide d_ffn
    assert B.STATUS[e.value.status] == "TASP_ERR_SHAPE"
    with pytest.raises(B.TaspError) as e:
        B.tasp_mask_workspace_bytes(d, 0)
    assert B.STATUS[e.value.status] == "TASP_ERR_SHAPE"


def _router(**kw):
    base = dict(n_bins=2048, proj_dim=256, hidden1=512, hidden2=256, n_tasks=5, temperature=1.0,
                tau=0.85)
    base.update(kw)
    fake = 4096                        # never dereferenced: every check runs before a launch
    return B.tasp_router(base["n_bins"], base["proj_dim"], base["hidden1"], base["hidden2"],
                         base["n_tasks"], base["temperature"], base["tau"], *([fake] * 7))


def test_router_workspace_and_argument_checks():
    _lib()
    one = B.tasp_router_workspace_bytes(_router(), 1)
    many = B.tasp_router_workspace_bytes(_router(), 64)
    # term frequencies, features and both hidden layers per prompt, plus one prompt's decision
    per = 4 * (2048 + 267 + 512 + 256)
    assert one >= per and many >= 64 * per and many > one
    for bad in (dict(n_bins=0), dict(n_bins=16385), dict(n_tasks=0), dict(n_tasks=17),
                dict(temperature=0.0), dict(temperature=float("nan")), dict(hidden1=0),
                dict(tau=float("inf"))):
        with pytest.raises(B.TaspError) as e:
            B.tasp_router_workspace_bytes(_router(**bad), 1)
        assert B.STATUS[e.value.status] == "TASP_ERR_INVALID_ARG", bad
    for n in (0, 65536):
        with pytest.raises(B.TaspError):
            B.tasp_router_workspace_bytes(_router(), n)
    r = _router()
    r.w2 = None
    with pytest.raises(B.TaspError):
        B.tasp_router_workspace_bytes(r, 1)
    # tasp_route rejects before launching: short or misaligned workspace, missing offsets
    r = _router()
    nb = B.tasp_router_workspace_bytes(r, 2)
    ws = 1 << 20
    with pytest.raises(B.TaspError) as e:
        B.tasp_route(r, 4096, 10, 4096, 2, 4096, ws, nb - 1, None, 4096, 4096, None)
    assert B.STATUS[e.value.status] == "TASP_ERR_WORKSPACE"
    with pytest.raises(B.TaspError) as e:
        B.tasp_route(r, 4096, 10, 4096, 2, 4096, ws + 8, nb, None, 4096, 4096, None)
    assert B.STATUS[e.value.status] == "TASP_ERR_WORKSPACE"
    with pytest.raises(B.TaspError) as e:
        B.tasp_route(r, 4096, 10, None, 2, 4096, ws, nb, None, 4096, 4096, None)
    assert B.STATUS[e.value.status] == "TASP_ERR_INVALID_ARG"
    with pytest.raises(B.TaspError) as e:
        B.tasp_route(r, 4096, -1, None, 1, 4096, ws, nb, None, 4096, 4096, None)
    assert B.STATUS[e.value.status] == "TASP_ERR_INVALID_ARG"


def test_shared_plan_host_checks():
    """Shared-store plans: mask-independent workspace that grows with the batch and prefill
    scratch, 128-divisible widths, and retained channels in aligned blocks of 16; all rejected
    before any GPU work."""
    _lib()
    d = _desc(d_model=512, d_ffn=1536, max_batch=1)
    n, ns = B.tasp_shared_plan_workspace_bytes(d)
    assert n > 0 and ns > 0 and n + ns < B.tasp_plan_workspace_bytes(d, None)
    big = _desc(d_model=512, d_ffn=1536, max_batch=4, max_prefill=64)
    nb, nbs = B.tasp_shared_plan_workspace_bytes(big)
    # the plan's own bytes do not depend on the batch or prefill scratch; the arena does
    assert nb == n and nbs > ns and nb + nbs < B.tasp_plan_workspace_bytes(big, None)
    for bad, status in ((dict(d_model=528), "TASP_ERR_SHAPE"),
                        (dict(d_ffn=1552), "TASP_ERR_SHAPE")):
        with pytest.raises(B.TaspError) as e:
            B.tasp_shared_plan_workspace_bytes(_desc(**{**dict(d_model=512, d_ffn=1536, max_batch=1), **bad}))
        assert B.STATUS[e.value.status] == status, bad
    fake = 1 << 20                          # never dereferenced: the checks run on the host
    lay = B.tasp_glayer(*([B.tasp_gqmat(fake, fake)] * 5), fake, fake)
    layers = (B.tasp_glayer * 1)(lay)
    store = B.tasp_gstore(layers, None, None)
    q = np.ones((1, 8), np.uint8)
    f = np.ones((1, 1536), np.uint8)
    f[0, 5] = 0                             # breaks the block of channels 0..15
    m = B.tasp_mask(q.ctypes.data, None, f.ctypes.data)
    with pytest.raises(B.TaspError) as e:
        B.tasp_compile_shared_plan(d, store, C.pointer(m), 1 << 30, n, 1 << 31, ns, None)
    assert B.STATUS[e.value.status] == "TASP_ERR_UNSUPPORTED"
    for ws, wsb, sc, scb in (((1 << 30) + 8, n, 1 << 31, ns),      # misaligned workspace
                             (1 << 30, n, (1 << 31) + 8, ns),      # misaligned scratch
                             (1 << 30, n, 1 << 31, ns - 1),        # short scratch
                             (1 << 30, n + ns - 1, None, 0),       # arena in the workspace: short
                             (1 << 30, n - 1, 1 << 31, ns)):       # short workspace
        with pytest.raises(B.TaspError) as e:
            B.tasp_compile_shared_plan(d, store, None, ws, wsb, sc, scb, None)
        assert B.STATUS[e.value.status] == "TASP_ERR_WORKSPACE", (ws, wsb, sc, scb)


def test_shared_store_memory_ledger_llama3_70b():
    """Memory of five Llama-3-70B masks over one groupwise store with the paper's request shape
    enabled (2,048-token prefill, 256 decode steps; paper, appendix "Backing-store semantics"
    and Table "memory"): the plans add metadata only, all five share one scratch arena, and the
    total stays far from five duplicated stores."""
    _lib()
    import synth
    sh = synth.LLAMA3_70B
    d = S.desc_from_shape(sh, max_batch=1, max_seq=2048 + 256, max_prefill=2048)
    plan, arena = B.tasp_shared_plan_workspace_bytes(d)
    dh, D, F = sh.head_dim, sh.d_model, sh.d_ffn
    per_layer = (sh.n_q_heads + 2 * sh.n_kv_heads) * dh * D + D * sh.n_q_heads * dh + 3 * F * D
    weights = sh.n_layers * per_layer
    scales = weights // 128 * 2
    kv = 2 * sh.n_layers * sh.n_kv_heads * (2048 + 256) * dh * 2
    five = weights + scales + 5 * plan + arena + kv
    one = weights + scales + plan + arena + kv
    assert five - one == 4 * plan
    assert 5 * plan < 0.1e9                      # metadata of five plans, decimal GB
    assert arena < 1.0e9                         # one prefill-sized scratch for all of them
    assert five < weights * 1.05 and five < 0.25 * 5 * weights
    # the decode-only desc needs the same plan bytes and a smaller arena
    p0, a0 = B.tasp_shared_plan_workspace_bytes(S.desc_from_shape(sh, max_batch=1, max_seq=2304))
    assert p0 == plan and a0 < arena
