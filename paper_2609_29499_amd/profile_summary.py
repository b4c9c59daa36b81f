"""Summaries of rocprofv3 result databases for the library's kernels.

    python -m paper_2609_29499_amd.profile_summary trace DB [--split KIND:GRID_X]
                                                               [--split-nth KIND:N] [--by-grid]
        per-kernel dispatch count / mean / median / min duration (us); with --split the run is cut
        at the first dispatch of KIND with that grid size in work-items, with --split-nth at the
        N-th dispatch of KIND (e.g. closure:2, the second plan compile: the benchmarks time the
        sparse plan first, then the dense one)
    python -m paper_2609_29499_amd.profile_summary traffic FETCH_DB WRITE_DB KIND
        HBM bytes per dispatch of KIND from a FETCH_SIZE and a WRITE_SIZE run, each scaled by what
        the same counter reads for the library's 1 GiB streaming copy in the same run
    python -m paper_2609_29499_amd.profile_summary pmc DB KIND [--grid G]
        mean of every collected counter per dispatch of KIND (of grid size G work-items)

Kernel kinds are read from the demangled names; GEMVs that share a template (O and down) are told
apart by their order inside a step (down follows gate/up).
"""
from __future__ import annotations

import argparse
import collections
import re
import sqlite3
import statistics

COPY_BYTES = 1 << 30


def kind_of(name: str) -> str | None:
    rules = [
        (r"attn_mfma_kernel", "attention"),
        (r"pf_attn_kernel", "prefill_attention"),
        (r"pf_rope_kernel", "rope_append"),
        (r"pf_prep_kernel|mfma_prep_kernel", "operand_prep"),
        (r"gemv_kernel<1, 0[,>]", "qkv_gemv"),
        (r"gemv_kernel<1, 2[,>]", "gateup_gemv"),
        (r"gemv_kernel<1, 1[,>]", "resid_gemv"),
        (r"gemv_kernel<1, 3[,>]", "lmhead_gemv"),
        (r"shared_gemv_kernel<0[,>]", "qkv_shared"),
        (r"shared_gemv_kernel<2[,>]", "gateup_shared"),
        (r"shared_gemv_kernel<1[,>]", "resid_shared"),
        (r"shared_maps_kernel", "shared_maps"),
        (r"mfma_gemv_kernel<0,", "qkv_mfma"),
        (r"mfma_gemv_kernel<2,", "gateup_mfma"),
        (r"mfma_gemv_kernel<1,", "resid_mfma"),
        (r"mfma_gemv_kernel<3,", "lmhead_mfma"),
        (r"pf_split_reduce_kernel<0>", "qkv_reduce"),
        (r"pf_split_reduce_kernel<1>", "resid_reduce"),
        (r"pf_(gemm|dma)_kernel<0,", "qkv_gemm"),
        (r"pf_(gemm|dma)_kernel<2,", "gateup_gemm"),
        (r"pf_(gemm|dma)_kernel<1,", "resid_gemm"),
        (r"pf_gemm_kernel<3,", "lmhead_gemm"),
        (r"router_features_kernel", "router_features"),
        (r"router_dense_kernel", "router_dense"),
        (r"router_head_kernel", "router_head"),
        (r"embed_kernel", "embed"),
        (r"argmax_kernel", "argmax"),
        (r"copy_kernel", "copy_probe"),
        (r"closure_kernel", "closure"),
    ]
    for pat, k in rules:
        if re.search(pat, name):
            return k
    return None


def _named(kinds):
    """Resolve resid_* into o_* / down_* by order: a residual GEMV right after gate/up is down;
    a split-K reduction takes the name of the GEMM it follows."""
    out, prev = [], None
    for k in kinds:
        if k and k.startswith("resid_"):
            suffix = k.split("_", 1)[1]
            if suffix == "reduce" and prev in ("o_gemm", "down_gemm"):
                k = prev.split("_", 1)[0] + "_reduce"
            else:
                k = ("down_" if prev and prev.startswith("gateup_") else "o_") + suffix
        out.append(k)
        if k:
            prev = k
    return out


def trace(db, split=None, by_grid=False, split_nth=None):
    con = sqlite3.connect(db)
    rows = con.execute("select name, grid_x, start, end from kernels order by start").fetchall()
    kinds = _named([kind_of(r[0]) for r in rows])
    t_split = None
    if split:
        sk, sg = split.split(":")
        cand = [r[2] for r, k in zip(rows, kinds) if k == sk and r[1] == int(sg)]
        t_split = min(cand) if cand else None
    if split_nth:
        sk, n = split_nth.split(":")
        cand = [r[2] for r, k in zip(rows, kinds) if k == sk]
        t_split = cand[int(n) - 1] if len(cand) >= int(n) else None
    stats = collections.defaultdict(list)
    for r, k in zip(rows, kinds):
        if not k or k in ("copy_probe", "closure"):
            continue
        phase = "all" if t_split is None else ("second" if r[2] >= t_split else "first")
        stats[(phase, k, r[1] if by_grid else "")].append((r[3] - r[2]) / 1000.0)
    print("| phase | kernel | grid | dispatches | mean us | median us | min us |")
    print("|---|---|---|---|---|---|---|")
    for (ph, k, g), v in stats.items():
        print(f"| {ph} | {k} | {g} | {len(v)} | {statistics.mean(v):.2f} | {statistics.median(v):.2f} | {min(v):.2f} |")


def _counter_rows(db):
    con = sqlite3.connect(db)
    return con.execute("select dispatch_id, kernel_name, grid_size_x, counter_name, value, start "
                       "from counters_collection order by start").fetchall()


def _per_dispatch(db):
    """dispatch id -> (kind, grid, {counter: value}) with the O/down naming resolved."""
    rows = _counter_rows(db)
    disp = collections.OrderedDict()
    for did, name, grid, cname, val, _ in rows:
        d = disp.setdefault(did, [name, grid, {}])
        d[2][cname] = d[2].get(cname, 0.0) + val
    names = _named([kind_of(v[0]) for v in disp.values()])
    return [(k, v[1], v[2]) for k, v in zip(names, disp.values())]


def _calibration(per, counter):
    """Bytes per counted KiB, from the 1 GiB copy-probe dispatches. The benchmarks run the probe
    last, so these are the copy dispatches after the last dispatch of any other kernel (plan
    compiles use the same copy kernel for their own buffers, the LM head copy among them)."""
    last_other = max((i for i, (k, g, c) in enumerate(per) if k not in (None, "copy_probe")),
                     default=-1)
    copies = [c[counter] for k, g, c in per[last_other + 1:] if k == "copy_probe" and counter in c]
    if not copies:
        raise SystemExit(f"no copy-probe dispatches with {counter} after the last other kernel")
    return COPY_BYTES / statistics.median(copies)


def traffic(fetch_db, write_db, kind):
    out = {}
    for db, counter, direction in ((fetch_db, "FETCH_SIZE", "read"), (write_db, "WRITE_SIZE", "write")):
        per = _per_dispatch(db)
        scale = _calibration(per, counter)
        vals = [c[counter] for k, g, c in per if k == kind and counter in c]
        kib = statistics.mean(vals)
        out[direction] = {"counter": counter, "dispatches": len(vals), "mean_KiB": round(kib, 1),
                          "copy_factor": round(scale / 1024.0, 4), "bytes": round(kib * scale)}
    out["bytes_per_launch"] = out["read"]["bytes"] + out["write"]["bytes"]
    return out


def pmc(db, kind, grid=None):
    per = _per_dispatch(db)
    acc = collections.defaultdict(list)
    for k, g, c in per:
        if k == kind and (grid is None or g == grid):
            for n, v in c.items():
                acc[n].append(v)
    return {n: {"dispatches": len(v), "mean": statistics.mean(v)} for n, v in acc.items()}


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    t = sub.add_parser("trace")
    t.add_argument("db")
    t.add_argument("--split")
    t.add_argument("--split-nth")
    t.add_argument("--by-grid", action="store_true", help="one row per (kernel, grid size)")
    f = sub.add_parser("traffic")
    f.add_argument("fetch_db")
    f.add_argument("write_db")
    f.add_argument("kind")
    p = sub.add_parser("pmc")
    p.add_argument("db")
    p.add_argument("kind")
    p.add_argument("--grid", type=int, help="only dispatches of this grid size (work-items)")
    a = ap.parse_args()
    if a.cmd == "trace":
        trace(a.db, a.split, a.by_grid, a.split_nth)
    elif a.cmd == "traffic":
        import json
        print(json.dumps(traffic(a.fetch_db, a.write_db, a.kind), indent=1))
    else:
        import json
        print(json.dumps(pmc(a.db, a.kind, a.grid), indent=1))


if __name__ == "__main__":
    main()
