"""Element-by-element comparison of the HIP estimator's cells with the oracle's.

Agreement rule: the iteration time of every cell within 1e-5 relative of the
oracle's (fp64) value, the plan (dp, tp, pp, m) and the stage cuts identical.
A cell whose plan or cuts differ is a near-tie when the GPU's plan, priced by
the oracle with the GPU's cuts, is within 1e-5 of the oracle's best (or sits
on the memory limit within 1e-5); anything else is a mismatch.
"""
from __future__ import annotations

import numpy as np

REL_T = 1e-5


def decode(w, ids):
    """Split cell indices into (job, type, count index)."""
    ids = np.asarray(ids, np.int64)
    ci = ids % w.n_counts
    g = (ids // w.n_counts) % w.n_types
    j = ids // (w.n_counts * w.n_types)
    return j, g, ci


def compare(w, gpu, ids, oracle, kappa_round=0, ref=None, rule=0, tables=None):
    """gpu: dict with t_iter, thr, dp, tp, pp, m, feasible, cuts (u8 rows) for `ids`,
    estimated under partition rule `rule`, or with communication latency from
    `tables` = (volumes, latencies).
    Returns a report dict; report['mismatch'] lists failing cells."""
    ids = np.asarray(ids, np.int64)
    if ref is None:
        ref = (oracle.cells(w, ids, kappa_round=kappa_round, rule=rule) if tables is None else
               oracle.cells_tab(w, ids, tables, kappa_round=kappa_round))

    def price(j, g, n, kap, dp, tp, pp, m, cuts=None):
        if tables is None:
            return oracle.eval_plan(w, j, g, n, kap, dp, tp, pp, m, cuts=cuts, rule=rule if cuts is None else 0)
        return oracle.eval_plan_tab(w, j, g, n, kap, dp, tp, pp, m, tables, cuts=cuts)

    J, G, CI = decode(w, ids)
    rep = dict(n=len(ids), exact=0, near_tie=0, mismatch=[], max_rel_T=0.0, max_rel_thr=0.0,
               infeasible=0)
    kap_all = w.kappa[kappa_round]
    for s in range(len(ids)):
        o_inf = not np.isfinite(ref["T"][s])
        g_inf = not bool(gpu["feasible"][s])
        gcuts = None
        if gpu.get("cuts") is not None:
            gcuts = np.asarray(gpu["cuts"][s])
        if o_inf and g_inf:
            ok = (np.isinf(gpu["t_iter"][s]) and gpu["thr"][s] == 0 and gpu["dp"][s] == 0)
            if gcuts is not None:
                ok = ok and (gcuts == 0xFF).all()
            if ok:
                rep["exact"] += 1
                rep["infeasible"] += 1
            else:
                rep["mismatch"].append((int(ids[s]), "infeasible cell has non-sentinel outputs"))
            continue
        j, g, ci = int(J[s]), int(G[s]), int(CI[s])
        n = int(w.counts[ci])
        kap = float(kap_all[g * w.n_counts + ci])
        if not g_inf:
            plan = (int(gpu["dp"][s]), int(gpu["tp"][s]), int(gpu["pp"][s]), int(gpu["m"][s]))
            pp = plan[2]
            if gcuts is not None:
                gc = [int(c) for c in gcuts[:pp - 1]]
                if not (gcuts[pp - 1:] == 0xFF).all():
                    rep["mismatch"].append((int(ids[s]), "cut row not padded with 0xFF"))
                    continue
            else:
                gc = None
        if not o_inf and not g_inf:
            oplan = (int(ref["dp"][s]), int(ref["tp"][s]), int(ref["pp"][s]), int(ref["m"][s]))
            ocuts = [int(c) for c in ref["cuts"][s][:oplan[2] - 1]]
            relT = abs(float(gpu["t_iter"][s]) - ref["T"][s]) / ref["T"][s]
            same = plan == oplan and (gc is None or gc == ocuts)
            if same:
                relthr = abs(float(gpu["thr"][s]) - ref["thr"][s]) / ref["thr"][s]
                rep["max_rel_T"] = max(rep["max_rel_T"], relT)
                rep["max_rel_thr"] = max(rep["max_rel_thr"], relthr)
                if relT <= REL_T and relthr <= REL_T:
                    rep["exact"] += 1
                else:
                    rep["mismatch"].append((int(ids[s]), f"T off by {relT:.3g}"))
                continue
        # differing decision: price the GPU's choice in the oracle
        if g_inf:
            # the oracle found a feasible plan; near-tie only if it sits on the memory limit
            e = price(j, g, n, kap, int(ref["dp"][s]), int(ref["tp"][s]), int(ref["pp"][s]), int(ref["m"][s]))
            if abs(e["mem_max"] - float(w.mem[g])) <= REL_T * float(w.mem[g]):
                rep["near_tie"] += 1
            else:
                rep["mismatch"].append((int(ids[s]), "GPU infeasible, oracle feasible"))
            continue
        e = price(j, g, n, kap, *plan, cuts=gc)
        on_mem_edge = abs(e["mem_max"] - float(w.mem[g])) <= REL_T * float(w.mem[g])
        if not e["feasible"] and not on_mem_edge:
            rep["mismatch"].append((int(ids[s]), f"GPU plan {plan} does not fit"))
            continue
        if abs(float(gpu["t_iter"][s]) - e["T"]) > REL_T * e["T"]:
            rep["mismatch"].append((int(ids[s]), "GPU T does not price its own plan"))
            continue
        if o_inf:
            if on_mem_edge:
                rep["near_tie"] += 1
            else:
                rep["mismatch"].append((int(ids[s]), "GPU feasible, oracle infeasible"))
            continue
        if abs(e["T"] - ref["T"][s]) <= REL_T * ref["T"][s] or on_mem_edge:
            rep["near_tie"] += 1
        else:
            rep["mismatch"].append((int(ids[s]), f"plan {plan} cuts {gc} vs oracle {oplan} {ocuts}: "
                                                 f"T {e['T']:.9g} vs {ref['T'][s]:.9g}"))
    return rep


def oracle_cells_parallel(oracle, w, ids, threads=None, **kw):
    """oracle.cells over `ids` split across host threads (the oracle's C
    calls keep no global state and release the interpreter lock)."""
    import os
    from concurrent.futures import ThreadPoolExecutor
    ids = np.asarray(ids, np.int64)
    threads = threads or max(1, min(16, os.cpu_count() or 1))
    chunks = [c for c in np.array_split(ids, threads) if len(c)]
    with ThreadPoolExecutor(max_workers=len(chunks)) as ex:
        parts = list(ex.map(lambda c: oracle.cells(w, c, **kw), chunks))
    return {k: np.concatenate([part[k] for part in parts]) for k in parts[0]}


def select(res, ids):
    """Rows `ids` of a full-matrix result dict (numpy)."""
    out = {}
    for k, v in res.items():
        if v is None:
            continue
        out[k] = v[ids]
    return out
