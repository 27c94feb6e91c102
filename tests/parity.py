"""Element-by-element comparison of a GPU search against the oracle.

The bar: ids and probe counts bit-exact, scores within 1e-4 absolute, except
on queries the oracle flags because a score lies within 1e-4 of tau
(TAU_EDGE: the fp32 and fp64 hit tests may disagree, which can change the
probe count and the candidate set) or within 1e-4 of the k-th score
(KTH_TIE: the k-th slot may go either way).  Such queries are counted and
their mismatches reported.  Where two returned scores are within 1e-4
(ORDER_TIE) the order of the tied entries is free, so the id sets and the
sorted score vectors are compared instead of the sequences.
"""
from __future__ import annotations

import numpy as np

import oracle

SCORE_TOL = 1e-4


def compare(ids, scores, probes, orc, tol=SCORE_TOL) -> dict:
    ids = np.asarray(ids)
    scores = np.asarray(scores, dtype=np.float64)
    probes = np.asarray(probes)
    nq = ids.shape[0]
    rep = {"queries": nq, "flag_tau_edge": 0, "flag_kth_tie": 0, "flag_order_tie": 0,
           "flagged_mismatch": 0, "mismatch": 0, "probe_mismatch": 0, "score_mismatch": 0,
           "max_score_err": 0.0, "examples": []}
    for i in range(nq):
        f = int(orc.flags[i])
        tau_edge = bool(f & oracle.FLAG_TAU_EDGE)
        kth = bool(f & oracle.FLAG_KTH_TIE)
        order_tie = bool(f & oracle.FLAG_ORDER_TIE)
        rep["flag_tau_edge"] += tau_edge
        rep["flag_kth_tie"] += kth
        rep["flag_order_tie"] += order_tie
        oi, osc = orc.ids[i], orc.scores[i]
        ok_probe = probes[i] == orc.probes[i]
        if order_tie:
            ok_ids = set(ids[i].tolist()) == set(oi.tolist())
        else:
            ok_ids = np.array_equal(ids[i], oi)
        fin = np.isfinite(osc)
        ok_pad = np.array_equal(np.isfinite(scores[i]), fin)
        err = float(np.max(np.abs(scores[i][fin] - osc[fin]))) if fin.any() else 0.0
        ok_sc = ok_pad and err <= tol
        good = ok_probe and ok_ids and ok_sc
        if tau_edge or kth:
            rep["flagged_mismatch"] += (not good)
            continue
        rep["max_score_err"] = max(rep["max_score_err"], err)
        if not good:
            rep["mismatch"] += 1
            rep["probe_mismatch"] += (not ok_probe)
            rep["score_mismatch"] += (not ok_sc)
            if len(rep["examples"]) < 5:
                rep["examples"].append({"q": i, "gpu_ids": ids[i].tolist(),
                                        "oracle_ids": oi.tolist(),
                                        "gpu_probes": int(probes[i]),
                                        "oracle_probes": int(orc.probes[i]),
                                        "score_err": err})
    return rep


def assert_parity(rep: dict):
    assert rep["mismatch"] == 0, rep
