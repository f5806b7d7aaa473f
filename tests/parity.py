"""Comparison of the GPU sampling outputs with the oracle (test helper).

Bar: token ids bit-exact except rows whose uniform lies within 1e-5 of a CDF boundary or whose top_p
lies within 1e-5 of the cumulative masses around the nucleus cut (both margins come from the
oracle); logprobs and probabilities within 1e-5 absolute; flags bit-exact; rows the oracle flags
BAD_INPUT (NaN / +inf logits) have unspecified outputs and are only checked for the flag.
"""
from __future__ import annotations

import numpy as np

TOL = 1e-5
BAND = 1e-5
ORACLE_FLAG_BITS = 1 | 2 | 4 | 8


def np_(t):
    return t.detach().cpu().numpy()


def compare_sample(ref: dict, out, rows=None, n_top: int = 0, check_flags: bool = True) -> dict:
    ids, lps, tids, tlps, flags = (np_(x) for x in out)
    if rows is not None:
        ids, lps, tids, tlps, flags = ids[rows], lps[rows], tids[rows], tlps[rows], flags[rows]
    rf = ref["flags"].astype(np.int64)
    gf = flags.astype(np.int64) & 0xFFFFFFFF
    if check_flags:
        bad = np.nonzero((gf & ORACLE_FLAG_BITS) != rf)[0]
        assert bad.size == 0, "flag mismatch rows %s: gpu %s oracle %s" % (bad[:8], gf[bad[:8]], rf[bad[:8]])
    bad_input = (rf & 4) != 0
    empty = (rf & 2) != 0
    assert (ids[empty & ~bad_input] == -1).all()
    band = (ref["cdf_margin"] < BAND) | (ref["topp_margin"] < BAND)
    cmp = ~bad_input & ~empty & ~band
    mism = np.nonzero(cmp & (ids != ref["ids"]))[0]
    assert mism.size == 0, "id mismatch rows %s: gpu %s oracle %s (margins %s %s)" % (
        mism[:8], ids[mism[:8]], ref["ids"][mism[:8]], ref["cdf_margin"][mism[:8]], ref["topp_margin"][mism[:8]])
    same = ~bad_input & ~empty & (ids == ref["ids"])
    dl = np.abs(lps[same].astype(np.float64) - ref["logprobs"][same])
    assert (dl <= TOL).all(), "logprob error %.3g at rows %s" % (dl.max(), np.nonzero(same)[0][np.argmax(dl)])
    if n_top:
        ok = ~bad_input
        assert np.array_equal(tids[ok], ref["top_ids"][ok]), "top-n ids differ"
        rt = ref["top_logprobs"][ok]
        gt = tlps[ok].astype(np.float64)
        fin = np.isfinite(rt)
        assert np.array_equal(np.isfinite(gt), fin)
        assert (np.abs(gt[fin] - rt[fin]) <= TOL).all(), "top-n logprob error %.3g" % np.abs(gt[fin] - rt[fin]).max()
    return dict(rows=int(len(ids)), compared=int(cmp.sum()), band=int(band.sum()),
                max_dlogprob=float(dl.max()) if dl.size else 0.0)
