"""Pins for the oracle's per-channel clip search (§5 Setup: linear search
over the squared error for the weights' clipping ratio; App. A.2): the
chosen clip minimizes the reconstruction error among the candidates when
the error is recomputed independently from the plain quantizer's codes,
one candidate reduces to plain RTN, and an outlier row is clipped."""
import numpy as np
import pytest

import workloads


def recon_err(orc, y, bits, clip):
    if bits == 4:
        q, s = orc.quant_sym_f32(y[None], clip)
        codes = orc.unpack_int4(q)[0].astype(np.float64)
    else:
        q, s = orc.quant_sym8_f32(y[None], clip, bits)
        codes = q[0].astype(np.float64)
    return float(np.sum((y.astype(np.float64) - codes * np.float64(s[0])) ** 2))


@pytest.mark.parametrize("bits", [4, 6, 8])
def test_choice_minimizes_error(orc, bits):
    w = workloads.random_rows(31 + bits, 12, 512, "student_t3", 0.02)
    q, s, c = orc.quant_search(w, rotate=True, bits=bits, n_candidates=30)
    y = orc.rotate_f16(w)
    cands = [np.float32((100 - j) / 100) for j in range(30)]
    for r in range(w.shape[0]):
        errs = [recon_err(orc, y[r], bits, float(cj)) for cj in cands]
        best = int(np.argmin(errs))
        assert c[r] == cands[best] or abs(errs[best] - errs[cands.index(c[r])]) <= 1e-12 * errs[best]
        # and the stored codes are the plain quantizer's at that clip
        if bits == 4:
            q2, s2 = orc.quant_sym_f32(y[r:r + 1], float(c[r]))
        else:
            q2, s2 = orc.quant_sym8_f32(y[r:r + 1], float(c[r]), bits)
        assert np.array_equal(q[r], q2[0]) and s[r] == s2[0]


def test_one_candidate_is_plain_rtn(orc):
    w = workloads.random_rows(5, 9, 4096, "normal", 0.02)
    q, s, c = orc.quant_search(w, rotate=True, bits=4, n_candidates=1)
    q2, s2 = orc.quant_int4(w, rotate=True, clip=1.0)
    assert np.all(c == 1.0) and np.array_equal(q, q2) and np.array_equal(s, s2)


def test_gaussian_rows_get_clipped(orc):
    """For 4-bit codes of Gaussian rows the squared error is smallest well
    inside the row maximum (the tail values are rare), so the search clips;
    with 8 bits the gain is small and the clip stays near 1."""
    w = workloads.random_rows(8, 6, 4096, "normal", 0.02)
    _, _, c4 = orc.quant_search(w, rotate=False, bits=4, n_candidates=50)
    _, _, c8 = orc.quant_search(w, rotate=False, bits=8, n_candidates=50)
    assert np.all(c4 < 0.9)
    assert np.all(c8 > c4)


def test_exact_ties_follow_the_defined_order(orc):
    """On rows whose two candidates' errors tie exactly (clip_ties), the
    oracle keeps candidate 1 only where the defined summation order makes
    its error strictly smaller, and these rows do depend on the order: a
    left-to-right sum would choose differently on some of them."""
    import clip_ties
    rows = clip_ties.tie_rows(orc, 96)
    _, _, c = orc.quant_search(rows, rotate=False, bits=4, n_candidates=2)
    differs = 0
    for r in range(rows.shape[0]):
        e0 = clip_ties.squared_errors(orc, rows[r], 1.0)
        e1 = clip_ties.squared_errors(orc, rows[r], clip_ties.C99)
        assert np.array_equal(np.sort(e0), np.sort(e1))  # an exact tie
        assert not np.array_equal(e0, e1)                # at different positions
        t0, t1 = clip_ties.sum_defined_order(e0), clip_ties.sum_defined_order(e1)
        pick = 1 if t1 < t0 else 0
        assert c[r] == (np.float32(clip_ties.C99) if pick else np.float32(1.0))
        l0, l1 = clip_ties.sum_left_to_right(e0), clip_ties.sum_left_to_right(e1)
        differs += pick != (1 if l1 < l0 else 0)
    assert differs >= 2
