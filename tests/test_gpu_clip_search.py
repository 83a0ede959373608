"""GPU parity of the weights' per-row clip search (§5 Setup, App. A.2)
through the C ABI against the CPU oracle: chosen clips, codes and scales
bit for bit.  Both sides sum the squared errors in the same defined
binary64 order, so the choice is the same on any input, including rows
whose candidates tie exactly (the order then decides)."""
import numpy as np
import pytest

import workloads
from test_gpu_parity import H, T, assert_same, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2404_00456_amd as q
    q.lib()
    return torch.device("cuda:0")


@pytest.mark.parametrize("n,rotate,bits,ncand", [
    (4096, True, 4, 20), (4096, True, 8, 20), (11008, True, 4, 30), (28672, True, 6, 10),
    (8192, False, 4, 50), (256, True, 4, 100), (56, True, 8, 5)])
def test_clip_search(dev, orc, n, rotate, bits, ncand):
    import paper_2404_00456_amd as q
    rows = 96 if n <= 8192 else 24
    say(f"clip search n={n} rotate={rotate} bits={bits} ncand={ncand}")
    w = workloads.random_rows(n * 3 + bits, rows, n, "student_t3", 0.02)
    w[0] = 0
    codes, scale, clip = q.quarot_quant_search(T(w, dev), rotate=rotate, bits=bits,
                                               n_candidates=ncand)
    rq, rs, rc = orc.quant_search(w, rotate=rotate, bits=bits, n_candidates=ncand)
    assert_same(H(clip), rc, "chosen clips")
    assert_same(H(codes).view(np.uint8), rq.view(np.uint8), "codes")
    assert_same(H(scale).view(np.uint16), rs.view(np.uint16), "scales")
    if ncand > 1 and bits == 4:
        assert (rc < 1).any()  # the search does move the clip on these rows


def test_clip_search_exact_ties(dev, orc):
    import clip_ties
    import paper_2404_00456_amd as q
    rows = clip_ties.tie_rows(orc, 256, seed=3)
    say(f"clip search on {rows.shape[0]} exactly tied rows, n={rows.shape[1]}")
    codes, scale, clip = q.quarot_quant_search(T(rows, dev), rotate=False, bits=4,
                                               n_candidates=2)
    rq, rs, rc = orc.quant_search(rows, rotate=False, bits=4, n_candidates=2)
    assert_same(H(clip), rc, "chosen clips")
    assert_same(H(codes).view(np.uint8), rq.view(np.uint8), "codes")
    assert_same(H(scale).view(np.uint16), rs.view(np.uint16), "scales")
    assert 0 < int((rc < 1).sum()) < rows.shape[0]  # both candidates win somewhere
