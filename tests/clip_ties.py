"""Rows whose two clip candidates tie exactly, for the clip-search tests
(§5 Setup / App. A.2: the weights' clip ratio picked by a linear search on
the squared error).

With candidates c_0 = 1 and c_1 = RN32(0.99) and scales s_A > s_B, a row
holding 7 s_A (its maximum: code 7, error 0 under s_A), 7 s_B (error 0
under s_B), pairs y + y' = k (s_A + s_B) coded k under both scales (the
error of y under one scale is minus the error of y' under the other), and
fillers below s_B / 2 (code 0, the same error under both) has the same
multiset of squared errors under both candidates, at swapped positions.
The exact errors tie; which candidate the binary64 sums prefer depends on
the order they are added in, so these rows check that a clip search sums
in the defined order.  The scales come from the oracle's quantizer.
"""
import numpy as np

C99 = float(np.float32(0.99))


def tie_scales(orc):
    """(s_A, s_B) fp16 pairs in [1, 8) with 7 s_A and 7 s_B exact in fp16,
    s_A the scale of max 7 s_A at clip 1 and s_B at clip RN32(0.99)."""
    sA = np.arange(0x3C00, 0x4800, dtype=np.uint16).view(np.float16).astype(np.float64)
    with np.errstate(over="ignore"):
        sA = sA[(7 * sA).astype(np.float16).astype(np.float64) == 7 * sA]
    rows = np.zeros((len(sA), 8), np.float32)
    rows[:, 0] = 7 * sA
    _, s1 = orc.quant_sym_f32(rows, 1.0)
    _, s2 = orc.quant_sym_f32(rows, C99)
    s1, s2 = s1.astype(np.float64), s2.astype(np.float64)
    with np.errstate(over="ignore"):
        good = (s1 == sA) & (s2 < s1) & ((7 * s2).astype(np.float16).astype(np.float64) == 7 * s2)
    return list(zip(sA[good], s2[good]))


def tie_rows(orc, count, n=2048, seed=0):
    """count fp16 rows of width n built as in the module docstring."""
    sc = tie_scales(orc)
    rng = np.random.default_rng(seed)
    out = np.empty((count, n), np.float16)
    for r in range(count):
        sA, sB = sc[int(rng.integers(len(sc)))]
        mag = np.exp(rng.uniform(np.log(2.0 ** -24), np.log(sB * 0.45), n))
        y = (mag * rng.choice([-1.0, 1.0], n)).astype(np.float16).astype(np.float64)
        pos = rng.permutation(n)
        y[pos[0]], y[pos[1]] = 7 * sA, 7 * sB
        for p in range(6):
            while True:
                k = int(rng.integers(1, 7)) * int(rng.choice([-1, 1]))
                a = np.float64(np.float16(k * sA + rng.uniform(-0.3, 0.3) * sB))
                b = k * (sA + sB) - a
                if np.float64(np.float16(b)) == b:
                    y[pos[2 + 2 * p]], y[pos[3 + 2 * p]] = a, b
                    break
        out[r] = y.astype(np.float16)
    return out


def squared_errors(orc, y, clip):
    """e_i = RN64((y_i - q_i s)^2) of the plain quantizer at this clip."""
    q, s = orc.quant_sym_f32(y.astype(np.float32)[None], clip)
    d = y.astype(np.float64) - orc.unpack_int4(q)[0].astype(np.float64) * np.float64(s[0])
    return d * d


def sum_defined_order(e):
    """256 interleaved partial sums, each in increasing index, then halved
    pairwise (P_t + P_{t+h}, h = 128 .. 1)."""
    n = len(e)
    e = np.concatenate([e, np.zeros((-n) % 256)])
    P = np.zeros(256)
    for c in range(len(e) // 256):
        P = P + e[c * 256:(c + 1) * 256]
    h = 128
    while h >= 1:
        P = P[:h] + P[h:2 * h]
        h //= 2
    return float(P[0])


def sum_left_to_right(e):
    s = 0.0
    for v in e:
        s += float(v)
    return s
