// Hadamard factors H_m for the Kronecker construction H_n = H_{2^k} (x) H_m
// (§3.1: n = 2^k m with H_m a known Hadamard matrix).  Built at compile time
// from the published constructions:
//   m = 12, 20, 108  Paley I   (prime q = m - 1 = 3 mod 4)
//   m = 28           Paley II  (prime q = 13 = 1 mod 4)
//   m = 172          Goethals-Seidel array of four circulants of order 43
//                    whose first rows are unions of order-6 cyclotomic
//                    classes of Z_43 (primitive root 3).
// Entry (r, s) is +1 or -1; H_m H_m^T = m I.
#pragma once

#include <cstdint>

namespace quarot {

// Quadratic character of a modulo the odd prime p, by Euler's criterion.
constexpr int quad_char(int a, int p)
{
    int r = ((a % p) + p) % p;
    if (r == 0)
        return 0;
    long long acc = 1, base = r;
    for (int e = (p - 1) / 2; e > 0; e >>= 1) {
        if (e & 1)
            acc = acc * base % p;
        base = base * base % p;
    }
    return acc == 1 ? 1 : -1;
}

// Paley I: H = I + S, S = [[0, j^T], [-j, Q]], Q[i][k] = chi(k - i).
constexpr int paley1_sign(int q, int r, int s)
{
    int core = 0;
    if (r == 0)
        core = (s == 0) ? 0 : 1;
    else if (s == 0)
        core = -1;
    else
        core = quad_char(s - r, q);
    return core + (r == s ? 1 : 0);
}

// Paley II with q = 13: conference matrix C = [[0, j^T], [j, Q]] (symmetric
// for q = 1 mod 4); H = C (x) [[1,1],[1,-1]] + I (x) [[1,-1],[-1,-1]].
constexpr int paley2_sign(int q, int r, int s)
{
    int R = r >> 1, S = s >> 1, u = r & 1, v = s & 1;
    int conf = 0;
    if (R == 0 || S == 0)
        conf = (R == S) ? 0 : 1;
    else
        conf = quad_char(S - R, q);
    int k = (u & v) ? -conf : conf;
    if (R == S)
        k += (u | v) ? -1 : 1;
    return k;
}

// The four first rows (A, B, C, D) of the order-172 Goethals-Seidel array.
// Position 0 has a fixed sign; any other j is -1 when its cyclotomic class
// (discrete log base 3, mod 6) is among the chosen ones.
struct Gs43Rows {
    int x[4][43];
    constexpr Gs43Rows() : x()
    {
        constexpr int p = 43;
        const int sign0[4] = {-1, 1, 1, 1};
        const int chosen[4] = {0b000011, 0b001011, 0b001011, 0b001101};  // class bitmasks
        int cls[p] = {};
        int v = 1;
        for (int t = 0; t < p - 1; ++t) {
            cls[v] = t % 6;
            v = v * 3 % p;
        }
        for (int w = 0; w < 4; ++w) {
            x[w][0] = sign0[w];
            for (int j = 1; j < p; ++j)
                x[w][j] = ((chosen[w] >> cls[j]) & 1) ? -1 : 1;
        }
    }
};

// Goethals-Seidel array, R the back-identity, X' the transpose:
//    A    B R    C R    D R
//  -B R   A     D'R   -C'R
//  -C R  -D'R    A     B'R
//  -D R   C'R  -B'R    A
constexpr int gs172_sign(const Gs43Rows &g, int r, int s)
{
    constexpr int p = 43;
    const int I = r / p, i = r % p, J = s / p, jcol = s % p;
    auto at = [&](int w, int j) { return g.x[w][((j % p) + p) % p]; };
    if (I == J)
        return at(0, jcol - i);  // circulant A on the diagonal
    // which sequence sits in block (I, J): the array is a Latin square
    const int seq[4][4] = {{0, 1, 2, 3}, {1, 0, 3, 2}, {2, 3, 0, 1}, {3, 2, 1, 0}};
    const int neg[4][4] = {{0, 0, 0, 0}, {1, 0, 0, 1}, {1, 1, 0, 0}, {1, 0, 1, 0}};
    const int trn[4][4] = {{0, 0, 0, 0}, {0, 0, 1, 1}, {0, 1, 0, 1}, {0, 1, 1, 0}};
    const int jr = p - 1 - jcol;  // column of X that the back-identity R selects
    // X[i][c] = x[c - i]; X'[i][c] = X[c][i] = x[i - c]
    const int e = trn[I][J] ? at(seq[I][J], i - jr) : at(seq[I][J], jr - i);
    return neg[I][J] ? -e : e;
}

constexpr int hm_sign(int m, int r, int s)
{
    if (m == 1)
        return 1;
    if (m == 12 || m == 20 || m == 108)
        return paley1_sign(m - 1, r, s);
    if (m == 28)
        return paley2_sign(13, r, s);
    if (m == 172)
        return gs172_sign(Gs43Rows(), r, s);
    return 0;
}

constexpr bool hm_supported(int m)
{
    return m == 1 || m == 12 || m == 20 || m == 28 || m == 108 || m == 172;
}

// Compile-time table as floats +-1.0 (what the kernels multiply by).
template <int M>
struct HmTable {
    float v[M][M];
    constexpr HmTable() : v()
    {
        const Gs43Rows g{};
        for (int r = 0; r < M; ++r)
            for (int s = 0; s < M; ++s)
                v[r][s] = (float)(M == 172 ? gs172_sign(g, r, s) : hm_sign(M, r, s));
    }
};

// H_m as the B operand of v_mfma_i32_16x16x64_i8 for the large-m kernels,
// which form the m-factor u = t . H_m on the int8 matrix cores: column tile
// ct (16 columns), k-block kb (64 inputs), lane l holds 16 bytes,
// byte e = H[kb*64 + (l/16)*16 + e][ct*16 + l%16] as int8 (+1 / -1), 0
// past the edge.  The A operand (digits of t) uses the same lane / byte -> k
// mapping, so the hardware's own k order within an instruction does not
// matter.  Stored as dwords, 4 per lane.
template <int M>
struct HmMfmaB {
    static constexpr int CT = (M + 15) / 16;
    static constexpr int KB = (M + 63) / 64;
    uint32_t w[CT][KB][64][4];
    constexpr HmMfmaB() : w()
    {
        const Gs43Rows g{};
        for (int ct = 0; ct < CT; ++ct)
            for (int kb = 0; kb < KB; ++kb)
                for (int l = 0; l < 64; ++l)
                    for (int q = 0; q < 4; ++q) {
                        uint32_t word = 0;
                        for (int j = 0; j < 4; ++j) {
                            const int r = kb * 64 + (l / 16) * 16 + 4 * q + j;
                            const int c = ct * 16 + l % 16;
                            int v = 0;
                            if (r < M && c < M)
                                v = M == 172 ? gs172_sign(g, r, c) : hm_sign(M, r, c);
                            word |= (uint32_t)(v & 0xFF) << (8 * j);
                        }
                        w[ct][kb][l][q] = word;
                    }
    }
};

}  // namespace quarot
