// Size rules of the kernels, host-only: which rotations each epilogue's
// kernels cover and how the decode attention splits a sequence.  Shared by
// the C ABI's argument checks and the launchers; no device code, so the
// host code of the ABI builds and runs on its own (the sanitizer test).
#include <algorithm>

#include "common.hpp"

namespace quarot {

bool rotate_supported(int epi, bool rotate, int k, int m, int n, int pro)
{
    if (n <= 0 || n % 8 != 0 || n > 32768)
        return false;
    if (pro == PRO_SWIGLU && ((epi != EPI_SYM && epi != EPI_E3M2) || !rotate))
        return false;
    if (epi == EPI_E3M2) {
        if (n % 128)
            return false;
        if (!rotate)
            return true;
        switch (m) {
        case 1: return k >= 7 && k <= 15;
        case 12: return k == 10 || k == 11;
        case 20:
        case 28: return k == 9 || k == 10;
        case 108: return k >= 5 && k <= 7;  // n a multiple of 128
        case 172: return k >= 5 && k <= 6;
        }
        return false;
    }
    if (!rotate)
        return epi == EPI_SYM || epi == EPI_SYM8 || (epi == EPI_KV && m == 1 && k >= 3 && k <= 9);
    if (epi == EPI_KV)
        return m == 1 && k >= 3 && k <= 9;
    switch (m) {
    case 1: return k >= 3 && k <= 15;
    case 12: return k >= 1 && k <= 11;
    case 20:
    case 28: return k >= 1 && k <= 10;
    case 108: return k >= 1 && k <= 7;
    case 172: return k >= 1 && k <= 6;
    }
    return false;
}

int kv_attn_splits(int64_t nq, int64_t seq_len)
{
    // about 2048 blocks in flight, chunks of at least 256 tokens
    const int64_t want = (2048 + nq - 1) / std::max<int64_t>(nq, 1);
    const int64_t most = (seq_len + 255) / 256;
    return (int)std::max<int64_t>(1, std::min(want, most));
}

}  // namespace quarot
