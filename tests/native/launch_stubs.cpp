// Stand-ins for the library's kernel launchers, for the host-only build of
// the C ABI (tests/test_sanitizers.py): every call is counted and fails, so
// the driver can check that no entry point tried to launch anything.
#include "../../paper_2404_00456_amd/csrc/common.hpp"

int quarot_stub_launches = 0;

namespace quarot {

static hipError_t stub()
{
    ++quarot_stub_launches;
    return hipErrorInvalidValue;
}

hipError_t launch_rotate(const RotArgs &, int, bool, int, int, hipStream_t, int) { return stub(); }
hipError_t launch_gemm(const GemmArgs &, hipStream_t, int) { return stub(); }
hipError_t launch_pack_e3m2(const uint8_t *, uint8_t *, int64_t, int, hipStream_t) { return stub(); }
hipError_t launch_gemm_grouped(const GemmArgs &, int, hipStream_t) { return stub(); }
hipError_t launch_gemm_grouped_e3m2(const GemmArgs &, int, hipStream_t) { return stub(); }
hipError_t launch_quant_grouped(const void *, bool, uint8_t *, uint16_t *, int64_t, int, int, float,
                                hipStream_t)
{
    return stub();
}
hipError_t launch_kv_dequant(const KvDeqArgs &, bool, hipStream_t) { return stub(); }
hipError_t launch_swiglu(const uint16_t *, const uint16_t *, uint16_t *, int64_t, hipStream_t)
{
    return stub();
}
hipError_t launch_quant_search(const SearchArgs &, int, bool, hipStream_t) { return stub(); }
hipError_t launch_kv_attention(const KvAttnArgs &, hipStream_t) { return stub(); }
hipError_t scratch_buffer(void **) { return stub(); }

}  // namespace quarot
