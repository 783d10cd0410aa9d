#include "launch.hpp"
namespace moe {
int gemm_block_m_fp8(int, int, int) { return 128; }
hipError_t launch_gemms_fp8(const GroupedGemm&, hipStream_t) { return hipErrorNotSupported; }
int gemm_block_m_int4(int, int, int) { return 64; }
hipError_t launch_gemms_int4(const GroupedGemm&, hipStream_t) { return hipErrorNotSupported; }
}
