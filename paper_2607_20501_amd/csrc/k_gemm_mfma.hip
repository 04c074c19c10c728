#include "dev.hpp"
namespace mk {
bool gemm_mfma_supported(int, const GemmArgs&) { return false; }
hipError_t launch_gemm_mfma(int, const GemmArgs&, hipStream_t) { return hipErrorInvalidValue; }
}
