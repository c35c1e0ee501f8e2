// Batched bf16 products (bf16 operands, float32 accumulation): not built yet.
#include "device_common.h"

namespace agn {
hipError_t launch_gemm_bf16(int, int, const GemmArgs&, hipStream_t) { return hipErrorInvalidValue; }
}  // namespace agn
