// verify_parallel.hip -- tree-masked factorised verification (SpecLA §4.2).
#include "device.hpp"
#include "kernels.hpp"

namespace sla {

bool parallel_supported(int, int, int) { return false; }

hipError_t launch_verify_parallel(const VerifyArgs &, int, hipStream_t) { return hipErrorInvalidConfiguration; }

}  // namespace sla
