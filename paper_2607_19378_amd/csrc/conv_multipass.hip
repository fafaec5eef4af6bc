// Multi-pass plans (filled in next): placeholders that report "unsupported".
#include "kernels.hpp"

namespace hyenand {
bool multipass_supported(const FftConvArgs&) { return false; }
size_t multipass_bytes_per_line(const FftConvArgs&) { return 0; }
hipError_t launch_multipass(const FftConvArgs&, int64_t, hipStream_t) { return hipErrorInvalidValue; }
bool fourstep_supported(const FftConvArgs&) { return false; }
size_t fourstep_bytes_per_line(const FftConvArgs&) { return 0; }
hipError_t launch_fourstep(const FftConvArgs&, int64_t, hipStream_t) { return hipErrorInvalidValue; }
}  // namespace hyenand
