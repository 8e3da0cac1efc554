// frac_bwd.hip -- chunked parallel scan, backward.
#include "frac_device.h"
#include "frac_kernels.h"

namespace frac {

size_t scan_bwd_workspace(const ScanParams&) { return 0; }

hipError_t launch_scan_bwd(const ScanParams&, void*, size_t, hipStream_t) { return hipErrorNotSupported; }

}  // namespace frac
