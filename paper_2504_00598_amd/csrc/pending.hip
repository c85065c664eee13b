// Entry points whose kernels are not built yet: they refuse loudly.
#include "cfp_internal.h"

namespace cfp {

hipError_t launch_scan(const cfp_chain_desc &, const int32_t *, uint8_t *, size_t, uint8_t *, int, SearchResult *,
                       const WsHeader *, int64_t *, int32_t *, hipStream_t) {
  return hipErrorNotSupported;
}
size_t scan_region_bytes(int, int, int) { return 0; }

}  // namespace cfp
