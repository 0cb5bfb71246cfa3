// Exact and relaxed tree acceptance by sampling (Sec. 3.1, Eq. 1).
#include "../launch.h"

namespace adt {

size_t accept_ws_bytes(int V) { return (size_t)V * 8 + 4096; }

adt_status launch_accept_sample(const float*, int64_t, int, const int32_t*, const int32_t*, const int32_t*,
                                const int32_t*, int, const adt_accept_cfg&, uint64_t, int32_t*, int32_t*, int32_t*,
                                void*, size_t, hipStream_t) {
  adt::set_error("sampling acceptance is not built yet");
  return ADT_E_UNSUPPORTED;
}

}  // namespace adt
