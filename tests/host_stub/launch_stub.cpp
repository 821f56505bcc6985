// Host-only stand-ins for the HIP launchers, so that the C ABI (abi.cpp, group_abi.cpp) and
// the host calibration (calibrate.cpp) can be built with a host compiler and its sanitizers
// and driven by the CPU tests.  Every launch reports a device error; the workspace size is the
// library's own layout.
#include "group.h"
#include "group_launch.h"
#include "launch.h"
#include "workspace.h"

namespace aatc {

aatc_status launch_encode(const void*, int, const void*, aatc_dtype, int64_t, int64_t,
                          aatc_layout, void*, uint16_t*, int64_t, int64_t, void*) {
  return AATC_E_DEVICE;
}

aatc_status launch_encode_last(const void*, int, int, const void*, aatc_dtype, aatc_layout,
                               void*, uint16_t*, int64_t, int, const int32_t*, void*) {
  return AATC_E_DEVICE;
}

size_t decode_workspace_bytes(int batch, int n_q_heads, int n_kv_heads, int64_t cap,
                              int counter_rows) {
  return ws_layout(batch, n_q_heads, n_kv_heads, cap, counter_rows).total;
}

aatc_status launch_decode(const void*, const void*, int, int, int, const void*, aatc_dtype,
                          const void*, const uint16_t*, const void*, const uint16_t*,
                          const int32_t*, int64_t, int, int, float, float*, void*, void*,
                          const void*, const void*, aatc_dtype, int, const void*, const void*,
                          aatc_dtype, const int32_t*, int) {
  return AATC_E_DEVICE;
}

aatc_status launch_group_encode(const void*, int, int, const void*, aatc_dtype, int64_t, int64_t,
                                void*, uint16_t*, int64_t, int64_t, void*) {
  return AATC_E_DEVICE;
}

size_t group_decode_workspace_bytes(int batch, int n_q_heads, int n_kv_heads, int gkv,
                                    int64_t cap) {
  const int n_groups = n_kv_heads / gkv;
  return group_ws_layout(batch, n_groups, n_q_heads / n_groups, 128 * gkv, cap).total;
}

aatc_status launch_group_decode(const void*, const void*, int, int, int, int, const void*,
                                aatc_dtype, const void*, const uint16_t*, const void*,
                                const uint16_t*, const int32_t*, int64_t, int, int, float,
                                float*, void*, void*) {
  return AATC_E_DEVICE;
}

aatc_status noalloc_scratch(void** ptr, void*) {
  *ptr = nullptr;
  return AATC_E_DEVICE;
}

}  // namespace aatc
