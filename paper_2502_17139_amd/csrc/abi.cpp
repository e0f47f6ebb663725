// C ABI housekeeping: version and status strings.
#include "fastcoder.h"

extern "C" int32_t fc_abi_version(void) { return 4; }

extern "C" const char* fc_status_string(fc_status s) {
  switch (s) {
    case FC_OK: return "FC_OK";
    case FC_ERR_INVALID: return "FC_ERR_INVALID: argument out of range or null pointer";
    case FC_ERR_WORKSPACE: return "FC_ERR_WORKSPACE: workspace missing or too small";
    case FC_ERR_DEVICE: return "FC_ERR_DEVICE: HIP launch/runtime error or device-side check failed";
    case FC_ERR_UNSUPPORTED: return "FC_ERR_UNSUPPORTED: request outside the library's limits";
  }
  return "FC_ERR_UNKNOWN";
}
