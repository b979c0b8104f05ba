// Status codes, thread-local error details and launch checking.
#include "bt_internal.h"

namespace bt {

static thread_local char g_err[512] = "";
static thread_local bt_status g_status = BT_OK;

bt_status fail(bt_status s, const char* fmt, ...) {
  g_status = s;
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return s;
}

void clear_error() {
  g_err[0] = 0;
  g_status = BT_OK;
}

bt_status check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(BT_EHIP, "%s launch failed: %s", what, hipGetErrorString(e));
  return BT_OK;
}

}  // namespace bt

extern "C" const char* bt_status_str(bt_status s) {
  switch (s) {
    case BT_OK: return "BT_OK";
    case BT_EINVAL: return "BT_EINVAL";
    case BT_ESHAPE: return "BT_ESHAPE";
    case BT_EALIGN: return "BT_EALIGN";
    case BT_EWORKSPACE: return "BT_EWORKSPACE";
    case BT_EHIP: return "BT_EHIP";
    case BT_ENONFINITE: return "BT_ENONFINITE";
  }
  return "BT_UNKNOWN";
}

extern "C" const char* bt_last_error(void) { return bt::g_err; }

extern "C" bt_status bt_last_status(void) { return bt::g_status; }

extern "C" const char* bt_version(void) { return "0.1.0"; }
