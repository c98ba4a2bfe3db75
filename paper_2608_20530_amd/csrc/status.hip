// Status strings of the C ABI.
#include "lilicorr.h"

extern "C" const char* lilicorr_status_string(lilicorr_status s) {
  switch (s) {
    case LILICORR_OK: return "ok";
    case LILICORR_ERR_INVALID_ARG: return "invalid argument";
    case LILICORR_ERR_UNSUPPORTED: return "unsupported size or parameter";
    case LILICORR_ERR_ALIGNMENT: return "pointer not 16-byte aligned";
    case LILICORR_ERR_WORKSPACE: return "workspace missing or too small";
    case LILICORR_ERR_HIP: return "HIP launch failed";
    case LILICORR_ERR_TIMEOUT: return "a bounded wait in a kernel gave up (outputs invalid)";
  }
  return "unknown status";
}
