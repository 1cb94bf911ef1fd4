// The library's version and return-code strings.  Plain host code with no
// device code, so that the host-only sanitizer build of the expert cache can
// link it too.
#include "../../include/draftexpert.h"

extern "C" {

int de_abi_version(void) { return DE_ABI_VERSION; }

const char* de_error_string(int code) {
  switch (code) {
    case DE_OK: return "ok";
    case DE_ERR_INVALID: return "invalid argument (null or misaligned pointer, or a size out of range)";
    case DE_ERR_UNSUPPORTED: return "unsupported dtype or option combination";
    case DE_ERR_HIP: return "HIP launch or runtime error";
    case DE_ERR_WORKSPACE: return "workspace missing, misaligned (256 B) or too small";
    case DE_ERR_NOT_RESIDENT: return "a needed routed expert had no valid slot (its term was dropped)";
    default: return "unknown error code";
  }
}

}  // extern "C"
