// Library-wide entry points of the C ABI: error strings and the version.
#include "common.h"

extern "C" const char* wedlm_strerror(int code) {
  switch (code) {
    case WEDLM_OK: return "ok";
    case WEDLM_E_ARG: return "invalid argument (null pointer or bad scalar)";
    case WEDLM_E_SHAPE: return "unsupported or inconsistent shape";
    case WEDLM_E_WORKSPACE: return "workspace too small";
    case WEDLM_E_LAUNCH: return "kernel launch failed";
    case WEDLM_E_DEVICE: return "no usable gfx950 device";
    case WEDLM_E_SCRATCH:
      return "needs more than the library's fixed scratch array";
    default: return "unknown error code";
  }
}

extern "C" int wedlm_version(void) { return WEDLM_VERSION_NUMBER; }
