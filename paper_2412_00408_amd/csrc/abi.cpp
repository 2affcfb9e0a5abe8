// abi.cpp — status strings and version of the libquake C ABI.
#include "quake.h"

extern "C" const char* quake_status_str(quake_status s) {
  switch (s) {
    case QUAKE_OK: return "QUAKE_OK";
    case QUAKE_EINVAL: return "QUAKE_EINVAL: invalid pointer, size, stride or scalar argument";
    case QUAKE_EDTYPE: return "QUAKE_EDTYPE: unknown quake_dtype";
    case QUAKE_EMODE: return "QUAKE_EMODE: unknown quake_mode";
    case QUAKE_EHIP: return "QUAKE_EHIP: HIP runtime call or kernel launch failed";
    case QUAKE_ENOSCRATCH:
      return "QUAKE_ENOSCRATCH: the shape needs more than the library's fixed split-row scratch";
  }
  return "QUAKE_?: unknown status";
}

extern "C" int quake_abi_version(void) { return QUAKE_ABI_VERSION; }
