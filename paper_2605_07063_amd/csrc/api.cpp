// Version and status strings of the C ABI (dr_api.h).
#include "dr_api.h"

extern "C" int dr_abi_version(void) { return DR_ABI_VERSION; }

extern "C" const char* dr_status_string(dr_status s) {
  switch (s) {
    case DR_OK: return "ok";
    case DR_ERR_ARG: return "invalid argument";
    case DR_ERR_DTYPE: return "unsupported dtype";
    case DR_ERR_NOT_SPD: return "matrix not positive definite";
    case DR_ERR_NOT_CONVERGED: return "iteration did not converge";
    case DR_ERR_NONFINITE: return "non-finite input";
    case DR_ERR_WORKSPACE: return "workspace missing or too small";
    case DR_ERR_HIP: return "HIP launch error";
    case DR_ERR_UNSUPPORTED: return "unsupported size";
    case DR_ERR_TOO_LARGE: return "problem needs more scratch than the no-allocation entry point holds";
  }
  return "unknown status";
}
