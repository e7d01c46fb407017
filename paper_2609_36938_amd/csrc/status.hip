// Status strings of the C ABI.
#include "janus.h"

extern "C" const char *janus_status_string(int status)
{
    switch (status) {
    case JANUS_OK: return "ok";
    case JANUS_ERR_INVALID_ARG: return "invalid argument";
    case JANUS_ERR_UNSUPPORTED: return "unsupported shape or dtype";
    case JANUS_ERR_WORKSPACE: return "workspace too small";
    case JANUS_ERR_DEVICE: return "device launch failed";
    default: return "unknown status";
    }
}
