// api.hip -- host-only entry points of libams: status text and build info.
#include "ams_device.h"

extern "C" const char *ams_status_str(ams_status s)
{
    switch (s) {
    case AMS_OK: return "ok";
    case AMS_ERR_NULL: return "a required pointer is NULL";
    case AMS_ERR_SIZE: return "a size is negative, too large, or inconsistent";
    case AMS_ERR_DTYPE: return "unknown storage dtype";
    case AMS_ERR_DIMS: return "unsupported layer widths";
    case AMS_ERR_WORKSPACE: return "workspace too small";
    case AMS_ERR_HIP: return "HIP launch or runtime error";
    case AMS_ERR_ID_RANGE: return "image ID out of range";
    case AMS_ERR_MODE: return "unknown pooling mode";
    }
    return "unknown status";
}

extern "C" const char *ams_build_info(void)
{
    return "libams 0.1.0 gfx950 wave64";
}
