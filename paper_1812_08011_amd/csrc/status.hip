#include "fp8train.h"

extern "C" const char* fp8t_status_string(int status) {
    switch (status) {
        case FP8T_OK: return "ok";
        case FP8T_EINVAL: return "invalid argument";
        case FP8T_EWORKSPACE: return "workspace too small";
        case FP8T_EHIP: return "HIP runtime error at launch";
        default: return "unknown status";
    }
}
