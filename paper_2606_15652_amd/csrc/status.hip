// Status strings and version of libmq.
#include "mq_device.h"

extern "C" const char* mq_status_string(mq_status s) {
    switch (s) {
        case MQ_OK: return "MQ_OK";
        case MQ_ERR_INVALID_ARG: return "MQ_ERR_INVALID_ARG: null pointer, negative size or bad budget";
        case MQ_ERR_UNSUPPORTED_SHAPE: return "MQ_ERR_UNSUPPORTED_SHAPE: K/N must be multiples of 128 within limits, leading dimensions large enough and multiples of 8";
        case MQ_ERR_MISALIGNED: return "MQ_ERR_MISALIGNED: pointer alignment rule violated";
        case MQ_ERR_WORKSPACE: return "MQ_ERR_WORKSPACE: workspace too small";
        case MQ_ERR_HIP: return "MQ_ERR_HIP: the HIP runtime reported an error";
        case MQ_ERR_SCRATCH_LIMIT: return "MQ_ERR_SCRATCH_LIMIT: the scratch-free call needs more than the library's 128 MiB scratch array";
    }
    return "MQ_ERR_UNKNOWN";
}

extern "C" int mq_version(void) { return 200; }
