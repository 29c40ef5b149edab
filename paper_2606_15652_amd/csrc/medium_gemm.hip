// The medium-M tiles of the streaming GEMM kernel (Section 3 Eq. (4); the
// kernel and its launcher are those of fused_gemm.hip), in a translation unit
// of their own so that the build can give them another instruction-scheduling
// strategy (build.py: maximum ILP).  Only launch_medium_tiles<RAW> is defined
// here; fused_gemm.hip calls it.
#define MQ_MEDIUM_TU
#include "fused_gemm.hip"
