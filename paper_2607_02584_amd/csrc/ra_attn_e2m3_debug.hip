// ra_attn_e2m3_debug.hip -- the debug-dump instantiations of the FP6
// attention kernel (the S, P-code and running-maximum dumps behind
// rotate_attn_attn_int4_debug), compiled from the same source as the plain
// kernels in a translation unit of their own.
#define RA_E2M3_DEBUG_TU 1
#include "ra_attn_e2m3.hip"
