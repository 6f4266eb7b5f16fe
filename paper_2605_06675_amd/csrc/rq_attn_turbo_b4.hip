// Decode-attention kernel variant: TurboQuant family, bit-widths up to 4
// (centroids looked up in register tables).
#include "rq_attn_impl.h"

RQ_DEFINE_ATTN_LAUNCHER(RQ_TURBO, 1, 4, launch_attn_turbo_b4)
