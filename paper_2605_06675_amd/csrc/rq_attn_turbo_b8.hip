// Decode-attention kernel variant: TurboQuant family, bit-widths up to 8
// (widths above 4 looked up in LDS centroid tables).
#include "rq_attn_impl.h"

RQ_DEFINE_ATTN_LAUNCHER(RQ_TURBO, 1, 8, launch_attn_turbo_b8)
