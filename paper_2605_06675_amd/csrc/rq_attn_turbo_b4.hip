// Decode-attention kernel variant: TurboQuant family, bit-widths up to 4
// (code pairs looked up in LDS pair tables).
#include "rq_attn_impl.h"

RQ_DEFINE_ATTN_LAUNCHER(RQ_TURBO, 1, 4, launch_attn_turbo_b4)
