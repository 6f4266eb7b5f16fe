// Decode-attention kernel variant: quarot family, 1 value-side A operand(s),
// bit-widths up to 4.
#include "rq_attn_impl.h"

RQ_DEFINE_ATTN_LAUNCHER(RQ_QUAROT, 1, 4, launch_attn_quarot_b4)
