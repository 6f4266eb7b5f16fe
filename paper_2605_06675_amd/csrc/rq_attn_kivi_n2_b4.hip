// Decode-attention kernel variant: kivi family, 2 value-side A operand(s),
// bit-widths up to 4.
#include "rq_attn_impl.h"

RQ_DEFINE_ATTN_LAUNCHER(RQ_KIVI, 2, 4, launch_attn_kivi_n2_b4)
