// Decode-attention kernel variant: kivi family, 2 value-side A operand(s),
// bit-widths up to 8.
#include "rq_attn_impl.h"

RQ_DEFINE_ATTN_LAUNCHER(RQ_KIVI, 2, 8, launch_attn_kivi_n2_b8)
