// Decode-attention kernel variant: kivi family, 1 value-side A operand(s),
// bit-widths up to 4.
#include "rq_attn_impl.h"

RQ_DEFINE_ATTN_LAUNCHER(RQ_KIVI, 1, 4, launch_attn_kivi_n1_b4)
