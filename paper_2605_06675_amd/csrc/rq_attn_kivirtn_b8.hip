// Decode-attention kernel variant: mixed family (KIVI keys, RTN values),
// bit-widths up to 8.
#include "rq_attn_impl.h"

RQ_DEFINE_ATTN_LAUNCHER(RQ_KIVI_RTN, 1, 8, launch_attn_kivirtn_b8)
