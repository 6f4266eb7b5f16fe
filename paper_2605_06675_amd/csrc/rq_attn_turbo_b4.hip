#include "rq_attn_impl.h"

RQ_DEFINE_ATTN_LAUNCHER(RQ_TURBO, 1, 4, launch_attn_turbo_b4)
