// host_ffn.h -- the host tier's split call (host_ffn.cpp), for the stack: begin hands one token's host-served
// experts to the pool's threads and returns at once; finish makes the caller join the remaining work and
// returns when y is complete.  moe_host_expert_ffn is begin + finish.  Plain C++ (no HIP types).
#pragma once

struct moe_host_tier;

namespace moe {
int host_ffn_begin(moe_host_tier *t, const float *x, int H, int I, int w_dtype, int n, const void *const *blobs,
                   const float *weights, float *y_out);
int host_ffn_finish(moe_host_tier *t);
}  // namespace moe
