// Host-side plan of one IMPALA-ResNet pass: parameter offsets in the flat buffer, the
// activation workspace layout, and the forward / backward launch sequences.
#pragma once

#include <stddef.h>
#include <stdint.h>
#include <string>

#include "../../include/cleanba_learner.h"

namespace cb {

struct ParamOffsets {
    int64_t conv_w[3][5], conv_b[3][5];   // [stage][0 = entry, 1 = res0.conv0, 2 = res0.conv1,
                                          //         3 = res1.conv0, 4 = res1.conv1]
    int64_t dense_w, dense_b, logits_w, logits_b, value_w, value_b;
    int64_t total;
};

struct NetPlan {
    impala_net_t net;
    int prec;               // Prec
    int es;                 // storage element size (2 bf16, 4 fp32)
    int64_t cap;            // frames the workspace is laid out for
    int training;
    int H[4], W[4], C[4];   // stage s reads [H[s], W[s], C[s]] and writes [H[s+1], W[s+1], C[s+1]]
    int flat, hidden, A;
    ParamOffsets po;
    // workspace byte offsets (each region 256-byte aligned)
    size_t c[3], idx[3], x[3][3], t[3][2], h;
    size_t g[3];            // gradient ping-pong buffers (backward)
    size_t wdb;             // bf16 copy of the dense weights [flat][hidden] (bf16 mode)
    size_t scratch;         // split-K / weight-gradient / head-gradient partials
    size_t scratch_bytes;
    size_t scratch_floats;  // the shared part; a second partial buffer for deferred reduces follows
    size_t total;
};

// Validation of the shape; returns an empty string when supported.
std::string check_net(const impala_net_t* net);
ParamOffsets param_offsets(const impala_net_t& net);
NetPlan make_plan(const impala_net_t& net, int prec, int64_t cap, int training);

// Launch sequences (argument validation done by the caller). n <= plan.cap frames.
// dense_bf16_ready: the bf16 copy of the dense weights in ws already holds params' values (an
// optimiser step wrote it), so the forward does not cast them again.
hipError_t run_forward(const NetPlan& p, const float* params, const uint8_t* obs,
                       const int32_t* row_idx, int64_t n, char* ws, float* logits, float* value,
                       hipStream_t s, bool dense_bf16_ready = false);
hipError_t run_backward(const NetPlan& p, const float* params, const uint8_t* obs,
                        const int32_t* row_idx, int64_t n, char* ws, const float* dlogits,
                        const float* dvalue, float* grads, hipStream_t s);
hipError_t fill_zero(float* p, int64_t n, hipStream_t s);

}  // namespace cb
