// Internal interface between the C-ABI entry points (tv_abi.cpp) and the
// kernel launchers (tv_kernels.hip). Not installed; callers use include/tv.h.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

namespace tv {

enum class Algo : int { kTraversal = 0, kTokenLevel = 1 };

struct VerifyArgs {
  int32_t batch;
  int32_t num_nodes;
  int32_t vocab;
  const int32_t* parents;
  const int32_t* tokens;
  const void* target;
  const void* draft;
  int32_t dtype;          // TV_DTYPE_*
  float temperature;
  const float* uniforms;
  int32_t mode;           // TV_SIBLINGS_*
  int32_t* accept_len;
  int32_t* accepted_node;
  int32_t* bonus_token;
  int32_t* status;
  int8_t* node_state;
  float* node_theta;
  float* p_init;
  int32_t* counters;
};

// Argument checks that need no GPU. Returns a tv_status_t.
int validate(const VerifyArgs& a, void* workspace, size_t workspace_bytes);

// Enqueue the verification kernel on `stream`. Arguments already validated.
// Returns a tv_status_t (TV_ERR_HIP if the launch failed).
int launch(const VerifyArgs& a, Algo algo, hipStream_t stream);

}  // namespace tv
