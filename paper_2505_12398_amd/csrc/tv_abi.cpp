// C-ABI entry points of libtv (declared in include/tv.h): argument validation
// on the host, then one kernel launch on the caller's stream. Nothing here
// touches the GPU before the arguments are known to be valid, so the
// validation paths run on machines without a GPU.
#include <math.h>
#include <stdint.h>

#include "tv.h"
#include "tv_launch.h"

namespace tv {

int validate(const VerifyArgs& a, void* workspace, size_t workspace_bytes) {
  const int st = validate_args(a);
  if (st != TV_OK || a.batch == 0) return st;
  if (!workspace || reinterpret_cast<uintptr_t>(workspace) % 256 ||
      workspace_bytes < workspace_layout(a.batch, a.vocab).bytes)
    return TV_ERR_WORKSPACE;
  return TV_OK;
}

int validate_args(const VerifyArgs& a) {
  if (a.batch < 0 || a.num_nodes < 1 || a.vocab < 2) return TV_ERR_INVALID_ARG;
  if (a.dtype != TV_DTYPE_BF16 && a.dtype != TV_DTYPE_F32) return TV_ERR_INVALID_ARG;
  if (a.mode != TV_SIBLINGS_WITHOUT_REPLACEMENT && a.mode != TV_SIBLINGS_WITH_REPLACEMENT)
    return TV_ERR_INVALID_ARG;
  if (!(a.temperature > 0.0f) || !isfinite(a.temperature)) return TV_ERR_INVALID_ARG;
  if (a.temperature < TV_MIN_TEMPERATURE || a.temperature > TV_MAX_TEMPERATURE)
    return TV_ERR_UNSUPPORTED;
  if (a.batch > TV_MAX_BATCH || a.num_nodes > TV_MAX_NODES || a.vocab > TV_MAX_VOCAB)
    return TV_ERR_UNSUPPORTED;
  if (a.dtype == TV_DTYPE_F32 && a.vocab > TV_MAX_VOCAB_F32) return TV_ERR_UNSUPPORTED;
  if (a.batch == 0) return TV_OK;
  if (!a.parents || !a.tokens || !a.target || !a.draft || !a.uniforms || !a.accept_len ||
      !a.accepted_node || !a.bonus_token || !a.status)
    return TV_ERR_INVALID_ARG;
  const size_t esize = a.dtype == TV_DTYPE_BF16 ? 2 : 4;
  const uintptr_t t = reinterpret_cast<uintptr_t>(a.target);
  const uintptr_t d = reinterpret_cast<uintptr_t>(a.draft);
  if (t % esize || d % esize) return TV_ERR_INVALID_ARG;
  if ((t & 15) != (d & 15)) return TV_ERR_UNSUPPORTED;
  const void* int_ptrs[] = {a.parents, a.tokens, a.uniforms, a.accept_len, a.accepted_node,
                            a.bonus_token, a.status, a.node_theta, a.p_init, a.counters};
  for (const void* p : int_ptrs)
    if (reinterpret_cast<uintptr_t>(p) % 4) return TV_ERR_INVALID_ARG;
  return TV_OK;
}

int validate_lmhead(const LmheadArgs& a, void* workspace, size_t workspace_bytes) {
  if (a.rows < 0 || a.hidden_size < 8 || a.vocab < 2) return TV_ERR_INVALID_ARG;
  if (a.hidden_size % 8) return TV_ERR_UNSUPPORTED;
  if (!(a.temperature > 0.0f) || !isfinite(a.temperature)) return TV_ERR_INVALID_ARG;
  if (a.temperature < TV_MIN_TEMPERATURE || a.temperature > TV_MAX_TEMPERATURE)
    return TV_ERR_UNSUPPORTED;
  if (a.rows > TV_MAX_LMHEAD_ROWS || a.hidden_size > TV_MAX_HIDDEN || a.vocab > TV_MAX_VOCAB)
    return TV_ERR_UNSUPPORTED;
  if (a.rows == 0) return TV_OK;
  if (!a.hidden || !a.weight || !a.logits || !a.row_max || !a.row_sum) return TV_ERR_INVALID_ARG;
  if (reinterpret_cast<uintptr_t>(a.hidden) % 16 || reinterpret_cast<uintptr_t>(a.weight) % 16 ||
      reinterpret_cast<uintptr_t>(a.logits) % 2 || reinterpret_cast<uintptr_t>(a.row_max) % 4 ||
      reinterpret_cast<uintptr_t>(a.row_sum) % 8)
    return TV_ERR_INVALID_ARG;
  if (!workspace || reinterpret_cast<uintptr_t>(workspace) % 256 ||
      workspace_bytes < lmhead_layout(a.rows, a.vocab).bytes)
    return TV_ERR_WORKSPACE;
  return TV_OK;
}

int validate_sample(const SampleArgs& a) {
  if (a.batch < 0 || a.num_nodes < 1 || a.vocab < 2) return TV_ERR_INVALID_ARG;
  if (a.dtype != TV_DTYPE_BF16 && a.dtype != TV_DTYPE_F32) return TV_ERR_INVALID_ARG;
  if (a.mode != TV_SIBLINGS_WITHOUT_REPLACEMENT && a.mode != TV_SIBLINGS_WITH_REPLACEMENT)
    return TV_ERR_INVALID_ARG;
  if (!(a.temperature > 0.0f) || !isfinite(a.temperature)) return TV_ERR_INVALID_ARG;
  if (a.temperature < TV_MIN_TEMPERATURE || a.temperature > TV_MAX_TEMPERATURE)
    return TV_ERR_UNSUPPORTED;
  if (a.batch > TV_MAX_BATCH || a.num_nodes > TV_MAX_NODES || a.vocab > TV_MAX_VOCAB)
    return TV_ERR_UNSUPPORTED;
  if (a.dtype == TV_DTYPE_F32 && a.vocab > TV_MAX_VOCAB_F32) return TV_ERR_UNSUPPORTED;
  if (a.batch == 0) return TV_OK;
  if (!a.parents || !a.draft || !a.uniforms || !a.tokens || !a.status) return TV_ERR_INVALID_ARG;
  const size_t esize = a.dtype == TV_DTYPE_BF16 ? 2 : 4;
  if (reinterpret_cast<uintptr_t>(a.draft) % esize) return TV_ERR_INVALID_ARG;
  const void* int_ptrs[] = {a.parents, a.uniforms, a.tokens, a.status};
  for (const void* p : int_ptrs)
    if (reinterpret_cast<uintptr_t>(p) % 4) return TV_ERR_INVALID_ARG;
  return TV_OK;
}

}  // namespace tv

namespace {

int verify_common(tv::Algo algo, int32_t batch, int32_t num_nodes, int32_t vocab,
                  const int32_t* parents, const int32_t* tokens, const void* target_logits,
                  const void* draft_logits, int32_t dtype, float temperature,
                  const float* uniforms, int32_t mode, int32_t* accept_len,
                  int32_t* accepted_node, int32_t* bonus_token, int32_t* status,
                  int8_t* node_state, float* node_theta, float* p_init, int32_t* counters,
                  void* workspace, size_t workspace_bytes, hipStream_t stream) {
  tv::VerifyArgs a{batch,       num_nodes,  vocab,  parents,  tokens,     target_logits,
                   draft_logits, dtype,      temperature, uniforms, mode,  accept_len,
                   accepted_node, bonus_token, status, node_state, node_theta, p_init,
                   counters};
  int st = tv::validate(a, workspace, workspace_bytes);
  if (st != TV_OK || batch == 0) return st;
  return tv::launch(a, algo, workspace, stream);
}

}  // namespace

extern "C" {

size_t tv_workspace_size(int32_t batch, int32_t num_nodes, int32_t vocab) {
  if (batch < 1 || batch > TV_MAX_BATCH || num_nodes < 1 || num_nodes > TV_MAX_NODES ||
      vocab < 2 || vocab > TV_MAX_VOCAB)
    return 0;
  return tv::workspace_layout(batch, vocab).bytes;
}

int tv_verify(int32_t batch, int32_t num_nodes, int32_t vocab, const int32_t* parents,
              const int32_t* tokens, const void* target_logits, const void* draft_logits,
              int32_t dtype, float temperature, const float* uniforms, int32_t mode,
              int32_t* accept_len, int32_t* accepted_node, int32_t* bonus_token,
              int32_t* status, int8_t* node_state, float* node_theta, float* p_init,
              int32_t* counters, void* workspace, size_t workspace_bytes,
              hipStream_t stream) {
  return verify_common(tv::Algo::kTraversal, batch, num_nodes, vocab, parents, tokens,
                       target_logits, draft_logits, dtype, temperature, uniforms, mode,
                       accept_len, accepted_node, bonus_token, status, node_state, node_theta,
                       p_init, counters, workspace, workspace_bytes, stream);
}

int tv_verify_tokenlevel(int32_t batch, int32_t num_nodes, int32_t vocab,
                         const int32_t* parents, const int32_t* tokens,
                         const void* target_logits, const void* draft_logits, int32_t dtype,
                         float temperature, const float* uniforms, int32_t mode,
                         int32_t* accept_len, int32_t* accepted_node, int32_t* bonus_token,
                         int32_t* status, int8_t* node_state, float* node_theta,
                         float* p_init, int32_t* counters, void* workspace,
                         size_t workspace_bytes, hipStream_t stream) {
  return verify_common(tv::Algo::kTokenLevel, batch, num_nodes, vocab, parents, tokens,
                       target_logits, draft_logits, dtype, temperature, uniforms, mode,
                       accept_len, accepted_node, bonus_token, status, node_state, node_theta,
                       p_init, counters, workspace, workspace_bytes, stream);
}

int tv_verify_noalloc(int32_t batch, int32_t num_nodes, int32_t vocab, const int32_t* parents,
                      const int32_t* tokens, const void* target_logits,
                      const void* draft_logits, int32_t dtype, float temperature,
                      const float* uniforms, int32_t mode, int32_t* accept_len,
                      int32_t* accepted_node, int32_t* bonus_token, int32_t* status,
                      int8_t* node_state, float* node_theta, float* p_init, int32_t* counters,
                      hipStream_t stream) {
  const tv::VerifyArgs a{batch,       num_nodes,  vocab,  parents,  tokens,     target_logits,
                         draft_logits, dtype,      temperature, uniforms, mode,  accept_len,
                         accepted_node, bonus_token, status, node_state, node_theta, p_init,
                         counters};
  const int st = tv::validate_args(a);
  if (st != TV_OK || batch == 0) return st;
  if (tv::workspace_layout(batch, vocab).bytes > tv::kStaticScratchBytes) return TV_ERR_UNSUPPORTED;
  void* scratch = nullptr;
  size_t scratch_bytes = 0;
  const int sst = tv::static_scratch(&scratch, &scratch_bytes);
  if (sst != TV_OK) return sst;
  return tv::launch(a, tv::Algo::kTraversal, scratch, stream);
}

int tv_verify_stats(int32_t batch, int32_t num_nodes, int32_t vocab, const int32_t* parents,
                    const int32_t* tokens, const void* target_logits, const void* draft_logits,
                    int32_t dtype, float temperature, const float* uniforms, int32_t mode,
                    const float* target_max, const double* target_sum, const float* draft_max,
                    const double* draft_sum, int32_t* accept_len, int32_t* accepted_node,
                    int32_t* bonus_token, int32_t* status, int8_t* node_state, float* node_theta,
                    float* p_init, int32_t* counters, void* workspace, size_t workspace_bytes,
                    hipStream_t stream) {
  tv::VerifyArgs a{batch,       num_nodes,  vocab,  parents,  tokens,     target_logits,
                   draft_logits, dtype,      temperature, uniforms, mode,  accept_len,
                   accepted_node, bonus_token, status, node_state, node_theta, p_init,
                   counters};
  a.target_max = target_max;
  a.target_sum = target_sum;
  a.draft_max = draft_max;
  a.draft_sum = draft_sum;
  const int st = tv::validate(a, workspace, workspace_bytes);
  if (st != TV_OK || batch == 0) return st;
  if (!target_max || !target_sum || !draft_max || !draft_sum) return TV_ERR_INVALID_ARG;
  if (reinterpret_cast<uintptr_t>(target_max) % 4 || reinterpret_cast<uintptr_t>(draft_max) % 4 ||
      reinterpret_cast<uintptr_t>(target_sum) % 8 || reinterpret_cast<uintptr_t>(draft_sum) % 8)
    return TV_ERR_INVALID_ARG;
  return tv::launch(a, tv::Algo::kTraversal, workspace, stream);
}

size_t tv_lmhead_workspace_size(int32_t rows, int32_t vocab) {
  if (rows < 1 || rows > TV_MAX_LMHEAD_ROWS || vocab < 2 || vocab > TV_MAX_VOCAB) return 0;
  return tv::lmhead_layout(rows, vocab).bytes;
}

int tv_lmhead_stats(int32_t rows, int32_t hidden_size, int32_t vocab, const void* hidden,
                    const void* weight, float temperature, void* logits, float* row_max,
                    double* row_sum, void* workspace, size_t workspace_bytes,
                    hipStream_t stream) {
  const tv::LmheadArgs a{rows, hidden_size, vocab, hidden, weight, temperature, logits, row_max,
                         row_sum};
  const int st = tv::validate_lmhead(a, workspace, workspace_bytes);
  if (st != TV_OK || rows == 0) return st;
  return tv::launch_lmhead(a, workspace, stream);
}

int tv_draft_tokens(int32_t batch, int32_t num_nodes, int32_t vocab, const int32_t* parents,
                    const void* draft_logits, int32_t dtype, float temperature,
                    const float* uniforms, int32_t mode, int32_t* tokens, int32_t* status,
                    hipStream_t stream) {
  const tv::SampleArgs a{batch, num_nodes, vocab, parents, draft_logits, dtype, temperature,
                         uniforms, mode, tokens, status};
  const int st = tv::validate_sample(a);
  if (st != TV_OK || batch == 0) return st;
  return tv::launch_sample(a, stream);
}

int tv_commit_paths(int32_t batch, int32_t num_nodes, const int32_t* parents,
                    const int32_t* tokens, const int32_t* accepted_node,
                    const int32_t* bonus_token, const int32_t* status, int32_t max_len,
                    int32_t* path_nodes, int32_t* path_tokens, int32_t* path_len,
                    hipStream_t stream) {
  if (batch < 0 || num_nodes < 1 || max_len < 0) return TV_ERR_INVALID_ARG;
  if (batch > TV_MAX_BATCH || num_nodes > TV_MAX_NODES || max_len > TV_MAX_NODES)
    return TV_ERR_UNSUPPORTED;
  if (batch == 0) return TV_OK;
  const void* ptrs[] = {parents, tokens, accepted_node, bonus_token, status, path_tokens,
                        path_len};
  for (const void* p : ptrs)
    if (!p || reinterpret_cast<uintptr_t>(p) % 4) return TV_ERR_INVALID_ARG;
  if ((max_len > 0 && !path_nodes) || reinterpret_cast<uintptr_t>(path_nodes) % 4)
    return TV_ERR_INVALID_ARG;
  const tv::CommitArgs a{batch, num_nodes, parents, tokens, accepted_node, bonus_token, status,
                         max_len, path_nodes, path_tokens, path_len};
  return tv::launch_commit(a, stream);
}

const char* tv_status_string(int code) {
  switch (code) {
    case TV_OK: return "ok";
    case TV_ERR_INVALID_ARG: return "invalid argument";
    case TV_ERR_UNSUPPORTED: return "unsupported size, temperature or pointer alignment";
    case TV_ERR_WORKSPACE: return "workspace missing, too small or misaligned";
    case TV_ERR_HIP: return "HIP kernel launch failed";
    default: return "unknown status";
  }
}

}  // extern "C"
