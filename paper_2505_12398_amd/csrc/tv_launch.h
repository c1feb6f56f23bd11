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
  // Row statistics given by the caller (tv_verify_stats), [batch][num_nodes]
  // each, or all NULL: the maximum of the row and sum exp((z - max) / T).
  const float* target_max = nullptr;
  const double* target_sum = nullptr;
  const float* draft_max = nullptr;
  const double* draft_sum = nullptr;
};

constexpr int kMaxGrid = 4096;        // workgroups of one launch
constexpr int kMaxGroup = 64;         // workgroups that verify one tree together
constexpr int kMaxBatchPasses = 8;    // passes computed together for one tree
constexpr int kSegPartBytes = 32;     // one contributor's partial result of one pass
constexpr int kGroupDescBytes = 128;  // a group's batch descriptor and helper count

// Device workspace: a header (the abort flag), the contributors' partial
// results, double buffered by batch parity, and one descriptor block per
// group. Groups times contributors never exceed kMaxGrid, nor batch times
// kMaxGroup.
struct WorkspaceLayout {
  size_t off_parts;        // partials [group][parity][pass][contributor]
  size_t parts_bytes;
  size_t off_desc;         // per group: a batch descriptor for helpers and the helper count
  size_t desc_bytes;
  size_t bytes;
};

inline size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

inline WorkspaceLayout workspace_layout(int32_t batch, int32_t vocab) {
  (void)vocab;
  WorkspaceLayout L{};
  const int64_t wg = static_cast<int64_t>(batch) * kMaxGroup < kMaxGrid
                         ? static_cast<int64_t>(batch) * kMaxGroup : kMaxGrid;
  size_t off = 256;                                    // header
  L.off_parts = off;
  L.parts_bytes = static_cast<size_t>(kSegPartBytes) * 2 * kMaxBatchPasses * (wg < 1 ? 1 : wg);
  off = align256(off + L.parts_bytes);
  const int64_t groups = batch < kMaxGrid ? batch : kMaxGrid;
  L.off_desc = off;
  L.desc_bytes = static_cast<size_t>(kGroupDescBytes) * (groups < 1 ? 1 : groups);
  off = align256(off + L.desc_bytes);
  L.bytes = off;
  return L;
}

// Argument checks that need no GPU, without / with the caller's workspace.
// Return a tv_status_t.
int validate_args(const VerifyArgs& a);
int validate(const VerifyArgs& a, void* workspace, size_t workspace_bytes);

// Bytes of the library's own device scratch (tv_verify_noalloc): more than the
// largest workspace any valid size needs (workspace_layout(TV_MAX_BATCH, .)).
constexpr size_t kStaticScratchBytes = size_t{3} << 20;

// This device's copy of the library's device scratch, its address looked up
// once per device with that device current. Returns a tv_status_t.
int static_scratch(void** ptr, size_t* bytes);

// LM head with fused row statistics (tv_lmhead_stats).
struct LmheadArgs {
  int32_t rows;           // M
  int32_t hidden_size;    // K
  int32_t vocab;          // N
  const void* hidden;     // bf16 [M][K]
  const void* weight;     // bf16 [N][K]
  float temperature;
  void* logits;           // bf16 [M][N]
  float* row_max;         // [M]
  double* row_sum;        // [M]
};

constexpr int kLmheadTileN = 256;   // logits columns per workgroup

// Workspace of tv_lmhead_stats: one (max, sum) partial per row and column tile.
struct LmheadLayout {
  int tiles_n;
  size_t off_max, off_sum, bytes;
};
inline LmheadLayout lmhead_layout(int32_t rows, int32_t vocab) {
  LmheadLayout L{};
  L.tiles_n = (vocab + kLmheadTileN - 1) / kLmheadTileN;
  const size_t n = static_cast<size_t>(rows) * static_cast<size_t>(L.tiles_n) * sizeof(float);
  L.off_max = 0;
  L.off_sum = align256(n);
  L.bytes = align256(L.off_sum + n);
  return L;
}

// Argument checks of the LM head that need no GPU. Returns a tv_status_t.
int validate_lmhead(const LmheadArgs& a, void* workspace, size_t workspace_bytes);

// Enqueue the LM head and the merge of its row statistics (arguments validated).
int launch_lmhead(const LmheadArgs& a, void* workspace, hipStream_t stream);

struct SampleArgs {
  int32_t batch;
  int32_t num_nodes;
  int32_t vocab;
  const int32_t* parents;
  const void* draft;
  int32_t dtype;          // TV_DTYPE_*
  float temperature;
  const float* uniforms;
  int32_t mode;           // TV_SIBLINGS_*
  int32_t* tokens;
  int32_t* status;
};

struct CommitArgs {
  int32_t batch;
  int32_t num_nodes;
  const int32_t* parents;
  const int32_t* tokens;
  const int32_t* accepted_node;
  const int32_t* bonus_token;
  const int32_t* status;
  int32_t max_len;
  int32_t* path_nodes;
  int32_t* path_tokens;
  int32_t* path_len;
};

// Enqueue the accepted-path commit on `stream` (arguments validated).
int launch_commit(const CommitArgs& a, hipStream_t stream);

// Argument checks of the sampler that need no GPU. Returns a tv_status_t.
int validate_sample(const SampleArgs& a);

// Enqueue the draft-tree token sampler on `stream` (arguments validated).
int launch_sample(const SampleArgs& a, hipStream_t stream);

// Enqueue the verification on `stream` (an initialisation kernel, then the
// cooperative verifier). Arguments already validated. Returns a tv_status_t.
int launch(const VerifyArgs& a, Algo algo, void* workspace, hipStream_t stream);

}  // namespace tv
