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

// A vocabulary pass over a node's rows is cut into segments of kSegVec 16-byte
// vectors; a segment is the unit of work any workgroup can claim, and the
// per-segment partial results are combined in segment order.
constexpr int kSegVec = 2048;
constexpr int kMaxSeg = 64;           // 2^20 bf16 or 2^19 fp32 logits: 131072 vectors
constexpr int kMaxGrid = 4096;        // workgroups of one launch (each may own one tree at a time)
constexpr int kSegPartBytes = 32;
constexpr int kMaxBatchPasses = 8;    // passes published together by one owner

// Segments per row: an upper bound over both dtypes and every alignment.
inline int max_segments(int32_t vocab) {
  const int64_t vec = (static_cast<int64_t>(vocab) + 3) / 4;       // fp32: 4 per vector
  int64_t s = (vec + kSegVec - 1) / kSegVec;
  if (s < 1) s = 1;
  return static_cast<int>(s > kMaxSeg ? kMaxSeg : s);
}

// Device workspace: a header with the launch-wide counters (trees left, abort
// flag, next tree to claim; each on its own 256-byte line), then per workgroup
// slot the work word, the completed-segment counter, the pass parameters and
// the per-segment partial results. All offsets are multiples of 256 bytes.
struct WorkspaceLayout {
  int32_t slots;           // workgroup slots: min(kMaxGrid, batch * segments)
  int32_t seg_stride;      // segments reserved per pass
  size_t off_words;        // uint64_t[slots]  work word (the pass the slot's tree offers)
  size_t off_done;         // uint32_t[slots]  segments of the slot's passes completed
  size_t off_desc;         // uint64_t[slots][8] batch descriptor
  size_t off_parts;        // slots * kMaxBatchPasses * seg_stride partial results
  size_t bytes;
};

inline size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

inline WorkspaceLayout workspace_layout(int32_t batch, int32_t vocab) {
  WorkspaceLayout L{};
  L.seg_stride = max_segments(vocab);
  const int64_t want = static_cast<int64_t>(batch) * L.seg_stride;
  L.slots = static_cast<int32_t>(want < kMaxGrid ? (want < 1 ? 1 : want) : kMaxGrid);
  size_t off = 1024;                                   // header
  L.off_words = off;
  off = align256(off + sizeof(uint64_t) * L.slots);
  L.off_done = off;
  off = align256(off + sizeof(uint32_t) * L.slots);
  L.off_desc = off;
  off = align256(off + 8 * sizeof(uint64_t) * L.slots);
  L.off_parts = off;
  off = align256(off + static_cast<size_t>(kSegPartBytes) * kMaxBatchPasses * L.seg_stride *
                           L.slots);
  L.bytes = off;
  return L;
}

// Argument checks that need no GPU. Returns a tv_status_t.
int validate(const VerifyArgs& a, void* workspace, size_t workspace_bytes);

// Enqueue the verification on `stream` (an initialisation kernel, then the
// verifier). Arguments already validated. Returns a tv_status_t.
int launch(const VerifyArgs& a, Algo algo, void* workspace, hipStream_t stream);

}  // namespace tv
