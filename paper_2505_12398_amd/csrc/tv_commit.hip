// Accepted-path commit (the step after verification): for every tree, the
// output of Def. def2 laid out for the next decoding cycle: the node indices
// of the accepted chain X^tau after the root, from the root down (the drafted
// positions whose cache entries are kept), and their tokens followed by Y.
#include <hip/hip_runtime.h>

#include "tv.h"
#include "tv_launch.h"

namespace {

// One thread per tree. The chain is found by walking from the accepted node
// to the root (each step to a smaller index, so at most num_nodes steps) and
// written in reverse; entries past it are -1.
__global__ void __launch_bounds__(256) commit_kernel(tv::CommitArgs a) {
  const int b = static_cast<int>(blockIdx.x * blockDim.x + threadIdx.x);
  if (b >= a.batch) return;
  const int n1 = a.num_nodes, L = a.max_len;
  const int32_t* par = a.parents + static_cast<size_t>(b) * n1;
  const int32_t* tok = a.tokens + static_cast<size_t>(b) * n1;
  int32_t* pn = a.path_nodes + static_cast<size_t>(b) * L;
  int32_t* pt = a.path_tokens + static_cast<size_t>(b) * (L + 1);
  for (int i = 0; i < L; ++i) pn[i] = -1;
  for (int i = 0; i <= L; ++i) pt[i] = -1;
  if (a.status[b] != TV_TREE_OK) {
    a.path_len[b] = 0;
    return;
  }
  const int acc = a.accepted_node[b];
  // depth of the accepted node; links must point backwards
  int depth = 0, bad = acc < 0 || acc >= n1;
  for (int x = acc; !bad && x > 0; ++depth) {
    const int p = par[x];
    if (p < 0 || p >= x) bad = 1;
    x = p;
  }
  if (bad) {
    a.path_len[b] = TV_COMMIT_INCONSISTENT;
    return;
  }
  if (depth > L) {
    a.path_len[b] = TV_COMMIT_OVERFLOW;
    return;
  }
  for (int x = acc, i = depth - 1; x > 0; --i) {
    pn[i] = x;
    pt[i] = tok[x];
    x = par[x];
  }
  pt[depth] = a.bonus_token[b];
  a.path_len[b] = depth + 1;
}

}  // namespace

namespace tv {

int launch_commit(const CommitArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(commit_kernel, dim3(static_cast<unsigned>((a.batch + 255) / 256)), dim3(256),
                     0, stream, a);
  return hipGetLastError() == hipSuccess ? TV_OK : TV_ERR_HIP;
}

}  // namespace tv
