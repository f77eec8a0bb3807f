// Ancestor-or-self bitmasks and depths of a packed draft tree.
//
// Sec. 3.1 "Tree Construction": a node sees itself and its ancestors,
// pi(v) = {v} u pi(P(v)), and its position comes from |pi(v)|.  Nodes are in
// topological order (parent[i] < i), so every walk up the parent chain visits
// strictly decreasing indices and ends in at most i+1 steps.
//
// One workgroup per sequence: the parent array is staged in LDS, then every
// thread walks the chains of its nodes there and assembles each row's 64-bit
// words from the highest word down, writing every word of the row once.
#include "ptd_common.hpp"
#include "ptd_internal.hpp"

namespace {

constexpr int kThreads = 256;

__global__ void __launch_bounds__(kThreads)
k_tree_mask(const int32_t* __restrict__ parent, const int32_t* __restrict__ tree_len,
            int T, int W, uint64_t* __restrict__ mask, int32_t* __restrict__ depth,
            int32_t* dev_status) {
  __shared__ int s_par[PTD_MAX_T];
  const int b = blockIdx.x;
  int n = T;
  if (tree_len) {
    n = tree_len[b];
    n = n < 0 ? 0 : (n > T ? T : n);
  }
  const int32_t* par = parent + static_cast<size_t>(b) * T;
  for (int i = threadIdx.x; i < n; i += kThreads) s_par[i] = par[i];
  __syncthreads();
  for (int i = threadIdx.x; i < T; i += kThreads) {
    uint64_t* row = mask + (static_cast<size_t>(b) * T + i) * W;
    if (i >= n) {
      for (int w = 0; w < W; ++w) row[w] = 0;
      if (depth) depth[static_cast<size_t>(b) * T + i] = 0;
      continue;
    }
    int cur = i >> 6;
    for (int w = cur + 1; w < W; ++w) row[w] = 0;
    uint64_t word = 0;
    int count = 0;
    int a = i;
    while (a != -1) {
      const int p = s_par[a];
      if (p < -1 || p >= a) {  // not topological: report and stop the walk
        ptd::report(dev_status, PTD_ERR_BAD_TREE);
        break;
      }
      const int wa = a >> 6;
      if (wa != cur) {
        row[cur] = word;
        for (int w = wa + 1; w < cur; ++w) row[w] = 0;
        cur = wa;
        word = 0;
      }
      word |= 1ull << (a & 63);
      ++count;
      a = p;
    }
    row[cur] = word;
    for (int w = 0; w < cur; ++w) row[w] = 0;
    if (depth) depth[static_cast<size_t>(b) * T + i] = count;
  }
}

}  // namespace

int ptd_launch_tree_mask(const int32_t* parent, const int32_t* tree_len, int B, int T,
                         uint64_t* mask, int32_t* depth, int32_t* dev_status,
                         hipStream_t stream) {
  const int W = ptd_cdiv(T, 64);
  hipLaunchKernelGGL(k_tree_mask, dim3(B), dim3(kThreads), 0, stream, parent, tree_len, T, W,
                     mask, depth, dev_status);
  return ptd_launch_status();
}

extern "C" int ptd_build_tree_mask(const int32_t* parent, const int32_t* tree_len,
                                   int32_t B, int32_t T, uint64_t* mask, int32_t* depth,
                                   int32_t* dev_status, void* stream) {
  PTD_RETURN_IF(!parent || !mask || !depth, PTD_ERR_NULL);
  PTD_RETURN_IF(B < 1 || T < 1 || T > PTD_MAX_T || B > 65535, PTD_ERR_SHAPE);
  return ptd_launch_tree_mask(parent, tree_len, B, T, mask, depth, dev_status,
                              static_cast<hipStream_t>(stream));
}
