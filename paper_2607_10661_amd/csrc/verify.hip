// Greedy verification of a packed token tree (Sec. 3.2 "Candidate
// Verification"; Alg. 1 steps 5-6).
//
// Edge (P(c), c) is eligible iff the verification token of P(c) -- the argmax
// of P(c)'s logits row -- equals the draft token of c.  A node is accepted when
// every edge on its root path is eligible; the longest accepted path (lowest
// terminal index on ties) is emitted with the terminal's verification token as
// the bonus token.
//
// One workgroup per sequence.  "All edges on the root path eligible" and the
// depth are computed together by pointer jumping over the parent array:
// after r rounds each node holds the AND of eligibility and the node count of
// the first 2^r nodes of its root path, so ceil(log2 T) rounds suffice.
#include "ptd_common.hpp"

namespace {

constexpr int kThreads = 256;
constexpr int kPer = PTD_MAX_T / kThreads;  // nodes per thread

__global__ void __launch_bounds__(kThreads)
k_verify(const int32_t* __restrict__ argmax, const int32_t* __restrict__ tokens,
         const int32_t* __restrict__ parent, const int32_t* __restrict__ tree_len,
         int T, int32_t* __restrict__ accept_len, int32_t* __restrict__ accept_nodes,
         int32_t* __restrict__ out_tokens, int32_t* dev_status) {
  __shared__ int s_par[PTD_MAX_T];
  __shared__ int s_tok[PTD_MAX_T];
  __shared__ int s_acc[2][PTD_MAX_T];
  __shared__ int s_dep[2][PTD_MAX_T];
  __shared__ int s_jmp[2][PTD_MAX_T];
  __shared__ int s_path[PTD_MAX_T];
  __shared__ int s_am[PTD_MAX_T + 1];
  __shared__ int s_red[kThreads / PTD_WAVE];

  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  int n = T;
  if (tree_len) {
    n = tree_len[b];
    n = n < 0 ? 0 : (n > T ? T : n);
  }
  const int32_t* am = argmax + static_cast<size_t>(b) * (T + 1);

  // stage the tree and the verification tokens (independent loads)
  int bad = 0;
  for (int i = tid; i <= T; i += kThreads) s_am[i] = am[i];
  for (int i = tid; i < n; i += kThreads) {
    const int p = parent[static_cast<size_t>(b) * T + i];
    s_par[i] = p;
    s_tok[i] = tokens[static_cast<size_t>(b) * T + i];
    bad |= (p < -1 || p >= i);
  }
  if (__syncthreads_or(bad)) {
    if (tid == 0) ptd::report(dev_status, PTD_ERR_BAD_TREE);
    for (int i = tid; i <= T; i += kThreads) {
      if (i < T) accept_nodes[static_cast<size_t>(b) * T + i] = -1;
      out_tokens[static_cast<size_t>(b) * (T + 1) + i] = -1;
    }
    if (tid == 0) accept_len[b] = 0;
    return;
  }

  for (int i = tid; i < n; i += kThreads) {
    const int p = s_par[i];
    s_acc[0][i] = (s_tok[i] == s_am[p + 1]) ? 1 : 0;  // eligibility of the edge into i
    s_dep[0][i] = 1;
    s_jmp[0][i] = p;
  }
  __syncthreads();

  // pointer jumping: combine the segment of i with the segment above it
  int cur = 0;
  for (int round = 0; round < 11; ++round) {
    int more = 0;
    for (int i = tid; i < n; i += kThreads) {
      const int j = s_jmp[cur][i];
      int acc = s_acc[cur][i], dep = s_dep[cur][i], jmp = j;
      if (j != -1) {
        acc &= s_acc[cur][j];
        dep += s_dep[cur][j];
        jmp = s_jmp[cur][j];
      }
      s_acc[cur ^ 1][i] = acc;
      s_dep[cur ^ 1][i] = dep;
      s_jmp[cur ^ 1][i] = jmp;
      more |= (jmp != -1);
    }
    cur ^= 1;
    if (!__syncthreads_or(more)) break;
  }

  // best accepted node: largest depth, then lowest index
  int best_key = -1;
  for (int i = tid; i < n; i += kThreads)
    if (s_acc[cur][i]) {
      const int key = s_dep[cur][i] * 2048 + (2047 - i);
      best_key = key > best_key ? key : best_key;
    }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const int other = __shfl_xor(best_key, o, PTD_WAVE);
    best_key = other > best_key ? other : best_key;
  }
  if ((tid & (PTD_WAVE - 1)) == 0) s_red[tid / PTD_WAVE] = best_key;
  __syncthreads();
  best_key = s_red[0];
  for (int w = 1; w < kThreads / PTD_WAVE; ++w) best_key = s_red[w] > best_key ? s_red[w] : best_key;

  const int k = best_key < 0 ? 0 : best_key / 2048;
  const int best = best_key < 0 ? -1 : 2047 - best_key % 2048;
  if (tid == 0) {
    int pos = k - 1;
    for (int c = best; c != -1 && pos >= 0; c = s_par[c]) s_path[pos--] = c;
    accept_len[b] = k;
  }
  __syncthreads();
  const int bonus = s_am[best + 1];  // row 0 (committed token) when nothing is accepted
  for (int t = tid; t <= T; t += kThreads) {
    int node = -1, tok = -1;
    if (t < k) {
      node = s_path[t];
      tok = s_tok[node];
    } else if (t == k) {
      tok = bonus;
    }
    if (t < T) accept_nodes[static_cast<size_t>(b) * T + t] = node;
    out_tokens[static_cast<size_t>(b) * (T + 1) + t] = tok;
  }
}

}  // namespace

extern "C" int ptd_verify(const int32_t* argmax, const int32_t* draft_tokens,
                          const int32_t* parent, const int32_t* tree_len, int32_t B,
                          int32_t T, int32_t* accept_len, int32_t* accept_nodes,
                          int32_t* out_tokens, int32_t* dev_status, void* stream) {
  PTD_RETURN_IF(!argmax || !draft_tokens || !parent || !accept_len || !accept_nodes ||
                    !out_tokens,
                PTD_ERR_NULL);
  PTD_RETURN_IF(B < 1 || T < 1 || T > PTD_MAX_T, PTD_ERR_SHAPE);
  static_assert(PTD_MAX_T <= 2048, "index packing in the best-node key");
  static_assert(kPer * kThreads == PTD_MAX_T, "node split");
  hipLaunchKernelGGL(k_verify, dim3(B), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), argmax, draft_tokens, parent,
                     tree_len, T, accept_len, accept_nodes, out_tokens, dev_status);
  return ptd_launch_status();
}
