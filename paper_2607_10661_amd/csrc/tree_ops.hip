// Tree bookkeeping of a Progressive Tree Drafting step on gfx950: greedy
// verification and progressive expansion, separately or fused in one launch.
//
// Verification (Sec. 3.2 "Candidate Verification"; Alg. 1 steps 5-6): edge
// (P(c), c) is eligible iff the verification token of P(c) -- the argmax of
// P(c)'s logits row -- equals the draft token of c.  A node is accepted when
// every edge on its root path is eligible; the longest accepted path (lowest
// terminal index on ties) is emitted with the terminal's verification token
// as the bonus token.  "All edges eligible" and the depth are computed
// together by pointer jumping: after r rounds each node holds the AND of
// eligibility and the node count of the first 2^r nodes of its root path.
//
// Expansion (Sec. 3.1 "Progressive Expansion": V^t = V^{t-1} u {d_v},
// E^t = E^{t-1} u {(v, d_v)}; "Overhead Constraints": width control and a
// depth threshold; App. A: top-k candidates instead of the single greedy
// token).  Node v (index order) offers topk_idx[v+1][0..k-1]:
//   - v of depth d grows only if d + 1 <= d_max and while its child count
//     (existing + added) is below width_sched[d];
//   - a candidate equal to the token of one of v's children, or to an earlier
//     candidate of v, is the same node and is skipped (merge by value, as in
//     Sec. 3.1 "Draft Extraction");
//   - the grown tree is renumbered breadth-first (depth, then the parent's new
//     index, then old children in index order before new children in candidate
//     order) and cut to the first T_max nodes.
// New children are never stored: a node's added tokens are a pure function of
// its row, its existing children and the caps, so they are counted once and
// regenerated when emitted.  Emission proceeds level by level with
// block-wide exclusive scans of child counts.
//
// One workgroup per sequence; the tree is staged in LDS once.
#include "ptd_async.hpp"
#include "ptd_common.hpp"

namespace {

constexpr int kThreads = 256;
constexpr int kTopkLds = 8192;  // top-k rows staged in LDS when (T+1)*k fits

struct WidthArg {
  int32_t w[PTD_MAX_DEPTH];
};

// Block-wide exclusive scan of vals[0..n) in place (n <= PTD_MAX_T); returns
// the total.  All threads must call it.
__device__ int block_exclusive_scan(int* vals, int n, int* s_part) {
  constexpr int PER = PTD_MAX_T / kThreads;
  const int tid = threadIdx.x;
  const int base = tid * PER;
  int local[PER];
  int sum = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int v = (base + j < n) ? vals[base + j] : 0;
    local[j] = sum;
    sum += v;
  }
  // inclusive scan of per-thread sums across the block
  const int lane = tid & 63, wave = tid >> 6;
  int x = sum;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, PTD_WAVE);
    if (lane >= o) x += y;
  }
  if (lane == 63) s_part[wave] = x;
  __syncthreads();
  int wave_off = 0, total = 0;
  for (int w = 0; w < kThreads / PTD_WAVE; ++w) {
    if (w < wave) wave_off += s_part[w];
    total += s_part[w];
  }
  const int excl = wave_off + x - sum;
#pragma unroll
  for (int j = 0; j < PER; ++j)
    if (base + j < n) vals[base + j] = excl + local[j];
  __syncthreads();
  return total;
}

struct ExpandCtx {
  const int* s_tok;
  const int* s_cstart;
  const int* s_ctok;  // tokens of each node's existing children, contiguous
  const int* s_ncld;
  const int* s_dep;
  const int32_t* row;  // topk_idx row of the node (k entries)
  int k, d_max;
  const int* width;  // width_sched in LDS
};

// Walk the candidates of node v; calls emit(position among added, token) for
// every added child and returns the number added.
template <typename F>
__device__ int grow(const ExpandCtx& c, int v, F&& emit) {
  const int d = c.s_dep[v];
  if (d + 1 > c.d_max) return 0;
  const int cap = c.width[d];
  int have = c.s_ncld[v];
  int added = 0;
  for (int r = 0; r < c.k; ++r) {
    if (have >= cap) break;
    const int cand = c.row[r];
    bool dup = false;
    const int cs = c.s_cstart[v], nc = c.s_ncld[v];
    for (int j = 0; j < nc && !dup; ++j) dup = c.s_ctok[cs + j] == cand;
    for (int r2 = 0; r2 < r && !dup; ++r2) dup = c.row[r2] == cand;
    if (dup) continue;
    emit(added, cand);
    ++added;
    ++have;
  }
  return added;
}

// Stage the live part of sequence b's tree in LDS; returns true (uniformly)
// if some parent[i] is outside [-1, i).
__device__ bool load_tree(const int32_t* __restrict__ parent, const int32_t* __restrict__ tokens,
                          int b, int T, int n, int* s_par, int* s_tok) {
  int bad = 0;
  for (int i = threadIdx.x; i < n; i += kThreads) {
    const int p = parent[static_cast<size_t>(b) * T + i];
    s_par[i] = p;
    s_tok[i] = tokens[static_cast<size_t>(b) * T + i];
    bad |= (p < -1 || p >= i);
  }
  return __syncthreads_or(bad) != 0;
}

__device__ int live_nodes(const int32_t* tree_len, int b, int T) {
  if (!tree_len) return T;
  const int n = tree_len[b];
  return n < 0 ? 0 : (n > T ? T : n);
}

struct VerifyLds {
  int acc[2][PTD_MAX_T], dep[2][PTD_MAX_T], jmp[2][PTD_MAX_T];
  int path[PTD_MAX_T];
  int red[kThreads / PTD_WAVE];
};

// s_am holds the sequence's T+1 verification tokens.
__device__ void verify_body(const int* s_par, const int* s_tok, const int* s_am, int n, int b,
                            int T, VerifyLds& L, int32_t* __restrict__ accept_len,
                            int32_t* __restrict__ accept_nodes, int32_t* __restrict__ out_tokens) {
  const int tid = threadIdx.x;
  for (int i = tid; i < n; i += kThreads) {
    const int p = s_par[i];
    L.acc[0][i] = (s_tok[i] == s_am[p + 1]) ? 1 : 0;  // eligibility of the edge into i
    L.dep[0][i] = 1;
    L.jmp[0][i] = p;
  }
  __syncthreads();
  // pointer jumping: combine the segment of i with the segment above it
  int cur = 0;
  for (int round = 0; round < 11; ++round) {
    int more = 0;
    for (int i = tid; i < n; i += kThreads) {
      const int j = L.jmp[cur][i];
      int acc = L.acc[cur][i], dep = L.dep[cur][i], jmp = j;
      if (j != -1) {
        acc &= L.acc[cur][j];
        dep += L.dep[cur][j];
        jmp = L.jmp[cur][j];
      }
      L.acc[cur ^ 1][i] = acc;
      L.dep[cur ^ 1][i] = dep;
      L.jmp[cur ^ 1][i] = jmp;
      more |= (jmp != -1);
    }
    cur ^= 1;
    if (!__syncthreads_or(more)) break;
  }
  // best accepted node: largest depth, then lowest index
  int best_key = -1;
  for (int i = tid; i < n; i += kThreads)
    if (L.acc[cur][i]) {
      const int key = L.dep[cur][i] * 2048 + (2047 - i);
      best_key = key > best_key ? key : best_key;
    }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const int other = __shfl_xor(best_key, o, PTD_WAVE);
    best_key = other > best_key ? other : best_key;
  }
  if ((tid & (PTD_WAVE - 1)) == 0) L.red[tid / PTD_WAVE] = best_key;
  __syncthreads();
  best_key = L.red[0];
  for (int w = 1; w < kThreads / PTD_WAVE; ++w) best_key = L.red[w] > best_key ? L.red[w] : best_key;

  const int k = best_key < 0 ? 0 : best_key / 2048;
  const int best = best_key < 0 ? -1 : 2047 - best_key % 2048;
  if (tid == 0) {
    int pos = k - 1;
    for (int c = best; c != -1 && pos >= 0; c = s_par[c]) L.path[pos--] = c;
    accept_len[b] = k;
  }
  __syncthreads();
  const int bonus = s_am[best + 1];  // row 0 (committed token) when nothing is accepted
  for (int t = tid; t <= T; t += kThreads) {
    int node = -1, tok = -1;
    if (t < k) {
      node = L.path[t];
      tok = s_tok[node];
    } else if (t == k) {
      tok = bonus;
    }
    if (t < T) accept_nodes[static_cast<size_t>(b) * T + t] = node;
    out_tokens[static_cast<size_t>(b) * (T + 1) + t] = tok;
  }
}

__device__ void verify_reject(int b, int T, int32_t* accept_len, int32_t* accept_nodes,
                              int32_t* out_tokens) {
  for (int i = threadIdx.x; i <= T; i += blockDim.x) {
    if (i < T) accept_nodes[static_cast<size_t>(b) * T + i] = -1;
    out_tokens[static_cast<size_t>(b) * (T + 1) + i] = -1;
  }
  if (threadIdx.x == 0) accept_len[b] = 0;
}

constexpr int kNewLds = 4096;  // new-child tokens stored when T*k fits

struct ExpandLds {
  int dep[PTD_MAX_T], ncld[PTD_MAX_T], cstart[PTD_MAX_T], clist[PTD_MAX_T], ctok[PTD_MAX_T];
  int newtok[kNewLds];
  int nnew[PTD_MAX_T], cnt[PTD_MAX_T];
  int oid[PTD_MAX_T], opar[PTD_MAX_T], otok[PTD_MAX_T];
  int part[kThreads / PTD_WAVE];
  int width[PTD_MAX_DEPTH];
  int topk[kTopkLds];
};

__device__ void expand_body(const int* s_par, const int* s_tok, int n, int b, int T,
                            const int32_t* __restrict__ topk_idx, int k, const WidthArg& ws,
                            int d_max, int T_max, ExpandLds& L,
                            int32_t* __restrict__ parent_next, int32_t* __restrict__ tokens_next,
                            int32_t* __restrict__ tree_len_next) {
  const int tid = threadIdx.x;
  int32_t* pn = parent_next + static_cast<size_t>(b) * T_max;
  int32_t* tn = tokens_next + static_cast<size_t>(b) * T_max;
  for (int d = tid; d < PTD_MAX_DEPTH; d += kThreads) L.width[d] = ws.w[d];
  const int32_t* topk_b = topk_idx + static_cast<size_t>(b) * (T + 1) * k;
  const bool staged = (T + 1) * k <= kTopkLds;
  if (staged)
    for (int x = tid; x < (T + 1) * k; x += kThreads) L.topk[x] = topk_b[x];
  const int32_t* rows = staged ? L.topk : topk_b;
  for (int i = tid; i < n; i += kThreads) L.ncld[i] = 0;
  __syncthreads();
  // depth (walk; parent[i] < i bounds every walk) and existing child counts
  for (int i = tid; i < n; i += kThreads) {
    int d = 0;
    for (int a = i; a != -1; a = s_par[a]) ++d;
    L.dep[i] = d;
    if (s_par[i] >= 0) atomicAdd(&L.ncld[s_par[i]], 1);
  }
  __syncthreads();
  // children lists in index order: offsets by scan, slot by rank among siblings
  for (int i = tid; i < n; i += kThreads) L.cstart[i] = L.ncld[i];
  __syncthreads();
  block_exclusive_scan(L.cstart, n, L.part);
  for (int i = tid; i < n; i += kThreads) {
    const int p = s_par[i];
    if (p < 0) continue;
    int rank = 0;
#pragma unroll 8
    for (int j = p + 1; j < i; ++j) rank += s_par[j] == p;
    L.clist[L.cstart[p] + rank] = i;
    L.ctok[L.cstart[p] + rank] = s_tok[i];
  }
  __syncthreads();

  ExpandCtx ctx{s_tok, L.cstart, L.ctok, L.ncld, L.dep, nullptr, k, d_max, L.width};
  const bool keep_new = n * k <= kNewLds;
  for (int v = tid; v < n; v += kThreads) {
    ExpandCtx c = ctx;
    c.row = rows + (v + 1) * k;
    int* dst = L.newtok + v * k;
    L.nnew[v] = grow(c, v, [&](int a, int tok) {
      if (keep_new) dst[a] = tok;
    });
  }
  // level 1: roots in index order
  for (int i = tid; i < n; i += kThreads) L.cnt[i] = s_par[i] < 0 ? 1 : 0;
  __syncthreads();
  const int nroots = block_exclusive_scan(L.cnt, n, L.part);
  for (int i = tid; i < n; i += kThreads)
    if (s_par[i] < 0 && L.cnt[i] < T_max) {
      L.oid[L.cnt[i]] = i;
      L.opar[L.cnt[i]] = -1;
      L.otok[L.cnt[i]] = s_tok[i];
    }
  __syncthreads();

  int lo = 0, hi = min(nroots, T_max);
  while (lo < hi && hi < T_max) {
    const int len = hi - lo;
    for (int e = tid; e < len; e += kThreads) {
      const int id = L.oid[lo + e];
      L.cnt[e] = id >= 0 ? L.ncld[id] + L.nnew[id] : 0;
    }
    __syncthreads();
    const int nchild = block_exclusive_scan(L.cnt, len, L.part);
    for (int e = tid; e < len; e += kThreads) {
      const int id = L.oid[lo + e];
      if (id < 0) continue;
      const int base = hi + L.cnt[e];
      const int nold = L.ncld[id];
      for (int j = 0; j < nold; ++j) {
        const int pos = base + j;
        if (pos >= T_max) break;
        const int c = L.clist[L.cstart[id] + j];
        L.oid[pos] = c;
        L.opar[pos] = lo + e;
        L.otok[pos] = s_tok[c];
      }
      const int parent_pos = lo + e;
      auto put = [&](int a, int tok) {
        const int pos = base + nold + a;
        if (pos < T_max) {
          L.oid[pos] = -1;  // new nodes are leaves in this step
          L.opar[pos] = parent_pos;
          L.otok[pos] = tok;
        }
      };
      if (keep_new) {
        for (int a = 0; a < L.nnew[id]; ++a) put(a, L.newtok[id * k + a]);
      } else {
        ExpandCtx c = ctx;
        c.row = rows + (id + 1) * k;
        grow(c, id, put);
      }
    }
    __syncthreads();
    lo = hi;
    hi = min(hi + nchild, T_max);
  }
  const int count = hi;
  for (int t = tid; t < T_max; t += kThreads) {
    pn[t] = t < count ? L.opar[t] : -1;
    tn[t] = t < count ? L.otok[t] : -1;
  }
  if (tid == 0) tree_len_next[b] = count;
}

__device__ void expand_reject(int b, int T_max, int32_t* parent_next, int32_t* tokens_next,
                              int32_t* tree_len_next) {
  for (int t = threadIdx.x; t < T_max; t += blockDim.x) {
    parent_next[static_cast<size_t>(b) * T_max + t] = -1;
    tokens_next[static_cast<size_t>(b) * T_max + t] = -1;
  }
  if (threadIdx.x == 0) tree_len_next[b] = 0;
}

__global__ void __launch_bounds__(kThreads)
k_verify(const int32_t* __restrict__ argmax, const int32_t* __restrict__ tokens,
         const int32_t* __restrict__ parent, const int32_t* __restrict__ tree_len, int T,
         int32_t* __restrict__ accept_len, int32_t* __restrict__ accept_nodes,
         int32_t* __restrict__ out_tokens, int32_t* dev_status) {
  __shared__ int s_par[PTD_MAX_T], s_tok[PTD_MAX_T], s_am[PTD_MAX_T + 1];
  __shared__ VerifyLds L;
  const int b = blockIdx.x;
  const int n = live_nodes(tree_len, b, T);
  for (int i = threadIdx.x; i <= T; i += kThreads) s_am[i] = argmax[static_cast<size_t>(b) * (T + 1) + i];
  if (load_tree(parent, tokens, b, T, n, s_par, s_tok)) {
    if (threadIdx.x == 0) ptd::report(dev_status, PTD_ERR_BAD_TREE);
    verify_reject(b, T, accept_len, accept_nodes, out_tokens);
    return;
  }
  verify_body(s_par, s_tok, s_am, n, b, T, L, accept_len, accept_nodes, out_tokens);
}

__global__ void __launch_bounds__(kThreads)
k_expand(const int32_t* __restrict__ parent, const int32_t* __restrict__ tokens,
         const int32_t* __restrict__ tree_len, int T, const int32_t* __restrict__ topk_idx,
         int k, WidthArg ws, int d_max, int T_max, int32_t* __restrict__ parent_next,
         int32_t* __restrict__ tokens_next, int32_t* __restrict__ tree_len_next,
         int32_t* dev_status) {
  __shared__ int s_par[PTD_MAX_T], s_tok[PTD_MAX_T];
  __shared__ ExpandLds L;
  const int b = blockIdx.x;
  const int n = live_nodes(tree_len, b, T);
  if (load_tree(parent, tokens, b, T, n, s_par, s_tok)) {
    if (threadIdx.x == 0) ptd::report(dev_status, PTD_ERR_BAD_TREE);
    expand_reject(b, T_max, parent_next, tokens_next, tree_len_next);
    return;
  }
  expand_body(s_par, s_tok, n, b, T, topk_idx, k, ws, d_max, T_max, L, parent_next,
              tokens_next, tree_len_next);
}

__global__ void __launch_bounds__(kThreads)
k_verify_expand(const int32_t* __restrict__ argmax, const int32_t* __restrict__ tokens,
                const int32_t* __restrict__ parent, const int32_t* __restrict__ tree_len, int T,
                const int32_t* __restrict__ topk_idx, int k, WidthArg ws, int d_max, int T_max,
                int32_t* __restrict__ accept_len, int32_t* __restrict__ accept_nodes,
                int32_t* __restrict__ out_tokens, int32_t* __restrict__ parent_next,
                int32_t* __restrict__ tokens_next, int32_t* __restrict__ tree_len_next,
                int32_t* dev_status) {
  __shared__ int s_par[PTD_MAX_T], s_tok[PTD_MAX_T], s_am[PTD_MAX_T + 1];
  __shared__ VerifyLds LV;
  __shared__ ExpandLds LE;
  const int b = blockIdx.x;
  const int n = live_nodes(tree_len, b, T);
  for (int i = threadIdx.x; i <= T; i += kThreads) s_am[i] = argmax[static_cast<size_t>(b) * (T + 1) + i];
  if (load_tree(parent, tokens, b, T, n, s_par, s_tok)) {
    if (threadIdx.x == 0) ptd::report(dev_status, PTD_ERR_BAD_TREE);
    verify_reject(b, T, accept_len, accept_nodes, out_tokens);
    expand_reject(b, T_max, parent_next, tokens_next, tree_len_next);
    return;
  }
  verify_body(s_par, s_tok, s_am, n, b, T, LV, accept_len, accept_nodes, out_tokens);
  expand_body(s_par, s_tok, n, b, T, topk_idx, k, ws, d_max, T_max, LE, parent_next,
              tokens_next, tree_len_next);
}

// ===========================================================================
// Trees of up to 64 * NPL nodes (NPL = 1, 2): one wave per sequence, node
// 64 x + lane in slot x of its lane, no workgroup barriers.  Same results as
// the workgroup kernels above.
//   - ancestor sets as NPL-word bit masks (word w: nodes 64 w .. 64 w + 63)
//     by pointer doubling over wave shuffles (anc = {i}, jump = parent;
//     anc |= anc[jump], jump = jump[jump] until every jump is -1);
//     depth = |anc|
//   - verification: a node is accepted iff anc contains no node whose edge is
//     ineligible (one ballot per word), the terminal is the wave maximum of
//     (depth, -index), and the path is the terminal's ancestor mask
//   - expansion: children masks by LDS atomic OR; a node's added candidates
//     as a bit set over its top-k row; breadth-first positions level by
//     level: the nodes of a level write their child counts at their
//     positions, a scan over the wave (DPP row shifts and broadcasts, one
//     per 64 positions) gives every node its first child's position, and
//     old children add their rank among their siblings to their parent's
// Wave reductions use DPP and the gfx950 lane swaps (VALU only); gathers
// from other lanes are the remaining LDS-latency steps.
// ===========================================================================
constexpr int kWaveNodes = 64;
constexpr int kWaveTree = 2 * kWaveNodes;  // trees (and cuts) the one-wave kernel takes

__device__ __forceinline__ uint64_t shfl64(uint64_t v, int src) {
  const uint32_t lo = __shfl(static_cast<uint32_t>(v), src, PTD_WAVE);
  const uint32_t hi = __shfl(static_cast<uint32_t>(v >> 32), src, PTD_WAVE);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Value of node j (0 <= j < 64 * NPL) from per-slot lane values v[x] (node
// 64 x + lane): lane j mod 64, slot j / 64.
template <int NPL, typename T>
__device__ __forceinline__ T gather_node(const T (&v)[NPL], int j) {
  T r = T{};
#pragma unroll
  for (int x = 0; x < NPL; ++x) {
    T t;
    if constexpr (sizeof(T) == 8) t = shfl64(v[x], j & 63);
    else t = __shfl(v[x], j & 63, PTD_WAVE);
    if ((j >> 6) == x) r = t;
  }
  return r;
}

// Maximum over the wave: within quads (quad permutes), half-rows and rows
// (mirrors), then across rows by v_permlane16_swap / v_permlane32_swap (with
// both operands holding the value, the two results are the lane's value and
// that of lane ^ 16, resp. lane ^ 32).
__device__ __forceinline__ int wave_max_i32(int x) {
  x = max(x, __builtin_amdgcn_update_dpp(x, x, 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
  x = max(x, __builtin_amdgcn_update_dpp(x, x, 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
  x = max(x, __builtin_amdgcn_update_dpp(x, x, 0x141, 0xF, 0xF, false));  // row_half_mirror
  x = max(x, __builtin_amdgcn_update_dpp(x, x, 0x140, 0xF, 0xF, false));  // row_mirror
  const auto r16 = __builtin_amdgcn_permlane16_swap(static_cast<uint32_t>(x), static_cast<uint32_t>(x), false, false);
  x = max(static_cast<int>(r16[0]), static_cast<int>(r16[1]));
  const auto r32 = __builtin_amdgcn_permlane32_swap(static_cast<uint32_t>(x), static_cast<uint32_t>(x), false, false);
  return max(static_cast<int>(r32[0]), static_cast<int>(r32[1]));
}

// Exclusive prefix sum over the lanes, and the total, on the vector ALU:
// an inclusive scan within each row of 16 lanes by row_shr 1, 2, 4, 8 (lanes
// shifted in from outside the row add 0), then the rows' totals carried by
// row_bcast:15 (lane 15 of a row into the next row: rows 1 and 3) and
// row_bcast:31 (lane 31 into rows 2 and 3).
__device__ __forceinline__ int wave_excl_scan(int c, int* total) {
  int x = c;
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, false);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, false);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, false);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, false);  // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false);  // row_bcast:15
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false);  // row_bcast:31
  *total = __builtin_amdgcn_readlane(x, 63);
  return x - c;
}

// Members of the NPL-word set m with a lower index than node 64 x + lane.
template <int NPL>
__device__ __forceinline__ int rank_below(const uint64_t (&m)[NPL], int x, uint64_t below) {
  int r = 0;
#pragma unroll
  for (int w = 0; w < NPL; ++w) r += w < x ? __popcll(m[w]) : w == x ? __popcll(m[w] & below) : 0;
  return r;
}

template <bool VERIFY, bool EXPAND, int KM, int NPL>
__global__ void __launch_bounds__(PTD_WAVE)
k_tree_wave(const int32_t* __restrict__ argmax, const int32_t* __restrict__ tokens,
            const int32_t* __restrict__ parent, const int32_t* __restrict__ tree_len, int T,
            const int32_t* __restrict__ topk_idx, int k, WidthArg ws, int d_max, int T_max,
            int32_t* __restrict__ accept_len, int32_t* __restrict__ accept_nodes,
            int32_t* __restrict__ out_tokens, int32_t* __restrict__ parent_next,
            int32_t* __restrict__ tokens_next, int32_t* __restrict__ tree_len_next,
            int32_t* dev_status) {
  constexpr int NN = NPL * kWaveNodes;  // nodes a wave holds
  static_assert(PTD_MAX_DEPTH == kWaveNodes, "one width entry per lane");
  __shared__ int s_cnt[NN];
  __shared__ uint64_t s_cm[NN][NPL];
  __shared__ uint32_t s_dup[NN];
  __shared__ int s_width[PTD_MAX_DEPTH];
  const int lane = threadIdx.x, b = blockIdx.x;
  const int n = live_nodes(tree_len, b, T);
  const uint64_t below = (1ull << lane) - 1ull;
  int node[NPL];
  bool live[NPL];
#pragma unroll
  for (int x = 0; x < NPL; ++x) {
    node[x] = x * kWaveNodes + lane;
    live[x] = node[x] < n;
  }

  // every global load first, none waiting for tree_len
  int par_in[NPL], tok_in[NPL];
#pragma unroll
  for (int x = 0; x < NPL; ++x) {
    par_in[x] = node[x] < T ? parent[static_cast<size_t>(b) * T + node[x]] : -1;
    tok_in[x] = node[x] < T ? tokens[static_cast<size_t>(b) * T + node[x]] : 0;
  }
  int am[NPL], am_last = 0;  // argmax rows 64 x + lane, and row NN
  if (VERIFY) {
    const int32_t* amb = argmax + static_cast<size_t>(b) * (T + 1);
#pragma unroll
    for (int x = 0; x < NPL; ++x) am[x] = node[x] <= T ? amb[node[x]] : 0;
    am_last = T >= NN ? amb[NN] : 0;
  }
  int cand[NPL][KM];
  if (EXPAND) {
#pragma unroll
    for (int x = 0; x < NPL; ++x) {
      const int32_t* row = topk_idx + (static_cast<size_t>(b) * (T + 1) + node[x] + 1) * k;
#pragma unroll
      for (int r = 0; r < KM; ++r) cand[x][r] = (node[x] < T && r < k) ? row[r] : 0;
    }
    s_width[lane] = ws.w[lane];
  }
  int par[NPL], tok[NPL];
  bool bad = false;
#pragma unroll
  for (int x = 0; x < NPL; ++x) {
    par[x] = live[x] ? par_in[x] : -1;
    tok[x] = live[x] ? tok_in[x] : 0;
    bad |= live[x] && (par[x] < -1 || par[x] >= node[x]);
#pragma unroll
    for (int w = 0; w < NPL; ++w) s_cm[node[x]][w] = 0ull;
    s_cnt[node[x]] = 0;
    s_dup[node[x]] = 0u;
  }

  if (__any(bad)) {  // not topological
    if (lane == 0) ptd::report(dev_status, PTD_ERR_BAD_TREE);
    if (VERIFY) verify_reject(b, T, accept_len, accept_nodes, out_tokens);
    if (EXPAND) expand_reject(b, T_max, parent_next, tokens_next, tree_len_next);
    return;
  }

  // ancestor masks and depths
  uint64_t anc[NPL][NPL];
  int jump[NPL], dep[NPL];
#pragma unroll
  for (int x = 0; x < NPL; ++x) {
#pragma unroll
    for (int w = 0; w < NPL; ++w) anc[x][w] = (live[x] && w == x) ? (1ull << lane) : 0ull;
    jump[x] = par[x];
  }
  for (;;) {
    bool any_jump = false;
#pragma unroll
    for (int x = 0; x < NPL; ++x) any_jump |= jump[x] >= 0;
    if (!__any(any_jump)) break;
    // gathers read the values before this round's updates
    uint64_t a2[NPL][NPL];
    int j2[NPL];
#pragma unroll
    for (int x = 0; x < NPL; ++x) {
      const int src = jump[x] >= 0 ? jump[x] : node[x];
#pragma unroll
      for (int w = 0; w < NPL; ++w) {
        uint64_t col[NPL];
#pragma unroll
        for (int y = 0; y < NPL; ++y) col[y] = anc[y][w];
        a2[x][w] = gather_node<NPL>(col, src);
      }
      j2[x] = gather_node<NPL>(jump, src);
    }
#pragma unroll
    for (int x = 0; x < NPL; ++x)
      if (jump[x] >= 0) {
#pragma unroll
        for (int w = 0; w < NPL; ++w) anc[x][w] |= a2[x][w];
        jump[x] = j2[x];
      }
  }
#pragma unroll
  for (int x = 0; x < NPL; ++x) {
    dep[x] = 0;
#pragma unroll
    for (int w = 0; w < NPL; ++w) dep[x] += __popcll(anc[x][w]);
  }

  if (VERIFY) {
    uint64_t elig[NPL];
#pragma unroll
    for (int x = 0; x < NPL; ++x) {
      const int pa = par[x] + 1;  // the parent's argmax row (0 for a root)
      // (the gather runs on every lane, outside the select)
      const int am_g = gather_node<NPL>(am, pa < NN ? pa : 0);
      const int am_par = pa < NN ? am_g : am_last;
      elig[x] = __ballot(live[x] && tok[x] == am_par);
    }
    int key = -1;
#pragma unroll
    for (int x = 0; x < NPL; ++x) {
      bool accepted = live[x];
#pragma unroll
      for (int w = 0; w < NPL; ++w) accepted &= (anc[x][w] & ~elig[w]) == 0ull;
      key = max(key, accepted ? dep[x] * 256 + (255 - node[x]) : -1);
    }
    key = wave_max_i32(key);
    const int klen = key < 0 ? 0 : key / 256;
    const int best = key < 0 ? -1 : 255 - key % 256;
    // best is uniform over the wave (a wave maximum): read its lane directly
    const int bl = __builtin_amdgcn_readfirstlane(best < 0 ? 0 : best & 63);
    const int bs = best < 0 ? 0 : best >> 6;
    uint64_t path[NPL];
#pragma unroll
    for (int w = 0; w < NPL; ++w) {
      path[w] = 0ull;
#pragma unroll
      for (int x = 0; x < NPL; ++x) {
        // (readlane returns int: widen through uint32_t, never sign-extend)
        const uint32_t phi = __builtin_amdgcn_readlane(static_cast<uint32_t>(anc[x][w] >> 32), bl);
        const uint32_t plo = __builtin_amdgcn_readlane(static_cast<uint32_t>(anc[x][w]), bl);
        const uint64_t pw = (static_cast<uint64_t>(phi) << 32) | plo;
        if (bs == x) path[w] = pw;
      }
    }
    const int bt = best + 1;  // the terminal's argmax row: the bonus token
    int bonus = am_last;
#pragma unroll
    for (int x = 0; x < NPL; ++x) {
      const int v = __builtin_amdgcn_readlane(am[x], __builtin_amdgcn_readfirstlane(bt & 63));
      if ((bt >> 6) == x) bonus = v;
    }
    int32_t* an = accept_nodes + static_cast<size_t>(b) * T;
    int32_t* ot = out_tokens + static_cast<size_t>(b) * (T + 1);
#pragma unroll
    for (int x = 0; x < NPL; ++x) {
      const bool on_path = best >= 0 && live[x] && ((path[x] >> lane) & 1ull);
      if (on_path) {
        an[dep[x] - 1] = node[x];
        ot[dep[x] - 1] = tok[x];
      }
      if (node[x] < T && node[x] >= klen) an[node[x]] = -1;
    }
    for (int t = lane; t <= T; t += PTD_WAVE) {
      if (t == klen) ot[t] = bonus;
      else if (t > klen) ot[t] = -1;
    }
    if (lane == 0) accept_len[b] = klen;
  }

  if (EXPAND) {
    // children masks, and each child marks the entries of its parent's top-k
    // row that repeat its own token (the parent's row gathered by shuffles)
#pragma unroll
    for (int x = 0; x < NPL; ++x) {
      uint32_t mydup = 0;
      const int psrc = par[x] >= 0 ? par[x] : node[x];
#pragma unroll
      for (int r = 0; r < KM; ++r) {
        int col[NPL];
#pragma unroll
        for (int y = 0; y < NPL; ++y) col[y] = cand[y][r];
        const int pc = gather_node<NPL>(col, psrc);
        mydup |= (pc == tok[x]) ? (1u << r) : 0u;
      }
      if (live[x] && par[x] >= 0) {
        atomicOr(reinterpret_cast<unsigned long long*>(&s_cm[par[x]][x]), 1ull << lane);
        atomicOr(&s_dup[par[x]], mydup);
      }
    }
    ptd::lds_barrier();  // LDS only: the global stores need no wait
    int ncld[NPL], nnew[NPL], srank[NPL];
    uint32_t sel[NPL];
#pragma unroll
    for (int x = 0; x < NPL; ++x) {
      ncld[x] = 0;
#pragma unroll
      for (int w = 0; w < NPL; ++w) ncld[x] += __popcll(s_cm[node[x]][w]);
      // candidates added under this node (bit r: topk row entry r)
      sel[x] = 0;
      if (live[x] && dep[x] + 1 <= d_max) {
        const int cap = s_width[dep[x]];
        const uint32_t dup = s_dup[node[x]];  // entries equal to an existing child's token
        int have = ncld[x];
#pragma unroll
        for (int r = 0; r < KM; ++r) {
          bool d = (dup >> r) & 1u;
#pragma unroll
          for (int r2 = 0; r2 < r; ++r2) d |= cand[x][r2] == cand[x][r];
          if (r < k && have < cap && !d) {
            sel[x] |= 1u << r;
            ++have;
          }
          if (have >= cap) break;
        }
      }
      nnew[x] = __popc(sel[x]);
      // an old child's rank among its siblings (children masks are complete)
      uint64_t sib[NPL];
#pragma unroll
      for (int w = 0; w < NPL; ++w) sib[w] = live[x] && par[x] >= 0 ? s_cm[par[x]][w] : 0ull;
      srank[x] = rank_below<NPL>(sib, x, below);
    }

    int32_t* pn = parent_next + static_cast<size_t>(b) * T_max;
    int32_t* tn = tokens_next + static_cast<size_t>(b) * T_max;
    uint64_t roots[NPL];
    int nroots = 0;
#pragma unroll
    for (int x = 0; x < NPL; ++x) {
      roots[x] = __ballot(live[x] && par[x] < 0);
      nroots += __popcll(roots[x]);
    }
    int pos[NPL];  // breadth-first position (-1: not placed, or cut at T_max)
#pragma unroll
    for (int x = 0; x < NPL; ++x) {
      pos[x] = -1;
      if (live[x] && par[x] < 0) {
        const int q = rank_below<NPL>(roots, x, below);
        if (q < T_max) {
          pos[x] = q;
          pn[q] = -1;
          tn[q] = tok[x];
        }
      }
    }
    int lo = 0, hi = min(nroots, T_max);
    for (int level = 1; lo < hi; ++level) {
      // positions [lo, hi) hold this level; slot x of lane p is position
      // lo + 64 x + p
      bool here[NPL];
#pragma unroll
      for (int x = 0; x < NPL; ++x) {
        here[x] = pos[x] >= 0 && dep[x] == level;
        if (here[x]) s_cnt[pos[x]] = ncld[x] + nnew[x];
      }
      ptd::lds_barrier();  // LDS only: the global stores need no wait
      int first[NPL], total = 0;
#pragma unroll
      for (int x = 0; x < NPL; ++x) {
        const int p = lo + x * kWaveNodes + lane;
        int t;
        first[x] = hi + total + wave_excl_scan(p < hi ? s_cnt[p] : 0, &t);
        total += t;
      }
      int pk[NPL];
#pragma unroll
      for (int x = 0; x < NPL; ++x) {
        const int start = gather_node<NPL>(first, here[x] ? pos[x] - lo : 0);  // valid where here
        if (here[x]) {  // added children: after the old ones, in candidate order
          int q = start + ncld[x];
#pragma unroll
          for (int r = 0; r < KM; ++r) {
            if ((sel[x] >> r) & 1u) {
              if (q < T_max) {
                pn[q] = pos[x];
                tn[q] = cand[x][r];
              }
              ++q;
            }
          }
        }
        // the node's first-child position and its own position packed for
        // one gather by its children (start < 2^16 and -1 <= pos < 2^15)
        pk[x] = (start & 0xFFFF) | ((pos[x] + 1) << 16);
      }
#pragma unroll
      for (int x = 0; x < NPL; ++x) {
        const int pkp = gather_node<NPL>(pk, par[x] >= 0 ? par[x] : node[x]);
        const int pstart = pkp & 0xFFFF;
        const int ppos = (pkp >> 16) - 1;
        if (live[x] && par[x] >= 0 && dep[x] == level + 1 && ppos >= 0) {  // the parent is on this level
          const int q = pstart + srank[x];
          if (q < T_max) {
            pos[x] = q;
            pn[q] = ppos;
            tn[q] = tok[x];
          }
        }
      }
      lo = hi;
      hi = min(hi + total, T_max);
    }
    for (int t = hi + lane; t < T_max; t += PTD_WAVE) {
      pn[t] = -1;
      tn[t] = -1;
    }
    if (lane == 0) tree_len_next[b] = hi;
  }
}

template <bool VERIFY, bool EXPAND>
void launch_wave(int B, int T, int T_max, int k, const int32_t* argmax, const int32_t* tokens,
                 const int32_t* parent, const int32_t* tree_len, const int32_t* topk_idx,
                 const WidthArg& ws, int d_max, int32_t* accept_len,
                 int32_t* accept_nodes, int32_t* out_tokens, int32_t* parent_next,
                 int32_t* tokens_next, int32_t* tree_len_next, int32_t* dev_status,
                 hipStream_t st) {
  const int npl = (T <= kWaveNodes && T_max <= kWaveNodes) ? 1 : 2;
#define PTD_WAVE_CASE(km, npl_)                                                                \
  hipLaunchKernelGGL((k_tree_wave<VERIFY, EXPAND, km, npl_>), dim3(B), dim3(PTD_WAVE), 0, st,  \
                     argmax, tokens, parent, tree_len, T, topk_idx, k, ws, d_max, T_max,        \
                     accept_len, accept_nodes, out_tokens, parent_next, tokens_next,            \
                     tree_len_next, dev_status)
#define PTD_WAVE_NPL(km) \
  if (npl == 1) PTD_WAVE_CASE(km, 1); else PTD_WAVE_CASE(km, 2);
  if (!EXPAND || k <= 4) { PTD_WAVE_NPL(4) }
  else if (k <= 8) { PTD_WAVE_NPL(8) }
  else { PTD_WAVE_NPL(16) }
#undef PTD_WAVE_NPL
#undef PTD_WAVE_CASE
}

bool expand_args_ok(int B, int T, int k, int d_max, int T_max) {
  return B >= 1 && T >= 1 && T <= PTD_MAX_T && k >= 1 && k <= PTD_MAX_K && d_max >= 1 &&
         d_max <= PTD_MAX_DEPTH && T_max >= 1 && T_max <= PTD_MAX_T;
}

WidthArg width_arg(const int32_t* width_sched, int d_max) {
  WidthArg ws;
  for (int d = 0; d < PTD_MAX_DEPTH; ++d) ws.w[d] = d < d_max ? width_sched[d] : 0;
  return ws;
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
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (T <= kWaveTree) {
    launch_wave<true, false>(B, T, 1, 1, argmax, draft_tokens, parent, tree_len, nullptr,
                             WidthArg{}, 1, accept_len, accept_nodes, out_tokens, nullptr,
                             nullptr, nullptr, dev_status, st);
  } else {
    hipLaunchKernelGGL(k_verify, dim3(B), dim3(kThreads), 0, st, argmax, draft_tokens, parent,
                       tree_len, T, accept_len, accept_nodes, out_tokens, dev_status);
  }
  return ptd_launch_status();
}

extern "C" int ptd_expand(const int32_t* parent, const int32_t* tokens,
                          const int32_t* tree_len, int32_t B, int32_t T,
                          const int32_t* topk_idx, int32_t k, const int32_t* width_sched,
                          int32_t d_max, int32_t T_max, int32_t* parent_next,
                          int32_t* tokens_next, int32_t* tree_len_next, int32_t* dev_status,
                          void* stream) {
  PTD_RETURN_IF(!parent || !tokens || !topk_idx || !width_sched || !parent_next ||
                    !tokens_next || !tree_len_next,
                PTD_ERR_NULL);
  PTD_RETURN_IF(!expand_args_ok(B, T, k, d_max, T_max), PTD_ERR_SHAPE);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (T <= kWaveTree && T_max <= kWaveTree) {
    launch_wave<false, true>(B, T, T_max, k, nullptr, tokens, parent, tree_len, topk_idx,
                             width_arg(width_sched, d_max), d_max, nullptr, nullptr,
                             nullptr, parent_next, tokens_next, tree_len_next, dev_status, st);
  } else {
    hipLaunchKernelGGL(k_expand, dim3(B), dim3(kThreads), 0, st, parent, tokens, tree_len, T,
                       topk_idx, k, width_arg(width_sched, d_max), d_max, T_max, parent_next,
                       tokens_next, tree_len_next, dev_status);
  }
  return ptd_launch_status();
}

extern "C" int ptd_verify_expand(const int32_t* argmax, const int32_t* draft_tokens,
                                 const int32_t* parent, const int32_t* tree_len, int32_t B,
                                 int32_t T, const int32_t* topk_idx, int32_t k,
                                 const int32_t* width_sched, int32_t d_max, int32_t T_max,
                                 int32_t* accept_len, int32_t* accept_nodes,
                                 int32_t* out_tokens, int32_t* parent_next,
                                 int32_t* tokens_next, int32_t* tree_len_next,
                                 int32_t* dev_status, void* stream) {
  PTD_RETURN_IF(!argmax || !draft_tokens || !parent || !topk_idx || !width_sched ||
                    !accept_len || !accept_nodes || !out_tokens || !parent_next ||
                    !tokens_next || !tree_len_next,
                PTD_ERR_NULL);
  PTD_RETURN_IF(!expand_args_ok(B, T, k, d_max, T_max), PTD_ERR_SHAPE);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (T <= kWaveTree && T_max <= kWaveTree) {
    launch_wave<true, true>(B, T, T_max, k, argmax, draft_tokens, parent, tree_len, topk_idx,
                            width_arg(width_sched, d_max), d_max, accept_len,
                            accept_nodes, out_tokens, parent_next, tokens_next, tree_len_next,
                            dev_status, st);
  } else {
    hipLaunchKernelGGL(k_verify_expand, dim3(B), dim3(kThreads), 0, st, argmax, draft_tokens,
                       parent, tree_len, T, topk_idx, k, width_arg(width_sched, d_max), d_max,
                       T_max, accept_len, accept_nodes, out_tokens, parent_next, tokens_next,
                       tree_len_next, dev_status);
  }
  return ptd_launch_status();
}
