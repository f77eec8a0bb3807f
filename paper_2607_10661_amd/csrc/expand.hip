// Progressive expansion of the draft tree with top-k children (Sec. 3.1
// "Progressive Expansion": V^t = V^{t-1} u {d_v}, E^t = E^{t-1} u {(v, d_v)};
// "Overhead Constraints": width control and a depth threshold; App. A: top-k
// candidates instead of the single greedy token).
//
// Rules (node v in index order, candidates topk_idx[v+1][0..k-1]):
//   - v of depth d grows only if d + 1 <= d_max and while its child count
//     (existing + added) is below width_sched[d];
//   - a candidate equal to the token of one of v's children, or to an earlier
//     candidate of v, is the same node and is skipped (merge by value, as in
//     Sec. 3.1 "Draft Extraction");
//   - the grown tree is renumbered breadth-first (depth, then the parent's new
//     index, then old children in index order before new children in candidate
//     order) and cut to the first T_max nodes.
//
// One workgroup per sequence.  New children are never stored: a node's list of
// added tokens is a pure function of its row, its existing children and the
// caps, so it is counted once and regenerated when the node's children are
// emitted.  Emission proceeds level by level with a block-wide exclusive scan
// of child counts over the current level.
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
  const int* s_clist;
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
    for (int j = 0; j < c.s_ncld[v] && !dup; ++j) dup = c.s_tok[c.s_clist[c.s_cstart[v] + j]] == cand;
    for (int r2 = 0; r2 < r && !dup; ++r2) dup = c.row[r2] == cand;
    if (dup) continue;
    emit(added, cand);
    ++added;
    ++have;
  }
  return added;
}

__global__ void __launch_bounds__(kThreads)
k_expand(const int32_t* __restrict__ parent, const int32_t* __restrict__ tokens,
         const int32_t* __restrict__ tree_len, int T, const int32_t* __restrict__ topk_idx,
         int k, WidthArg ws, int d_max, int T_max, int32_t* __restrict__ parent_next,
         int32_t* __restrict__ tokens_next, int32_t* __restrict__ tree_len_next,
         int32_t* dev_status) {
  __shared__ int s_par[PTD_MAX_T], s_tok[PTD_MAX_T], s_dep[PTD_MAX_T];
  __shared__ int s_ncld[PTD_MAX_T], s_cstart[PTD_MAX_T], s_clist[PTD_MAX_T];
  __shared__ int s_nnew[PTD_MAX_T], s_cnt[PTD_MAX_T];
  __shared__ int s_oid[PTD_MAX_T], s_opar[PTD_MAX_T], s_otok[PTD_MAX_T];
  __shared__ int s_part[kThreads / PTD_WAVE];
  __shared__ int s_width[PTD_MAX_DEPTH];
  __shared__ int s_topk[kTopkLds];

  const int b = blockIdx.x, tid = threadIdx.x;
  int n = T;
  if (tree_len) {
    n = tree_len[b];
    n = n < 0 ? 0 : (n > T ? T : n);
  }
  int32_t* pn = parent_next + static_cast<size_t>(b) * T_max;
  int32_t* tn = tokens_next + static_cast<size_t>(b) * T_max;

  for (int d = tid; d < PTD_MAX_DEPTH; d += kThreads) s_width[d] = ws.w[d];
  const int32_t* topk_b = topk_idx + static_cast<size_t>(b) * (T + 1) * k;
  const bool staged = (T + 1) * k <= kTopkLds;
  if (staged)
    for (int x = tid; x < (T + 1) * k; x += kThreads) s_topk[x] = topk_b[x];
  const int32_t* rows = staged ? s_topk : topk_b;
  int bad = 0;
  for (int i = tid; i < n; i += kThreads) {
    const int p = parent[static_cast<size_t>(b) * T + i];
    s_par[i] = p;
    s_tok[i] = tokens[static_cast<size_t>(b) * T + i];
    s_ncld[i] = 0;
    if (p < -1 || p >= i) bad = 1;
  }
  if (__syncthreads_or(bad)) {
    if (tid == 0) {
      ptd::report(dev_status, PTD_ERR_BAD_TREE);
      tree_len_next[b] = 0;
    }
    for (int t = tid; t < T_max; t += kThreads) pn[t] = tn[t] = -1;
    return;
  }
  // depth (walk; parent[i] < i bounds every walk) and existing child counts
  for (int i = tid; i < n; i += kThreads) {
    int d = 0;
    for (int a = i; a != -1; a = s_par[a]) ++d;
    s_dep[i] = d;
    if (s_par[i] >= 0) atomicAdd(&s_ncld[s_par[i]], 1);
  }
  __syncthreads();
  // children lists in index order: offsets by scan, slot by rank among siblings
  for (int i = tid; i < n; i += kThreads) s_cstart[i] = s_ncld[i];
  __syncthreads();
  block_exclusive_scan(s_cstart, n, s_part);
  for (int i = tid; i < n; i += kThreads) {
    const int p = s_par[i];
    if (p < 0) continue;
    int rank = 0;
    for (int j = p + 1; j < i; ++j) rank += s_par[j] == p;
    s_clist[s_cstart[p] + rank] = i;
  }
  __syncthreads();

  ExpandCtx ctx{s_tok, s_cstart, s_clist, s_ncld, s_dep, nullptr, k, d_max, s_width};
  for (int v = tid; v < n; v += kThreads) {
    ExpandCtx c = ctx;
    c.row = rows + (v + 1) * k;
    s_nnew[v] = grow(c, v, [](int, int) {});
  }
  // level 1: roots in index order
  for (int i = tid; i < n; i += kThreads) s_cnt[i] = s_par[i] < 0 ? 1 : 0;
  __syncthreads();
  const int nroots = block_exclusive_scan(s_cnt, n, s_part);
  for (int i = tid; i < n; i += kThreads)
    if (s_par[i] < 0 && s_cnt[i] < T_max) {
      s_oid[s_cnt[i]] = i;
      s_opar[s_cnt[i]] = -1;
      s_otok[s_cnt[i]] = s_tok[i];
    }
  __syncthreads();

  int lo = 0, hi = min(nroots, T_max);
  while (lo < hi && hi < T_max) {
    const int len = hi - lo;
    for (int e = tid; e < len; e += kThreads) {
      const int id = s_oid[lo + e];
      s_cnt[e] = id >= 0 ? s_ncld[id] + s_nnew[id] : 0;
    }
    __syncthreads();
    const int nchild = block_exclusive_scan(s_cnt, len, s_part);
    for (int e = tid; e < len; e += kThreads) {
      const int id = s_oid[lo + e];
      if (id < 0) continue;
      const int base = hi + s_cnt[e];
      const int nold = s_ncld[id];
      for (int j = 0; j < nold; ++j) {
        const int pos = base + j;
        if (pos >= T_max) break;
        const int c = s_clist[s_cstart[id] + j];
        s_oid[pos] = c;
        s_opar[pos] = lo + e;
        s_otok[pos] = s_tok[c];
      }
      ExpandCtx c = ctx;
      c.row = rows + (id + 1) * k;
      const int parent_pos = lo + e;
      grow(c, id, [&](int a, int tok) {
        const int pos = base + nold + a;
        if (pos < T_max) {
          s_oid[pos] = -1;  // new nodes are leaves in this step
          s_opar[pos] = parent_pos;
          s_otok[pos] = tok;
        }
      });
    }
    __syncthreads();
    lo = hi;
    hi = min(hi + nchild, T_max);
  }
  const int count = hi;
  for (int t = tid; t < T_max; t += kThreads) {
    pn[t] = t < count ? s_opar[t] : -1;
    tn[t] = t < count ? s_otok[t] : -1;
  }
  if (tid == 0) tree_len_next[b] = count;
}

}  // namespace

extern "C" int ptd_expand(const int32_t* parent, const int32_t* tokens,
                          const int32_t* tree_len, int32_t B, int32_t T,
                          const int32_t* topk_idx, int32_t k, const int32_t* width_sched,
                          int32_t d_max, int32_t T_max, int32_t* parent_next,
                          int32_t* tokens_next, int32_t* tree_len_next, int32_t* dev_status,
                          void* stream) {
  PTD_RETURN_IF(!parent || !tokens || !topk_idx || !width_sched || !parent_next ||
                    !tokens_next || !tree_len_next,
                PTD_ERR_NULL);
  PTD_RETURN_IF(B < 1 || T < 1 || T > PTD_MAX_T || k < 1 || k > PTD_MAX_K || d_max < 1 ||
                    d_max > PTD_MAX_DEPTH || T_max < 1 || T_max > PTD_MAX_T,
                PTD_ERR_SHAPE);
  WidthArg ws;
  for (int d = 0; d < PTD_MAX_DEPTH; ++d) ws.w[d] = d < d_max ? width_sched[d] : 0;
  hipLaunchKernelGGL(k_expand, dim3(B), dim3(kThreads), 0, static_cast<hipStream_t>(stream),
                     parent, tokens, tree_len, T, topk_idx, k, ws, d_max, T_max, parent_next,
                     tokens_next, tree_len_next, dev_status);
  return ptd_launch_status();
}
