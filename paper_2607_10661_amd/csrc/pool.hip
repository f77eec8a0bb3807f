// Depth control of the draft forest and the value-keyed candidate pool.
//
// Sec. 3.1 "Overhead Constraints" (Stepping Mechanism) and Alg. 1 step 3:
// when a sub-tree is deeper than d_max, its earliest-added (lowest-index)
// child's sub-tree replaces it and the other branches are pruned, repeatedly,
// so a chain keeps its last d_max nodes.  Sec. 3.1 "Draft Extraction via
// Merging" and Alg. 1 steps 1 and 4: every sub-tree of the draft is merged by
// M into the pool tree keyed by its root's token; the candidate tree of the
// next step is the pool tree keyed by the last committed token.
//
// Draft trees have at most 128 nodes and pool trees at most 129 (their root
// included), one node per thread:
//   k_step_prune     one workgroup of 64 or 128 threads per sequence:
//                    ancestor masks by pointer jumping through LDS, sub-tree
//                    depths, the new root of every sub-tree along its chain
//                    of lowest-index children, and breadth-first renumbering
//                    of the kept forest level by level (ranks counted over
//                    the level's mask).
//   k_pool_merge     one workgroup per sequence.  The sequence's hash table
//                    (token -> tree) is staged in LDS; every draft node's
//                    token is looked up, the missing tokens get new trees in
//                    index order of their first occurrence (while there is
//                    room) and are inserted.  The touched trees are staged in
//                    LDS with sibling links, up to 64 at a time; thread j
//                    merges every sub-tree whose root token keys staged tree
//                    j, the sub-tree's nodes in index order (the trees are
//                    independent and proceed together).  The appended nodes,
//                    the trees' node counts, the new slots and the tree count
//                    are written back (a merge never changes a stored node).
//   k_pool_retrieve  one workgroup of 192 threads per sequence: 64 hash slots
//                    from the token's home slot in one load, the tree's nodes
//                    one per thread, breadth-first order by levels.
//
// Pool layout per sequence (ptd_pool_bytes): int32 ntrees, padded to 16
// bytes; int32 slot_key[H]; int32 slot_tree[H] (-1 empty); int32 count[e_max];
// int2 node[e_max][n_cap] = (token, parent index in the tree; -1 at the root,
// which is node 0).  H is the power of two >= 2 e_max (at least 64).  Nodes
// of a tree are stored in insertion order, so a parent precedes its children.
#include "ptd_common.hpp"

namespace {

constexpr int kMaxNodes = 128;            // draft nodes per sequence
constexpr int kMaxCap = kMaxNodes + 1;    // pool tree capacity, root included
constexpr int kMaxTrees = 2048;           // pool trees per sequence
constexpr int kMaxSlots = 4096;
constexpr int kMergeThreads = 256;
constexpr int kStageTrees = 64;           // pool trees staged in LDS at a time
constexpr int kStageSlots = kStageTrees * kMaxCap;
constexpr int kRetrieveThreads = 192;     // >= kMaxCap, whole waves
constexpr int kRW = kRetrieveThreads / PTD_WAVE;

struct PoolGeom {
  int e_max, n_cap, H, hbits;
  size_t seq_bytes, off_key, off_tree, off_count, off_node;
};

inline bool pool_geom(int e_max, int n_cap, PoolGeom* g) {
  if (e_max < 1 || e_max > kMaxTrees || n_cap < 1 || n_cap > kMaxCap) return false;
  int H = 64, hb = 6;
  while (H < 2 * e_max) {
    H <<= 1;
    ++hb;
  }
  g->e_max = e_max;
  g->n_cap = n_cap;
  g->H = H;
  g->hbits = hb;
  g->off_key = 16;
  g->off_tree = g->off_key + 4 * static_cast<size_t>(H);
  g->off_count = g->off_tree + 4 * static_cast<size_t>(H);
  g->off_node = (g->off_count + 4 * static_cast<size_t>(e_max) + 15) & ~static_cast<size_t>(15);
  g->seq_bytes = (g->off_node + 8 * static_cast<size_t>(e_max) * n_cap + 255) & ~static_cast<size_t>(255);
  return true;
}

struct PoolView {
  int32_t* ntrees;
  int32_t* key;
  int32_t* tree;
  int32_t* count;
  int2* node;
};
__device__ __forceinline__ PoolView view(void* pool, const PoolGeom& g, int b) {
  char* base = static_cast<char*>(pool) + static_cast<size_t>(b) * g.seq_bytes;
  return PoolView{reinterpret_cast<int32_t*>(base), reinterpret_cast<int32_t*>(base + g.off_key),
                  reinterpret_cast<int32_t*>(base + g.off_tree),
                  reinterpret_cast<int32_t*>(base + g.off_count),
                  reinterpret_cast<int2*>(base + g.off_node)};
}

__device__ __forceinline__ int home_slot(int token, int hbits) {
  return static_cast<int>((static_cast<uint32_t>(token) * 0x9E3779B1u) >> (32 - hbits));
}

__device__ __forceinline__ uint64_t below_mask(int lane) { return (1ull << lane) - 1ull; }

// Rank of node v among the nodes of a level mask (NW words over nodes
// 0 .. 64*NW-1) ordered by (key, index); keys read from s_key.
template <int NW>
__device__ __forceinline__ int level_rank(const uint64_t* s_lvl, const int* s_key, int v, int key) {
  int rank = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w)
    for (uint64_t m = s_lvl[w]; m;) {  // eight members at a time, their keys read together
      int u[8], ku[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        u[q] = m ? 64 * w + __builtin_ctzll(m) : -1;
        m &= m - 1ull;
      }
#pragma unroll
      for (int q = 0; q < 8; ++q) ku[q] = u[q] >= 0 ? s_key[u[q]] : 0;
#pragma unroll
      for (int q = 0; q < 8; ++q)
        if (u[q] >= 0 && (ku[q] < key || (ku[q] == key && u[q] < v))) ++rank;
    }
  return rank;
}

template <int NW>
__device__ __forceinline__ int mask_count(const uint64_t* s_m) {
  int c = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) c += __popcll(s_m[w]);
  return c;
}

// ---------------------------------------------------------------------------
// stepping (NW = 1: trees of up to 64 nodes, 2: up to 128)
// ---------------------------------------------------------------------------
template <int NW>
__global__ void __launch_bounds__(PTD_WAVE * NW)
k_step_prune(const int32_t* __restrict__ parent, const int32_t* __restrict__ tokens,
             const int32_t* __restrict__ tree_len, int T, int d_max, int T_max,
             int32_t* __restrict__ parent_next, int32_t* __restrict__ tokens_next,
             int32_t* __restrict__ tree_len_next, int32_t* dev_status) {
  constexpr int N = PTD_WAVE * NW;
  __shared__ uint64_t s_anc[N][NW];
  __shared__ uint64_t s_U[N + 1][NW];
  __shared__ uint64_t s_cm[N][NW];
  __shared__ int s_jump[N], s_h[N], s_fc[N], s_rootof[N], s_out[N], s_key[N];
  __shared__ uint64_t s_nr[NW], s_keep[NW], s_lvl[NW];
  const int v = threadIdx.x, lane = v & 63, wv = v >> 6, b = blockIdx.x;
  int n = T;
  if (tree_len) {
    n = tree_len[b];
    n = n < 0 ? 0 : (n > T ? T : n);
  }
  int32_t* pn = parent_next + static_cast<size_t>(b) * T_max;
  int32_t* tn = tokens_next + static_cast<size_t>(b) * T_max;
  const bool live = v < n;
  const int par = live ? parent[static_cast<size_t>(b) * T + v] : -1;
  const int tok = live ? tokens[static_cast<size_t>(b) * T + v] : -1;
  if (__syncthreads_or(live && (par < -1 || par >= v))) {
    if (v == 0) {
      ptd::report(dev_status, PTD_ERR_BAD_TREE);
      tree_len_next[b] = 0;
    }
    for (int t = v; t < T_max; t += N) {
      pn[t] = -1;
      tn[t] = -1;
    }
    return;
  }
  // ancestor-or-self masks by pointer jumping
  uint64_t anc[NW];
#pragma unroll
  for (int w = 0; w < NW; ++w) anc[w] = (live && w == wv) ? (1ull << lane) : 0ull;
  int jump = par;
  for (;;) {
#pragma unroll
    for (int w = 0; w < NW; ++w) s_anc[v][w] = anc[w];
    s_jump[v] = jump;
    if (!__syncthreads_or(jump >= 0)) break;
    if (jump >= 0) {
#pragma unroll
      for (int w = 0; w < NW; ++w) anc[w] |= s_anc[jump][w];
      jump = s_jump[jump];
    }
    __syncthreads();
  }
  int dep = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) dep += __popcll(anc[w]);
  // depth of the sub-tree under each node: max over its descendants x of
  // dep(x) - dep(v) + 1.  U[d], the union of the ancestor-or-self sets of the
  // nodes at depth d, holds exactly the nodes with a descendant at depth d;
  // v's descendants fill every level from dep(v) down to its deepest one,
  // so h(v) counts the consecutive levels d >= dep(v) with v in U[d].
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    s_U[v][w] = 0ull;
    s_cm[v][w] = 0ull;
    if (v == 0) {
      s_U[N][w] = 0ull;
      s_nr[w] = 0ull;
    }
  }
  __syncthreads();
  if (live) {
#pragma unroll
    for (int w = 0; w < NW; ++w)
      if (anc[w]) atomicOr(&s_U[dep][w], static_cast<unsigned long long>(anc[w]));
    if (par >= 0) atomicOr(&s_cm[par][wv], 1ull << lane);
  }
  __syncthreads();
  int h = 0;
  if (live) {
    int d = dep;  // v itself is in U[dep]; levels examined eight at a time
    for (bool more = true; more;) {
      bool in[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) in[q] = d + 1 + q <= N && ((s_U[min(d + 1 + q, N)][wv] >> lane) & 1ull);
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        more &= in[q];
        d += more ? 1 : 0;
      }
    }
    h = d - dep + 1;
  }
  s_h[v] = h;
  int fc = -1;
#pragma unroll
  for (int w = NW - 1; w >= 0; --w)
    if (s_cm[v][w]) fc = 64 * w + __builtin_ctzll(s_cm[v][w]);
  s_fc[v] = fc;
  __syncthreads();
  // every old root steps down its lowest-index children while too deep
  if (live && par < 0) {
    int x = v;
    while (s_h[x] > d_max) x = s_fc[x];
    s_rootof[x] = v;
    atomicOr(&s_nr[x >> 6], 1ull << (x & 63));
  }
  __syncthreads();
  bool keep = false;
#pragma unroll
  for (int w = 0; w < NW; ++w) keep |= live && (anc[w] & s_nr[w]) != 0ull;
  const uint64_t kb = __ballot(keep);
  if (lane == 0) s_keep[wv] = kb;
  __syncthreads();
  int nd = 0;  // depth in the kept forest
#pragma unroll
  for (int w = 0; w < NW; ++w) nd += __popcll(anc[w] & s_keep[w]);
  const int kept = mask_count<NW>(s_keep);
  const bool is_root = keep && nd == 1;
  // breadth-first numbering: level 1 by the old root they replace, deeper
  // levels by (parent's number, old index)
  int outid = -1, ppid = -1, base = 0;
  for (int L = 1; base < kept && L <= N; ++L) {  // uniform
    const bool here = keep && nd == L;
    __syncthreads();  // numbers of level L - 1 written; s_lvl, s_key free
    const uint64_t lb = __ballot(here);
    if (lane == 0) s_lvl[wv] = lb;
    int key = 0;
    if (here) key = L == 1 ? s_rootof[v] : s_out[par];
    s_key[v] = key;
    __syncthreads();
    if (here) {
      outid = base + level_rank<NW>(s_lvl, s_key, v, key);
      ppid = L == 1 ? -1 : key;
      s_out[v] = outid;
    }
    base += mask_count<NW>(s_lvl);
  }
  for (int t = v; t < T_max; t += N) {
    pn[t] = -1;
    tn[t] = -1;
  }
  __syncthreads();
  if (keep && outid < T_max) {
    pn[outid] = is_root ? -1 : ppid;
    tn[outid] = tok;
  }
  if (v == 0) tree_len_next[b] = min(kept, T_max);
}

// ---------------------------------------------------------------------------
// pool
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(kMergeThreads) k_pool_init(void* pool, PoolGeom g) {
  const int b = blockIdx.x;
  PoolView P = view(pool, g, b);
  for (int i = threadIdx.x; i < g.H; i += kMergeThreads) {
    P.key[i] = 0;
    P.tree[i] = -1;
  }
  if (threadIdx.x == 0) *P.ntrees = 0;
}

struct MergeLds {
  alignas(16) int key[kMaxSlots];
  alignas(16) int tree[kMaxSlots];
  // draft nodes
  int par[kMaxNodes];
  alignas(16) int tok[kMaxNodes];
  int firstof[kMaxNodes];  // first node in index order with the same token
  int newid[kMaxNodes];    // tree id given to a missing token's first node
  int jof[kMaxNodes];      // index among the touched trees (first nodes)
  int jump[kMaxNodes];
  int newslot[kMaxNodes];
  uint64_t anc[kMaxNodes][2];
  uint64_t desc[kMaxNodes][2];  // descendants-or-self of each draft node
  // touched trees, in order of first use
  int dtree[kMaxNodes], dkey[kMaxNodes], dnew[kMaxNodes];
  uint64_t gmask[kMaxNodes][2];  // draft nodes whose sub-trees go to each
  uint64_t wm[2];                // per-wave ballots
  int ntrees, nd;
  // staged trees of one batch: node k of staged tree j at j * n_cap + k
  int cnt[kStageTrees], cnt0[kStageTrees];
  int ntok[kStageSlots];
  short npar[kStageSlots], fc[kStageSlots], ns[kStageSlots];
  short map[kStageTrees][kMaxNodes];  // draft node -> staged node (-1: dropped)
};

// index of node v among the nodes whose flag is set, in index order, from
// the per-wave ballots in wm (threads 0 .. 127)
__device__ __forceinline__ int rank_below(const uint64_t* wm, int v) {
  const int w = v >> 6;
  return (w ? __popcll(wm[0]) : 0) + __popcll(wm[w] & below_mask(v & 63));
}

__global__ void __launch_bounds__(kMergeThreads)
k_pool_merge(void* pool, PoolGeom g, const int32_t* __restrict__ parent,
             const int32_t* __restrict__ tokens, const int32_t* __restrict__ tree_len, int T,
             int32_t* dev_status) {
  __shared__ MergeLds L;
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const bool nodes = tid < kMaxNodes;  // waves 0 and 1 hold one draft node each
  PoolView P = view(pool, g, b);
  int n = T;
  if (tree_len) {
    n = tree_len[b];
    n = n < 0 ? 0 : (n > T ? T : n);
  }
  const bool live = tid < n;
  bool bad = false;
  int par = -1, t = 0;
  if (live) {
    par = parent[static_cast<size_t>(b) * T + tid];
    t = tokens[static_cast<size_t>(b) * T + tid];
    bad = par < -1 || par >= tid;
    L.par[tid] = par;
    L.tok[tid] = t;
  }
  if (nodes) {
    L.gmask[tid][0] = 0ull;
    L.gmask[tid][1] = 0ull;
    L.desc[tid][0] = 0ull;
    L.desc[tid][1] = 0ull;
    L.newslot[tid] = -1;
  }
  {  // the hash table in 16-byte chunks, all of a thread's loads in flight
     // (named registers: arrays here were moved to LDS and scratch)
    static_assert(kMaxSlots == 16 * kMergeThreads, "four chunks of keys per thread");
    const int nq = g.H / 4;
    const int4* gk = reinterpret_cast<const int4*>(P.key);
    const int4* gt = reinterpret_cast<const int4*>(P.tree);
    int4* lk = reinterpret_cast<int4*>(L.key);
    int4* lt = reinterpret_cast<int4*>(L.tree);
    const int q0 = tid, q1 = tid + kMergeThreads, q2 = tid + 2 * kMergeThreads,
              q3 = tid + 3 * kMergeThreads;
    int4 k0, t0, k1, t1, k2, t2, k3, t3;
    if (q0 < nq) { k0 = gk[q0]; t0 = gt[q0]; }
    if (q1 < nq) { k1 = gk[q1]; t1 = gt[q1]; }
    if (q2 < nq) { k2 = gk[q2]; t2 = gt[q2]; }
    if (q3 < nq) { k3 = gk[q3]; t3 = gt[q3]; }
    if (q0 < nq) { lk[q0] = k0; lt[q0] = t0; }
    if (q1 < nq) { lk[q1] = k1; lt[q1] = t1; }
    if (q2 < nq) { lk[q2] = k2; lt[q2] = t2; }
    if (q3 < nq) { lk[q3] = k3; lt[q3] = t3; }
  }
  if (tid == 0) L.ntrees = min(max(*P.ntrees, 0), g.e_max);
  if (__syncthreads_or(bad)) {
    if (tid == 0) ptd::report(dev_status, PTD_ERR_BAD_TREE);
    return;  // the pool is left as it was
  }
  const int H = g.H, hb = g.hbits;
  const int ntrees0 = L.ntrees;

  // lookups; the first node (index order) of every token
  int e = -1, first = tid;
  if (live) {
    for (int s = home_slot(t, hb), k = 0; k < H; ++k, s = (s + 1) & (H - 1)) {
      const int tr = L.tree[s];
      if (tr < 0) break;
      if (L.key[s] == t) {
        e = tr < g.e_max ? tr : -1;  // an id out of range (a pool not initialised) reads as absent
        break;
      }
    }
    // four tokens per LDS read (the draft tokens start 16-byte aligned)
    const int4* tk4 = reinterpret_cast<const int4*>(L.tok);
    for (int u4 = 0; 4 * u4 < tid && first == tid; ++u4) {
      const int4 q = tk4[u4];
      const int u = 4 * u4;
      if (q.w == t && u + 3 < tid) first = u + 3;
      if (q.z == t && u + 2 < tid) first = u + 2;
      if (q.y == t && u + 1 < tid) first = u + 1;
      if (q.x == t) first = u;
    }
    L.firstof[tid] = first;
  }
  // new trees for the missing tokens, in index order of their first node
  const bool newfirst = live && e < 0 && first == tid;
  if (nodes) {
    const uint64_t bm = __ballot(newfirst);
    if (lane == 0) L.wm[wave] = bm;
  }
  __syncthreads();
  if (newfirst) {
    const int id = ntrees0 + rank_below(L.wm, tid);
    L.newid[tid] = id < g.e_max ? id : -1;
  }
  const int nnew = __popcll(L.wm[0]) + __popcll(L.wm[1]);
  __syncthreads();
  bool created = false;
  if (live && e < 0) {
    e = L.newid[first];
    created = e >= 0;
  }
  if (newfirst && e >= 0) {  // insert token -> tree; slots claimed by compare-and-swap
    for (int s = home_slot(t, hb), k = 0; k < H; ++k, s = (s + 1) & (H - 1)) {
      if (atomicCAS(&L.tree[s], -1, e) == -1) {
        L.key[s] = t;
        L.newslot[tid] = s;
        break;
      }
    }
  }
  // touched trees in order of first use (the first node of their token)
  const bool firstuse = live && e >= 0 && first == tid;
  if (nodes) {
    const uint64_t bm = __ballot(firstuse);
    if (lane == 0) L.wm[wave] = bm;
  }
  __syncthreads();
  if (firstuse) {
    const int j = rank_below(L.wm, tid);
    L.jof[tid] = j;
    L.dtree[j] = e;
    L.dkey[j] = t;
    L.dnew[j] = created ? 1 : 0;
  }
  if (tid == 0) {
    L.nd = __popcll(L.wm[0]) + __popcll(L.wm[1]);
    L.ntrees = min(ntrees0 + nnew, g.e_max);
  }
  // ancestor-or-self masks by pointer jumping
  uint64_t anc0 = (live && wave == 0) ? (1ull << lane) : 0ull;
  uint64_t anc1 = (live && wave == 1) ? (1ull << lane) : 0ull;
  int jump = live ? par : -1;
  for (;;) {
    if (nodes) {
      L.anc[tid][0] = anc0;
      L.anc[tid][1] = anc1;
      L.jump[tid] = jump;
    }
    if (!__syncthreads_or(jump >= 0)) break;
    if (jump >= 0) {
      anc0 |= L.anc[jump][0];
      anc1 |= L.anc[jump][1];
      jump = L.jump[jump];
    }
    __syncthreads();
  }
  if (live && e >= 0) {
    const int j = L.jof[first];
    atomicOr(&L.gmask[j][wave], 1ull << lane);
  }
  // descendant-or-self masks: every node sets its bit in the mask of each
  // node of its ancestor-or-self set
  if (live) {
    for (uint64_t m = anc0; m; m &= m - 1ull)
      atomicOr(reinterpret_cast<unsigned long long*>(&L.desc[__builtin_ctzll(m)][wave]), 1ull << lane);
    for (uint64_t m = anc1; m; m &= m - 1ull)
      atomicOr(reinterpret_cast<unsigned long long*>(&L.desc[64 + __builtin_ctzll(m)][wave]), 1ull << lane);
  }
  __syncthreads();
  const int nd = L.nd, n_cap = g.n_cap;

  for (int j0 = 0; j0 < nd; j0 += kStageTrees) {
    const int nb = min(kStageTrees, nd - j0);
    // stage the batch's trees (new ones start as a lone root); a thread's
    // two loads of a pass are issued before either is used
    {
      const int total = nb * n_cap;
      auto load = [&](int i, int2& v, int& c0) {
        v = make_int2(0, -1);
        c0 = 0;
        if (i < total) {
          const int jl = i / n_cap, k = i - jl * n_cap;
          if (!L.dnew[j0 + jl]) {
            const int et = L.dtree[j0 + jl];
            v = P.node[static_cast<size_t>(et) * n_cap + k];
            if (k == 0) c0 = P.count[et];
          }
        }
      };
      auto store = [&](int i, int2 v, int c0) {
        if (i >= total) return;
        const int jl = i / n_cap, k = i - jl * n_cap;
        if (L.dnew[j0 + jl]) {
          if (k == 0) {
            L.ntok[i] = L.dkey[j0 + jl];
            L.npar[i] = -1;
            L.cnt[jl] = 1;
          }
        } else {
          L.ntok[i] = v.x;
          L.npar[i] = static_cast<short>(v.y < 0 || v.y >= k ? -1 : v.y);
          if (k == 0) L.cnt[jl] = min(max(c0, 1), n_cap);
        }
        L.fc[i] = -1;
        L.ns[i] = -1;
      };
      constexpr int kInFlight = 8;  // loads of a thread issued before any is used
      for (int i = tid; i < total; i += kInFlight * kMergeThreads) {
        int2 v[kInFlight];
        int c[kInFlight];
#pragma unroll
        for (int q = 0; q < kInFlight; ++q) load(i + q * kMergeThreads, v[q], c[q]);
#pragma unroll
        for (int q = 0; q < kInFlight; ++q) store(i + q * kMergeThreads, v[q], c[q]);
      }
    }
    __syncthreads();
    // sibling links of the staged nodes, in insertion order: one thread per
    // staged tree prepends every node to its parent's list, last node first
    // (the staging left every link at -1)
    if (tid < nb) {
      const int base = tid * n_cap, c = L.cnt[tid];
      L.cnt0[tid] = L.dnew[j0 + tid] ? 0 : c;  // records below cnt0 are unchanged
      for (int k = c - 1; k >= 1; --k) {
        const int p = L.npar[base + k];
        if (p < 0) continue;  // parents precede their children
        L.ns[base + k] = L.fc[base + p];
        L.fc[base + p] = static_cast<short>(k);
      }
    }
    __syncthreads();

    // thread jl merges every sub-tree keyed by staged tree jl; a sub-tree's
    // nodes are visited in index order from its descendant mask, so a
    // node's parent is mapped before the node
    if (tid < nb) {
      const int jl = tid, j = j0 + jl, base = jl * n_cap;
      int cnt = L.cnt[jl];
#pragma unroll
      for (int gw = 0; gw < 2; ++gw)
        for (uint64_t gm = L.gmask[j][gw]; gm; gm &= gm - 1ull) {  // sub-tree roots, in order
          const int u = 64 * gw + __builtin_ctzll(gm);
          L.map[jl][u] = 0;
#pragma unroll
          for (int dw = 0; dw < 2; ++dw) {
            uint64_t m = L.desc[u][dw];
            if (dw == (u >> 6)) m &= ~below_mask(u & 63) & ~(1ull << (u & 63));
            else if (dw < (u >> 6)) m = 0ull;
            for (; m; m &= m - 1ull) {
              const int c = 64 * dw + __builtin_ctzll(m);
              const int pnode = L.map[jl][L.par[c]];
              if (pnode < 0) {
                L.map[jl][c] = -1;
                continue;
              }
              const int tc = L.tok[c];
              int k = L.fc[base + pnode], last = -1;
              while (k >= 0 && L.ntok[base + k] != tc) {
                last = k;
                k = L.ns[base + k];
              }
              if (k < 0 && cnt < n_cap) {  // append as the last child of pnode
                k = cnt++;
                L.ntok[base + k] = tc;
                L.npar[base + k] = static_cast<short>(pnode);
                L.fc[base + k] = -1;
                L.ns[base + k] = -1;
                if (last < 0) L.fc[base + pnode] = static_cast<short>(k);
                else L.ns[base + last] = static_cast<short>(k);
              }
              L.map[jl][c] = static_cast<short>(k);  // -1: full, skipped with its sub-tree
            }
          }
        }
      L.cnt[jl] = cnt;
    }
    __syncthreads();

    // write back
    for (int i = tid; i < nb * n_cap; i += kMergeThreads) {
      const int jl = i / n_cap, k = i - jl * n_cap;
      const int et = L.dtree[j0 + jl];
      if (k >= L.cnt0[jl] && k < L.cnt[jl])  // a merge only appends
        P.node[static_cast<size_t>(et) * n_cap + k] = make_int2(L.ntok[i], L.npar[i]);
      if (k == 0) P.count[et] = L.cnt[jl];
    }
    __syncthreads();  // the staged arrays are reused by the next batch
  }
  if (nodes) {
    const int s = L.newslot[tid];
    if (s >= 0) {
      P.key[s] = L.key[s];
      P.tree[s] = L.tree[s];
    }
  }
  if (tid == 0) *P.ntrees = L.ntrees;
}

__global__ void __launch_bounds__(kRetrieveThreads)
k_pool_retrieve(const void* pool, PoolGeom g, const int32_t* __restrict__ last_token,
                int T_max, int32_t* __restrict__ parent_out, int32_t* __restrict__ tokens_out,
                int32_t* __restrict__ tree_len_out) {
  __shared__ int s_dist[kRetrieveThreads], s_nxt[kRetrieveThreads], s_ok[kRetrieveThreads];
  __shared__ int s_out[kRetrieveThreads], s_key[kRetrieveThreads];
  __shared__ uint64_t s_lvl[kRW], s_all[kRW];
  __shared__ int s_e;
  const int k = threadIdx.x, lane = k & 63, wv = k >> 6, b = blockIdx.x;
  const PoolView P = view(const_cast<void*>(pool), g, b);
  int32_t* po = parent_out + static_cast<size_t>(b) * T_max;
  int32_t* to = tokens_out + static_cast<size_t>(b) * T_max;
  for (int t = k; t < T_max; t += kRetrieveThreads) {
    po[t] = -1;
    to[t] = -1;
  }
  if (wv == 0) {  // probe 64 slots at a time from the home slot
    const int key = last_token[b];
    int e = -1;
    const int home = home_slot(key, g.hbits);
    for (int k0 = 0; k0 < g.H; k0 += PTD_WAVE) {
      const int s = (home + k0 + lane) & (g.H - 1);
      const int tr = P.tree[s];
      const int ky = P.key[s];
      const uint64_t hit = __ballot(tr >= 0 && ky == key);
      const uint64_t empty = __ballot(tr < 0);
      const int fh = hit ? __builtin_ctzll(hit) : PTD_WAVE;
      const int fe = empty ? __builtin_ctzll(empty) : PTD_WAVE;
      if (fh < fe) {
        e = __shfl(tr, fh, PTD_WAVE);
        if (e >= g.e_max) e = -1;  // out of range: a pool not initialised
        break;
      }
      if (fe < PTD_WAVE) break;  // an empty slot ends the probe: absent
    }
    if (lane == 0) s_e = e;
  }
  __syncthreads();
  const int e = s_e;
  if (e < 0) {
    if (k == 0) tree_len_out[b] = 0;
    return;
  }
  const int cnt = min(max(P.count[e], 1), g.n_cap);
  const int2 nd = k < cnt ? P.node[static_cast<size_t>(e) * g.n_cap + k] : make_int2(0, -1);
  const bool live = k < cnt && (k == 0 || (nd.y >= 0 && nd.y < k));
  const int par = live && k > 0 ? nd.y : -1;
  // depth below the root by pointer jumping; a node under a dead one is
  // unreachable (only in a pool that was not initialised)
  int dist = par >= 0 ? 1 : 0, nxt = par;
  bool ok = live;
  for (;;) {
    s_dist[k] = dist;
    s_nxt[k] = nxt;
    s_ok[k] = ok;
    if (!__syncthreads_or(nxt >= 0)) break;
    if (nxt >= 0) {
      dist += s_dist[nxt];
      ok = ok && s_ok[nxt];
      nxt = s_nxt[nxt];
    }
    __syncthreads();
  }
  const bool reach = ok && k > 0;
  const uint64_t rb = __ballot(reach);
  if (lane == 0) s_all[wv] = rb;
  // breadth first by levels: level 1 = the root's children in insertion
  // order; deeper levels by (parent's number, insertion index)
  int outid = -1, ppid = -1, base = 0;
  __syncthreads();
  const int total = mask_count<kRW>(s_all);
  for (int lv = 1; base < total && lv < kRetrieveThreads; ++lv) {  // uniform
    const bool here = reach && dist == lv;
    __syncthreads();  // numbers of level lv - 1 written; s_lvl, s_key free
    const uint64_t lb = __ballot(here);
    if (lane == 0) s_lvl[wv] = lb;
    int key = 0;
    if (here) key = lv == 1 ? 0 : s_out[par];
    s_key[k] = key;
    __syncthreads();
    if (here) {
      outid = base + level_rank<kRW>(s_lvl, s_key, k, key);
      ppid = lv == 1 ? -1 : key;
      s_out[k] = outid;
    }
    base += mask_count<kRW>(s_lvl);
  }
  __syncthreads();
  if (outid >= 0 && outid < T_max) {
    po[outid] = ppid;
    to[outid] = nd.x;
  }
  if (k == 0) tree_len_out[b] = min(total, T_max);
}

}  // namespace

extern "C" size_t ptd_pool_bytes(int32_t B, int32_t e_max, int32_t n_cap) {
  PoolGeom g;
  if (B < 1 || !pool_geom(e_max, n_cap, &g)) return 0;
  return static_cast<size_t>(B) * g.seq_bytes;
}

extern "C" int ptd_pool_init(void* pool, size_t pool_bytes, int32_t B, int32_t e_max,
                             int32_t n_cap, void* stream) {
  PTD_RETURN_IF(!pool, PTD_ERR_NULL);
  PoolGeom g;
  PTD_RETURN_IF(B < 1 || !pool_geom(e_max, n_cap, &g), PTD_ERR_SHAPE);
  PTD_RETURN_IF(pool_bytes < static_cast<size_t>(B) * g.seq_bytes, PTD_ERR_WORKSPACE);
  PTD_RETURN_IF(!ptd_aligned(pool, 256), PTD_ERR_ALIGN);
  hipLaunchKernelGGL(k_pool_init, dim3(B), dim3(kMergeThreads), 0,
                     static_cast<hipStream_t>(stream), pool, g);
  return ptd_launch_status();
}

extern "C" int ptd_pool_merge(void* pool, size_t pool_bytes, int32_t B, int32_t e_max,
                              int32_t n_cap, const int32_t* parent, const int32_t* tokens,
                              const int32_t* tree_len, int32_t T, int32_t* dev_status,
                              void* stream) {
  PTD_RETURN_IF(!pool || !parent || !tokens, PTD_ERR_NULL);
  PoolGeom g;
  PTD_RETURN_IF(B < 1 || !pool_geom(e_max, n_cap, &g) || T < 1 || T > kMaxNodes, PTD_ERR_SHAPE);
  PTD_RETURN_IF(pool_bytes < static_cast<size_t>(B) * g.seq_bytes, PTD_ERR_WORKSPACE);
  PTD_RETURN_IF(!ptd_aligned(pool, 256), PTD_ERR_ALIGN);
  hipLaunchKernelGGL(k_pool_merge, dim3(B), dim3(kMergeThreads), 0,
                     static_cast<hipStream_t>(stream), pool, g, parent, tokens, tree_len, T,
                     dev_status);
  return ptd_launch_status();
}

extern "C" int ptd_pool_retrieve(const void* pool, size_t pool_bytes, int32_t B, int32_t e_max,
                                 int32_t n_cap, const int32_t* last_token, int32_t T_max,
                                 int32_t* parent_out, int32_t* tokens_out,
                                 int32_t* tree_len_out, void* stream) {
  PTD_RETURN_IF(!pool || !last_token || !parent_out || !tokens_out || !tree_len_out,
                PTD_ERR_NULL);
  PoolGeom g;
  PTD_RETURN_IF(B < 1 || !pool_geom(e_max, n_cap, &g) || T_max < 1 || T_max > PTD_MAX_T,
                PTD_ERR_SHAPE);
  PTD_RETURN_IF(pool_bytes < static_cast<size_t>(B) * g.seq_bytes, PTD_ERR_WORKSPACE);
  PTD_RETURN_IF(!ptd_aligned(pool, 256), PTD_ERR_ALIGN);
  hipLaunchKernelGGL(k_pool_retrieve, dim3(B), dim3(kRetrieveThreads), 0,
                     static_cast<hipStream_t>(stream), pool, g, last_token, T_max, parent_out,
                     tokens_out, tree_len_out);
  return ptd_launch_status();
}

extern "C" int ptd_step_prune(const int32_t* parent, const int32_t* tokens,
                              const int32_t* tree_len, int32_t B, int32_t T, int32_t d_max,
                              int32_t T_max, int32_t* parent_next, int32_t* tokens_next,
                              int32_t* tree_len_next, int32_t* dev_status, void* stream) {
  PTD_RETURN_IF(!parent || !tokens || !parent_next || !tokens_next || !tree_len_next,
                PTD_ERR_NULL);
  PTD_RETURN_IF(B < 1 || T < 1 || T > kMaxNodes || d_max < 1 || T_max < 1 ||
                    T_max > PTD_MAX_T,
                PTD_ERR_SHAPE);
  if (T <= PTD_WAVE)
    hipLaunchKernelGGL(k_step_prune<1>, dim3(B), dim3(PTD_WAVE), 0,
                       static_cast<hipStream_t>(stream), parent, tokens, tree_len, T, d_max, T_max,
                       parent_next, tokens_next, tree_len_next, dev_status);
  else
    hipLaunchKernelGGL(k_step_prune<2>, dim3(B), dim3(2 * PTD_WAVE), 0,
                       static_cast<hipStream_t>(stream), parent, tokens, tree_len, T, d_max, T_max,
                       parent_next, tokens_next, tree_len_next, dev_status);
  return ptd_launch_status();
}
