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
// All three kernels work on trees of at most 64 nodes (one node per lane):
//   k_step_prune     one wave per sequence: ancestor masks by pointer jumping
//                    over shuffles, sub-tree depths, the new root of every
//                    sub-tree along its chain of lowest-index children, and
//                    breadth-first renumbering of the kept forest level by
//                    level (ranks counted over the level's lanes).
//   k_pool_merge     one workgroup per sequence.  The sequence's hash table
//                    (token -> tree) is staged in LDS; wave 0 looks every
//                    draft node's token up, gives the missing tokens new trees
//                    in index order of their first occurrence (while there is
//                    room) and inserts them.  The touched trees are staged in
//                    LDS with sibling links; lane j of wave 0 merges every
//                    sub-tree whose root token keys tree j, the sub-tree's
//                    nodes in index order (the lanes' trees are independent
//                    and proceed together).  Trees, slots and the tree count
//                    are written back.
//   k_pool_retrieve  one wave per sequence: 64 hash slots from the token's
//                    home slot in one load, the tree's nodes one per lane,
//                    breadth-first order by levels.
//
// Pool layout per sequence (ptd_pool_bytes): int32 ntrees, padded to 16
// bytes; int32 slot_key[H]; int32 slot_tree[H] (-1 empty); int32 count[e_max];
// int2 node[e_max][n_cap] = (token, parent index in the tree; -1 at the root,
// which is node 0).  H is the power of two >= 2 e_max (at least 64).  Nodes
// of a tree are stored in insertion order, so a parent precedes its children.
#include "ptd_common.hpp"

namespace {

constexpr int kMaxNodes = 64;    // draft nodes per sequence, pool tree capacity
constexpr int kMaxTrees = 2048;  // pool trees per sequence
constexpr int kMaxSlots = 4096;
constexpr int kMergeThreads = 256;

struct PoolGeom {
  int e_max, n_cap, H, hbits;
  size_t seq_bytes, off_key, off_tree, off_count, off_node;
};

inline bool pool_geom(int e_max, int n_cap, PoolGeom* g) {
  if (e_max < 1 || e_max > kMaxTrees || n_cap < 1 || n_cap > kMaxNodes) return false;
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

// value of lane src (src uniform over the wave): v_readlane, no LDS round trip
__device__ __forceinline__ int rl(int v, int src) { return __builtin_amdgcn_readlane(v, src); }
__device__ __forceinline__ uint64_t rl64(uint64_t v, int src) {
  const uint32_t lo = __builtin_amdgcn_readlane(static_cast<uint32_t>(v), src);
  const uint32_t hi = __builtin_amdgcn_readlane(static_cast<uint32_t>(v >> 32), src);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src) {
  const uint32_t lo = __shfl(static_cast<uint32_t>(v), src, PTD_WAVE);
  const uint32_t hi = __shfl(static_cast<uint32_t>(v >> 32), src, PTD_WAVE);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// ---------------------------------------------------------------------------
// stepping
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(PTD_WAVE)
k_step_prune(const int32_t* __restrict__ parent, const int32_t* __restrict__ tokens,
             const int32_t* __restrict__ tree_len, int T, int d_max, int T_max,
             int32_t* __restrict__ parent_next, int32_t* __restrict__ tokens_next,
             int32_t* __restrict__ tree_len_next, int32_t* dev_status) {
  __shared__ int s_h[kMaxNodes], s_fc[kMaxNodes], s_rootof[kMaxNodes];
  __shared__ unsigned long long s_cm[kMaxNodes];
  __shared__ unsigned long long s_U[kMaxNodes + 1];
  __shared__ unsigned long long s_nr;
  const int lane = threadIdx.x, b = blockIdx.x;
  int n = T;
  if (tree_len) {
    n = tree_len[b];
    n = n < 0 ? 0 : (n > T ? T : n);
  }
  int32_t* pn = parent_next + static_cast<size_t>(b) * T_max;
  int32_t* tn = tokens_next + static_cast<size_t>(b) * T_max;
  const bool live = lane < n;
  const int par = live ? parent[static_cast<size_t>(b) * T + lane] : -1;
  const int tok = live ? tokens[static_cast<size_t>(b) * T + lane] : -1;
  if (__any(live && (par < -1 || par >= lane))) {
    if (lane == 0) {
      ptd::report(dev_status, PTD_ERR_BAD_TREE);
      tree_len_next[b] = 0;
    }
    for (int t = lane; t < T_max; t += PTD_WAVE) {
      pn[t] = -1;
      tn[t] = -1;
    }
    return;
  }
  // ancestor-or-self masks by pointer jumping
  uint64_t anc = live ? (1ull << lane) : 0ull;
  int jump = par;
  while (__any(jump >= 0)) {
    const int src = jump >= 0 ? jump : lane;
    const uint64_t a2 = shfl_u64(anc, src);
    const int j2 = __shfl(jump, src, PTD_WAVE);
    if (jump >= 0) {
      anc |= a2;
      jump = j2;
    }
  }
  const int dep = __popcll(anc);
  // depth of the sub-tree under each node: max over its descendants w of
  // dep(w) - dep(v) + 1.  U[d], the union of the ancestor-or-self sets of the
  // nodes at depth d, holds exactly the nodes with a descendant at depth d;
  // v's descendants fill every level from dep(v) down to its deepest one,
  // so h(v) counts the consecutive levels d >= dep(v) with v in U[d].
  s_U[lane] = 0ull;
  if (lane == 0) s_U[kMaxNodes] = 0ull;
  __syncthreads();
  if (live) atomicOr(&s_U[dep], static_cast<unsigned long long>(anc));
  __syncthreads();
  int h = 0;
  if (live) {
    int d = dep;  // v itself is in U[dep]
    while (d < kMaxNodes && ((s_U[d + 1] >> lane) & 1ull)) ++d;
    h = d - dep + 1;
  }
  s_h[lane] = h;
  s_cm[lane] = 0ull;
  if (lane == 0) s_nr = 0ull;
  __syncthreads();
  if (live && par >= 0) atomicOr(&s_cm[par], 1ull << lane);
  __syncthreads();
  const uint64_t cm = s_cm[lane];
  s_fc[lane] = cm ? __builtin_ctzll(cm) : -1;
  __syncthreads();
  // every old root steps down its lowest-index children while too deep
  if (live && par < 0) {
    int x = lane;
    while (s_h[x] > d_max) x = s_fc[x];
    s_rootof[x] = lane;
    atomicOr(&s_nr, 1ull << x);
  }
  __syncthreads();
  const uint64_t NR = s_nr;
  const bool keep = live && (anc & NR) != 0ull;
  const uint64_t KEEP = __ballot(keep);
  const int nd = __popcll(anc & KEEP);  // depth in the kept forest
  const bool is_root = keep && nd == 1;
  const int rootof = is_root ? s_rootof[lane] : 0;
  // breadth-first numbering: level 1 by the old root they replace, deeper
  // levels by (parent's number, old index)
  int outid = -1;
  int base = 0;
  {
    const uint64_t lvl = __ballot(is_root);
    int rank = 0;
    for (uint64_t m = lvl; m; m &= m - 1ull) {
      const int w = __builtin_ctzll(m);
      const int rw = rl(rootof, w);
      if (is_root && rw < rootof) ++rank;
    }
    if (is_root) outid = rank;
    base = __popcll(lvl);
  }
  for (int L = 2; base < __popcll(KEEP) && L <= kMaxNodes; ++L) {
    const bool here = keep && nd == L;
    const uint64_t lvl = __ballot(here);
    const int pid = __shfl(outid, here ? par : lane, PTD_WAVE);  // parent numbered one level up
    int rank = 0;
    for (uint64_t m = lvl; m; m &= m - 1ull) {
      const int w = __builtin_ctzll(m);
      const int pw = rl(pid, w);
      if (here && (pw < pid || (pw == pid && w < lane))) ++rank;
    }
    if (here) outid = base + rank;
    base += __popcll(lvl);
  }
  const int ppid = __shfl(outid, par >= 0 ? par : lane, PTD_WAVE);
  const int kept = __popcll(KEEP);
  for (int t = lane; t < T_max; t += PTD_WAVE) {
    pn[t] = -1;
    tn[t] = -1;
  }
  __syncthreads();
  if (keep && outid < T_max) {
    pn[outid] = is_root ? -1 : ppid;
    tn[outid] = tok;
  }
  if (lane == 0) tree_len_next[b] = min(kept, T_max);
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
  int par[kMaxNodes], tok[kMaxNodes], e[kMaxNodes];
  int dtree[kMaxNodes];          // distinct trees touched, in order of first use
  unsigned long long gmask[kMaxNodes];  // draft nodes whose sub-trees go to each
  int dnew[kMaxNodes];           // 1: created by this call
  int cnt[kMaxNodes];            // staged node counts
  int2 node[kMaxNodes][kMaxNodes];
  signed char fc[kMaxNodes][kMaxNodes], ns[kMaxNodes][kMaxNodes], lc[kMaxNodes][kMaxNodes];
  signed char map[kMaxNodes][kMaxNodes];
  unsigned long long desc[kMaxNodes];  // descendants-or-self of each draft node
  int newslot[kMaxNodes];
  int ntrees, nd;
};

__global__ void __launch_bounds__(kMergeThreads)
k_pool_merge(void* pool, PoolGeom g, const int32_t* __restrict__ parent,
             const int32_t* __restrict__ tokens, const int32_t* __restrict__ tree_len, int T,
             int32_t* dev_status) {
  __shared__ MergeLds L;
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  PoolView P = view(pool, g, b);
  int n = T;
  if (tree_len) {
    n = tree_len[b];
    n = n < 0 ? 0 : (n > T ? T : n);
  }
  bool bad = false;
  if (tid < n) {
    const int p = parent[static_cast<size_t>(b) * T + tid];
    bad = p < -1 || p >= tid;
    L.par[tid] = p;
    L.tok[tid] = tokens[static_cast<size_t>(b) * T + tid];
  }
  {  // the hash table in 16-byte chunks, all of a thread's loads in flight
    constexpr int R = kMaxSlots / 4 / kMergeThreads;
    const int nq = g.H / 4;
    const int4* gk = reinterpret_cast<const int4*>(P.key);
    const int4* gt = reinterpret_cast<const int4*>(P.tree);
    int4 vk[R], vt[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int q = tid + r * kMergeThreads;
      if (q < nq) {
        vk[r] = gk[q];
        vt[r] = gt[q];
      }
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int q = tid + r * kMergeThreads;
      if (q < nq) {
        reinterpret_cast<int4*>(L.key)[q] = vk[r];
        reinterpret_cast<int4*>(L.tree)[q] = vt[r];
      }
    }
  }
  if (tid == 0) L.ntrees = min(max(*P.ntrees, 0), g.e_max);
  if (__syncthreads_or(bad)) {
    if (tid == 0) ptd::report(dev_status, PTD_ERR_BAD_TREE);
    return;  // the pool is left as it was
  }
  const int H = g.H, hb = g.hbits;

  // lookups; new trees for the missing tokens, in index order of first occurrence
  if (wave == 0) {
    const bool live = lane < n;
    const int t = live ? L.tok[lane] : 0;
    int e = -1;
    if (live) {
      for (int s = home_slot(t, hb), k = 0; k < H; ++k, s = (s + 1) & (H - 1)) {
        const int tr = L.tree[s];
        if (tr < 0) break;
        if (L.key[s] == t) {
          e = tr < g.e_max ? tr : -1;  // an id out of range (a pool not initialised) reads as absent
          break;
        }
      }
    }
    const uint64_t miss = __ballot(live && e < 0);
    int ntrees = L.ntrees;
    bool first = false;
    uint64_t todo = miss;
    while (todo) {  // uniform
      const int src = __builtin_ctzll(todo);
      const int ts = __builtin_amdgcn_readlane(t, src);
      const uint64_t same = __ballot(live && e < 0 && t == ts) & todo;
      const int id = ntrees < g.e_max ? ntrees : -1;
      if ((same >> lane) & 1ull) e = id;
      if (lane == src) first = id >= 0;
      if (id >= 0) ++ntrees;
      todo &= ~same;
    }
    L.newslot[lane] = -1;
    if (first) {  // insert token -> tree; slots claimed by compare-and-swap
      for (int s = home_slot(t, hb), k = 0; k < H; ++k, s = (s + 1) & (H - 1)) {
        if (atomicCAS(&L.tree[s], -1, e) == -1) {
          L.key[s] = t;
          L.newslot[lane] = s;
          break;
        }
      }
    }
    if (lane < n) L.e[lane] = e;
    // distinct trees touched, in order of first use
    const uint64_t has = __ballot(live && e >= 0);
    bool firstuse = false;
    uint64_t mymask = 0ull;
    todo = has;
    while (todo) {
      const int src = __builtin_ctzll(todo);
      const int es = __builtin_amdgcn_readlane(e, src);
      const uint64_t same = __ballot(live && e == es) & todo;
      if (lane == src) {
        firstuse = true;
        mymask = same;
      }
      todo &= ~same;
    }
    const uint64_t fu = __ballot(firstuse);
    if (firstuse) {
      const int j = __popcll(fu & below_mask(lane));
      L.dtree[j] = e;
      L.dnew[j] = first ? 1 : 0;
      L.gmask[j] = mymask;
    }
    if (lane == 0) {
      L.nd = __popcll(fu);
      L.ntrees = ntrees;
    }
    // ancestor-or-self masks by pointer jumping, then the descendant masks
    const int par = live ? L.par[lane] : -1;
    uint64_t anc = live ? (1ull << lane) : 0ull;
    int jump = par;
    while (__any(jump >= 0)) {
      const int src = jump >= 0 ? jump : lane;
      const uint64_t a2 = shfl_u64(anc, src);
      const int j2 = __shfl(jump, src, PTD_WAVE);
      if (jump >= 0) {
        anc |= a2;
        jump = j2;
      }
    }
    for (int u = 0; u < n; ++u) {
      const uint64_t d = __ballot((anc >> u) & 1ull);
      if (lane == 0) L.desc[u] = d;
    }
  }
  __syncthreads();
  const int nd = L.nd, n_cap = g.n_cap;

  // stage the touched trees (new ones start as a lone root); all of a
  // thread's loads are issued before any is used
  {
    constexpr int R = kMaxNodes * kMaxNodes / kMergeThreads;
    const int total = nd * n_cap;
    int2 v[R];
    int c0[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int i = tid + r * kMergeThreads;
      c0[r] = 0;
      if (i < total) {
        const int j = i / n_cap, k = i - j * n_cap;
        const int e = L.dtree[j];
        if (!L.dnew[j]) {
          v[r] = P.node[static_cast<size_t>(e) * n_cap + k];
          if (k == 0) c0[r] = P.count[e];
        }
      }
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int i = tid + r * kMergeThreads;
      if (i >= total) continue;
      const int j = i / n_cap, k = i - j * n_cap;
      if (L.dnew[j]) {
        if (k == 0) {
          int tkey = 0;
          for (int u = 0; u < n; ++u)
            if (L.e[u] == L.dtree[j]) {
              tkey = L.tok[u];
              break;
            }
          L.node[j][0] = make_int2(tkey, -1);
          L.cnt[j] = 1;
        }
      } else {
        L.node[j][k] = v[r];
        if (k == 0) L.cnt[j] = min(max(c0[r], 1), n_cap);
      }
      L.fc[j][k] = -1;
      L.lc[j][k] = -1;
      L.ns[j][k] = -1;
    }
  }
  __syncthreads();
  // sibling links of the staged nodes, in insertion order
  for (int i = tid; i < nd * n_cap; i += kMergeThreads) {
    const int j = i / n_cap, k = i % n_cap;
    if (k == 0 || k >= L.cnt[j]) continue;
    const int p = L.node[j][k].y;
    if (p < 0 || p >= k) continue;  // parents precede their children
    int nx = -1;
    for (int k2 = k + 1; k2 < L.cnt[j]; ++k2)
      if (L.node[j][k2].y == p) {
        nx = k2;
        break;
      }
    L.ns[j][k] = static_cast<signed char>(nx);
    bool firstk = true, lastk = nx < 0;
    for (int k2 = 1; k2 < k; ++k2)
      if (L.node[j][k2].y == p) {
        firstk = false;
        break;
      }
    if (firstk) L.fc[j][p] = static_cast<signed char>(k);
    if (lastk) L.lc[j][p] = static_cast<signed char>(k);
  }
  __syncthreads();

  // lane j merges every sub-tree keyed by tree j; a sub-tree's nodes are
  // visited in index order from its descendant mask, so a node's parent is
  // mapped before the node
  if (wave == 0 && lane < nd) {
    const int j = lane;
    int cnt = L.cnt[j];
    for (uint64_t gm = L.gmask[j]; gm; gm &= gm - 1ull) {  // this tree's sub-tree roots, in order
      const int u = __builtin_ctzll(gm);
      L.map[j][u] = 0;
      for (uint64_t m = L.desc[u] & ~(1ull << u); m; m &= m - 1ull) {
        const int c = __builtin_ctzll(m);
        const int pnode = L.map[j][L.par[c]];
        if (pnode < 0) {
          L.map[j][c] = -1;
          continue;
        }
        const int tc = L.tok[c];
        int k = L.fc[j][pnode];
        while (k >= 0 && L.node[j][k].x != tc) k = L.ns[j][k];
        if (k < 0 && cnt < n_cap) {  // append as the last child of pnode
          k = cnt++;
          L.node[j][k] = make_int2(tc, pnode);
          L.fc[j][k] = -1;
          L.lc[j][k] = -1;
          L.ns[j][k] = -1;
          const int last = L.lc[j][pnode];
          if (last < 0) L.fc[j][pnode] = static_cast<signed char>(k);
          else L.ns[j][last] = static_cast<signed char>(k);
          L.lc[j][pnode] = static_cast<signed char>(k);
        }
        L.map[j][c] = static_cast<signed char>(k);  // -1: full, skipped with its sub-tree
      }
    }
    L.cnt[j] = cnt;
  }
  __syncthreads();

  // write back
  for (int i = tid; i < nd * n_cap; i += kMergeThreads) {
    const int j = i / n_cap, k = i % n_cap;
    if (k < L.cnt[j]) P.node[static_cast<size_t>(L.dtree[j]) * n_cap + k] = L.node[j][k];
    if (k == 0) P.count[L.dtree[j]] = L.cnt[j];
  }
  if (tid < PTD_WAVE) {
    const int s = L.newslot[tid];
    if (s >= 0) {
      P.key[s] = L.key[s];
      P.tree[s] = L.tree[s];
    }
  }
  if (tid == 0) *P.ntrees = L.ntrees;
}

__global__ void __launch_bounds__(PTD_WAVE)
k_pool_retrieve(const void* pool, PoolGeom g, const int32_t* __restrict__ last_token,
                int T_max, int32_t* __restrict__ parent_out, int32_t* __restrict__ tokens_out,
                int32_t* __restrict__ tree_len_out) {
  const int lane = threadIdx.x, b = blockIdx.x;
  const PoolView P = view(const_cast<void*>(pool), g, b);
  int32_t* po = parent_out + static_cast<size_t>(b) * T_max;
  int32_t* to = tokens_out + static_cast<size_t>(b) * T_max;
  for (int t = lane; t < T_max; t += PTD_WAVE) {
    po[t] = -1;
    to[t] = -1;
  }
  const int key = last_token[b];
  // probe 64 slots at a time from the home slot
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
  if (e < 0) {
    if (lane == 0) tree_len_out[b] = 0;
    return;
  }
  const int cnt = min(max(P.count[e], 1), g.n_cap);
  const int2 nd = lane < cnt ? P.node[static_cast<size_t>(e) * g.n_cap + lane] : make_int2(0, -1);
  const bool live = lane < cnt && (lane == 0 || (nd.y >= 0 && nd.y < lane));
  const int par = live ? nd.y : -1;
  // breadth first by levels: level 1 = the root's children in insertion
  // order; deeper levels by (parent's number, insertion index)
  int outid = -1;
  int base = 0;
  uint64_t prev = 1ull;  // level 0: the root (node 0)
  for (;;) {
    const bool here = live && lane > 0 && par >= 0 && ((prev >> par) & 1ull);
    const uint64_t lvl = __ballot(here);
    if (!lvl) break;
    const int pid = __shfl(outid, here ? par : lane, PTD_WAVE);
    int rank = 0;
    for (uint64_t m = lvl; m; m &= m - 1ull) {
      const int w = __builtin_ctzll(m);
      const int pw = rl(pid, w);
      if (here && (pw < pid || (pw == pid && w < lane))) ++rank;
    }
    if (here) outid = base + rank;
    base += __popcll(lvl);
    prev = lvl;
  }
  const int ppid = __shfl(outid, par > 0 ? par : lane, PTD_WAVE);
  if (outid >= 0 && outid < T_max) {
    po[outid] = par == 0 ? -1 : ppid;
    to[outid] = nd.x;
  }
  if (lane == 0) tree_len_out[b] = min(cnt - 1, T_max);
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
  hipLaunchKernelGGL(k_pool_retrieve, dim3(B), dim3(PTD_WAVE), 0,
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
  hipLaunchKernelGGL(k_step_prune, dim3(B), dim3(PTD_WAVE), 0, static_cast<hipStream_t>(stream),
                     parent, tokens, tree_len, T, d_max, T_max, parent_next, tokens_next,
                     tree_len_next, dev_status);
  return ptd_launch_status();
}
