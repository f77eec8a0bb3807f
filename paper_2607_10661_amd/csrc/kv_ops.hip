// Positions of the tree nodes with the rotary embedding of their queries and
// keys, and the commit of the accepted path into the KV cache.
//
// Sec. 3.1 "Tree Construction": the position of node v is given by |pi(v)|,
// and a root's parent is the last committed token, so node i of sequence b
// sits at kv_len[b] + |pi(i)| - 1.  The rotary embedding (Su et al.,
// RoFormer) turns dimension pair p by pos * inv_freq[p].
// Sec. 3.2: the accepted sequence X' = (n_0, n_1, ..., n_k, V_{n_k}); the
// draft nodes n_1..n_k become committed tokens, node n_j moving from cache row
// kv_len + n_j to row kv_len + j - 1.  A node at depth j was rotated at
// kv_len + j - 1, so the committed rows carry the rotation of their own row.
//
// Kernels
//   k_tree_rope    one workgroup per (node, sequence).  The sequence's parent
//                  array is staged in LDS and every node's |pi| is found by
//                  pointer doubling (about log2(depth) rounds), which also
//                  checks the tree.  The node's D/2 angles and their sine and
//                  cosine are computed in fp64 into LDS; then every thread
//                  turns 16-byte chunks of the node's Hq query heads and Hkv
//                  key rows in fp32 and writes them back rounded to the input
//                  dtype.
//   k_kv_commit    one workgroup per (KV head, K or V, sequence): the path is
//                  checked, then rows move in passes of 256 16-byte chunks;
//                  each pass loads all its source chunks before a barrier and
//                  stores after it.  A later destination never holds an
//                  earlier-unread source (node ids increase along the path, so
//                  kv_len + n_j >= kv_len + j, and a destination row kv_len + j
//                  can only be the source of an earlier, already-read node).
#include <limits.h>
#include <math.h>

#include "ptd_common.hpp"

namespace {

constexpr int kThreads = 256;
constexpr int kMaxHalf = 64;  // D/2 for D <= 128

using u32x4 = uint32_t __attribute__((ext_vector_type(4)));

struct RopeArgs {
  void* q;                 // [B][T][Hq][D] or null
  void* k;                 // [B][Hkv][L_cap][D] or null
  const int32_t* kv_len;   // [B]
  const int32_t* parent;   // [B][T]
  int32_t* pos_out;        // [B][T] or null
  int32_t* dev_status;
  int T, Hq, Hkv, D, L_cap;
  double inv_freq[kMaxHalf];
};

// fp32 view of a 16-byte chunk: 8 bf16 or 4 fp32 values
template <bool BF16>
__device__ __forceinline__ void unpack(const u32x4& c, float (&x)[BF16 ? 8 : 4]) {
  if constexpr (BF16) {
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      x[2 * w] = ptd::bf16_lo(c[w]);
      x[2 * w + 1] = ptd::bf16_hi(c[w]);
    }
  } else {
#pragma unroll
    for (int w = 0; w < 4; ++w) x[w] = __uint_as_float(c[w]);
  }
}
template <bool BF16>
__device__ __forceinline__ u32x4 pack(const float (&x)[BF16 ? 8 : 4]) {
  u32x4 c;
  if constexpr (BF16) {
#pragma unroll
    for (int w = 0; w < 4; ++w) c[w] = ptd::cvt_pk_bf16(x[2 * w], x[2 * w + 1]);
  } else {
#pragma unroll
    for (int w = 0; w < 4; ++w) c[w] = __float_as_uint(x[w]);
  }
  return c;
}

template <bool BF16, bool INTERLEAVED>
__global__ void __launch_bounds__(kThreads) k_tree_rope(RopeArgs a) {
  constexpr int E = BF16 ? 8 : 4;  // elements per 16-byte chunk
  __shared__ int s_anc[2][PTD_MAX_T];
  __shared__ int s_len[2][PTD_MAX_T];
  __shared__ float2 s_cs[kMaxHalf];
  const int i = blockIdx.x, b = blockIdx.y, tid = threadIdx.x, T = a.T;
  const int kv = a.kv_len[b];
  // uniform: nothing of this sequence is touched.  Without keys only the
  // positions must stay representable.
  if (kv < 0 || kv > (a.k ? a.L_cap : INT_MAX) - T) {
    if (tid == 0) ptd::report(a.dev_status, PTD_ERR_KV_LEN);
    return;
  }

  // |pi(v)| of every node by pointer doubling: len[v] counts the nodes from v
  // up to (excluding) anc[v]; each round adds the segment above anc[v].
  const int32_t* par = a.parent + static_cast<size_t>(b) * T;
  bool bad = false;
  for (int v = tid; v < T; v += kThreads) {
    const int p = par[v];
    bad |= p < -1 || p >= v;
    s_anc[0][v] = p;
    s_len[0][v] = 1;
  }
  if (__syncthreads_or(bad)) {
    if (tid == 0) ptd::report(a.dev_status, PTD_ERR_BAD_TREE);
    return;
  }
  int cur = 0;
  for (;;) {
    bool more = false;
    for (int v = tid; v < T; v += kThreads) {
      const int u = s_anc[cur][v];
      int l = s_len[cur][v], w = u;
      if (u >= 0) {
        l += s_len[cur][u];
        w = s_anc[cur][u];
      }
      s_anc[cur ^ 1][v] = w;
      s_len[cur ^ 1][v] = l;
      more |= w >= 0;
    }
    cur ^= 1;
    if (!__syncthreads_or(more)) break;
  }
  const int pos = kv + s_len[cur][i] - 1;
  if (a.pos_out && tid == 0) a.pos_out[static_cast<size_t>(b) * T + i] = pos;

  const int H2 = a.D / 2;
  if (tid < H2) {
    double s, c;
    sincos(static_cast<double>(pos) * a.inv_freq[tid], &s, &c);
    s_cs[tid] = make_float2(static_cast<float>(c), static_cast<float>(s));
  }
  __syncthreads();

  // work items: (head, chunk).  Half pairing: chunk c covers pairs
  // [c*E, c*E + E) and reads one chunk from each half of the head.
  // Interleaved: chunk c holds pairs c*E/2 .. c*E/2 + E/2 - 1 in place.
  const int per_head = INTERLEAVED ? a.D / E : H2 / E;
  const int nq = a.q ? a.Hq : 0, nk = a.k ? a.Hkv : 0;
  const int items = (nq + nk) * per_head;
  for (int it = tid; it < items; it += kThreads) {
    const int h = it / per_head, c = it % per_head;
    char* row;
    if (h < nq) {
      row = static_cast<char*>(a.q) + ((static_cast<size_t>(b) * T + i) * a.Hq + h) *
                                          static_cast<size_t>(a.D) * (BF16 ? 2 : 4);
    } else {
      const int g = h - nq;
      row = static_cast<char*>(a.k) +
            ((static_cast<size_t>(b) * a.Hkv + g) * a.L_cap + kv + i) *
                static_cast<size_t>(a.D) * (BF16 ? 2 : 4);
    }
    u32x4* rc = reinterpret_cast<u32x4*>(row);
    if constexpr (INTERLEAVED) {
      float x[E];
      unpack<BF16>(rc[c], x);
#pragma unroll
      for (int e = 0; e < E; e += 2) {
        const float2 cs = s_cs[(c * E + e) / 2];
        const float xa = x[e], xb = x[e + 1];
        x[e] = xa * cs.x - xb * cs.y;
        x[e + 1] = xa * cs.y + xb * cs.x;
      }
      rc[c] = pack<BF16>(x);
    } else {
      const int hc = H2 / E;  // chunks per half
      float xa[E], xb[E];
      unpack<BF16>(rc[c], xa);
      unpack<BF16>(rc[c + hc], xb);
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const float2 cs = s_cs[c * E + e];
        const float u = xa[e], w = xb[e];
        xa[e] = u * cs.x - w * cs.y;
        xb[e] = u * cs.y + w * cs.x;
      }
      rc[c] = pack<BF16>(xa);
      rc[c + hc] = pack<BF16>(xb);
    }
  }
}

struct CommitArgs {
  void* k;                      // [B][Hkv][L_cap][D]
  void* v;
  const int32_t* kv_len;        // [B]
  const int32_t* accept_len;    // [B]
  const int32_t* accept_nodes;  // [B][T]
  int32_t* kv_len_next;         // [B]
  int32_t* dev_status;
  int T, Hkv, L_cap, row_chunks;  // row_chunks = 16-byte chunks per row
};

__global__ void __launch_bounds__(kThreads) k_kv_commit(CommitArgs a) {
  __shared__ int s_node[PTD_MAX_T];
  const int g = blockIdx.x, which = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
  const int T = a.T;
  const int kv = a.kv_len[b];
  const int n = a.accept_len[b];
  const bool writer = g == 0 && which == 0 && tid == 0;
  if (kv < 0 || kv > a.L_cap - T) {  // uniform
    if (writer) {
      ptd::report(a.dev_status, PTD_ERR_KV_LEN);
      a.kv_len_next[b] = kv;
    }
    return;
  }
  bool bad = n < 0 || n > T;
  if (!bad) {
    const int32_t* nodes = a.accept_nodes + static_cast<size_t>(b) * T;
    for (int j = tid; j < n; j += kThreads) {
      const int x = nodes[j];
      const int prev = j > 0 ? nodes[j - 1] : -1;
      bad |= x < 0 || x >= T || x <= prev;
      s_node[j] = x;
    }
  }
  if (__syncthreads_or(bad)) {
    if (writer) {
      ptd::report(a.dev_status, PTD_ERR_BAD_PATH);
      a.kv_len_next[b] = kv;
    }
    return;
  }
  if (writer) a.kv_len_next[b] = kv + n;

  u32x4* head = reinterpret_cast<u32x4*>(which == 0 ? a.k : a.v) +
                (static_cast<size_t>(b) * a.Hkv + g) * a.L_cap * a.row_chunks;
  const int rows_per_pass = kThreads / a.row_chunks;
  const int j_off = tid / a.row_chunks, ch = tid % a.row_chunks;
  for (int j0 = 0; j0 < n; j0 += rows_per_pass) {
    const int j = j0 + j_off;
    const bool move = j < n && s_node[j] != j;  // rows already in place stay
    u32x4 val;
    if (move) val = head[static_cast<size_t>(kv + s_node[j]) * a.row_chunks + ch];
    __syncthreads();  // every source chunk of this pass is in registers
    if (move) head[static_cast<size_t>(kv + j) * a.row_chunks + ch] = val;
    __syncthreads();  // later passes read rows this pass may have written
  }
}

bool rope_shape_ok(const ptd_attn_shape* s, int T) {
  return s && s->B >= 1 && s->Hq >= 1 && s->Hkv >= 1 && (s->D == 64 || s->D == 128) &&
         T >= 1 && T <= PTD_MAX_T && s->L_cap >= T &&
         (s->in_dtype == PTD_BF16 || s->in_dtype == PTD_F32);
}

}  // namespace

extern "C" int ptd_tree_rope(void* q, void* k_cache, const int32_t* kv_len,
                             const int32_t* parent, int32_t T, const ptd_attn_shape* shape,
                             double theta, const double* inv_freq, int32_t pairing,
                             int32_t* pos_out, int32_t* dev_status, void* stream) {
  PTD_RETURN_IF(!shape || !kv_len || !parent || (!q && !k_cache && !pos_out), PTD_ERR_NULL);
  PTD_RETURN_IF(shape->in_dtype != PTD_BF16 && shape->in_dtype != PTD_F32, PTD_ERR_DTYPE);
  PTD_RETURN_IF(!rope_shape_ok(shape, T), PTD_ERR_SHAPE);
  PTD_RETURN_IF(pairing != PTD_ROPE_HALF && pairing != PTD_ROPE_INTERLEAVED, PTD_ERR_SHAPE);
  PTD_RETURN_IF(!inv_freq && !(theta > 0.0 && theta < INFINITY), PTD_ERR_SHAPE);
  PTD_RETURN_IF((q && !ptd_aligned(q, 16)) || (k_cache && !ptd_aligned(k_cache, 16)),
                PTD_ERR_ALIGN);
  RopeArgs a;
  a.q = q;
  a.k = k_cache;
  a.kv_len = kv_len;
  a.parent = parent;
  a.pos_out = pos_out;
  a.dev_status = dev_status;
  a.T = T;
  a.Hq = shape->Hq;
  a.Hkv = shape->Hkv;
  a.D = shape->D;
  a.L_cap = shape->L_cap;
  for (int p = 0; p < kMaxHalf; ++p) {
    if (p < shape->D / 2) {
      a.inv_freq[p] = inv_freq ? inv_freq[p] : pow(theta, -2.0 * p / shape->D);
      PTD_RETURN_IF(!(fabs(a.inv_freq[p]) < INFINITY), PTD_ERR_SHAPE);
    } else {
      a.inv_freq[p] = 0.0;
    }
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  const dim3 grid(T, shape->B);
  const bool bf16 = shape->in_dtype == PTD_BF16, il = pairing == PTD_ROPE_INTERLEAVED;
  if (bf16 && il) hipLaunchKernelGGL((k_tree_rope<true, true>), grid, dim3(kThreads), 0, st, a);
  else if (bf16) hipLaunchKernelGGL((k_tree_rope<true, false>), grid, dim3(kThreads), 0, st, a);
  else if (il) hipLaunchKernelGGL((k_tree_rope<false, true>), grid, dim3(kThreads), 0, st, a);
  else hipLaunchKernelGGL((k_tree_rope<false, false>), grid, dim3(kThreads), 0, st, a);
  return ptd_launch_status();
}

extern "C" int ptd_kv_commit(void* k_cache, void* v_cache, const int32_t* kv_len,
                             const int32_t* accept_len, const int32_t* accept_nodes,
                             int32_t T, const ptd_attn_shape* shape, int32_t* kv_len_next,
                             int32_t* dev_status, void* stream) {
  PTD_RETURN_IF(!shape || !k_cache || !v_cache || !kv_len || !accept_len || !accept_nodes ||
                    !kv_len_next,
                PTD_ERR_NULL);
  PTD_RETURN_IF(shape->in_dtype != PTD_BF16 && shape->in_dtype != PTD_F32, PTD_ERR_DTYPE);
  PTD_RETURN_IF(!rope_shape_ok(shape, T), PTD_ERR_SHAPE);
  PTD_RETURN_IF(kv_len_next == kv_len, PTD_ERR_SHAPE);
  PTD_RETURN_IF(!ptd_aligned(k_cache, 16) || !ptd_aligned(v_cache, 16), PTD_ERR_ALIGN);
  CommitArgs a;
  a.k = k_cache;
  a.v = v_cache;
  a.kv_len = kv_len;
  a.accept_len = accept_len;
  a.accept_nodes = accept_nodes;
  a.kv_len_next = kv_len_next;
  a.dev_status = dev_status;
  a.T = T;
  a.Hkv = shape->Hkv;
  a.L_cap = shape->L_cap;
  a.row_chunks = shape->D * (shape->in_dtype == PTD_BF16 ? 2 : 4) / 16;  // 8, 16 or 32
  hipLaunchKernelGGL(k_kv_commit, dim3(shape->Hkv, 2, shape->B), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), a);
  return ptd_launch_status();
}
