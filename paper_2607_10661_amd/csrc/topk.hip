// Per-row argmax and top-k of the verification logits (Sec. 3.2: greedy
// verification tokens are the highest-probability predictions; App. A: top-k
// candidates for the draft-tree expansion).
//
// Order: value descending, equal values by the lower vocabulary index, -0.0
// equal to +0.0.  Each element becomes one 64-bit key
//   key = orderable(value) << 32 | ~index
// so the required order is plain unsigned comparison of keys, and every key of
// a row is distinct.
//
// Kernels
//   k_topk_row      one workgroup per (row, vocabulary slice), a slice being
//                   at most 16 loads of 16 bytes per lane (131072 bf16 values):
//                   a cheap lower bound of the KMAX-th best value leaves a few
//                   candidates, selected by one wave (details below).
//   k_topk_scalar   rows that are not 16-byte aligned: one wave per (row,
//                   slice) with element loads; each lane keeps a sorted list
//                   of its KMAX best keys in registers.
// Sorted lists are merged by a butterfly of 6 steps per wave, each merging two
// sorted lists with a bitonic network.
//   k_topk_merge    one wave per row merges the slice results the same way
//                   (only when a row spans several slices).
// The selected values are re-read from the logits, so topk_val carries the
// row's own values (including the sign of a zero).
#include "ptd_common.hpp"

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ uint64_t make_key(uint32_t bits, uint32_t idx) {
  if (bits == 0x80000000u) bits = 0u;  // -0.0 ties with +0.0
  const uint32_t ord = (bits & 0x80000000u) ? ~bits : (bits | 0x80000000u);
  return (static_cast<uint64_t>(ord) << 32) | static_cast<uint32_t>(~idx);
}
__device__ __forceinline__ uint32_t key_index(uint64_t key) {
  return ~static_cast<uint32_t>(key);
}

// Order-preserving image of a float (the upper half of a key): larger value
// <=> larger image, -0 maps like +0.  Empty list slots hold 0, below every
// real value (including -inf).
__device__ __forceinline__ uint32_t ord_of(float x) {
  uint32_t bits = __float_as_uint(x);
  if (bits == 0x80000000u) bits = 0u;
  return (bits & 0x80000000u) ? ~bits : (bits | 0x80000000u);
}
template <int KMAX>
__device__ __forceinline__ void insert(uint64_t (&l)[KMAX], uint64_t key) {
  if (key > l[KMAX - 1]) {
    l[KMAX - 1] = key;
#pragma unroll
    for (int j = KMAX - 1; j > 0; --j) {
      if (l[j] > l[j - 1]) {
        const uint64_t t = l[j];
        l[j] = l[j - 1];
        l[j - 1] = t;
      }
    }
  }
}

// Top-KMAX of two descending lists, left in `a` (descending): the
// elementwise max of a and reversed b is a bitonic sequence holding the top
// KMAX, which a bitonic merge network sorts.
template <int KMAX>
__device__ __forceinline__ void merge_lists(uint64_t (&a)[KMAX], const uint64_t (&b)[KMAX]) {
#pragma unroll
  for (int i = 0; i < KMAX; ++i) a[i] = a[i] > b[KMAX - 1 - i] ? a[i] : b[KMAX - 1 - i];
#pragma unroll
  for (int j = KMAX / 2; j > 0; j >>= 1)
#pragma unroll
    for (int i = 0; i < KMAX; ++i)
      if ((i & j) == 0 && a[i] < a[i + j]) {
        const uint64_t t = a[i];
        a[i] = a[i + j];
        a[i + j] = t;
      }
}

// After the butterfly every lane holds the wave's top KMAX, descending.
template <int KMAX>
__device__ __forceinline__ void wave_merge(uint64_t (&l)[KMAX]) {
#pragma unroll
  for (int o = 1; o < PTD_WAVE; o <<= 1) {
    uint64_t other[KMAX];
#pragma unroll
    for (int i = 0; i < KMAX; ++i) other[i] = ptd::shfl_xor_u64(l[i], o);
    merge_lists<KMAX>(l, other);
  }
}

template <bool BF16>
__device__ __forceinline__ uint32_t elem_bits(const void* base, size_t i) {
  if constexpr (BF16) return static_cast<uint32_t>(static_cast<const uint16_t*>(base)[i]) << 16;
  else return static_cast<const uint32_t*>(base)[i];
}

template <bool BF16>
__device__ __forceinline__ float elem_value(const void* base, size_t i) {
  return __uint_as_float(elem_bits<BF16>(base, i));
}

// Final results of one row from its KMAX best keys (key r held by lane r).
// (k <= V makes every emitted key a real element; the bound check only keeps
// the value re-read inside the row whatever the key.)
template <bool BF16>
__device__ __forceinline__ void emit(uint64_t key, int lane, int k, int V, const void* row_base,
                                     int row, int32_t* argmax, int32_t* topk_idx,
                                     float* topk_val) {
  const uint32_t idx = key_index(key);
  const bool real = idx < static_cast<uint32_t>(V);
  if (lane == 0) argmax[row] = real ? static_cast<int32_t>(idx) : -1;
  if (lane < k) {
    if (topk_idx) topk_idx[static_cast<size_t>(row) * k + lane] = real ? static_cast<int32_t>(idx) : -1;
    if (topk_val) topk_val[static_cast<size_t>(row) * k + lane] = real ? elem_value<BF16>(row_base, idx) : 0.f;
  }
}

// One workgroup (16 waves) per (row, slice), a slice being at most kRowLoads
// 16-byte loads per lane, all issued before any is consumed.
//   1. Every lane takes the maximum of each of its chunks and of all of them.
//   2. A lower bound tau of the slice's KMAX-th best value: the lanes of a
//      wave form KMAX groups; each group's largest lane maximum is a distinct
//      element, so the least of the KMAX group maxima is at most the KMAX-th
//      best value.  The bound of the slice is the largest bound of its waves.
//   3. Elements whose image reaches tau (few, for any spread of values) are
//      appended to a candidate list in LDS, and one wave selects the KMAX
//      best of the list.  If the list overflows (many values tied at the
//      top), every lane instead keeps a sorted list of its best keys among
//      those elements, re-read from memory, and the lists are merged.
constexpr int kRowThreads = 1024;
constexpr int kRowLoads = 16;   // 16-byte loads per lane per slice
constexpr int kCandCap = 1024;  // LDS candidate list

template <int KMAX, bool BF16>
__device__ __forceinline__ void chunk_elems(const uint4& c, float (&x)[BF16 ? 8 : 4]) {
  const uint32_t ws[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
  for (int e = 0; e < (BF16 ? 8 : 4); ++e) {
    if constexpr (BF16) x[e] = (e & 1) ? ptd::bf16_hi(ws[e >> 1]) : ptd::bf16_lo(ws[e >> 1]);
    else x[e] = __uint_as_float(ws[e]);
  }
}

template <int KMAX, bool BF16>
__global__ void __launch_bounds__(kRowThreads)
k_topk_row(const void* __restrict__ logits, int V, long long ld, int slices, int slice_len,
           int k, int32_t* __restrict__ argmax, int32_t* __restrict__ topk_idx,
           float* __restrict__ topk_val, uint64_t* __restrict__ part) {
  constexpr int E = BF16 ? 8 : 4;  // elements per 16-byte chunk
  constexpr int NW = kRowThreads / PTD_WAVE;
  constexpr int GL = PTD_WAVE / KMAX;  // lanes per group
  __shared__ uint64_t s_cand[kCandCap];
  __shared__ uint32_t s_tau[NW];
  __shared__ int s_cnt;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int row = blockIdx.x / slices, s = blockIdx.x % slices;
  const int v0 = s * slice_len;
  const int v1 = min(V, v0 + slice_len);
  const void* rb = BF16 ? static_cast<const void*>(static_cast<const uint16_t*>(logits) + row * ld)
                        : static_cast<const void*>(static_cast<const float*>(logits) + row * ld);
  const int nfull = (v1 - v0) / E;  // whole chunks; chunk j = tid + u * kRowThreads
  const int vt = v0 + nfull * E + tid;  // the slice's last partial chunk, one element per lane
  const bool tail = vt < v1;
  if (tid == 0) s_cnt = 0;
  uint4 w[kRowLoads];
#pragma unroll
  for (int u = 0; u < kRowLoads; ++u) {
    const int j = tid + u * kRowThreads;
    if (j < nfull) {
      const int v = v0 + j * E;
      w[u] = BF16 ? *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(rb) + v)
                  : *reinterpret_cast<const uint4*>(static_cast<const float*>(rb) + v);
    }
  }
  const float xt = tail ? __uint_as_float(elem_bits<BF16>(rb, vt)) : 0.f;

  // 1. chunk and lane maxima, as images (0 = no element)
  uint32_t cm[kRowLoads];
  uint32_t lm = tail ? ord_of(xt) : 0u;
#pragma unroll
  for (int u = 0; u < kRowLoads; ++u) {
    cm[u] = 0;
    if (tid + u * kRowThreads < nfull) {
      float x[E];
      chunk_elems<KMAX, BF16>(w[u], x);
      float m = x[0];
#pragma unroll
      for (int e = 1; e < E; ++e) m = fmaxf(m, x[e]);
      cm[u] = ord_of(m);
      lm = max(lm, cm[u]);
    }
  }
  // 2. the bound: max over the lane groups, then min over the groups
  uint32_t g = lm;
#pragma unroll
  for (int o = 1; o < GL; o <<= 1) g = max(g, static_cast<uint32_t>(__shfl_xor(static_cast<int>(g), o, PTD_WAVE)));
#pragma unroll
  for (int o = GL; o < PTD_WAVE; o <<= 1) g = min(g, static_cast<uint32_t>(__shfl_xor(static_cast<int>(g), o, PTD_WAVE)));
  if (lane == 0) s_tau[wave] = g;
  __syncthreads();
  uint32_t tau = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) tau = max(tau, s_tau[i]);

  // 3. collect the elements that reach tau
#pragma unroll
  for (int u = 0; u < kRowLoads; ++u) {
    if (cm[u] >= tau && cm[u] != 0) {
      float x[E];
      chunk_elems<KMAX, BF16>(w[u], x);
      const int v = v0 + (tid + u * kRowThreads) * E;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        if (ord_of(x[e]) >= tau) {
          const int pos = atomicAdd(&s_cnt, 1);
          if (pos < kCandCap) s_cand[pos] = make_key(__float_as_uint(x[e]), static_cast<uint32_t>(v + e));
        }
      }
    }
  }
  if (tail && ord_of(xt) >= tau) {
    const int pos = atomicAdd(&s_cnt, 1);
    if (pos < kCandCap) s_cand[pos] = make_key(__float_as_uint(xt), static_cast<uint32_t>(vt));
  }
  __syncthreads();
  int n = s_cnt;
  uint64_t l[KMAX];
#pragma unroll
  for (int j = 0; j < KMAX; ++j) l[j] = 0;
  if (n > kCandCap) {  // uniform over the workgroup
    for (int j = tid; j < nfull; j += kRowThreads) {
      const int v = v0 + j * E;
      const uint4 c = BF16 ? *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(rb) + v)
                           : *reinterpret_cast<const uint4*>(static_cast<const float*>(rb) + v);
      float x[E];
      chunk_elems<KMAX, BF16>(c, x);
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const uint64_t key = make_key(__float_as_uint(x[e]), static_cast<uint32_t>(v + e));
        if (ord_of(x[e]) >= tau && key > l[KMAX - 1]) insert<KMAX>(l, key);
      }
    }
    if (tail) {
      const uint64_t key = make_key(__float_as_uint(xt), static_cast<uint32_t>(vt));
      if (key > l[KMAX - 1]) insert<KMAX>(l, key);
    }
    wave_merge<KMAX>(l);
    if (lane < KMAX) {
      uint64_t mine = 0;
#pragma unroll
      for (int r = 0; r < KMAX; ++r) mine = (lane == r) ? l[r] : mine;
      s_cand[wave * KMAX + lane] = mine;
    }
    __syncthreads();
    n = NW * KMAX;
#pragma unroll
    for (int j = 0; j < KMAX; ++j) l[j] = 0;
  }
  if (wave != 0) return;
  for (int i = lane; i < n; i += PTD_WAVE) insert<KMAX>(l, s_cand[i]);
  wave_merge<KMAX>(l);
  uint64_t mine = 0;
#pragma unroll
  for (int r = 0; r < KMAX; ++r) mine = (lane == r) ? l[r] : mine;
  if (slices == 1) {
    emit<BF16>(mine, lane, k, V, rb, row, argmax, topk_idx, topk_val);
  } else if (lane < KMAX) {
    part[static_cast<size_t>(blockIdx.x) * KMAX + lane] = mine;
  }
}

// Rows that are not 16-byte aligned: one wave per (row, slice), element loads.
template <int KMAX, bool BF16>
__global__ void __launch_bounds__(kThreads)
k_topk_scalar(const void* __restrict__ logits, int R, int V, long long ld, int slices,
              int slice_len, int k, int32_t* __restrict__ argmax, int32_t* __restrict__ topk_idx,
              float* __restrict__ topk_val, uint64_t* __restrict__ part) {
  const int lane = threadIdx.x & 63;
  const int item = blockIdx.x * (kThreads / PTD_WAVE) + (threadIdx.x >> 6);
  if (item >= R * slices) return;  // whole wave
  const int row = item / slices, s = item % slices;
  const int v0 = s * slice_len;
  const int v1 = min(V, v0 + slice_len);
  const void* rb = BF16 ? static_cast<const void*>(static_cast<const uint16_t*>(logits) + row * ld)
                        : static_cast<const void*>(static_cast<const float*>(logits) + row * ld);
  uint64_t l[KMAX];
#pragma unroll
  for (int j = 0; j < KMAX; ++j) l[j] = 0;
  for (int v = v0 + lane; v < v1; v += PTD_WAVE) {
    const uint64_t key = make_key(elem_bits<BF16>(rb, v), static_cast<uint32_t>(v));
    if (key > l[KMAX - 1]) insert<KMAX>(l, key);
  }
  wave_merge<KMAX>(l);
  uint64_t mine = 0;
#pragma unroll
  for (int r = 0; r < KMAX; ++r) mine = (lane == r) ? l[r] : mine;
  if (slices == 1) {
    emit<BF16>(mine, lane, k, V, rb, row, argmax, topk_idx, topk_val);
  } else if (lane < KMAX) {
    part[static_cast<size_t>(item) * KMAX + lane] = mine;
  }
}

template <int KMAX, bool BF16>
__global__ void __launch_bounds__(kThreads)
k_topk_merge(const void* __restrict__ logits, int R, int V, long long ld, int slices, int k,
             const uint64_t* __restrict__ part, int32_t* __restrict__ argmax,
             int32_t* __restrict__ topk_idx, float* __restrict__ topk_val) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * (kThreads / PTD_WAVE) + (threadIdx.x >> 6);
  if (row >= R) return;  // whole wave
  uint64_t l[KMAX];
#pragma unroll
  for (int j = 0; j < KMAX; ++j) l[j] = 0;
  const uint64_t* pr = part + static_cast<size_t>(row) * slices * KMAX;
  for (int j = lane; j < slices * KMAX; j += PTD_WAVE) insert<KMAX>(l, pr[j]);
  wave_merge<KMAX>(l);
  uint64_t mine = 0;
#pragma unroll
  for (int r = 0; r < KMAX; ++r) mine = (lane == r) ? l[r] : mine;
  const void* rb = BF16 ? static_cast<const void*>(static_cast<const uint16_t*>(logits) + row * ld)
                        : static_cast<const void*>(static_cast<const float*>(logits) + row * ld);
  emit<BF16>(mine, lane, k, V, rb, row, argmax, topk_idx, topk_val);
}

struct TopkPlan {
  int kmax, slices, slice_len;
  bool vec;  // 16-byte aligned rows: k_topk_row, else k_topk_scalar
  size_t ws_bytes;
};

bool make_topk_plan(int R, int V, int k, int elem_bytes, bool vec, TopkPlan* p) {
  if (R < 1 || V < 1 || k < 1 || k > PTD_MAX_K || k > V) return false;
  p->kmax = k <= 1 ? 1 : k <= 2 ? 2 : k <= 4 ? 4 : k <= 8 ? 8 : 16;
  p->vec = vec;
  const int E = 16 / elem_bytes;
  // a slice is at most one batch of loads per lane: a whole row per
  // workgroup when it fits, so that no merge launch follows
  const long long max_len = static_cast<long long>(kRowThreads) * kRowLoads * E;
  int s = static_cast<int>((V + max_len - 1) / max_len);
  int len = (V + s - 1) / s;
  len = (len + 7) & ~7;  // keep slice starts 16-byte aligned
  s = (V + len - 1) / len;
  if (static_cast<long long>(R) * s > (1LL << 30)) return false;
  p->slices = s;
  p->slice_len = len;
  p->ws_bytes = s > 1 ? static_cast<size_t>(R) * s * p->kmax * sizeof(uint64_t) : 0;
  return true;
}

template <int KMAX, bool BF16>
void launch(const TopkPlan& pl, const void* logits, int R, int V, long long ld, int k,
            int32_t* am, int32_t* ti, float* tv, uint64_t* part, hipStream_t st) {
  constexpr int WPB = kThreads / PTD_WAVE;
  if (pl.vec)
    hipLaunchKernelGGL((k_topk_row<KMAX, BF16>), dim3(R * pl.slices), dim3(kRowThreads), 0, st,
                       logits, V, ld, pl.slices, pl.slice_len, k, am, ti, tv, part);
  else
    hipLaunchKernelGGL((k_topk_scalar<KMAX, BF16>), dim3((R * pl.slices + WPB - 1) / WPB),
                       dim3(kThreads), 0, st, logits, R, V, ld, pl.slices, pl.slice_len, k, am,
                       ti, tv, part);
  if (pl.slices > 1)
    hipLaunchKernelGGL((k_topk_merge<KMAX, BF16>), dim3((R + WPB - 1) / WPB), dim3(kThreads), 0,
                       st, logits, R, V, ld, pl.slices, k, part, am, ti, tv);
}

template <bool BF16>
void dispatch(const TopkPlan& pl, const void* logits, int R, int V, long long ld, int k,
              int32_t* am, int32_t* ti, float* tv, uint64_t* part, hipStream_t st) {
  switch (pl.kmax) {
    case 1: launch<1, BF16>(pl, logits, R, V, ld, k, am, ti, tv, part, st); break;
    case 2: launch<2, BF16>(pl, logits, R, V, ld, k, am, ti, tv, part, st); break;
    case 4: launch<4, BF16>(pl, logits, R, V, ld, k, am, ti, tv, part, st); break;
    case 8: launch<8, BF16>(pl, logits, R, V, ld, k, am, ti, tv, part, st); break;
    default: launch<16, BF16>(pl, logits, R, V, ld, k, am, ti, tv, part, st); break;
  }
}

}  // namespace

extern "C" size_t ptd_topk_workspace_bytes(int32_t R, int32_t V, int32_t k) {
  // the dtype is not known here: size for the larger of the bf16 and fp32 plans
  TopkPlan p2, p4;
  if (!make_topk_plan(R, V, k, 2, true, &p2) || !make_topk_plan(R, V, k, 4, true, &p4)) return 0;
  return p2.ws_bytes > p4.ws_bytes ? p2.ws_bytes : p4.ws_bytes;
}

extern "C" int ptd_topk_argmax(const void* logits, ptd_dtype dtype, int32_t R, int32_t V,
                               int64_t ld, int32_t k, int32_t* argmax, int32_t* topk_idx,
                               float* topk_val, void* workspace, size_t workspace_bytes,
                               void* stream) {
  PTD_RETURN_IF(!logits || !argmax, PTD_ERR_NULL);
  PTD_RETURN_IF(dtype != PTD_F32 && dtype != PTD_BF16, PTD_ERR_DTYPE);
  PTD_RETURN_IF(ld < V, PTD_ERR_SHAPE);
  const size_t es = dtype == PTD_BF16 ? 2 : 4;
  PTD_RETURN_IF(!ptd_aligned(logits, es), PTD_ERR_ALIGN);
  const bool vec = ptd_aligned(logits, 16) && (static_cast<size_t>(ld) * es) % 16 == 0;
  TopkPlan pl;
  PTD_RETURN_IF(!make_topk_plan(R, V, k, static_cast<int>(es), vec, &pl), PTD_ERR_SHAPE);
  if (pl.ws_bytes) {
    PTD_RETURN_IF(!workspace || workspace_bytes < pl.ws_bytes, PTD_ERR_WORKSPACE);
    PTD_RETURN_IF(!ptd_aligned(workspace, 8), PTD_ERR_ALIGN);
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint64_t* part = static_cast<uint64_t*>(workspace);
  if (dtype == PTD_BF16)
    dispatch<true>(pl, logits, R, V, ld, k, argmax, topk_idx, topk_val, part, st);
  else
    dispatch<false>(pl, logits, R, V, ld, k, argmax, topk_idx, topk_val, part, st);
  return ptd_launch_status();
}
