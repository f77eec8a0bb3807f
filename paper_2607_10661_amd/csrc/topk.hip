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
//   k_topk_partial  one wave per (row, vocabulary slice): each lane keeps a
//                   sorted list of its KMAX best keys in registers while it
//                   streams the slice with 16-byte loads (four in flight);
//                   the 64 lists are then merged by a butterfly of 6 steps,
//                   each merging two sorted lists with a bitonic network.
//   k_topk_merge    one wave per row merges the slice results the same way.
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

template <int KMAX, bool BF16, bool VEC>
__global__ void __launch_bounds__(kThreads)
k_topk_partial(const void* __restrict__ logits, int R, int V, long long ld, int slices,
               int slice_len, int k, int32_t* __restrict__ argmax,
               int32_t* __restrict__ topk_idx, float* __restrict__ topk_val,
               uint64_t* __restrict__ part) {
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

  if constexpr (VEC) {
    // 16-byte chunks j = lane, lane + 64, ...; U chunks per batch are loaded
    // (predicated) before any is consumed, so U loads are in flight per lane
    constexpr int E = BF16 ? 8 : 4;  // elements per 16-byte load
    constexpr int U = 4;
    const int nfull = (v1 - v0) / E;
    for (int j0 = 0; j0 < nfull; j0 += U * PTD_WAVE) {
      uint4 w[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = j0 + u * PTD_WAVE + lane;
        if (j < nfull) {
          const int v = v0 + j * E;
          w[u] = BF16 ? *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(rb) + v)
                      : *reinterpret_cast<const uint4*>(static_cast<const float*>(rb) + v);
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = j0 + u * PTD_WAVE + lane;
        if (j >= nfull) continue;
        const int v = v0 + j * E;
        const uint32_t ws[4] = {w[u].x, w[u].y, w[u].z, w[u].w};
#pragma unroll
        for (int e = 0; e < E; ++e) {
          uint32_t bits;
          if constexpr (BF16) bits = (e & 1) ? (ws[e >> 1] & 0xFFFF0000u) : (ws[e >> 1] << 16);
          else bits = ws[e];
          insert<KMAX>(l, make_key(bits, static_cast<uint32_t>(v + e)));
        }
      }
    }
    // the last partial chunk, one element per lane
    const int vt = v0 + nfull * E + lane;
    if (vt < v1) insert<KMAX>(l, make_key(elem_bits<BF16>(rb, vt), static_cast<uint32_t>(vt)));
  } else {
    for (int v = v0 + lane; v < v1; v += PTD_WAVE)
      insert<KMAX>(l, make_key(elem_bits<BF16>(rb, v), static_cast<uint32_t>(v)));
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
  size_t ws_bytes;
};

bool make_topk_plan(int R, int V, int k, TopkPlan* p) {
  if (R < 1 || V < 1 || k < 1 || k > PTD_MAX_K || k > V) return false;
  p->kmax = k <= 1 ? 1 : k <= 2 ? 2 : k <= 4 ? 4 : k <= 8 ? 8 : 16;
  // one wave per slice of ~4096 elements (eight 16-byte bf16 loads per lane)
  int s = (V + 4095) / 4096;
  if (s < 1) s = 1;
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
void launch(const TopkPlan& pl, bool vec, const void* logits, int R, int V, long long ld,
            int k, int32_t* am, int32_t* ti, float* tv, uint64_t* part, hipStream_t st) {
  constexpr int WPB = kThreads / PTD_WAVE;
  const dim3 grid((R * pl.slices + WPB - 1) / WPB);
  if (vec)
    hipLaunchKernelGGL((k_topk_partial<KMAX, BF16, true>), grid, dim3(kThreads), 0, st, logits, R,
                       V, ld, pl.slices, pl.slice_len, k, am, ti, tv, part);
  else
    hipLaunchKernelGGL((k_topk_partial<KMAX, BF16, false>), grid, dim3(kThreads), 0, st, logits,
                       R, V, ld, pl.slices, pl.slice_len, k, am, ti, tv, part);
  if (pl.slices > 1)
    hipLaunchKernelGGL((k_topk_merge<KMAX, BF16>), dim3((R + WPB - 1) / WPB), dim3(kThreads), 0,
                       st, logits, R, V, ld, pl.slices, k, part, am, ti, tv);
}

template <bool BF16>
void dispatch(const TopkPlan& pl, bool vec, const void* logits, int R, int V, long long ld, int k,
              int32_t* am, int32_t* ti, float* tv, uint64_t* part, hipStream_t st) {
  switch (pl.kmax) {
    case 1: launch<1, BF16>(pl, vec, logits, R, V, ld, k, am, ti, tv, part, st); break;
    case 2: launch<2, BF16>(pl, vec, logits, R, V, ld, k, am, ti, tv, part, st); break;
    case 4: launch<4, BF16>(pl, vec, logits, R, V, ld, k, am, ti, tv, part, st); break;
    case 8: launch<8, BF16>(pl, vec, logits, R, V, ld, k, am, ti, tv, part, st); break;
    default: launch<16, BF16>(pl, vec, logits, R, V, ld, k, am, ti, tv, part, st); break;
  }
}

}  // namespace

extern "C" size_t ptd_topk_workspace_bytes(int32_t R, int32_t V, int32_t k) {
  TopkPlan pl;
  if (!make_topk_plan(R, V, k, &pl)) return 0;
  return pl.ws_bytes;
}

extern "C" int ptd_topk_argmax(const void* logits, ptd_dtype dtype, int32_t R, int32_t V,
                               int64_t ld, int32_t k, int32_t* argmax, int32_t* topk_idx,
                               float* topk_val, void* workspace, size_t workspace_bytes,
                               void* stream) {
  PTD_RETURN_IF(!logits || !argmax, PTD_ERR_NULL);
  PTD_RETURN_IF(dtype != PTD_F32 && dtype != PTD_BF16, PTD_ERR_DTYPE);
  PTD_RETURN_IF(ld < V, PTD_ERR_SHAPE);
  TopkPlan pl;
  PTD_RETURN_IF(!make_topk_plan(R, V, k, &pl), PTD_ERR_SHAPE);
  const size_t es = dtype == PTD_BF16 ? 2 : 4;
  PTD_RETURN_IF(!ptd_aligned(logits, es), PTD_ERR_ALIGN);
  if (pl.ws_bytes) {
    PTD_RETURN_IF(!workspace || workspace_bytes < pl.ws_bytes, PTD_ERR_WORKSPACE);
    PTD_RETURN_IF(!ptd_aligned(workspace, 8), PTD_ERR_ALIGN);
  }
  const bool vec = ptd_aligned(logits, 16) && (static_cast<size_t>(ld) * es) % 16 == 0;
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint64_t* part = static_cast<uint64_t*>(workspace);
  if (dtype == PTD_BF16)
    dispatch<true>(pl, vec, logits, R, V, ld, k, argmax, topk_idx, topk_val, part, st);
  else
    dispatch<false>(pl, vec, logits, R, V, ld, k, argmax, topk_idx, topk_val, part, st);
  return ptd_launch_status();
}
