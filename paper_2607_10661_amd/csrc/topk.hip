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
//                   at most 4096 chunks of 16 bytes (32768 bf16 or 16384
//                   fp32 values; 6144 chunks for a few long rows) held in
//                   registers (1024 threads x 4 or 6 chunks, or 512 x 8 when
//                   there are many slices): a cheap lower
//                   bound of the KMAX-th best value leaves a few candidates,
//                   ranked by counting (details below).
//   k_topk_scalar   rows that are not 16-byte aligned: one wave per (row,
//                   slice) with element loads; each lane keeps a sorted list
//                   of its KMAX best keys in registers.
// Sorted lists are merged by a butterfly of 6 steps per wave, each merging two
// sorted lists with a bitonic network.
//   k_topk_merge    one workgroup per row ranks the slice results by counting
//                   (only when a row spans several slices).
// A slice result is KMAX (key, value bits) pairs in the workspace.  topk_val
// carries the row's own values (including the sign of a zero): candidates
// keep their bits; the rare paths that hold only keys re-read the logits.
#include <algorithm>

#include "ptd_async.hpp"
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

// Slot r of slice result `item` from a key alone (value bits re-read).
template <bool BF16>
__device__ __forceinline__ void store_part(uint64_t* part, int item, int kmax, int r, uint64_t key,
                                           const void* row_base) {
  uint64_t* q = part + (static_cast<size_t>(item) * kmax + r) * 2;
  q[0] = key;
  q[1] = key ? elem_bits<BF16>(row_base, key_index(key)) : 0u;
}

// One workgroup of NT threads per (row, slice), a slice being at most one
// batch of NL chunks of 16 bytes per lane (NT * NL * 16 bytes), loaded
// straight into registers.
//   1. Every lane takes the image of each of its chunks (bf16 images are 16
//      bits wide and computed two at a time with packed 16-bit integer
//      operations) and their maximum.
//   2. A lower bound tau of the slice's KMAX-th best value: the lanes of a
//      wave form KMAX groups; each group's largest lane maximum is a distinct
//      element, so the least of the KMAX group maxima is at most the KMAX-th
//      best value.  The bound of the slice is the largest bound of its waves.
//   3. Chunks whose image reaches tau are copied with their index to a list
//      in LDS, then the workgroup examines the listed chunks a thread per
//      element and appends the elements that reach tau to a candidate list.
//      The slice's last partial chunk (fewer than one chunk of elements) is
//      read with plain loads and checked the same way.
//   4. The candidates are ranked by counting: the list is cut into parts,
//      each thread counts the keys of one part above one candidate, and the
//      counts are summed in LDS.  The candidates of rank below k are the
//      result.  If either list overflows (many values tied at the top), every
//      lane keeps a sorted list of its best keys among its own elements that
//      reach tau, and the lists are merged.
// Only listed chunks pass through LDS, so the slice is read from memory once
// and LDS carries a few KB.  The kernel's loops stay rolled, which keeps its
// code small: its instructions are fetched once per CU, cold.
constexpr int kCandCap = 256;                            // LDS candidate list
constexpr int kListCap = 256;                            // LDS chunk list

using s16x2 = short __attribute__((ext_vector_type(2)));

// Images: order-preserving integers, 0 reserved for "no element".
//   fp32: ord_of (-0 maps like +0).
//   bf16: 0x8001 + v, v the 16-bit signed-order value (sign-magnitude turned
//         into two's complement order by flipping the magnitude bits of
//         negative values).  -0 maps one below +0, so a bound equal to the
//         image of +0 is lowered to that of -0 before elements are compared.
constexpr uint32_t kImgPosZeroBf16 = 0x8001u;
__device__ __forceinline__ s16x2 sorder2(uint32_t d) {
  const s16x2 v = __builtin_bit_cast(s16x2, d);
  const s16x2 sg = v >> static_cast<short>(15);
  return __builtin_bit_cast(s16x2, d ^ (__builtin_bit_cast(uint32_t, sg) & 0x7FFF7FFFu));
}
template <bool BF16>
__device__ __forceinline__ uint32_t elem_img(uint32_t bits32) {  // bits of the fp32 value
  if constexpr (BF16) {
    const short h = static_cast<short>(bits32 >> 16);
    const short o = static_cast<short>(h ^ ((h >> 15) & 0x7FFF));
    return static_cast<uint32_t>(static_cast<int>(o) + 0x8001);
  } else {
    return ord_of(__uint_as_float(bits32));
  }
}
template <bool BF16>
__device__ __forceinline__ uint32_t chunk_img(const uint4& c) {
  if constexpr (BF16) {
    const s16x2 m = __builtin_elementwise_max(__builtin_elementwise_max(sorder2(c.x), sorder2(c.y)),
                                              __builtin_elementwise_max(sorder2(c.z), sorder2(c.w)));
    return static_cast<uint32_t>(max(static_cast<int>(m.x), static_cast<int>(m.y)) + 0x8001);
  } else {
    return ord_of(fmaxf(fmaxf(__uint_as_float(c.x), __uint_as_float(c.y)),
                        fmaxf(__uint_as_float(c.z), __uint_as_float(c.w))));
  }
}
// fp32 bits of element e of a chunk
template <bool BF16>
__device__ __forceinline__ uint32_t chunk_bits(const uint4& c, int e) {
  const uint32_t ws[4] = {c.x, c.y, c.z, c.w};
  if constexpr (BF16) return (e & 1) ? (ws[e >> 1] & 0xFFFF0000u) : (ws[e >> 1] << 16);
  else return ws[e];
}
// bound used in comparisons (see the bf16 image above)
template <bool BF16>
__device__ __forceinline__ uint32_t cmp_bound(uint32_t tau) {
  return (BF16 && tau == kImgPosZeroBf16) ? tau - 1 : tau;
}

// Cross-lane steps of a wave on the vector ALU, level j pairing lanes that
// differ in bit j: quad permutes (j = 0, 1), the half-row and row mirrors
// (j = 2, 3: once the value is uniform over blocks of 2^j lanes, the mirror
// partner lies in the other block), v_permlane16_swap / v_permlane32_swap
// (j = 4, 5: with both operands holding the value, the two results are the
// lane's value and its partner's).
template <bool MAX, int J>
__device__ __forceinline__ uint32_t lane_step(uint32_t x) {
  constexpr int kCtrl[4] = {0xB1, 0x4E, 0x141, 0x140};  // quad_perm 1032, 2301, half-row, row mirror
  if constexpr (J < 4) {
    const uint32_t y = static_cast<uint32_t>(
        __builtin_amdgcn_update_dpp(static_cast<int>(x), static_cast<int>(x), kCtrl[J], 0xF, 0xF, false));
    return MAX ? max(x, y) : min(x, y);
  } else {
    const auto r = J == 4 ? __builtin_amdgcn_permlane16_swap(x, x, false, false)
                          : __builtin_amdgcn_permlane32_swap(x, x, false, false);
    return MAX ? max(r[0], r[1]) : min(r[0], r[1]);
  }
}
// Maximum over aligned groups of GL lanes, then minimum over the groups.
template <int GL>
__device__ __forceinline__ uint32_t group_max_min(uint32_t x) {
  if constexpr (GL > 1) x = lane_step<true, 0>(x); else x = lane_step<false, 0>(x);
  if constexpr (GL > 2) x = lane_step<true, 1>(x); else x = lane_step<false, 1>(x);
  if constexpr (GL > 4) x = lane_step<true, 2>(x); else x = lane_step<false, 2>(x);
  if constexpr (GL > 8) x = lane_step<true, 3>(x); else x = lane_step<false, 3>(x);
  if constexpr (GL > 16) x = lane_step<true, 4>(x); else x = lane_step<false, 4>(x);
  if constexpr (GL > 32) x = lane_step<true, 5>(x); else x = lane_step<false, 5>(x);
  return x;
}

template <int KMAX, bool BF16, int NT, int NL>
__global__ void __launch_bounds__(NT)
k_topk_row(const void* __restrict__ logits, int V, long long ld, int slices, int slice_len,
           int k, int32_t* __restrict__ argmax, int32_t* __restrict__ topk_idx,
           float* __restrict__ topk_val, uint64_t* __restrict__ part) {
  constexpr int E = BF16 ? 8 : 4;  // elements per 16-byte chunk
  constexpr int ES = BF16 ? 2 : 4;
  constexpr int NW = NT / PTD_WAVE;
  static_assert(NT >= kCandCap && NW % 4 == 0 && NT * NL <= 65536, "workgroup shape");
  static_assert((NT & (NT - 1)) == 0, "KMAX groups of NT / KMAX lanes");
  constexpr int GL = PTD_WAVE / KMAX;  // lanes per group inside a wave
  constexpr int GW = NT / KMAX;        // lanes per group across the workgroup
  constexpr int GWL = GW < PTD_WAVE ? GW : PTD_WAVE;  // ... of them inside one wave
  constexpr int WPG = GW / GWL;        // waves per workgroup-wide group
  __shared__ __attribute__((aligned(16))) uint4 s_ldata[kListCap];
  __shared__ uint64_t s_cand[kCandCap];
  __shared__ uint32_t s_bits[kCandCap];
  __shared__ uint32_t s_rank[kCandCap];
  __shared__ uint16_t s_list[kListCap];
  __shared__ __attribute__((aligned(16))) uint32_t s_tau[NW];
  __shared__ __attribute__((aligned(16))) uint32_t s_tau2[NW];
  __shared__ int s_nlist, s_cnt;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int row = blockIdx.x / slices, s = blockIdx.x % slices;
  const int v0 = s * slice_len;
  const int v1 = min(V, v0 + slice_len);
  const char* rb = static_cast<const char*>(logits) + static_cast<size_t>(row) * ld * ES;
  const char* sb = rb + static_cast<size_t>(v0) * ES;  // the slice, 16-byte aligned
  const int nfull = (v1 - v0) / E;  // whole chunks of the slice (at most NT * NL)
  const int vt = v0 + nfull * E + tid;  // the last partial chunk, one element per lane
  const bool tail = vt < v1;

  // Chunk u of a lane is u * NT + tid (past the end: the slice's
  // last chunk, never examined); all loads are issued before any wait.
  uint4 cw[NL];
  if (nfull > 0) {
    const uint4* src = reinterpret_cast<const uint4*>(sb);
#pragma unroll
    for (int u = 0; u < NL; ++u) cw[u] = src[min(u * NT + tid, nfull - 1)];
  } else {
#pragma unroll
    for (int u = 0; u < NL; ++u) cw[u] = make_uint4(0u, 0u, 0u, 0u);
  }
  const uint32_t bt = tail ? elem_bits<BF16>(rb, vt) : 0u;
  if (tid < kCandCap) s_rank[tid] = 0;
  if (tid == 0) {
    s_cnt = 0;
    s_nlist = 0;
  }

  // 1. chunk images and the lane maximum
  uint32_t cm[NL];
  uint32_t lm = tail ? elem_img<BF16>(bt) : 0u;
#pragma unroll
  for (int u = 0; u < NL; ++u) {
    cm[u] = u * NT + tid < nfull ? chunk_img<BF16>(cw[u]) : 0u;
    lm = max(lm, cm[u]);
  }
  // 2. the bound, the larger of two: per wave, max over groups of GL lanes
  //    then min over the wave's KMAX groups, and the largest of these over
  //    the waves; and min over KMAX groups of NT / KMAX lanes spanning the
  //    workgroup of the group maxima (much closer to the KMAX-th best value
  //    of the slice, hence few candidates; the first stays positive where a
  //    short slice leaves whole workgroup-wide groups empty)
  const uint32_t g = group_max_min<GL>(lm);
  const uint32_t g2 = group_max_min<GWL>(lm);  // GWL = 64: the wave's maximum
  if (lane == 0) {
    s_tau[wave] = g;
    s_tau2[wave] = g2;
  }
  ptd::lds_barrier();
  uint32_t tau = 0;
#pragma unroll
  for (int i = 0; i < NW; i += 4) {
    const uint4 t4 = *reinterpret_cast<const uint4*>(s_tau + i);
    tau = max(max(tau, max(t4.x, t4.y)), max(t4.z, t4.w));
  }
  uint32_t tau2 = ~0u;
#pragma unroll
  for (int j = 0; j < NW / WPG; ++j) {
    uint32_t gm = 0;
#pragma unroll
    for (int w = 0; w < WPG; ++w) gm = max(gm, s_tau2[j * WPG + w]);
    tau2 = min(tau2, gm);
  }
  tau = max(tau, tau2);
  const uint32_t tc = cmp_bound<BF16>(tau);

  // 3. list the chunks that reach the bound, then examine them
  auto append = [&](uint32_t bits, int v) {
    const int pos = atomicAdd(&s_cnt, 1);
    if (pos < kCandCap) {
      s_cand[pos] = make_key(bits, static_cast<uint32_t>(v));
      s_bits[pos] = bits;
    }
  };
#pragma unroll
  for (int u = 0; u < NL; ++u) {
    if (cm[u] != 0 && cm[u] >= tc) {
      const int pos = atomicAdd(&s_nlist, 1);
      if (pos < kListCap) {
        s_ldata[pos] = cw[u];
        s_list[pos] = static_cast<uint16_t>(u * NT + tid);
      }
    }
  }
  if (tail && elem_img<BF16>(bt) >= tc) append(bt, vt);
  ptd::lds_barrier();
  const int nl = s_nlist;
  if (nl <= kListCap) {  // uniform
    for (int i0 = 0; i0 < nl; i0 += NT / E) {
      const int i = i0 + tid / E;
      if (i < nl) {
        const int c = s_list[i], e = tid & (E - 1);
        const uint32_t bits = BF16 ? static_cast<uint32_t>(reinterpret_cast<const uint16_t*>(s_ldata + i)[e]) << 16
                                   : reinterpret_cast<const uint32_t*>(s_ldata + i)[e];
        if (elem_img<BF16>(bits) >= tc) append(bits, v0 + c * E + e);
      }
    }
  }
  __syncthreads();
  const int n = s_cnt;

  // 4. selection
  if (nl <= kListCap && n <= kCandCap) {  // uniform over the workgroup
    int n2 = PTD_WAVE;  // candidates per part-set: a power of two >= n
    while (n2 < n) n2 <<= 1;
    const int parts = NT / n2;
    const int i = tid & (n2 - 1), p = tid / n2;  // p is uniform over a wave
    const int len = (n + parts - 1) / parts;
    const int j0 = p * len, j1 = min(n, j0 + len);
    const uint64_t mine = i < n ? s_cand[i] : ~0ull;
    uint32_t above = 0;
    for (int j = j0; j < j1; ++j) above += s_cand[j] > mine ? 1u : 0u;
    if (above) atomicAdd(&s_rank[i], above);
    __syncthreads();
    if (tid < n) {
      const uint32_t rank = s_rank[tid];
      const uint64_t key = s_cand[tid];
      if (slices == 1) {
        const int32_t idx = static_cast<int32_t>(key_index(key));
        if (rank == 0) argmax[row] = idx;
        if (rank < static_cast<uint32_t>(k)) {
          if (topk_idx) topk_idx[static_cast<size_t>(row) * k + rank] = idx;
          if (topk_val) topk_val[static_cast<size_t>(row) * k + rank] = __uint_as_float(s_bits[tid]);
        }
      } else if (rank < static_cast<uint32_t>(KMAX)) {
        uint64_t* q = part + (static_cast<size_t>(blockIdx.x) * KMAX + rank) * 2;
        q[0] = key;
        q[1] = s_bits[tid];
      }
    } else if (slices > 1 && tid < KMAX) {  // fewer candidates than KMAX: empty slots
      uint64_t* q = part + (static_cast<size_t>(blockIdx.x) * KMAX + tid) * 2;
      q[0] = 0;
      q[1] = 0;
    }
    return;
  }

  // overflow: per-lane sorted lists of the lane's own elements that reach tau
  uint64_t l[KMAX];
#pragma unroll
  for (int j = 0; j < KMAX; ++j) l[j] = 0;
#pragma unroll
  for (int u = 0; u < NL; ++u) {
    const int c = u * NT + tid;
    if (c < nfull) {
      const int v = v0 + c * E;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const uint32_t bits = chunk_bits<BF16>(cw[u], e);
        const uint64_t key = make_key(bits, static_cast<uint32_t>(v + e));
        if (elem_img<BF16>(bits) >= tc && key > l[KMAX - 1]) insert<KMAX>(l, key);
      }
    }
  }
  if (tail) {
    const uint64_t key = make_key(bt, static_cast<uint32_t>(vt));
    if (key > l[KMAX - 1]) insert<KMAX>(l, key);
  }
  wave_merge<KMAX>(l);
  if (lane < KMAX) {
    uint64_t mine = 0;
#pragma unroll
    for (int r = 0; r < KMAX; ++r) mine = (lane == r) ? l[r] : mine;
    s_cand[wave * KMAX + lane] = mine;  // every wave is past its reads of s_cand
  }
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int j = 0; j < KMAX; ++j) l[j] = 0;
  for (int i = lane; i < NW * KMAX; i += PTD_WAVE) insert<KMAX>(l, s_cand[i]);
  wave_merge<KMAX>(l);
  uint64_t mine = 0;
#pragma unroll
  for (int r = 0; r < KMAX; ++r) mine = (lane == r) ? l[r] : mine;
  if (slices == 1) emit<BF16>(mine, lane, k, V, rb, row, argmax, topk_idx, topk_val);
  else if (lane < KMAX) store_part<BF16>(part, blockIdx.x, KMAX, lane, mine, rb);
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
  if (slices == 1) emit<BF16>(mine, lane, k, V, rb, row, argmax, topk_idx, topk_val);
  else if (lane < KMAX) store_part<BF16>(part, item, KMAX, lane, mine, rb);
}

// One workgroup per row: the row's slices * KMAX (key, bits) pairs are ranked
// by counting like the candidates of k_topk_row (empty slots hold key 0,
// below every element, so they never reach a rank below k <= V).  Beyond
// kThreads pairs, wave 0 merges sorted lists instead.
template <int KMAX, bool BF16>
__global__ void __launch_bounds__(kThreads)
k_topk_merge(const void* __restrict__ logits, int V, long long ld, int slices, int k,
             const uint64_t* __restrict__ part, int32_t* __restrict__ argmax,
             int32_t* __restrict__ topk_idx, float* __restrict__ topk_val) {
  __shared__ uint64_t s_key[kThreads];
  __shared__ uint32_t s_rank[kThreads];
  const int tid = threadIdx.x, lane = tid & 63, row = blockIdx.x;
  const int n = slices * KMAX;
  const uint64_t* pr = part + static_cast<size_t>(row) * n * 2;
  if (n <= kThreads) {  // uniform
    uint64_t key = 0;
    uint32_t bits = 0;
    if (tid < n) {
      key = pr[2 * tid];
      bits = static_cast<uint32_t>(pr[2 * tid + 1]);
      s_key[tid] = key;
    }
    s_rank[tid] = 0;
    __syncthreads();
    int n2 = PTD_WAVE;
    while (n2 < n) n2 <<= 1;
    const int parts = kThreads / n2;
    const int i = tid & (n2 - 1), p = tid / n2;
    const int len = (n + parts - 1) / parts;
    const int j0 = p * len, j1 = min(n, j0 + len);
    const uint64_t mine = i < n ? s_key[i] : ~0ull;
    uint32_t above = 0;
    for (int j = j0; j < j1; ++j) above += s_key[j] > mine ? 1u : 0u;
    if (above) atomicAdd(&s_rank[i], above);
    __syncthreads();
    if (tid < n) {
      const uint32_t rank = s_rank[tid];
      if (rank < static_cast<uint32_t>(k)) {
        const int32_t idx = static_cast<int32_t>(key_index(key));
        if (rank == 0) argmax[row] = idx;
        if (topk_idx) topk_idx[static_cast<size_t>(row) * k + rank] = idx;
        if (topk_val) topk_val[static_cast<size_t>(row) * k + rank] = __uint_as_float(bits);
      }
    }
    return;
  }
  if (tid >= PTD_WAVE) return;
  uint64_t l[KMAX];
#pragma unroll
  for (int j = 0; j < KMAX; ++j) l[j] = 0;
  for (int j = lane; j < n; j += PTD_WAVE) insert<KMAX>(l, pr[2 * j]);
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
  int nt, nl;  // k_topk_row: threads per workgroup, 16-byte chunks per lane
  bool vec;  // 16-byte aligned rows: k_topk_row, else k_topk_scalar
  size_t ws_bytes;
};

// Workgroup shape of k_topk_row for R rows of V elements (E per chunk).
void topk_shape(int R, int V, int E, int* nt, int* nl) {
  // Many slices (at least four per CU): 512 threads of 8 chunks each, three
  // workgroups resident per CU and every lane's loads in flight at once
  // (measured on 1040 rows x 128256 bf16: 53.2 us against 72.9 us for
  // 1024 x 4).  Fewer: 1024 threads of 4 chunks, the shortest latency for a
  // slice (65 rows x 32000: 5.1 us against 5.1-7.2 us for the others), or of
  // 6 chunks when that leaves one slice per CU where 4 chunks would not
  // (65 rows x 128256: 3 slices per row, 9.2 against 9.9 us with the merge).
  const long long s4 = (static_cast<long long>(V) + 4096LL * E - 1) / (4096LL * E);
  if (static_cast<long long>(R) * s4 >= 4 * 256) {
    *nt = 512;
    *nl = 8;
  } else {
    const long long s6 = (static_cast<long long>(V) + 6144LL * E - 1) / (6144LL * E);
    *nt = 1024;
    *nl = (R * s4 > 256 && R * s6 <= 256) ? 6 : 4;
  }
}

bool make_topk_plan(int R, int V, int k, int elem_bytes, bool vec, TopkPlan* p) {
  if (R < 1 || V < 1 || k < 1 || k > PTD_MAX_K || k > V) return false;
  p->kmax = k <= 1 ? 1 : k <= 2 ? 2 : k <= 4 ? 4 : k <= 8 ? 8 : 16;
  p->vec = vec;
  const int E = 16 / elem_bytes;
  topk_shape(R, V, E, &p->nt, &p->nl);
  // A slice is at most nt * nl whole chunks (plus, for the last, a partial
  // chunk): rows longer than that are split and merged afterwards.
  const long long max_len = static_cast<long long>(p->nt) * p->nl * E;
  int s = static_cast<int>((V + max_len - 1) / max_len);
  int len = (V + s - 1) / s;
  len = (len + 7) & ~7;  // keep slice starts 16-byte aligned
  s = (V + len - 1) / len;
  if (static_cast<long long>(R) * s > (1LL << 30)) return false;
  p->slices = s;
  p->slice_len = len;
  p->ws_bytes = s > 1 ? static_cast<size_t>(R) * s * p->kmax * 2 * sizeof(uint64_t) : 0;
  return true;
}

template <int KMAX, bool BF16>
void launch(const TopkPlan& pl, const void* logits, int R, int V, long long ld, int k,
            int32_t* am, int32_t* ti, float* tv, uint64_t* part, hipStream_t st) {
  constexpr int WPB = kThreads / PTD_WAVE;
  if (pl.vec) {
#define PTD_TOPK_ROW(nt_, nl_)                                                                   \
  if (pl.nt == nt_ && pl.nl == nl_)                                                              \
    hipLaunchKernelGGL((k_topk_row<KMAX, BF16, nt_, nl_>), dim3(R * pl.slices), dim3(nt_), 0, st, \
                       logits, V, ld, pl.slices, pl.slice_len, k, am, ti, tv, part);
    PTD_TOPK_ROW(1024, 4) PTD_TOPK_ROW(1024, 6) PTD_TOPK_ROW(512, 8)
#undef PTD_TOPK_ROW
  } else
    hipLaunchKernelGGL((k_topk_scalar<KMAX, BF16>), dim3((R * pl.slices + WPB - 1) / WPB),
                       dim3(kThreads), 0, st, logits, R, V, ld, pl.slices, pl.slice_len, k, am,
                       ti, tv, part);
  if (pl.slices > 1)
    hipLaunchKernelGGL((k_topk_merge<KMAX, BF16>), dim3(R), dim3(kThreads), 0, st, logits, V, ld,
                       pl.slices, k, part, am, ti, tv);
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
