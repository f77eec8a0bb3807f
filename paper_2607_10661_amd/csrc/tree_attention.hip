// Tree-masked attention for one Progressive Tree Drafting step on gfx950.
//
// Sec. 3.1 "Tree Construction" + Sec. 3.2: every packed tree node attends to
// the committed prefix and to its own ancestors (pi(v) = {v} u pi(P(v))) only.
// For sequence b, KV head g and query row r = i*G + hg (node i, query head
// h = g*G + hg), the keys are cache rows [0, kv_len) plus kv_len + a for every
// ancestor-or-self a of node i; node i's own K/V row is kv_len + i.
//
// Kernels
//   k_attn_mfma    bf16 q/k/v.  One workgroup = (b, g, row pass, KV split);
//                  8 waves (2 per SIMD), each owning up to 32 query rows.  K/V
//                  stream HBM -> LDS with asynchronous copies into a ring of
//                  ten 32-key sub-tiles (all 160 KB of LDS), shared by every
//                  query row of the GQA group; V is read transposed straight
//                  from its natural layout with ds_read_b64_tr_b16.  Scores
//                  are computed transposed, S^T = K Q^T, and the output as
//                  O^T = V^T P^T, so each lane owns one query column in both
//                  accumulators and the online-softmax rescale is lane-local;
//                  the softmax row sums are one more MFMA of P with an
//                  all-ones operand.  MFMA: v_mfma_f32_16x16x32_bf16, fp32
//                  accumulation.
//                  Trees of up to 128 nodes need no mask pass: each lane
//                  holds two parent[] entries and walks its rows' ancestor
//                  chains with wave shuffles.  With the keys split over
//                  several workgroups, each writes fp32 partials (m, l, O).
//   k_attn_combine merges split-KV partials in a fixed split order.
//   k_attn_valu    fp32 (or bf16) inputs on the vector ALUs, fp32 throughout.
#include <math.h>

#include <mutex>
#include <type_traits>

#include "ptd_async.hpp"
#include "ptd_common.hpp"
#include "ptd_internal.hpp"

namespace {

using ptd::dma16;
using ptd::dma16_s;
using ptd::dma4;
using ptd::lds_addr;
using ptd::lds_barrier;
using ptd::wait_vmcnt;
using ptd::wait_vmcnt_le;

using bf16x8 = __bf16 __attribute__((ext_vector_type(8)));
using f32x4 = float __attribute__((ext_vector_type(4)));
using u32x4 = uint32_t __attribute__((ext_vector_type(4)));
using u32x2 = uint32_t __attribute__((ext_vector_type(2)));

constexpr int kThreads = 512;   // 8 waves: two per SIMD
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegBig = -1.0e30f;  // running-max start: finite, below any score
// A query block of a tile in which some softmax weight p exceeds this
// fraction of its query row's sum so far carries p into the PV product as
// bf16 hi + lo rather than bf16 (see k_attn_mfma).
constexpr float kPreciseFrac = 1.0f / 16.0f;

struct AttnParams {
  const void* q;
  const void* k;
  const void* v;
  const int32_t* kv_len;
  const int32_t* parent;  // [B][T]
  const int32_t* tree_len;  // [B] or null: nodes at index >= tree_len[b] are padding
  const float* k_scale;     // [Hkv] or null (8-bit caches): key = code value * k_scale[g]
  const float* v_scale;     // [Hkv] or null: value = code value * v_scale[g]
  const uint64_t* mask;   // [B][T][W] ancestor words (trees of more than 128 nodes, fp32 path)
  void* out;
  float* part_o;    // [S][B][Hkv][M][D]
  float2* part_ml;  // [S][B][Hkv][M]: (running max * c, sum of p)
  int32_t* dev_status;
  int B, T, Hq, Hkv, G, M, L_cap, W;
  int splits, passes, rows_per_pass;
  // paged caches: k and v are [num_pages][Hkv][2^page_shift][D] and row r of
  // sequence b lives in page page_table[b][r >> page_shift]; null: contiguous
  const int32_t* page_table;
  int page_shift, max_pages, num_pages;
  float scale;  // softmax scale
  float c;      // scale * log2(e)
  int out_bf16;
};

// Keys of a sequence are [0, N), N = kv_len + T, cut into `splits` chunks of
// this size (a multiple of 32, the key granularity of one MFMA step).
__host__ __device__ inline int chunk_size(int N, int splits) {
  const int c = (N + splits - 1) / splits;
  return (c + 31) & ~31;
}

// Live nodes of sequence b (the rest of the T slots are padding).
__device__ inline int live_nodes(const AttnParams& p, int b) {
  return p.tree_len ? min(max(p.tree_len[b], 0), p.T) : p.T;
}

__device__ inline void logical_block(int nblocks, int npairs, bool by_size, int& id) {
  // Workgroups are dealt round-robin over the 8 XCDs (block i to XCD i mod 8)
  // and each XCD runs its share in block order.  The items of one (b, g) pair
  // (its row passes and KV splits) share keys and query rows, so they stay on
  // one XCD (one L2), consecutive.  With the sequences ordered by size
  // (by_size), the pairs are dealt round-robin over the XCDs too (pair q to
  // XCD q mod 8), so every XCD gets a like share of long and short sequences
  // and runs its own largest first; otherwise each XCD takes a contiguous
  // range of pairs.
  const int bid = blockIdx.x;
  if (by_size && (npairs & 7) == 0 && (nblocks & 7) == 0) {
    const int ips = nblocks / npairs;  // items per pair
    const int x = bid & 7, j = bid >> 3;
    id = (x + 8 * (j / ips)) * ips + j % ips;
  } else if ((nblocks & 7) == 0) {
    id = (bid & 7) * (nblocks >> 3) + (bid >> 3);
  } else {
    id = bid;
  }
}

// ===========================================================================
// MFMA path
// ===========================================================================
// Max / sum of a lane's value and that of lane ^ 32 (or ^ 16), on the VALU
// (gfx950 v_permlane32_swap / v_permlane16_swap: with both operands holding
// the value, the two results are the value of the lane and of its partner).
__device__ __forceinline__ float max_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_xor16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float sum_xor16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

using i16x4 = short __attribute__((ext_vector_type(4)));

__device__ __forceinline__ i16x4 lds_read_tr16(const unsigned char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((PTD_LDS i16x4*)p);
}

using i32x2 = int __attribute__((ext_vector_type(2)));
// Transpose read of bytes (ds_read_b64_tr_b8): in each 16-lane group, lane i
// receives byte i mod 8 of the 8 bytes read by the group's lanes 2j + i / 8,
// j = 0..7, as its bytes j.
__device__ __forceinline__ u32x2 lds_read_tr8(const unsigned char* p) {
  return __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr8_b64_v2i32((PTD_LDS i32x2*)p));
}
// Eight OCP E4M3 values (bytes 0..7 of w) as eight bf16, exactly (every E4M3
// value is a bf16 value): gfx950 v_cvt_scalef32_pk_bf16_fp8 with scale 1.
__device__ __forceinline__ bf16x8 e4m3x8_to_bf16(u32x2 w) {
  const u32x4 r = {
      __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[0], 1.0f, false)),
      __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[0], 1.0f, true)),
      __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[1], 1.0f, false)),
      __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[1], 1.0f, true))};
  return __builtin_bit_cast(bf16x8, r);
}

// LDS layout of one 32-key sub-tile: K rows then V rows, each [32][D] of
// ES-byte elements (bf16, or E4M3 for 8-bit caches), row-major with the
// 16-byte chunks of row r stored XOR-permuted (CH = D*ES/16 chunks per row).
// bf16, D = 128 (16 chunks): K rows by r mod 16, V rows by f(r) = ((r mod 8)
// << 1) | bit 3 of r.  The K-operand reads (ds_read_b128: 16 rows x one
// chunk per 16 lanes) are then conflict-free -- measured 205 B/clk per CU
// against 113 with f, which leaves them 2-way bank-conflicted -- and f >> 1
// is distinct over rows 0..7 and over rows 8..15, so each half-wave of a V
// transpose read (8 rows x 2 adjacent chunks) covers all 16 chunk positions
// once (177 B/clk).  Otherwise (bf16 D = 64, E4M3 D = 128: 8 chunks) both
// use r mod 8.
template <int D, int ES, int NT = kThreads>
struct Ring {
  static constexpr int RB = D * ES;                  // bytes per row
  static constexpr int CH = RB / 16;                 // 16-byte chunks per row
  static constexpr int SUB = 32;                     // keys per sub-tile
  static constexpr int PART = SUB * RB;              // bytes of K (or V) per sub-tile
  static constexpr int SLOT = 2 * PART;              // K + V
  // sub-tiles in the ring: all of LDS for bf16 with 512-thread workgroups
  // (10), half of it with 256-thread ones (two workgroups per CU: 5); 10 for
  // E4M3 (80 KB) either way: a deeper ring, every slot requested at the
  // start, made the first sub-tiles land later (measured 1-6 % slower calls)
  static constexpr int NS = ES == 1 ? 10 : (160 * 1024 / (kThreads / NT)) / SLOT;
  static constexpr int DPS = 2 * SUB * CH / NT;  // copies per thread per sub-tile
  static constexpr int BYTES = NS * SLOT;
  static_assert((DPS == 1 || DPS % 2 == 0) && (2 * SUB * CH) % NT == 0, "sub-tile split");
  __device__ static int swz_k(int row, int chunk) { return chunk ^ (row & (CH - 1)); }
  __device__ static int swz_v(int row, int chunk) {
    if constexpr (CH == 16) return chunk ^ (((row & 7) << 1) | ((row >> 3) & 1));
    else return chunk ^ (row & (CH - 1));
  }
};

// 16-byte global load into VGPRs, issued from inline asm like the copies, so
// that the compiler does not track it: the caller waits with an explicit
// vmcnt and then fences the registers (vector-memory operations retire in
// issue order, so the loads issued before the copies complete first).
__device__ __forceinline__ u32x4 gload16(const void* p) {
  u32x4 v;
  asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(v) : "v"(p) : "memory");
  return v;
}
// Orders every later use of v after the preceding (volatile) wait.
__device__ __forceinline__ void reg_fence(u32x4& v) { asm volatile("" : "+v"(v)); }

template <int D, int QB, int WR, bool F8, int NT = kThreads>
__global__ void __launch_bounds__(NT, kThreads / NT) k_attn_mfma(AttnParams p) {
  // F8: keys and values are OCP E4M3 codes (scaled per KV head), widened to
  // bf16 exactly after the LDS reads; everything else is the bf16 kernel
  using KV = std::conditional_t<F8, uint8_t, uint16_t>;
  constexpr int ES = F8 ? 1 : 2;
  using R = Ring<D, ES, NT>;
  constexpr int WK = (NT / PTD_WAVE) / WR;  // key groups: sub-tiles per round
  constexpr int DB = D / 32;                      // 32-wide d blocks (QK^T k-dim)
  constexpr int DT = D / 16;                      // 16-wide d tiles (PV output rows)
  constexpr int PARK_O = WK > 1 ? WR * WK * QB * DT * 64 * 16 : 0;  // parked fragments
  constexpr int PARK_BYTES = PARK_O + (WK > 1 ? WR * WK * QB * 64 * 8 : 0);
  constexpr int SMEM = R::BYTES > PARK_BYTES ? R::BYTES : PARK_BYTES;
  static_assert(R::NS >= 2 * WK, "ring must hold two rounds");
  static_assert(QB * DB + 2 + R::NS * R::DPS <= 63, "vector-memory counter range");
  __shared__ __attribute__((aligned(16))) unsigned char smem[SMEM];

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int wr = wave % WR;
  const int kg = wave / WR;
  const int l16 = lane & 15;
  const int l4 = lane >> 4;

  // A batch of up to 64 sequences is taken largest first (size = committed
  // keys + tree nodes; ties in index order): the longest workgroups start
  // first and the short ones fill in at the end.  Work item b names the b-th
  // largest sequence; each wave ranks the sizes with shuffles.
  const bool by_size = p.B > 1 && p.B <= PTD_WAVE;
  int id;
  logical_block(gridDim.x, p.B * p.Hkv, by_size, id);
  const int split = id % p.splits;
  int rest = id / p.splits;
  const int pass = rest % p.passes;
  rest /= p.passes;
  const int g = rest % p.Hkv;
  int b = rest / p.Hkv;
  if (by_size) {
    const int bl = b;
    int nl = -1;
    if (lane < p.B) {  // clamped: an invalid kv_len is reported below, not summed
      const int kv = p.kv_len[lane];
      nl = (kv < 0 ? -1 : min(kv, p.L_cap)) + live_nodes(p, lane);
    }
    int rank = 0;
    for (int j = 0; j < p.B; ++j) {
      const int nj = __shfl(nl, j, PTD_WAVE);
      rank += (nj > nl || (nj == nl && j < lane)) ? 1 : 0;
    }
    // the ranks of lanes < B are a permutation of 0 .. B-1: one lane hits
    const uint64_t hit = __ballot(lane < p.B && rank == bl);
    b = hit ? __builtin_ctzll(hit) : bl;
  }

  const int n_kv = p.kv_len[b];
  const int tl = live_nodes(p, b);
  if (n_kv < 0 || n_kv > p.L_cap - tl) {  // (no overflow near the int range)
    if (tid == 0) ptd::report(p.dev_status, PTD_ERR_KV_LEN);
    return;
  }
  const int N = n_kv + tl;
  const int csz = chunk_size(N, p.splits);
  const int start = split * csz;
  const int end = min(N, start + csz);
  if (start >= end) {  // empty split: the combine skips it
    if (p.splits == 1) {  // no keys at all (every node padding): zero rows
      const int r0 = pass * p.rows_per_pass, r1 = min(p.M, r0 + p.rows_per_pass);
      for (int x = tid; x < (r1 - r0) * D; x += NT) {
        const int r = r0 + x / D, d = x % D;
        const size_t off = ((static_cast<size_t>(b) * p.T + r / p.G) * p.Hq + g * p.G + r % p.G) * D + d;
        if (p.out_bf16) static_cast<uint16_t*>(p.out)[off] = 0;
        else static_cast<float*>(p.out)[off] = 0.f;
      }
    }
    return;
  }

  const bool paged = p.page_table != nullptr;  // uniform
  const KV* kbase = static_cast<const KV*>(p.k) +
                    (paged ? 0 : (static_cast<size_t>(b) * p.Hkv + g) * p.L_cap * D);
  const KV* vbase = static_cast<const KV*>(p.v) +
                    (paged ? 0 : (static_cast<size_t>(b) * p.Hkv + g) * p.L_cap * D);
  // paged: the split's first 256 page ids, one per lane and register, loaded
  // untracked ahead of the query rows
  const int first_page = paged ? (start >> p.page_shift) : 0;
  u32x4 pg = {0u, 0u, 0u, 0u};
  if (paged) {
    const int npg = ((end - 1) >> p.page_shift) - first_page + 1;
    const int32_t* pt = p.page_table + static_cast<size_t>(b) * p.max_pages + first_page;
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (r * PTD_WAVE + lane < npg) pg[r] = ptd::gload4(pt + r * PTD_WAVE + lane);
  }
  const int pr0 = pass * p.rows_per_pass;
  const int rowbase = pr0 + wr * 16 * QB;
  const bool wave_live = rowbase < p.M;  // padding waves only copy and sync

  // ---- query fragments straight to VGPRs (B operand of S^T = K Q^T): lane
  //      holds Q[row l16][d = 32*db + 8*l4 .. +8]; issued before every copy
  u32x4 qraw[QB][DB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int r = min(rowbase + qb * 16 + l16, p.M - 1);
    const int i = r / p.G, hg = r % p.G;
    const uint16_t* src = static_cast<const uint16_t*>(p.q) +
                          ((static_cast<size_t>(b) * p.T + i) * p.Hq + g * p.G + hg) * D + 8 * l4;
#pragma unroll
    for (int db = 0; db < DB; ++db) qraw[qb][db] = gload16(src + 32 * db);
  }
  if (paged) {  // the page ids (issued before the query rows) are needed by the first copy
    wait_vmcnt_le(QB * DB);
    reg_fence(pg);
    const int npg = ((end - 1) >> p.page_shift) - first_page + 1;
    bool bad = false;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const bool used = r * PTD_WAVE + lane < npg;
      bad |= used && pg[r] >= static_cast<uint32_t>(p.num_pages);
      if (!used || pg[r] >= static_cast<uint32_t>(p.num_pages)) pg[r] = 0u;  // read page 0 instead
    }
    if (__any(bad) && tid == 0) ptd::report(p.dev_status, PTD_ERR_PAGE);
  }

  // ---- sub-tile copies: thread tid moves chunks u*512 + tid of the
  //      sub-tile's 2*32*CH chunks (K rows, then V rows); chunk u of a thread
  //      is K or V for the whole wave (SUB*CH is a multiple of 64)
  const uint32_t ring = lds_addr(smem);
  uint32_t cp_voff[R::DPS], cp_lds[R::DPS];
  int cp_row[R::DPS], cp_off[R::DPS];
  bool cp_v[R::DPS];
#pragma unroll
  for (int u = 0; u < R::DPS; ++u) {
    const int c = u * NT + tid;
    cp_v[u] = (u * NT + wave * PTD_WAVE) / (R::SUB * R::CH) != 0;
    const int local = c % (R::SUB * R::CH);
    cp_row[u] = local / R::CH;
    cp_off[u] = (cp_v[u] ? R::swz_v(cp_row[u], local % R::CH)
                         : R::swz_k(cp_row[u], local % R::CH)) * (16 / ES);  // elements
    cp_voff[u] = static_cast<uint32_t>((cp_row[u] * D + cp_off[u]) * ES);
    cp_lds[u] = static_cast<uint32_t>((u * NT + wave * PTD_WAVE) * 16);
  }
  // element offset of key row `row0` (a multiple of 32): contiguous, or in
  // its page (a page holds a multiple of 32 rows, so the sub-tile's 32 rows
  // are consecutive there)
  auto tile_offset = [&](int row0) __attribute__((always_inline)) -> size_t {
    if (!paged) return static_cast<size_t>(row0) * D;
    const int ti = (row0 >> p.page_shift) - first_page;  // uniform
    uint32_t phys;
    if (ti < 4 * PTD_WAVE) {
      const uint32_t v0 = __builtin_amdgcn_readlane(pg[0], ti & 63);
      const uint32_t v1 = __builtin_amdgcn_readlane(pg[1], ti & 63);
      const uint32_t v2 = __builtin_amdgcn_readlane(pg[2], ti & 63);
      const uint32_t v3 = __builtin_amdgcn_readlane(pg[3], ti & 63);
      const int k = ti >> 6;
      phys = k == 0 ? v0 : k == 1 ? v1 : k == 2 ? v2 : v3;
    } else {  // beyond the staged ids: a scalar load (checked the same way)
      phys = static_cast<uint32_t>(
          p.page_table[static_cast<size_t>(b) * p.max_pages + (row0 >> p.page_shift)]);
      if (phys >= static_cast<uint32_t>(p.num_pages)) {
        if (tid == 0) ptd::report(p.dev_status, PTD_ERR_PAGE);
        phys = 0u;
      }
    }
    const size_t prow = ((static_cast<size_t>(phys) * p.Hkv + g) << p.page_shift) +
                        (row0 & ((1 << p.page_shift) - 1));
    return prow * D;
  };
  // copy sub-tile t (keys start + 32t ..) into ring slot `slot`
  auto issue = [&](int t, int slot) __attribute__((always_inline)) {
    const uint32_t slot_lds = ring + slot * R::SLOT;
    const int row0 = start + t * R::SUB;
    const size_t tile = tile_offset(row0);
    if (row0 + R::SUB <= N) {  // whole sub-tile inside the keys: scalar base
      if constexpr (R::DPS == 1) {
        dma16_s((cp_v[0] ? vbase : kbase) + tile, cp_voff[0], slot_lds + cp_lds[0]);
      } else {
#pragma unroll
        for (int u = 0; u < R::DPS; u += 2)
          ptd::dma16_s2((cp_v[u] ? vbase : kbase) + tile, cp_voff[u], slot_lds + cp_lds[u],
                        (cp_v[u + 1] ? vbase : kbase) + tile, cp_voff[u + 1], slot_lds + cp_lds[u + 1]);
      }
    } else {  // last sub-tile: rows past the keys re-read the last key
#pragma unroll
      for (int u = 0; u < R::DPS; ++u) {
        const int grow = min(row0 + cp_row[u], N - 1);
        dma16((cp_v[u] ? vbase : kbase) + tile + static_cast<size_t>(grow - row0) * D + cp_off[u],
              slot_lds + cp_lds[u]);
      }
    }
  };

  const int ntiles = (end - start + R::SUB - 1) / R::SUB;
  const int nrounds = (ntiles + WK - 1) / WK;
  const int ninit = min(ntiles, R::NS);

  // ---- parent[] entries for deriving ancestor words in-kernel (trees of
  //      <= 128 nodes: two per lane), loaded untracked like the query rows
  //      and, like them, before any copy
  const bool small_tree = p.W <= 2;
  u32x4 par_raw = {0xFFFFFFFFu, 0xFFFFFFFFu, 0u, 0u};  // (parent[lane], parent[lane + 64])
  if (small_tree) {
    const int32_t* pb = p.parent + static_cast<size_t>(b) * p.T;
    // 4-byte untracked loads; lanes past T keep -1
    if (lane < p.T) par_raw[0] = ptd::gload4(pb + lane);
    if (lane + 64 < p.T) par_raw[1] = ptd::gload4(pb + lane + 64);
  }
  int par_lo = -1, par_hi = -1;
  bf16x8 qf[QB][DB];  // set from qraw once the first wait has covered the loads

  // per-lane LDS byte offsets inside a sub-tile (the row's swizzle is the
  // same for both 16-row halves, which therefore differ by a constant)
  int koff[DB], voff[DT];
  if constexpr (F8) {
    // K: lane (l16, l4) reads the 8 bytes d = 32*db + 8*l4 .. of key l16.
    // V: source lane l16 = 2j + h of group l4 points at key slot j's row
    // (keys 4*l4 + j, j < 4, and 16 + 4*l4 + j - 4), bytes 16*dt + 8h ..;
    // the transpose read gives lane l16 the 8 keys' values at d = 16*dt + l16.
#pragma unroll
    for (int db = 0; db < DB; ++db)
      koff[db] = l16 * R::RB + R::swz_k(l16, 2 * db + (l4 >> 1)) * 16 + (l4 & 1) * 8;
    const int j = l16 >> 1, h = l16 & 1;
    const int key0 = j < 4 ? 4 * l4 + j : 16 + 4 * l4 + (j - 4);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) voff[dt] = key0 * R::RB + R::swz_v(key0, dt) * 16 + h * 8;
  } else {
#pragma unroll
    for (int db = 0; db < DB; ++db)
      koff[db] = l16 * R::RB + R::swz_k(l16, db * 4 + l4) * 16;
    const int tj = l16 >> 2, tq = l16 & 3;
    const int key0 = 4 * l4 + tj;  // this lane's source key for the transpose reads
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
      voff[dt] = key0 * R::RB + R::swz_v(key0, 2 * dt + (tq >> 1)) * 16 + (tq & 1) * 8;
  }

  struct Tile {
    f32x4 s[2][QB];
  };
  struct KFrag {
    bf16x8 k[DB][2];
  };
  // K fragments of the sub-tile in `slot` (A operand: 16 keys x 32 d)
  auto read_k = [&](int slot) __attribute__((always_inline)) -> KFrag {
    KFrag f;
    const unsigned char* ks = smem + slot * R::SLOT;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        if constexpr (F8)
          f.k[db][kb] = e4m3x8_to_bf16(*reinterpret_cast<const u32x2*>(ks + kb * 16 * R::RB + koff[db]));
        else
          f.k[db][kb] = __builtin_bit_cast(
              bf16x8, *reinterpret_cast<const u32x4*>(ks + kb * 16 * R::RB + koff[db]));
      }
    return f;
  };
  // S^T (keys x queries) = K Q^T; lane: query l16, keys 16*kb + 4*l4 + e
  auto qk = [&](const KFrag& f) __attribute__((always_inline)) -> Tile {
    Tile x;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) x.s[kb][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
          x.s[kb][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.k[db][kb], qf[qb][db], x.s[kb][qb], 0, 0, 0);
    return x;
  };
  // V^T fragments (A operand of O^T += V^T P^T).  K-slot j of lane group l4
  // is key 4*l4 + j (j < 4) or 16 + 4*l4 + (j - 4), matching the S^T layout;
  // source lane 4*j + q of a 16-lane group points at V[key_j][16*dt + 4q],
  // and lane i of the group receives V[key_0..3][16*dt + i].
  struct VFrag {
    bf16x8 v[DT];
  };
  auto read_v = [&](int slot) __attribute__((always_inline)) -> VFrag {
    VFrag f;
    const unsigned char* vs = smem + slot * R::SLOT + R::PART;
    if constexpr (F8) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) f.v[dt] = e4m3x8_to_bf16(lds_read_tr8(vs + voff[dt]));
      return f;
    }
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const i16x4 lo = lds_read_tr16(vs + voff[dt]);
      const i16x4 hi = lds_read_tr16(vs + 16 * R::RB + voff[dt]);
      const u32x2 l2 = __builtin_bit_cast(u32x2, lo);
      const u32x2 h2 = __builtin_bit_cast(u32x2, hi);
      const u32x4 vv = {l2[0], l2[1], h2[0], h2[1]};
      f.v[dt] = __builtin_bit_cast(bf16x8, vv);
    }
    return f;
  };

  // ---- scores of keys past the chunk end, or of tree keys that are not
  //      ancestors, become -inf.  For trees of <= 128 nodes the ancestor words
  //      of the rows' nodes are derived here, at each sub-tile with tree keys
  //      (only the last few of a sequence): every lane follows the parent
  //      chains of its rows' nodes (parent[a] read from lane a % 64 by
  //      shuffles, all lanes active); each step moves to a lower index, so
  //      128 steps end every walk.  Larger trees read the mask pass's rows.
  // first sub-tile reaching past the committed keys or the chunk end
  const int t_mask0 = max(0, (min(n_kv, end) - start) / R::SUB);
  auto mask_tile = [&](Tile& x, int t) __attribute__((always_inline)) {
    if (t < t_mask0) return;
    const int abs0 = start + t * R::SUB;
    int node[QB];
    uint64_t mw0[QB], mw1[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      node[qb] = min(rowbase + qb * 16 + l16, p.M - 1) / p.G;
      mw0[qb] = 0ull;
      mw1[qb] = 0ull;
    }
    if (small_tree && abs0 + R::SUB > n_kv) {
      int a[QB];  // padding nodes see no tree keys (and their parents are not read)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) a[qb] = node[qb] < tl ? node[qb] : -1;
      for (int step = 0; step < 128; ++step) {
        bool live = false;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) live |= a[qb] >= 0;
        if (!__any(live)) break;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
          const int xa = a[qb];
          const uint64_t bit = 1ull << (xa & 63);  // branchless: no indexed word pair
          mw0[qb] |= (xa >= 0 && xa < 64) ? bit : 0ull;
          mw1[qb] |= (xa >= 64) ? bit : 0ull;
          const int plo = __shfl(par_lo, xa & 63, PTD_WAVE);
          const int phi = __shfl(par_hi, xa & 63, PTD_WAVE);
          int nx = xa >= 64 ? phi : plo;
          if (xa < 0) {
            nx = -1;
          } else if (nx < -1 || nx >= xa) {  // not topological
            ptd::report(p.dev_status, PTD_ERR_BAD_TREE);
            nx = -1;
          }
          a[qb] = nx;
        }
      }
    }
    // visibility as selects only: per-element branches writing the tile
    // through this lambda's reference were miscompiled
    if (small_tree) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int key = abs0 + kb * 16 + l4 * 4 + e;
          const int a = key - n_kv;
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) {
            const uint64_t word = a >= 64 ? mw1[qb] : mw0[qb];
            const bool anc = ((word >> (a & 63)) & 1ull) != 0;
            const bool vis = key < end && (key < n_kv || anc);
            x.s[kb][qb][e] = vis ? x.s[kb][qb][e] : -INFINITY;
          }
        }
    } else {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int key = abs0 + kb * 16 + l4 * 4 + e;
          const int a = min(max(key - n_kv, 0), p.T - 1);  // in-range row word for any key
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) {
            const uint64_t word = p.mask[(static_cast<size_t>(b) * p.T + node[qb]) * p.W + (a >> 6)];
            const bool anc = ((word >> (a & 63)) & 1ull) != 0;
            const bool vis = key < end && (key < n_kv || anc);
            x.s[kb][qb][e] = vis ? x.s[kb][qb][e] : -INFINITY;
          }
        }
    }
  };

  // ---- online softmax state.  Scores become p = 2^(s*c - m*c) against a
  //      reference maximum m per query row that moves lazily: while no p of a
  //      sub-tile exceeds 2^16, O and l stay far inside the fp32 range and m
  //      is kept.  Otherwise (the first keys a row sees, m still at its start
  //      value, or a score well above m) the rows' maxima are formed, m moves
  //      up to them, O and l are rescaled and the sub-tile's p are recomputed.
  //      The row sums l run on the matrix cores: an MFMA of the bf16 P
  //      fragment with an all-ones A operand gives every output row the sums
  //      of P's columns over the 32 keys, so each lane holds its query
  //      column's l with no cross-lane reduction (two MFMAs per sub-tile
  //      against about thirty vector instructions for dot products and
  //      cross-lane sums).
  f32x4 o[QB][DT];
  float m[QB], nmc[QB];
  f32x4 ls[QB];  // row sums of p (all four elements: the lane's query column)
  // score scale in the exp2 domain; 8-bit keys carry their head's scale
  const float c = F8 && p.k_scale ? p.c * p.k_scale[g] : p.c;
  const float vsc = F8 && p.v_scale ? p.v_scale[g] : 1.0f;  // value scale
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m[qb] = kNegBig;
    nmc[qb] = -kNegBig * c;
    ls[qb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[qb][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // exponentials of a tile, and the largest of each lane's eight
  auto exp_tile = [&](const Tile& x, float (&pv)[QB][8], float (&pm)[QB]) __attribute__((always_inline)) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        pv[qb][e] = __builtin_amdgcn_exp2f(fmaf(x.s[0][qb][e], c, nmc[qb]));
        pv[qb][4 + e] = __builtin_amdgcn_exp2f(fmaf(x.s[1][qb][e], c, nmc[qb]));
      }
      pm[qb] = fmaxf(fmaxf(fmaxf(pv[qb][0], pv[qb][1]), fmaxf(pv[qb][2], pv[qb][3])),
                     fmaxf(fmaxf(pv[qb][4], pv[qb][5]), fmaxf(pv[qb][6], pv[qb][7])));
    }
  };
  // bf16 ones: A operand of the row-sum MFMA (every output row = the sum of
  // the B operand's column over the 32 keys)
  const bf16x8 ones8 = __builtin_bit_cast(bf16x8, u32x4{0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u});
  // rare: move the reference of rows whose maximum passed it (uniform over
  // the row's four lanes).  Every lane runs the same instructions (a factor
  // of 1 where the reference stays): rescaling accumulators under a per-lane
  // branch returned wrong row sums in some builds.
  auto move_ref = [&](const Tile& x) __attribute__((always_inline)) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float mx = fmaxf(fmaxf(fmaxf(x.s[0][qb][0], x.s[0][qb][1]), fmaxf(x.s[0][qb][2], x.s[0][qb][3])),
                       fmaxf(fmaxf(x.s[1][qb][0], x.s[1][qb][1]), fmaxf(x.s[1][qb][2], x.s[1][qb][3])));
      mx = max_xor32(max_xor16(mx));
      const bool up = mx > m[qb];
      const float alpha = up ? __builtin_amdgcn_exp2f((m[qb] - mx) * c) : 1.0f;  // 0 for the first keys
      m[qb] = up ? mx : m[qb];
      nmc[qb] = up ? -mx * c : nmc[qb];
      ls[qb] *= alpha;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) o[qb][dt] *= alpha;
    }
  };
  // p of a tile as bf16 MFMA operands (B of O^T += V^T P^T: lane holds its
  // query column's 8 keys); for precise query blocks also the rounding
  // residue p - bf16(p)
  struct PFrag {
    bf16x8 hi[QB], lo[QB];
  };
  auto pv_acc = [&](const VFrag& v, const PFrag& f, unsigned precise) __attribute__((always_inline)) {
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
        o[qb][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v.v[dt], f.hi[qb], o[qb][dt], 0, 0, 0);
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) ls[qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones8, f.hi[qb], ls[qb], 0, 0, 0);
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
      if (precise & (1u << qb)) {
        ls[qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones8, f.lo[qb], ls[qb], 0, 0, 0);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          o[qb][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v.v[dt], f.lo[qb], o[qb][dt], 0, 0, 0);
      }
  };

  // ---- rounds.  Round rd holds sub-tiles rd*WK .. rd*WK + WK - 1 (wave kg
  //      takes rd*WK + kg).  Software pipeline (PIPE): during round rd a wave
  //      issues the QK^T MFMAs of its round rd + 1 sub-tile interleaved with
  //      the softmax of its round rd sub-tile (scores kept in registers from
  //      the round before), then the PV MFMAs of round rd.  Round rd thus
  //      reads K of round rd + 1 and V of round rd, the data of round rd + 1
  //      is waited for at the barrier of round rd, and the slots of round
  //      rd - 1 are free there and refilled right away.  Round rd + 1's data
  //      is then issued by round rd - 1, which needs 3*WK ring slots; with
  //      more key groups a round computes its own sub-tile start to end.
  //      The denominator adds the same bf16 p that enter O, so that O is
  //      the exact average of V under the rounded weights.  A query block
  //      of a tile in which some p exceeds kPreciseFrac of its row's sum so
  //      far (this wave's keys, from the row-sum accumulator)
  //      carries p as bf16 hi + lo (residue at most 2^-16 p instead of
  //      2^-8 p): every key carried as plain bf16 then weighs at most
  //      kPreciseFrac of its row's final sum, so the 2^-8 relative rounding
  //      of a dominant key, or of a few large ones, never reaches O.
  constexpr bool PIPE = 3 * WK <= R::NS;
  static_assert((2 + (PIPE ? 1 : 0)) * WK <= R::NS, "round data issued one round ahead");
  // bf16 p of scores x (exponentials pv and lane maxima pm computed);
  // returns the mask of precise query blocks (residues in f.lo)
  auto to_p = [&](const Tile& x, float (&pv)[QB][8], float (&pm)[QB], PFrag& f)
      __attribute__((always_inline)) -> unsigned {
    bool over = false;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) over |= !(pm[qb] <= 65536.0f);
    if (__any(over)) {
      move_ref(x);
      exp_tile(x, pv, pm);
    }
    unsigned pmask = 0;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
      pmask |= __any(!(pm[qb] <= kPreciseFrac * ls[qb][0])) ? (1u << qb) : 0u;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const bool precise = pmask & (1u << qb);
      u32x4 ph, pl;
#pragma unroll
      for (int w = 0; w < 4; ++w) ph[w] = ptd::cvt_pk_bf16(pv[qb][2 * w], pv[qb][2 * w + 1]);
      f.hi[qb] = __builtin_bit_cast(bf16x8, ph);
      if (precise) {
#pragma unroll
        for (int w = 0; w < 4; ++w)
          pl[w] = ptd::cvt_pk_bf16(pv[qb][2 * w] - static_cast<float>(f.hi[qb][2 * w]),
                                   pv[qb][2 * w + 1] - static_cast<float>(f.hi[qb][2 * w + 1]));
        f.lo[qb] = __builtin_bit_cast(bf16x8, pl);
      }
    }
    return pmask;
  };

  for (int t = 0; t < ninit; ++t) issue(t, t);
  wait_vmcnt_le((ninit - min(ntiles, WK)) * R::DPS);  // round 0 (query rows, parents) landed
  lds_barrier();
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      reg_fence(qraw[qb][db]);
      qf[qb][db] = __builtin_bit_cast(bf16x8, qraw[qb][db]);
    }
  reg_fence(par_raw);
  par_lo = static_cast<int>(par_raw[0]);
  par_hi = static_cast<int>(par_raw[1]);

  // rounds whose wait count is the steady-state constant: every refill so far
  // issued in full (R::NS + (rd - 1) * WK <= ntiles)
  const int steady_end = ntiles >= R::NS ? (ntiles - R::NS) / WK + 1 : -1;
  int cs = kg;  // ring slot of this wave's sub-tile of the current round
  int rs = 0;   // slot refilled next (round rd - 1's slots, in order)
  Tile sc;      // PIPE: scores of the current round's sub-tile
  if (PIPE && wave_live && kg < ntiles) {
    sc = qk(read_k(cs));
    mask_tile(sc, kg);
  }
  // a round in general: waits by the count of copies issued so far, refills
  // (whole or last sub-tiles, contiguous or paged caches), masked sub-tiles
  auto round = [&](int rd) __attribute__((always_inline)) {
      const bool do_wait = PIPE ? rd + 1 < nrounds : rd >= 1;
      if (do_wait) {
        if (rd >= 1 && rd <= steady_end) {
          wait_vmcnt<(R::NS - (2 + (PIPE ? 1 : 0)) * WK) * R::DPS>();
        } else {
          const int issued = min(ntiles, R::NS + max(0, rd - 1) * WK);
          const int needed = min(ntiles, (rd + 1 + (PIPE ? 1 : 0)) * WK);
          wait_vmcnt_le((issued - needed) * R::DPS);
        }
        lds_barrier();
        if (rd >= 1) {
#pragma unroll
          for (int w = 0; w < WK; ++w) {
            const int tt = R::NS + (rd - 1) * WK + w;
            if (tt < ntiles) issue(tt, rs);
            rs = rs + 1 == R::NS ? 0 : rs + 1;
          }
        }
      }
      int ns = cs + WK;
      if (ns >= R::NS) ns -= R::NS;
      const int j = rd * WK + kg;
      if (wave_live && j < ntiles) {
        float pv[QB][8], pm[QB];
        if constexpr (PIPE) {
          // next K reads in flight while this sub-tile's exponentials run (they
          // overlap the previous round's PV MFMAs, still executing); then the
          // next QK^T and this PV back to back on the matrix cores.  After the
          // wave's last sub-tile the next-tile QK^T works on whatever the slot
          // holds and its result is dropped: one code path keeps the register
          // allocation of this loop within the two-waves-per-SIMD budget.
          const KFrag kf = read_k(ns);
          exp_tile(sc, pv, pm);
          PFrag pf;
          const unsigned precise = to_p(sc, pv, pm, pf);
          Tile sn = qk(kf);
          const VFrag vf = read_v(cs);
          pv_acc(vf, pf, precise);
          if (j + WK < ntiles) mask_tile(sn, j + WK);
          sc = sn;
        } else {
          sc = qk(read_k(cs));
          mask_tile(sc, j);
          const VFrag vf = read_v(cs);
          exp_tile(sc, pv, pm);
          PFrag pf;
          const unsigned precise = to_p(sc, pv, pm, pf);
          pv_acc(vf, pf, precise);
        }
      }
      cs = ns;
  };
  // Steady rounds: every refill of the round is a whole sub-tile of a
  // contiguous cache below t_mask0, so this round's and the next round's
  // sub-tiles need no masking either; the wait count is the constant, the
  // tile address scalar arithmetic, and the general round's tests drop out
  // (with and without the software pipeline; without it, 34.9 against 36.7 us
  // per call on 40 heads x 96 rows x 4192 keys).
  // The scalar instructions of a round are issued by the CU's one scalar unit
  // for every wave, and the two waves of a SIMD reach the refills together:
  // measured on 8 KV heads x 256 rows x 32832 keys, 70.7 against 76.0 us per
  // call; on ragged-16, 156.2 against 171.2.  A steady round also splits the
  // hi + lo P of the general round: the bf16 P and its PV and row-sum MFMAs
  // always, the residues and their MFMAs after them in a rarely taken branch,
  // so the main path is one block the scheduling groups below can interleave
  // (the precise test still reads the row sums before this sub-tile, and
  // every accumulator receives hi before lo as in the general round).
  const int steady_hi =
      (!paged && t_mask0 >= R::NS + WK) ? (t_mask0 - R::NS - WK) / WK + 1 : 0;
  auto round_steady = [&](int rd) __attribute__((always_inline)) {
    wait_vmcnt<(R::NS - (2 + (PIPE ? 1 : 0)) * WK) * R::DPS>();
    lds_barrier();
#pragma unroll
    for (int w = 0; w < WK; ++w) {
      const int tt = R::NS + (rd - 1) * WK + w;
      const size_t tile = static_cast<size_t>(start + tt * R::SUB) * D;
      const uint32_t slot_lds = ring + rs * R::SLOT;
      if constexpr (R::DPS == 1) {
        dma16_s((cp_v[0] ? vbase : kbase) + tile, cp_voff[0], slot_lds + cp_lds[0]);
      } else {
#pragma unroll
        for (int u = 0; u < R::DPS; u += 2)
          ptd::dma16_s2((cp_v[u] ? vbase : kbase) + tile, cp_voff[u], slot_lds + cp_lds[u],
                        (cp_v[u + 1] ? vbase : kbase) + tile, cp_voff[u + 1],
                        slot_lds + cp_lds[u + 1]);
      }
      rs = rs + 1 == R::NS ? 0 : rs + 1;
    }
    int ns = cs + WK;
    if (ns >= R::NS) ns -= R::NS;
    if constexpr (PIPE) {
      if (wave_live) {
        float pv[QB][8], pm[QB];
        const KFrag kf = read_k(ns);
        exp_tile(sc, pv, pm);
        Tile sn = qk(kf);
        // the K reads, a few exponentials, then one QK^T MFMA per three
        // vector instructions (scheduling groups: 0x100 LDS reads, 0x002
        // vector ALU, 0x008 MFMA)
        __builtin_amdgcn_sched_group_barrier(0x100, 2 * DB, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);
#pragma unroll
        for (int i = 0; i < 2 * QB * DB; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);
        }
        bool over = false;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) over |= !(pm[qb] <= 65536.0f);
        if (__any(over)) {
          move_ref(sc);
          exp_tile(sc, pv, pm);
        }
        unsigned pmask = 0;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
          pmask |= __any(!(pm[qb] <= kPreciseFrac * ls[qb][0])) ? (1u << qb) : 0u;
        PFrag pf;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
          u32x4 ph;
#pragma unroll
          for (int w = 0; w < 4; ++w) ph[w] = ptd::cvt_pk_bf16(pv[qb][2 * w], pv[qb][2 * w + 1]);
          pf.hi[qb] = __builtin_bit_cast(bf16x8, ph);
        }
        const VFrag vf = read_v(cs);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
            o[qb][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf.v[dt], pf.hi[qb], o[qb][dt], 0, 0, 0);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) ls[qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones8, pf.hi[qb], ls[qb], 0, 0, 0);
        // the V reads, then one PV MFMA per two vector instructions
        __builtin_amdgcn_sched_group_barrier(0x100, 2 * DT, 1);
#pragma unroll
        for (int i = 0; i < DT * QB; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
          __builtin_amdgcn_sched_group_barrier(0x002, 2, 1);
        }
        if (pmask) {
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
            if (pmask & (1u << qb)) {
              u32x4 pl;
#pragma unroll
              for (int w = 0; w < 4; ++w)
                pl[w] = ptd::cvt_pk_bf16(pv[qb][2 * w] - static_cast<float>(pf.hi[qb][2 * w]),
                                         pv[qb][2 * w + 1] - static_cast<float>(pf.hi[qb][2 * w + 1]));
              pf.lo[qb] = __builtin_bit_cast(bf16x8, pl);
              ls[qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones8, pf.lo[qb], ls[qb], 0, 0, 0);
#pragma unroll
              for (int dt = 0; dt < DT; ++dt)
                o[qb][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf.v[dt], pf.lo[qb], o[qb][dt], 0, 0, 0);
            }
        }
        sc = sn;
      }
    } else {
      if (wave_live) {
        float pv[QB][8], pm[QB];
        sc = qk(read_k(cs));
        const VFrag vf = read_v(cs);
        exp_tile(sc, pv, pm);
        PFrag pf;
        const unsigned precise = to_p(sc, pv, pm, pf);
        pv_acc(vf, pf, precise);
      }
    }
    cs = ns;
  };
  int rd0 = 0;
  if (steady_hi >= 1) {
    round(0);
    for (int rd = 1; rd <= steady_hi; ++rd) round_steady(rd);
    rd0 = steady_hi + 1;
  }
  for (int rd = rd0; rd < nrounds; ++rd) round(rd);
  wait_vmcnt<0>();
  lds_barrier();  // every copy landed and every wave is done with the ring


  // ---- softmax denominators (each lane: its query column's)
  float lsum[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) lsum[qb] = ls[qb][0];

  // ---- epilogue.  The key groups of a row group hold their fragments in the
  //      same lane layout (lane: query column l16, d = 16*dt + 4*l4 + 0..3), so
  //      the merge is lane-local: every wave parks its fragments and (m, l)
  //      per column in LDS, then wave (wr, kg) merges the key groups (fixed
  //      order) for d-tiles [kg*DPW, (kg+1)*DPW) of its row group and stores
  //      them.  With one key group the fragments are stored directly.
  constexpr int DPW = DT / WK;  // d-tiles merged and stored per wave
  static_assert(DT % WK == 0, "d-tiles per wave");
  const bool all_rows = rowbase + 16 * QB <= p.M;  // uniform: the common case
  auto store_tile = [&](int qb, int dt, f32x4 acc, float mc, float den) {
    const int r = rowbase + qb * 16 + l16;
    if (!all_rows && r >= p.M) return;
    if (p.splits == 1) {
      const int i = r / p.G, hg = r % p.G;
      const size_t off = ((static_cast<size_t>(b) * p.T + i) * p.Hq + g * p.G + hg) * D +
                         16 * dt + 4 * l4;
      const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
      const f32x4 v = i < tl ? acc * (vsc / den) : zero;
      if (p.out_bf16) {
        const u32x2 w2 = {ptd::cvt_pk_bf16(v[0], v[1]), ptd::cvt_pk_bf16(v[2], v[3])};
        *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(p.out) + off) = w2;
      } else {
        *reinterpret_cast<f32x4*>(static_cast<float*>(p.out) + off) = v;
      }
    } else {
      const size_t prow = ((static_cast<size_t>(split) * p.B + b) * p.Hkv + g) * p.M + r;
      *reinterpret_cast<f32x4*>(p.part_o + prow * D + 16 * dt + 4 * l4) = F8 ? acc * vsc : acc;
      if (dt == 0 && l4 == 0) p.part_ml[prow] = make_float2(mc, den);
    }
  };
  if constexpr (WK == 1) {
    if (!wave_live) return;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) store_tile(qb, dt, o[qb][dt], m[qb] * c, lsum[qb]);
  } else {
    f32x4* so = reinterpret_cast<f32x4*>(smem);  // [WR][WK][QB][DT][64]
    float2* sml = reinterpret_cast<float2*>(smem + PARK_O);  // [WR][WK][QB][64]
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) so[(((wr * WK + kg) * QB + qb) * DT + dt) * 64 + lane] = o[qb][dt];
      sml[((wr * WK + kg) * QB + qb) * 64 + lane] = make_float2(m[qb], lsum[qb]);
    }
    lds_barrier();
    if (!wave_live) return;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float mk[WK], w[WK];
      float mm = kNegBig, den = 0.f;
#pragma unroll
      for (int k2 = 0; k2 < WK; ++k2) {
        mk[k2] = sml[((wr * WK + k2) * QB + qb) * 64 + lane].x;
        mm = fmaxf(mm, mk[k2]);
      }
#pragma unroll
      for (int k2 = 0; k2 < WK; ++k2) {
        w[k2] = __builtin_amdgcn_exp2f((mk[k2] - mm) * c);
        den += w[k2] * sml[((wr * WK + k2) * QB + qb) * 64 + lane].y;
      }
#pragma unroll
      for (int j = 0; j < DPW; ++j) {
        const int dt = kg * DPW + j;
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int k2 = 0; k2 < WK; ++k2) acc += so[(((wr * WK + k2) * QB + qb) * DT + dt) * 64 + lane] * w[k2];
        store_tile(qb, dt, acc, mm * c, den);
      }
    }
  }
}

// ===========================================================================
// split-KV combine: out = sum_s w_s O_s / sum_s w_s l_s, w_s = 2^(mc_s - max mc),
// one thread per (b, g, row, 4 columns), online in the split index (fixed
// order, so the result is deterministic).  A workgroup covers 256 / (D/4)
// consecutive rows of one (b, g): everything per (b, g) is uniform (scalar
// loads and arithmetic) and a thread's row and columns are shifts of its id.
// ===========================================================================
template <int D, int U>
__global__ void __launch_bounds__(256) k_attn_combine(AttnParams p) {
  constexpr int D4 = D / 4;
  constexpr int RPB = 256 / D4;  // rows per workgroup
  const int nrb = (p.M + RPB - 1) / RPB;
  const int bg = static_cast<int>(blockIdx.x) / nrb;  // uniform
  const int rb = static_cast<int>(blockIdx.x) - bg * nrb;
  const int b = bg / p.Hkv;
  const int g = bg - b * p.Hkv;
  const int d4 = threadIdx.x % D4;
  const int r = rb * RPB + static_cast<int>(threadIdx.x) / D4;
  if (r >= p.M) return;
  // The partials are loaded, U splits at a time, without waiting for kv_len
  // (the workspace holds all p.splits of them); the updates by empty splits,
  // whose partials were never written, are discarded with selects.
  const size_t stride = static_cast<size_t>(p.B) * p.Hkv * p.M;
  const size_t row0 = (static_cast<size_t>(b) * p.Hkv + g) * p.M + r;
  float2 ml[U];
  f32x4 ov[U];
  auto load_group = [&](int s0) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const size_t pr = row0 + static_cast<size_t>(min(s0 + u, p.splits - 1)) * stride;
      ml[u] = p.part_ml[pr];
      ov[u] = *reinterpret_cast<const f32x4*>(p.part_o + pr * D + d4 * 4);
    }
  };
  const int n_kv = p.kv_len[b];
  const int tl = live_nodes(p, b);
  load_group(0);
  const bool valid = n_kv >= 0 && n_kv <= p.L_cap - tl;  // else reported by the attention kernel
  const int N = valid ? n_kv + tl : 1;
  const int csz = chunk_size(max(N, 1), p.splits);
  const int nsp = (N + csz - 1) / csz;  // non-empty splits
  float mrun = kNegBig, den = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  auto merge_group = [&](int s0) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool live = s0 + u < nsp;
      const float mn = fmaxf(mrun, ml[u].x);
      const float a = __builtin_amdgcn_exp2f(mrun - mn);
      const float w = __builtin_amdgcn_exp2f(ml[u].x - mn);
      const f32x4 na = acc * a + ov[u] * w;
      den = live ? den * a + w * ml[u].y : den;
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[e] = live ? na[e] : acc[e];
      mrun = live ? mn : mrun;
    }
  };
  merge_group(0);  // the first group outside the loop: its loads stay ahead of every wait
  for (int s0 = U; s0 < nsp; s0 += U) {
    load_group(s0);
    merge_group(s0);
  }
  if (!valid) return;
  const int i = r / p.G, hg = r % p.G;
  const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
  const f32x4 v = i < tl ? acc * (1.0f / den) : zero;  // padding nodes: zero
  const size_t off = ((static_cast<size_t>(b) * p.T + i) * p.Hq + g * p.G + hg) * D + d4 * 4;
  if (p.out_bf16) {
    const u32x2 w = {ptd::cvt_pk_bf16(v[0], v[1]), ptd::cvt_pk_bf16(v[2], v[3])};
    *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(p.out) + off) = w;
  } else {
    *reinterpret_cast<f32x4*>(static_cast<float*>(p.out) + off) = v;
  }
}

// ===========================================================================
// vector-ALU path (fp32 inputs): one workgroup of 256 threads per (b, g, pass
// of 32 rows); 64-key tiles; lane j of a wave scores key j of the tile for one
// query row at a time; the running state of every row lives in LDS.
// ===========================================================================
constexpr int kValuThreads = 256;
constexpr int kValuRows = 32;

template <int D>
__global__ void __launch_bounds__(kValuThreads) k_attn_valu(AttnParams p) {
  constexpr int KT = 64;
  constexpr int DU = D / 64;  // output columns per lane
  __shared__ float ks[KT][D + 1];
  __shared__ float vs[KT][D];
  __shared__ float qs[kValuRows][D];
  __shared__ float acc[kValuRows][D];
  __shared__ float sm[kValuRows], sl[kValuRows];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int pass = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int n_kv = p.kv_len[b];
  const int tl = live_nodes(p, b);
  if (n_kv < 0 || n_kv > p.L_cap - tl) {  // (no overflow near the int range)
    if (tid == 0) ptd::report(p.dev_status, PTD_ERR_KV_LEN);
    return;
  }
  const int N = n_kv + tl;
  const int r0 = pass * kValuRows;
  const float* qg = static_cast<const float*>(p.q);
  const float* kg = static_cast<const float*>(p.k);
  const float* vg = static_cast<const float*>(p.v);
  for (int x = tid; x < kValuRows * D; x += kValuThreads) {
    const int rl = x / D, d = x % D, r = r0 + rl;
    float v = 0.f;
    if (r < p.M) {
      const int i = r / p.G, hg = r % p.G;
      v = qg[((static_cast<size_t>(b) * p.T + i) * p.Hq + g * p.G + hg) * D + d];
    }
    qs[rl][d] = v;
    acc[rl][d] = 0.f;
  }
  if (tid < kValuRows) {
    sm[tid] = kNegBig;
    sl[tid] = 0.f;
  }
  const size_t kvoff = (static_cast<size_t>(b) * p.Hkv + g) * p.L_cap * D;
  for (int t0 = 0; t0 < N; t0 += KT) {
    __syncthreads();
    for (int x = tid; x < KT * D; x += kValuThreads) {
      const int kk = x / D, d = x % D;
      const int row = min(t0 + kk, N - 1);
      ks[kk][d] = kg[kvoff + static_cast<size_t>(row) * D + d];
      vs[kk][d] = vg[kvoff + static_cast<size_t>(row) * D + d];
    }
    __syncthreads();
    const int key = t0 + lane;
#pragma unroll 1
    for (int rl = wave; rl < kValuRows; rl += kValuThreads / PTD_WAVE) {
      const int r = r0 + rl;
      if (r >= p.M) break;
      const int i = r / p.G;
      bool vis = key < N;
      if (vis && key >= n_kv) {
        const int a = key - n_kv;
        vis = (p.mask[(static_cast<size_t>(b) * p.T + i) * p.W + (a >> 6)] >> (a & 63)) & 1ull;
      }
      float s = -INFINITY;
      if (vis) {
        float dot = 0.f;
#pragma unroll 8
        for (int d = 0; d < D; ++d) dot = fmaf(qs[rl][d], ks[lane][d], dot);
        s = dot * p.scale;
      }
      const float m_old = sm[rl];
      const float m_new = fmaxf(m_old, ptd::wave_max(s));
      const float alpha = expf(m_old - m_new);
      const float pj = expf(s - m_new);
      const float psum = ptd::wave_sum(pj);
      float a[DU];
#pragma unroll
      for (int u = 0; u < DU; ++u) a[u] = acc[rl][lane + 64 * u] * alpha;
#pragma unroll 4
      for (int j = 0; j < KT; ++j) {
        const float pb = __shfl(pj, j, PTD_WAVE);
#pragma unroll
        for (int u = 0; u < DU; ++u) a[u] = fmaf(pb, vs[j][lane + 64 * u], a[u]);
      }
#pragma unroll
      for (int u = 0; u < DU; ++u) acc[rl][lane + 64 * u] = a[u];
      if (lane == 0) {
        sl[rl] = sl[rl] * alpha + psum;
        sm[rl] = m_new;
      }
    }
  }
  __syncthreads();
  for (int x = tid; x < kValuRows * D; x += kValuThreads) {
    const int rl = x / D, d = x % D, r = r0 + rl;
    if (r >= p.M) continue;
    const int i = r / p.G, hg = r % p.G;
    const size_t off = ((static_cast<size_t>(b) * p.T + i) * p.Hq + g * p.G + hg) * D + d;
    const float v = i < tl ? acc[rl][d] / sl[rl] : 0.f;  // padding nodes: zero
    if (p.out_bf16) static_cast<uint16_t*>(p.out)[off] = static_cast<uint16_t>(ptd::f32_to_bf16_rne(v));
    else static_cast<float*>(p.out)[off] = v;
  }
}

// ===========================================================================
// host planning
// ===========================================================================
struct Plan {
  bool mfma;
  int QB, WR, passes, rows_per_pass, splits;
  int nt;  // threads per k_attn_mfma workgroup (512, or 256 with two workgroups per CU)
  bool needs_mask;  // mask rows read from memory (fp32 path, trees over 128 nodes)
  // workspace: [partials][mask rows], each 256-byte aligned
  size_t partial_bytes, mask_bytes, total_bytes;
};

size_t align256(size_t n) { return (n + 255) & ~static_cast<size_t>(255); }

constexpr int kTargetBlocks = 256;  // one resident workgroup per CU on MI355X

bool make_plan(const ptd_attn_shape* s, int T, Plan* pl) {
  if (!s || s->B < 1 || s->Hq < 1 || s->Hkv < 1 || s->Hq % s->Hkv) return false;
  if (s->D != 64 && s->D != 128) return false;
  if (T < 1 || T > PTD_MAX_T || s->L_cap < 1) return false;  // (L_cap >= T: per entry point)
  if ((s->in_dtype != PTD_F32 && s->in_dtype != PTD_BF16) ||
      (s->out_dtype != PTD_F32 && s->out_dtype != PTD_BF16))
    return false;
  const long long M = static_cast<long long>(T) * (s->Hq / s->Hkv);
  if (M > (1 << 24)) return false;
  pl->mfma = s->in_dtype == PTD_BF16;
  if (pl->mfma) {
    const int mp = static_cast<int>(M < 256 ? M : 256);
    const int nblk = (mp + 15) / 16;
    // 8 waves: WR row groups of 16*QB rows (QB <= 2) x (8/WR) key groups.
    // Up to 64 rows: passes of 32 rows (QB = 1), so that the workgroups of a
    // (b, g) split its keys half as many ways: half the split partials for
    // the combine, with each key read by two passes sharing one L2
    // (measured on 32 heads x 64 rows x 2112 keys: 14.3 + 4.7 us against
    // 16.3 + 4.7 us for one 64-row pass and twice the splits).
    if (nblk <= 4) { pl->WR = 2; pl->QB = 1; }
    // 65-128 rows: passes of 64 (WR = 2, QB = 2), fewer waves reading each
    // sub-tile than one 128-row pass (measured on 40 KV heads x 96 rows x
    // 4192 keys: 33.3 against 35.2 us).
    else if (nblk <= 8) { pl->WR = 2; pl->QB = 2; }
    // More than 128 rows: passes of 128 (WR = 4, QB = 2) rather than one
    // pass of up to 256 rows over eight row groups.  Every row-group wave
    // reads each K/V sub-tile from LDS, so four waves halve the LDS reads per
    // key; the passes share the keys through one XCD's L2 (measured on 8
    // KV heads x 256 rows x 32832 keys: 64.1 against 69.4 us).
    else { pl->WR = 4; pl->QB = 2; }
    // A batch of sequences in 128-row passes runs 256-thread workgroups (the
    // four row groups, one key group, a five-sub-tile ring in half of LDS),
    // two resident per CU: one's prologue and tail overlap the other's rounds
    // instead of following them, and their rounds drift apart instead of
    // meeting at one barrier (measured on ragged-16: 136.5 against 146.2 us
    // with three KV splits per sequence, 141.2 with two; a single sequence
    // was not faster: 68.1 against 67.3 us on 8 KV heads x 32832 keys).
    pl->nt = (pl->WR == 4 && s->B > 1) ? 256 : kThreads;
    pl->rows_per_pass = 16 * pl->QB * pl->WR;
    pl->passes = static_cast<int>((M + pl->rows_per_pass - 1) / pl->rows_per_pass);
    const long long items = static_cast<long long>(s->B) * s->Hkv * pl->passes;
    // Several sequences may differ in length (kv_len is not known here):
    // twice the workgroups, so the dispatcher can even out long and short
    // ones (measured on 16 sequences of 512-8192 keys: 151-158 against
    // 167-171 us; a single sequence was slower with it).
    const int target = pl->nt == 256 ? 3 * kTargetBlocks : s->B > 1 ? 2 * kTargetBlocks : kTargetBlocks;
    int sp = static_cast<int>(target / items);
    const int max_by_len = (s->L_cap + 255) / 256;  // at least ~256 keys per split
    if (sp > max_by_len) sp = max_by_len;
    if (sp < 1) sp = 1;
    if (sp > 64) sp = 64;
    pl->splits = sp;
  } else {
    pl->WR = pl->QB = 0;
    pl->nt = kValuThreads;
    pl->rows_per_pass = kValuRows;
    pl->passes = static_cast<int>((M + kValuRows - 1) / kValuRows);
    pl->splits = 1;
  }
  if (static_cast<long long>(s->B) * s->Hkv * pl->passes * pl->splits > 0x7FFFFFFFLL) return false;
  // the combine's grid: one workgroup per 8 (D = 128) or 16 (D = 64) rows of a (b, g)
  if (pl->splits > 1 && static_cast<long long>(s->B) * s->Hkv * ((M + 7) / 8) > 0x7FFFFFFFLL) return false;
  pl->needs_mask = !pl->mfma || T > 128;
  pl->partial_bytes = pl->splits > 1
      ? align256(static_cast<size_t>(pl->splits) * s->B * s->Hkv * M * (s->D + 2) * sizeof(float))
      : 0;
  pl->mask_bytes = align256(static_cast<size_t>(s->B) * T * ((T + 63) / 64) * sizeof(uint64_t));
  pl->total_bytes = pl->partial_bytes + (pl->needs_mask ? pl->mask_bytes : 0);
  return true;
}

template <int D, bool F8>
void launch_mfma(const Plan& pl, const AttnParams& prm, hipStream_t st) {
  const dim3 grid(prm.B * prm.Hkv * pl.passes * pl.splits);
  if (pl.nt == 256) {
    hipLaunchKernelGGL((k_attn_mfma<D, 2, 4, F8, 256>), grid, dim3(256), 0, st, prm);
    return;
  }
  const dim3 block(kThreads);
#define PTD_MFMA_CASE(qb_, wr_) \
  if (pl.QB == qb_ && pl.WR == wr_) { hipLaunchKernelGGL((k_attn_mfma<D, qb_, wr_, F8>), grid, block, 0, st, prm); return; }
  PTD_MFMA_CASE(1, 2) PTD_MFMA_CASE(2, 2) PTD_MFMA_CASE(2, 4)
#undef PTD_MFMA_CASE
}

}  // namespace

extern "C" size_t ptd_tree_attention_workspace_bytes(const ptd_attn_shape* shape, int32_t T) {
  Plan pl;
  if (!make_plan(shape, T, &pl)) return 0;
  return pl.total_bytes;
}

// ---------------------------------------------------------------------------
// Allocation-free variant: the scratch is a fixed device array.  In host code
// `scratch` names a host-side stand-in, never the device memory: its device
// address is looked up once per GPU (hipGetSymbolAddress with that GPU
// current) and only that address is handed to kernels.
// ---------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[PTD_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};

// Device address of the current GPU's scratch array (null on failure).
void* scratch_device_ptr() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxScratchDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
      (void)hipGetLastError();  // clear the sticky error of the failed lookup
      return nullptr;
    }
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

namespace {

// The attention call on contiguous caches (page_table null) or paged ones.
int attention_impl(const void* q, const void* k_cache, const void* v_cache,
                   const int32_t* kv_len, const int32_t* tree_len, const int32_t* parent,
                   int32_t T, void* out,
                   const ptd_attn_shape* shape, const uint64_t* mask, void* workspace,
                   size_t workspace_bytes, int32_t* dev_status, void* stream,
                   const int32_t* page_table, int page_shift, int max_pages, int num_pages,
                   bool f8 = false, const float* k_scale = nullptr,
                   const float* v_scale = nullptr, bool noalloc = false) {
  PTD_RETURN_IF(!q || !k_cache || !v_cache || !kv_len || !parent || !out || !shape,
                PTD_ERR_NULL);
  if (shape->in_dtype != PTD_F32 && shape->in_dtype != PTD_BF16) return PTD_ERR_DTYPE;
  if (shape->out_dtype != PTD_F32 && shape->out_dtype != PTD_BF16) return PTD_ERR_DTYPE;
  Plan pl;
  PTD_RETURN_IF(!make_plan(shape, T, &pl), PTD_ERR_SHAPE);
  // every tree row must fit unless tree sizes come with the call
  PTD_RETURN_IF(!tree_len && shape->L_cap < T, PTD_ERR_SHAPE);
  PTD_RETURN_IF(!ptd_aligned(q, 16) || !ptd_aligned(k_cache, 16) || !ptd_aligned(v_cache, 16) ||
                    !ptd_aligned(out, 16) || (mask && !ptd_aligned(mask, 8)),
                PTD_ERR_ALIGN);
  const bool build_mask = pl.needs_mask && !mask;
  const size_t need = pl.partial_bytes + (build_mask ? pl.mask_bytes : 0);
  if (noalloc && need > 0) {  // the fixed scratch array stands in for the workspace
    PTD_RETURN_IF(need > PTD_NOALLOC_SCRATCH_BYTES, PTD_ERR_SCRATCH);
    workspace = scratch_device_ptr();
    PTD_RETURN_IF(!workspace, PTD_ERR_HIP);
    workspace_bytes = PTD_NOALLOC_SCRATCH_BYTES;
  }
  if (need > 0) {
    PTD_RETURN_IF(!workspace, PTD_ERR_WORKSPACE);
    PTD_RETURN_IF(workspace_bytes < need, PTD_ERR_WORKSPACE);
    PTD_RETURN_IF(!ptd_aligned(workspace, 256), PTD_ERR_ALIGN);
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  if (build_mask) {
    uint64_t* mws = reinterpret_cast<uint64_t*>(ws + pl.partial_bytes);
    const int rc = ptd_launch_tree_mask(parent, tree_len, shape->B, T, mws, nullptr, dev_status, st);
    if (rc != PTD_OK) return rc;
    mask = mws;
  }
  AttnParams prm;
  prm.q = q;
  prm.k = k_cache;
  prm.v = v_cache;
  prm.kv_len = kv_len;
  prm.parent = parent;
  prm.tree_len = tree_len;
  prm.k_scale = k_scale;
  prm.v_scale = v_scale;
  prm.mask = pl.needs_mask ? mask : nullptr;
  prm.out = out;
  prm.part_o = pl.splits > 1 ? reinterpret_cast<float*>(ws) : nullptr;
  prm.part_ml = nullptr;
  prm.dev_status = dev_status;
  prm.B = shape->B;
  prm.T = T;
  prm.Hq = shape->Hq;
  prm.Hkv = shape->Hkv;
  prm.G = shape->Hq / shape->Hkv;
  prm.M = T * prm.G;
  prm.L_cap = shape->L_cap;
  prm.W = (T + 63) / 64;
  prm.splits = pl.splits;
  prm.passes = pl.passes;
  prm.rows_per_pass = pl.rows_per_pass;
  prm.scale = shape->scale > 0.f ? shape->scale : 1.0f / sqrtf(static_cast<float>(shape->D));
  prm.c = prm.scale * kLog2e;
  prm.out_bf16 = shape->out_dtype == PTD_BF16;
  prm.page_table = page_table;
  prm.page_shift = page_shift;
  prm.max_pages = max_pages;
  prm.num_pages = num_pages;
  if (pl.splits > 1) {
    const size_t rows = static_cast<size_t>(pl.splits) * prm.B * prm.Hkv * prm.M;
    prm.part_ml = reinterpret_cast<float2*>(prm.part_o + rows * shape->D);
  }
  if (pl.mfma) {
    if (f8) launch_mfma<128, true>(pl, prm, st);  // (D = 128 checked by the entry point)
    else if (shape->D == 128) launch_mfma<128, false>(pl, prm, st);
    else launch_mfma<64, false>(pl, prm, st);
    if (pl.splits > 1) {
      const int rpb = 256 / (shape->D / 4);  // rows per combine workgroup
      const dim3 grid(static_cast<unsigned>(static_cast<long long>(prm.B) * prm.Hkv *
                                            ((prm.M + rpb - 1) / rpb)));
      // U = splits loaded at once: the fewest of 2, 4, 8, 16 covering them
      // (16 splits in one group of loads rather than two: 72.4 against 76.4
      // us per call on 8 KV heads x 256 rows x 32832 keys)
      const int u = pl.splits <= 2 ? 2 : pl.splits <= 4 ? 4 : pl.splits <= 8 ? 8 : 16;
#define PTD_COMBINE(d_, u_) \
  if (shape->D == d_ && u == u_) hipLaunchKernelGGL((k_attn_combine<d_, u_>), grid, dim3(256), 0, st, prm);
      PTD_COMBINE(128, 2) PTD_COMBINE(128, 4) PTD_COMBINE(128, 8) PTD_COMBINE(128, 16)
      PTD_COMBINE(64, 2) PTD_COMBINE(64, 4) PTD_COMBINE(64, 8) PTD_COMBINE(64, 16)
#undef PTD_COMBINE
    }
  } else {
    const dim3 grid(pl.passes, prm.Hkv, prm.B);
    PTD_RETURN_IF(prm.Hkv > 65535 || prm.B > 65535, PTD_ERR_SHAPE);
    if (shape->D == 128) hipLaunchKernelGGL(k_attn_valu<128>, grid, dim3(kValuThreads), 0, st, prm);
    else hipLaunchKernelGGL(k_attn_valu<64>, grid, dim3(kValuThreads), 0, st, prm);
  }
  return ptd_launch_status();
}

}  // namespace

extern "C" int ptd_tree_attention(const void* q, const void* k_cache, const void* v_cache,
                                  const int32_t* kv_len, const int32_t* parent, int32_t T,
                                  void* out, const ptd_attn_shape* shape,
                                  const uint64_t* mask, void* workspace,
                                  size_t workspace_bytes, int32_t* dev_status,
                                  void* stream) {
  return attention_impl(q, k_cache, v_cache, kv_len, nullptr, parent, T, out, shape, mask,
                        workspace, workspace_bytes, dev_status, stream, nullptr, 0, 0, 0);
}

extern "C" int ptd_tree_attention_ragged(const void* q, const void* k_cache, const void* v_cache,
                                         const int32_t* kv_len, const int32_t* tree_len,
                                         const int32_t* parent, int32_t T, void* out,
                                         const ptd_attn_shape* shape, const uint64_t* mask,
                                         void* workspace, size_t workspace_bytes,
                                         int32_t* dev_status, void* stream) {
  return attention_impl(q, k_cache, v_cache, kv_len, tree_len, parent, T, out, shape, mask,
                        workspace, workspace_bytes, dev_status, stream, nullptr, 0, 0, 0);
}

extern "C" int ptd_tree_attention_noalloc(const void* q, const void* k_cache, const void* v_cache,
                                          const int32_t* kv_len, const int32_t* tree_len,
                                          const int32_t* parent, int32_t T, void* out,
                                          const ptd_attn_shape* shape, const uint64_t* mask,
                                          int32_t* dev_status, void* stream) {
  return attention_impl(q, k_cache, v_cache, kv_len, tree_len, parent, T, out, shape, mask,
                        nullptr, 0, dev_status, stream, nullptr, 0, 0, 0, false, nullptr, nullptr,
                        true);
}

extern "C" int ptd_tree_attention_fp8kv(const void* q, const void* k_cache, const void* v_cache,
                                        const float* k_scale, const float* v_scale,
                                        const int32_t* kv_len, const int32_t* tree_len,
                                        const int32_t* parent, int32_t T, void* out,
                                        const ptd_attn_shape* shape, void* workspace,
                                        size_t workspace_bytes, int32_t* dev_status,
                                        void* stream) {
  PTD_RETURN_IF(!shape, PTD_ERR_NULL);
  PTD_RETURN_IF(shape->in_dtype != PTD_BF16, PTD_ERR_DTYPE);  // bf16 queries (the MFMA path)
  PTD_RETURN_IF(shape->D != 128, PTD_ERR_SHAPE);
  PTD_RETURN_IF((k_scale && !ptd_aligned(k_scale, 4)) || (v_scale && !ptd_aligned(v_scale, 4)),
                PTD_ERR_ALIGN);
  return attention_impl(q, k_cache, v_cache, kv_len, tree_len, parent, T, out, shape, nullptr,
                        workspace, workspace_bytes, dev_status, stream, nullptr, 0, 0, 0, true,
                        k_scale, v_scale);
}

namespace {

// Checks of a page description; the page-size shift on success.
int paged_args(const ptd_kv_pages* kv, const ptd_attn_shape* shape, int* shift) {
  PTD_RETURN_IF(!kv || !shape, PTD_ERR_NULL);
  PTD_RETURN_IF(!kv->k_pages || !kv->v_pages || !kv->page_table, PTD_ERR_NULL);
  PTD_RETURN_IF(shape->in_dtype != PTD_BF16, PTD_ERR_DTYPE);  // the MFMA path only
  const int ps = kv->page_size;
  PTD_RETURN_IF(ps < 32 || ps > (1 << 20) || (ps & (ps - 1)) != 0, PTD_ERR_SHAPE);
  PTD_RETURN_IF(kv->max_pages < 1 || kv->num_pages < 1, PTD_ERR_SHAPE);
  PTD_RETURN_IF(static_cast<long long>(kv->max_pages) * ps != shape->L_cap, PTD_ERR_SHAPE);
  int sh = 0;
  while ((1 << sh) < ps) ++sh;
  *shift = sh;
  return PTD_OK;
}

}  // namespace

extern "C" int ptd_tree_attention_paged(const void* q, const ptd_kv_pages* kv,
                                        const int32_t* kv_len, const int32_t* tree_len,
                                        const int32_t* parent, int32_t T,
                                        void* out, const ptd_attn_shape* shape,
                                        const uint64_t* mask, void* workspace,
                                        size_t workspace_bytes, int32_t* dev_status,
                                        void* stream) {
  int shift = 0;
  const int rc = paged_args(kv, shape, &shift);
  if (rc != PTD_OK) return rc;
  return attention_impl(q, kv->k_pages, kv->v_pages, kv_len, tree_len, parent, T, out, shape, mask,
                        workspace, workspace_bytes, dev_status, stream, kv->page_table, shift,
                        kv->max_pages, kv->num_pages);
}

extern "C" int ptd_tree_attention_paged_fp8kv(const void* q, const ptd_kv_pages* kv,
                                              const float* k_scale, const float* v_scale,
                                              const int32_t* kv_len, const int32_t* tree_len,
                                              const int32_t* parent, int32_t T, void* out,
                                              const ptd_attn_shape* shape, void* workspace,
                                              size_t workspace_bytes, int32_t* dev_status,
                                              void* stream) {
  int shift = 0;
  const int rc = paged_args(kv, shape, &shift);
  if (rc != PTD_OK) return rc;
  PTD_RETURN_IF(shape->D != 128, PTD_ERR_SHAPE);
  PTD_RETURN_IF((k_scale && !ptd_aligned(k_scale, 4)) || (v_scale && !ptd_aligned(v_scale, 4)),
                PTD_ERR_ALIGN);
  return attention_impl(q, kv->k_pages, kv->v_pages, kv_len, tree_len, parent, T, out, shape,
                        nullptr, workspace, workspace_bytes, dev_status, stream, kv->page_table,
                        shift, kv->max_pages, kv->num_pages, true, k_scale, v_scale);
}
