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
//                  8 waves (2 per SIMD), each owning up to 32 query rows and a
//                  share of every key tile.  K/V tiles of 128 keys are streamed
//                  HBM -> VGPR -> LDS (double buffered, one barrier per tile)
//                  and shared by every query row of the GQA group.  Scores are computed
//                  transposed, S^T = K Q^T, and the output as O^T = V^T P^T,
//                  so each lane owns one query column in both accumulators and
//                  the online-softmax rescale is lane-local.  MFMA:
//                  v_mfma_f32_16x16x32_bf16, fp32 accumulation.
//   k_attn_valu    fp32 (or bf16) inputs on the vector ALUs, fp32 throughout.
//   k_attn_combine merges split-KV partials (m, l, O) in a fixed split order.
#include <math.h>

#include "ptd_common.hpp"
#include "ptd_internal.hpp"

namespace {

using bf16x8 = __bf16 __attribute__((ext_vector_type(8)));
using f32x4 = float __attribute__((ext_vector_type(4)));
using u32x4 = uint32_t __attribute__((ext_vector_type(4)));
using u32x2 = uint32_t __attribute__((ext_vector_type(2)));

constexpr int kThreads = 512;   // 8 waves
constexpr int kKT = 128;        // keys per LDS tile
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegBig = -1.0e30f;  // running-max start: finite, below any score

struct AttnParams {
  const void* q;
  const void* k;
  const void* v;
  const int32_t* kv_len;
  const uint64_t* mask;
  void* out;
  float* part_o;    // [S][B][Hkv][M][D]
  float2* part_ml;  // [S][B][Hkv][M]: (running max * c, sum of p)
  int32_t* dev_status;
  int B, T, Hq, Hkv, G, M, L_cap, W;
  int splits, passes, rows_per_pass;
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

__device__ inline void logical_block(int nblocks, int& id) {
  // Work items that share K/V and queries (the splits of one (b, g)) get
  // consecutive logical ids; blocks are dealt round-robin over the 8 XCDs, so
  // map each XCD to one contiguous range of logical ids (same L2).
  const int bid = blockIdx.x;
  if ((nblocks & 7) == 0) {
    id = (bid & 7) * (nblocks >> 3) + (bid >> 3);
  } else {
    id = bid;
  }
}

// ===========================================================================
// MFMA path
// ===========================================================================
template <int D>
struct TileLayout {
  static constexpr int KS = D + 8;    // K tile row stride (bf16 elements)
  static constexpr int VS = kKT + 8;  // V^T tile row stride
  static constexpr int K_ELEMS = kKT * KS;
  static constexpr int V_ELEMS = D * VS;
  static constexpr int STAGE_ELEMS = K_ELEMS + V_ELEMS;
  static constexpr int KCHUNKS = kKT * D / 8;     // 16-byte K chunks per tile
  static constexpr int VUNITS = (kKT / 4) * (D / 8);  // (4 keys x 8 d) V units per tile
  static constexpr int KU = (KCHUNKS + kThreads - 1) / kThreads;
  static constexpr int VU = (VUNITS + kThreads - 1) / kThreads;
};

template <int D, int QB, int WR>
__global__ void __launch_bounds__(kThreads, 1) k_attn_mfma(AttnParams p) {
  using L = TileLayout<D>;
  constexpr int WK = (kThreads / PTD_WAVE) / WR;  // key groups
  constexpr int KPW = kKT / WK;         // keys per wave per tile
  constexpr int SUBS = KPW / 32;        // 32-key MFMA steps per wave per tile
  constexpr int DB = D / 32;            // 32-wide d blocks (QK^T k-dim)
  constexpr int DT = D / 16;            // 16-wide d tiles (PV output rows)
  constexpr int STAGE_BYTES = L::STAGE_ELEMS * 2;
  constexpr int COMB_BYTES = (WK - 1) * WR * (QB * DT * 64 * 16 + QB * 64 * 8);
  constexpr int SMEM = (2 * STAGE_BYTES > COMB_BYTES) ? 2 * STAGE_BYTES : COMB_BYTES;
  __shared__ __attribute__((aligned(16))) unsigned char smem[SMEM];

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int wr = wave % WR;
  const int kg = wave / WR;
  const int l16 = lane & 15;
  const int l4 = lane >> 4;

  int id;
  logical_block(gridDim.x, id);
  const int split = id % p.splits;
  int rest = id / p.splits;
  const int pass = rest % p.passes;
  rest /= p.passes;
  const int g = rest % p.Hkv;
  const int b = rest / p.Hkv;

  const int n_kv = p.kv_len[b];
  if (n_kv < 0 || n_kv + p.T > p.L_cap) {
    if (tid == 0) ptd::report(p.dev_status, PTD_ERR_KV_LEN);
    return;
  }
  const int N = n_kv + p.T;
  const int csz = chunk_size(N, p.splits);
  const int start = split * csz;
  const int end = min(N, start + csz);
  if (start >= end) return;  // empty split: the combine skips it

  const uint16_t* kbase = static_cast<const uint16_t*>(p.k) +
                          (static_cast<size_t>(b) * p.Hkv + g) * p.L_cap * D;
  const uint16_t* vbase = static_cast<const uint16_t*>(p.v) +
                          (static_cast<size_t>(b) * p.Hkv + g) * p.L_cap * D;
  const int rowbase = pass * p.rows_per_pass + wr * 16 * QB;
  const bool wave_live = rowbase < p.M;  // padding waves only join the barriers

  // ---- query fragments (B operand of S^T = K Q^T): lane holds
  //      Q[row l16][d = 32*db + 8*l4 .. +8]
  bf16x8 qf[QB][DB];
  const uint64_t* mrow[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int r = rowbase + qb * 16 + l16;
    const bool live = r < p.M;
    const int i = live ? r / p.G : 0;
    const int hg = live ? r % p.G : 0;
    mrow[qb] = p.mask + (static_cast<size_t>(b) * p.T + i) * p.W;
    const uint16_t* qrow = static_cast<const uint16_t*>(p.q) +
                           ((static_cast<size_t>(b) * p.T + i) * p.Hq + g * p.G + hg) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (live) v = *reinterpret_cast<const u32x4*>(qrow + db * 32 + l4 * 8);
      qf[qb][db] = __builtin_bit_cast(bf16x8, v);
    }
  }

  f32x4 o[QB][DT];
  float m[QB], lsum[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m[qb] = kNegBig;
    lsum[qb] = 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[qb][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // ---- tile staging: HBM -> registers -> LDS
  u32x4 kreg[L::KU];
  u32x4 vreg[L::VU][4];
  auto load_tile = [&](int t0) {
#pragma unroll
    for (int u = 0; u < L::KU; ++u) {
      const int c = tid + kThreads * u;
      if (L::KCHUNKS % kThreads && c >= L::KCHUNKS) break;
      const int key = c / (D / 8), dch = c % (D / 8);
      const int row = min(t0 + key, N - 1);
      kreg[u] = *reinterpret_cast<const u32x4*>(kbase + static_cast<size_t>(row) * D + dch * 8);
    }
#pragma unroll
    for (int u = 0; u < L::VU; ++u) {
      const int unit = tid + kThreads * u;
      if (L::VUNITS % kThreads && unit >= L::VUNITS) break;
      const int kgrp = unit / (D / 8), dch = unit % (D / 8);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = min(t0 + 4 * kgrp + e, N - 1);
        vreg[u][e] = *reinterpret_cast<const u32x4*>(vbase + static_cast<size_t>(row) * D + dch * 8);
      }
    }
  };
  auto store_tile = [&](int stage) {
    uint16_t* ks = reinterpret_cast<uint16_t*>(smem) + stage * L::STAGE_ELEMS;
    uint16_t* vt = ks + L::K_ELEMS;
#pragma unroll
    for (int u = 0; u < L::KU; ++u) {
      const int c = tid + kThreads * u;
      if (L::KCHUNKS % kThreads && c >= L::KCHUNKS) break;
      const int key = c / (D / 8), dch = c % (D / 8);
      *reinterpret_cast<u32x4*>(ks + key * L::KS + dch * 8) = kreg[u];
    }
#pragma unroll
    for (int u = 0; u < L::VU; ++u) {
      const int unit = tid + kThreads * u;
      if (L::VUNITS % kThreads && unit >= L::VUNITS) break;
      const int kgrp = unit / (D / 8), dch = unit % (D / 8);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int w = j >> 1;
        uint32_t a0 = vreg[u][0][w], a1 = vreg[u][1][w], a2 = vreg[u][2][w], a3 = vreg[u][3][w];
        u32x2 pk;
        if (j & 1) {
          pk[0] = (a0 >> 16) | (a1 & 0xFFFF0000u);
          pk[1] = (a2 >> 16) | (a3 & 0xFFFF0000u);
        } else {
          pk[0] = (a0 & 0xFFFFu) | (a1 << 16);
          pk[1] = (a2 & 0xFFFFu) | (a3 << 16);
        }
        *reinterpret_cast<u32x2*>(vt + (dch * 8 + j) * L::VS + 4 * kgrp) = pk;
      }
    }
  };

  const int ntiles = (end - start + kKT - 1) / kKT;
  load_tile(start);
  store_tile(0);
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const int t0 = start + t * kKT;
    const bool more = t + 1 < ntiles;
    if (more) load_tile(t0 + kKT);

    const uint16_t* ks = reinterpret_cast<const uint16_t*>(smem) + (t & 1) * L::STAGE_ELEMS;
    const uint16_t* vt = ks + L::K_ELEMS;
#pragma unroll
    for (int sub = 0; sub < SUBS; ++sub) {
      const int ko = kg * KPW + sub * 32;  // key offset inside the tile
      const int abs0 = t0 + ko;
      if (abs0 >= end || !wave_live) break;

      // ---- S^T (keys x queries) = K Q^T; lane: query l16, keys 4*l4 + e
      f32x4 s[2][QB];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) s[kb][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int db = 0; db < DB; ++db) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          const u32x4 kv = *reinterpret_cast<const u32x4*>(
              ks + (ko + kb * 16 + l16) * L::KS + db * 32 + l4 * 8);
          const bf16x8 kf = __builtin_bit_cast(bf16x8, kv);
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
            s[kb][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[qb][db], s[kb][qb], 0, 0, 0);
        }
      }

      // ---- visibility: past the chunk end, or a tree key that is not an ancestor
      if (abs0 + 32 > n_kv || abs0 + 32 > end) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int key = abs0 + kb * 16 + l4 * 4 + e;
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) {
              bool vis = key < end;
              if (vis && key >= n_kv) {
                const int a = key - n_kv;
                vis = (mrow[qb][a >> 6] >> (a & 63)) & 1ull;
              }
              if (!vis) s[kb][qb][e] = -INFINITY;
            }
          }
      }

      // ---- online softmax (exp2 domain), lane-local per query column
      bf16x8 pf[QB], pfl[QB];
      bool rescale = false;
      float alpha[QB];
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        float mx = fmaxf(fmaxf(fmaxf(s[0][qb][0], s[0][qb][1]), fmaxf(s[0][qb][2], s[0][qb][3])),
                         fmaxf(fmaxf(s[1][qb][0], s[1][qb][1]), fmaxf(s[1][qb][2], s[1][qb][3])));
        mx = fmaxf(mx, __shfl_xor(mx, 16, PTD_WAVE));
        mx = fmaxf(mx, __shfl_xor(mx, 32, PTD_WAVE));
        const float m_new = fmaxf(m[qb], mx);
        alpha[qb] = __builtin_amdgcn_exp2f((m[qb] - m_new) * p.c);
        rescale |= m_new != m[qb];
        m[qb] = m_new;
        const float mc = m_new * p.c;
        float pv[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          pv[e] = __builtin_amdgcn_exp2f(fmaf(s[0][qb][e], p.c, -mc));
          pv[4 + e] = __builtin_amdgcn_exp2f(fmaf(s[1][qb][e], p.c, -mc));
        }
        // p = hi + lo with hi = bf16(p), lo = bf16(p - hi): the PV product
        // then sees p to ~2^-17 relative instead of bf16's 2^-9
        u32x4 ph, pl;
        float ps = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          ph[w] = ptd::pack_bf16x2(pv[2 * w], pv[2 * w + 1]);
          pl[w] = ptd::pack_bf16x2(pv[2 * w] - ptd::bf16_lo(ph[w]),
                                   pv[2 * w + 1] - ptd::bf16_hi(ph[w]));
          ps += pv[2 * w] + pv[2 * w + 1];
        }
        lsum[qb] = lsum[qb] * alpha[qb] + ps;
        pf[qb] = __builtin_bit_cast(bf16x8, ph);
        pfl[qb] = __builtin_bit_cast(bf16x8, pl);
      }
      if (__any(rescale)) {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) o[qb][dt] *= alpha[qb];
      }

      // ---- O^T (d x queries) += V^T P^T; k-slot j of lane group l4 is key
      //      4*l4 + j (j < 4) or 16 + 4*l4 + (j - 4), matching the S^T layout
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const uint16_t* vrow = vt + (dt * 16 + l16) * L::VS + ko + l4 * 4;
        const u32x2 lo = *reinterpret_cast<const u32x2*>(vrow);
        const u32x2 hi = *reinterpret_cast<const u32x2*>(vrow + 16);
        const u32x4 vv = {lo[0], lo[1], hi[0], hi[1]};
        const bf16x8 vf = __builtin_bit_cast(bf16x8, vv);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
          o[qb][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[qb], o[qb][dt], 0, 0, 0);
          o[qb][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pfl[qb], o[qb][dt], 0, 0, 0);
        }
      }
    }

    if (more) store_tile((t + 1) & 1);
    __syncthreads();
  }

  // ---- per-column totals of the softmax denominator
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    lsum[qb] += __shfl_xor(lsum[qb], 16, PTD_WAVE);
    lsum[qb] += __shfl_xor(lsum[qb], 32, PTD_WAVE);
  }

  // ---- merge the key groups of the workgroup (fixed order kg = 1..WK-1)
  if constexpr (WK > 1) {
    constexpr int OBYTES = QB * DT * 64 * 16;
    constexpr int SLOT = OBYTES + QB * 64 * 8;
    if (kg > 0) {
      unsigned char* slot = smem + ((kg - 1) * WR + wr) * SLOT;
      f32x4* so = reinterpret_cast<f32x4*>(slot);
      float2* sml = reinterpret_cast<float2*>(slot + OBYTES);
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) so[(qb * DT + dt) * 64 + lane] = o[qb][dt];
        sml[qb * 64 + lane] = make_float2(m[qb], lsum[qb]);
      }
    }
    __syncthreads();
    if (kg > 0) return;
#pragma unroll
    for (int k2 = 1; k2 < WK; ++k2) {
      const unsigned char* slot = smem + ((k2 - 1) * WR + wr) * SLOT;
      const f32x4* so = reinterpret_cast<const f32x4*>(slot);
      const float2* sml = reinterpret_cast<const float2*>(slot + OBYTES);
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const float2 ml = sml[qb * 64 + lane];
        const float mn = fmaxf(m[qb], ml.x);
        const float w0 = __builtin_amdgcn_exp2f((m[qb] - mn) * p.c);
        const float w1 = __builtin_amdgcn_exp2f((ml.x - mn) * p.c);
        m[qb] = mn;
        lsum[qb] = lsum[qb] * w0 + ml.y * w1;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[qb][dt] = o[qb][dt] * w0 + so[(qb * DT + dt) * 64 + lane] * w1;
      }
    }
  }

  // ---- write: lane holds O^T[d = 16*dt + 4*l4 + 0..3][query l16]
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int r = rowbase + qb * 16 + l16;
    if (r >= p.M) continue;
    if (p.splits == 1) {
      const int i = r / p.G, hg = r % p.G;
      const size_t off = ((static_cast<size_t>(b) * p.T + i) * p.Hq + g * p.G + hg) * D;
      const float inv = 1.0f / lsum[qb];
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const int d0 = dt * 16 + l4 * 4;
        const f32x4 v = o[qb][dt] * inv;
        if (p.out_bf16) {
          u32x2 w = {ptd::pack_bf16x2(v[0], v[1]), ptd::pack_bf16x2(v[2], v[3])};
          *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(p.out) + off + d0) = w;
        } else {
          *reinterpret_cast<f32x4*>(static_cast<float*>(p.out) + off + d0) = v;
        }
      }
    } else {
      const size_t prow = ((static_cast<size_t>(split) * p.B + b) * p.Hkv + g) * p.M + r;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        *reinterpret_cast<f32x4*>(p.part_o + prow * D + dt * 16 + l4 * 4) = o[qb][dt];
      if (l4 == 0) p.part_ml[prow] = make_float2(m[qb] * p.c, lsum[qb]);
    }
  }
}

// ===========================================================================
// split-KV combine: out = sum_s w_s O_s / sum_s w_s l_s, w_s = 2^(mc_s - max mc)
// ===========================================================================
template <int D>
__global__ void __launch_bounds__(256) k_attn_combine(AttnParams p) {
  const size_t idx = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  constexpr int D4 = D / 4;
  const size_t total = static_cast<size_t>(p.B) * p.Hkv * p.M * D4;
  if (idx >= total) return;
  const int d4 = static_cast<int>(idx % D4);
  size_t rest = idx / D4;
  const int r = static_cast<int>(rest % p.M);
  rest /= p.M;
  const int g = static_cast<int>(rest % p.Hkv);
  const int b = static_cast<int>(rest / p.Hkv);
  const int n_kv = p.kv_len[b];
  if (n_kv < 0 || n_kv + p.T > p.L_cap) return;  // reported by the attention kernel
  const int N = n_kv + p.T;
  const int csz = chunk_size(N, p.splits);
  const int nsp = (N + csz - 1) / csz;  // non-empty splits
  const size_t stride = static_cast<size_t>(p.B) * p.Hkv * p.M;
  const size_t row0 = (static_cast<size_t>(b) * p.Hkv + g) * p.M + r;
  float mx = kNegBig;
  for (int s = 0; s < nsp; ++s) mx = fmaxf(mx, p.part_ml[row0 + s * stride].x);
  float den = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < nsp; ++s) {
    const float2 ml = p.part_ml[row0 + s * stride];
    const float w = __builtin_amdgcn_exp2f(ml.x - mx);
    den += w * ml.y;
    acc += w * *reinterpret_cast<const f32x4*>(p.part_o + (row0 + s * stride) * D + d4 * 4);
  }
  const f32x4 v = acc * (1.0f / den);
  const int i = r / p.G, hg = r % p.G;
  const size_t off = ((static_cast<size_t>(b) * p.T + i) * p.Hq + g * p.G + hg) * D + d4 * 4;
  if (p.out_bf16) {
    u32x2 w = {ptd::pack_bf16x2(v[0], v[1]), ptd::pack_bf16x2(v[2], v[3])};
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
  if (n_kv < 0 || n_kv + p.T > p.L_cap) {
    if (tid == 0) ptd::report(p.dev_status, PTD_ERR_KV_LEN);
    return;
  }
  const int N = n_kv + p.T;
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
    const float v = acc[rl][d] / sl[rl];
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
  size_t partial_bytes, mask_bytes, total_bytes;
};

constexpr int kTargetBlocks = 256;  // one resident workgroup per CU on MI355X

bool make_plan(const ptd_attn_shape* s, int T, Plan* pl) {
  if (!s || s->B < 1 || s->Hq < 1 || s->Hkv < 1 || s->Hq % s->Hkv) return false;
  if (s->D != 64 && s->D != 128) return false;
  if (T < 1 || T > PTD_MAX_T || s->L_cap < T) return false;
  if ((s->in_dtype != PTD_F32 && s->in_dtype != PTD_BF16) ||
      (s->out_dtype != PTD_F32 && s->out_dtype != PTD_BF16))
    return false;
  const long long M = static_cast<long long>(T) * (s->Hq / s->Hkv);
  if (M > (1 << 24)) return false;
  pl->mfma = s->in_dtype == PTD_BF16;
  if (pl->mfma) {
    const int mp = static_cast<int>(M < 256 ? M : 256);
    const int nblk = (mp + 15) / 16;
    // 8 waves: WR row groups of 16*QB rows (QB <= 2) x (8/WR) key groups,
    // each key group at least 32 keys of the 128-key tile
    if (nblk <= 4) { pl->WR = 2; pl->QB = (nblk + 1) / 2; }
    else if (nblk <= 8) { pl->WR = 4; pl->QB = (nblk + 3) / 4; }
    else { pl->WR = 8; pl->QB = (nblk + 7) / 8; }
    pl->rows_per_pass = 16 * pl->QB * pl->WR;
    pl->passes = static_cast<int>((M + pl->rows_per_pass - 1) / pl->rows_per_pass);
    const long long items = static_cast<long long>(s->B) * s->Hkv * pl->passes;
    int sp = static_cast<int>(kTargetBlocks / items);
    const int max_by_len = (s->L_cap + 255) / 256;  // at least ~256 keys per split
    if (sp > max_by_len) sp = max_by_len;
    if (sp < 1) sp = 1;
    if (sp > 64) sp = 64;
    pl->splits = sp;
  } else {
    pl->WR = pl->QB = 0;
    pl->rows_per_pass = kValuRows;
    pl->passes = static_cast<int>((M + kValuRows - 1) / kValuRows);
    pl->splits = 1;
  }
  if (static_cast<long long>(s->B) * s->Hkv * pl->passes * pl->splits > 0x7FFFFFFFLL) return false;
  pl->partial_bytes = pl->splits > 1
      ? static_cast<size_t>(pl->splits) * s->B * s->Hkv * M * (s->D + 2) * sizeof(float)
      : 0;
  pl->partial_bytes = (pl->partial_bytes + 255) & ~static_cast<size_t>(255);
  pl->mask_bytes = static_cast<size_t>(s->B) * T * ((T + 63) / 64) * sizeof(uint64_t);
  pl->mask_bytes = (pl->mask_bytes + 255) & ~static_cast<size_t>(255);
  pl->total_bytes = pl->partial_bytes + pl->mask_bytes;
  return true;
}

template <int D>
void launch_mfma(const Plan& pl, const AttnParams& prm, hipStream_t st) {
  const dim3 grid(prm.B * prm.Hkv * pl.passes * pl.splits);
  const dim3 block(kThreads);
#define PTD_MFMA_CASE(qb_, wr_) \
  if (pl.QB == qb_ && pl.WR == wr_) { hipLaunchKernelGGL((k_attn_mfma<D, qb_, wr_>), grid, block, 0, st, prm); return; }
  PTD_MFMA_CASE(1, 2) PTD_MFMA_CASE(2, 2)
  PTD_MFMA_CASE(1, 4) PTD_MFMA_CASE(2, 4)
  PTD_MFMA_CASE(1, 8) PTD_MFMA_CASE(2, 8)
#undef PTD_MFMA_CASE
}

}  // namespace

extern "C" size_t ptd_tree_attention_workspace_bytes(const ptd_attn_shape* shape, int32_t T) {
  Plan pl;
  if (!make_plan(shape, T, &pl)) return 0;
  return pl.total_bytes;
}

extern "C" int ptd_tree_attention(const void* q, const void* k_cache, const void* v_cache,
                                  const int32_t* kv_len, const int32_t* parent, int32_t T,
                                  void* out, const ptd_attn_shape* shape,
                                  const uint64_t* mask, void* workspace,
                                  size_t workspace_bytes, int32_t* dev_status,
                                  void* stream) {
  PTD_RETURN_IF(!q || !k_cache || !v_cache || !kv_len || !parent || !out || !shape,
                PTD_ERR_NULL);
  if (shape->in_dtype != PTD_F32 && shape->in_dtype != PTD_BF16) return PTD_ERR_DTYPE;
  if (shape->out_dtype != PTD_F32 && shape->out_dtype != PTD_BF16) return PTD_ERR_DTYPE;
  Plan pl;
  PTD_RETURN_IF(!make_plan(shape, T, &pl), PTD_ERR_SHAPE);
  PTD_RETURN_IF(!ptd_aligned(q, 16) || !ptd_aligned(k_cache, 16) || !ptd_aligned(v_cache, 16) ||
                    !ptd_aligned(out, 16) || (mask && !ptd_aligned(mask, 8)),
                PTD_ERR_ALIGN);
  const size_t need = mask ? pl.partial_bytes : pl.total_bytes;
  if (need > 0) {
    PTD_RETURN_IF(!workspace, PTD_ERR_WORKSPACE);
    PTD_RETURN_IF(workspace_bytes < need, PTD_ERR_WORKSPACE);
    PTD_RETURN_IF(!ptd_aligned(workspace, 256), PTD_ERR_ALIGN);
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  if (!mask) {
    uint64_t* mws = reinterpret_cast<uint64_t*>(ws + pl.partial_bytes);
    const int rc = ptd_launch_tree_mask(parent, nullptr, shape->B, T, mws, nullptr, dev_status, st);
    if (rc != PTD_OK) return rc;
    mask = mws;
  }
  AttnParams prm;
  prm.q = q;
  prm.k = k_cache;
  prm.v = v_cache;
  prm.kv_len = kv_len;
  prm.mask = mask;
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
  if (pl.splits > 1) {
    const size_t rows = static_cast<size_t>(pl.splits) * prm.B * prm.Hkv * prm.M;
    prm.part_ml = reinterpret_cast<float2*>(prm.part_o + rows * shape->D);
  }
  if (pl.mfma) {
    if (shape->D == 128) launch_mfma<128>(pl, prm, st);
    else launch_mfma<64>(pl, prm, st);
    if (pl.splits > 1) {
      const size_t total = static_cast<size_t>(prm.B) * prm.Hkv * prm.M * (shape->D / 4);
      const dim3 grid(static_cast<unsigned>((total + 255) / 256));
      if (shape->D == 128) hipLaunchKernelGGL(k_attn_combine<128>, grid, dim3(256), 0, st, prm);
      else hipLaunchKernelGGL(k_attn_combine<64>, grid, dim3(256), 0, st, prm);
    }
  } else {
    const dim3 grid(pl.passes, prm.Hkv, prm.B);
    PTD_RETURN_IF(prm.Hkv > 65535 || prm.B > 65535, PTD_ERR_SHAPE);
    if (shape->D == 128) hipLaunchKernelGGL(k_attn_valu<128>, grid, dim3(kValuThreads), 0, st, prm);
    else hipLaunchKernelGGL(k_attn_valu<64>, grid, dim3(kValuThreads), 0, st, prm);
  }
  return ptd_launch_status();
}
