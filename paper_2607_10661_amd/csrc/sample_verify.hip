// Sampling verification of a draft tree (Sec. 3.2 "sampling decoding
// strategy"; App. E recursive candidate-tree sampling; App. F proof of
// distributional consistency).
//
// P_v = softmax(logits row of v / temperature); row 0 is the last committed
// token n_0 (the parent of every root), row v + 1 is node v.  From n_0 the
// children of the current node are examined in index order; child n (token
// t_n) is accepted iff u_node[n] < P_v[t_n] / S, S being the mass of P_v not
// yet rejected at this node (App. F divides by it).  A rejected token's
// probability becomes 0, so a later sibling with the same token is rejected.
// On acceptance the walk moves to n; when every child is rejected the node is
// the terminal and the bonus token is drawn by inverse CDF (index order) from
// the residual distribution with u_bonus[row].
//
// Kernels
//   k_block_stats    one wave per (block of 2048 vocabulary entries, logits
//                    row), four per workgroup (k_block_stats_wg: one
//                    workgroup per block, for calls with few blocks): the
//                    block maximum m_b and
//                    z_b = sum exp((l - m_b) / temperature) over the block,
//                    each term an fp32 exponential with its argument's
//                    rounding compensated (~1.2e-7 relative), added in fp64.
//   k_verify_sample  one workgroup of 1024 threads per sequence.  Each row's
//                    maximum m and normalizer z = sum_b z_b e^((m_b - m)/t)
//                    are formed in LDS; the tree, the uniforms and every
//                    node's probability under its parent's row (numerator in
//                    fp64) are staged.  Each level of the walk lists the
//                    current node's children in index order with ballots, and
//                    one thread takes the accept / reject decisions in order;
//                    rejected tokens are marked in an LDS bitmap (one bit per
//                    vocabulary entry).  Bonus draw: the block sums of the
//                    terminal's row, less the rejected terms, locate the block
//                    where the running total passes u * W; that block's 2048
//                    terms are recomputed (the same arithmetic) and scanned by
//                    all threads.
#include <math.h>

#include "ptd_common.hpp"

namespace {

constexpr int kStatThreads = 256;
constexpr int kBlock = 2048;  // vocabulary entries per statistics block
constexpr int kWalkThreads = 1024;
constexpr int kWalkWaves = kWalkThreads / PTD_WAVE;
constexpr int kMaxVocab = 262144;  // LDS bitmap of rejected tokens: 32 KB
constexpr int kMaxBlocks = kMaxVocab / kBlock;

template <bool BF16>
__device__ __forceinline__ float logit(const void* row, int y) {
  if constexpr (BF16) return ptd::bf16_to_f32(static_cast<const uint16_t*>(row)[y]);
  else return static_cast<const float*>(row)[y];
}

__device__ __forceinline__ double shfl_up_f64(double x, int d) {
  const uint64_t u = __double_as_longlong(x);
  const uint32_t lo = __shfl_up(static_cast<uint32_t>(u), d, PTD_WAVE);
  const uint32_t hi = __shfl_up(static_cast<uint32_t>(u >> 32), d, PTD_WAVE);
  return __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(hi) << 32) | lo));
}
// One DPP step of a wave scan on an fp64 value (both halves moved with the
// same control; lanes outside the row or the row mask receive +0.0).
template <int CTRL, int ROWS>
__device__ __forceinline__ double dpp_f64(double x) {
  const uint64_t u = __double_as_longlong(x);
  const uint32_t lo = static_cast<uint32_t>(
      __builtin_amdgcn_update_dpp(0, static_cast<int>(static_cast<uint32_t>(u)), CTRL, ROWS, 0xF, false));
  const uint32_t hi = static_cast<uint32_t>(
      __builtin_amdgcn_update_dpp(0, static_cast<int>(static_cast<uint32_t>(u >> 32)), CTRL, ROWS, 0xF, false));
  return __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(hi) << 32) | lo));
}
// Inclusive prefix sum over the wave on the vector ALU: row_shr 1, 2, 4, 8
// within rows of 16 lanes, then row_bcast:15 (into rows 1 and 3) and
// row_bcast:31 (into rows 2 and 3).
__device__ __forceinline__ double wave_incl_scan_f64(double x) {
  x += dpp_f64<0x111, 0xF>(x);
  x += dpp_f64<0x112, 0xF>(x);
  x += dpp_f64<0x114, 0xF>(x);
  x += dpp_f64<0x118, 0xF>(x);
  x += dpp_f64<0x142, 0xA>(x);
  x += dpp_f64<0x143, 0xC>(x);
  return x;
}
__device__ __forceinline__ double readlane_f64(double x, int lane) {
  const uint64_t u = __double_as_longlong(x);
  const uint32_t lo = __builtin_amdgcn_readlane(static_cast<uint32_t>(u), lane);
  const uint32_t hi = __builtin_amdgcn_readlane(static_cast<uint32_t>(u >> 32), lane);
  return __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(hi) << 32) | lo));
}
__device__ __forceinline__ double shfl_xor_f64(double x, int d) {
  const uint64_t u = __double_as_longlong(x);
  const uint32_t lo = __shfl_xor(static_cast<uint32_t>(u), d, PTD_WAVE);
  const uint32_t hi = __shfl_xor(static_cast<uint32_t>(u >> 32), d, PTD_WAVE);
  return __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(hi) << 32) | lo));
}

struct RowStat {
  double m, z;
};

// exp((l - m) / temperature) as 2^(x) with x = (l - m) * c, c = c_hi + c_lo =
// log2(e) / temperature.  The difference l - m is kept exactly as d_hi + d_lo
// (TwoSum) and the rounding of x is carried to first order, so each term is
// within about one ulp of v_exp_f32 (~1.2e-7 relative) of the exact value.
__device__ __forceinline__ float exp_term(float l, float m, float c_hi, float c_lo) {
  const float d = l - m;
  const float bb = d - l;
  const float d_lo = (l - (d - bb)) + (-m - bb);
  const float x = d * c_hi;
  const float err = fmaf(d, c_hi, -x) + fmaf(d, c_lo, d_lo * c_hi);
  // (x <= 0 here; v_exp_f32 differs from exp2f only where 2^x is subnormal,
  // terms negligible against a sum of at least 1)
  return __builtin_amdgcn_exp2f(x) * fmaf(err, 0.69314718f, 1.0f);
}

using u32x4 = uint32_t __attribute__((ext_vector_type(4)));

// the values of a 16-byte chunk of a row
template <bool BF16>
__device__ __forceinline__ void chunk_vals(const u32x4& c, float (&x)[BF16 ? 8 : 4]) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    if constexpr (BF16) {
      x[2 * w] = ptd::bf16_lo(c[w]);
      x[2 * w + 1] = ptd::bf16_hi(c[w]);
    } else {
      x[w] = __uint_as_float(c[w]);
    }
  }
}

// Block maximum, then the block's sum of terms relative to it: one wave per
// (block, row), four blocks per workgroup, no workgroup barrier.  A 16-byte
// aligned row is read in 16-byte chunks (4 per lane for bf16, 8 for fp32,
// lane-interleaved and all issued before the first is used) plus a scalar
// tail in the last block; other rows element by element.
template <bool BF16>
__global__ void __launch_bounds__(kStatThreads)
k_block_stats(const void* __restrict__ logits, int V, long long ld, int nblk, float c_hi,
              float c_lo, RowStat* __restrict__ stats) {
  constexpr int E = BF16 ? 8 : 4;
  constexpr int CPL = kBlock / E / PTD_WAVE;  // chunks per lane: 4 (bf16) or 8 (fp32)
  const int lane = threadIdx.x & 63;
  const int blk = blockIdx.x * (kStatThreads / PTD_WAVE) + (threadIdx.x >> 6);
  const int r = blockIdx.y;
  if (blk >= nblk) return;  // whole wave
  const char* row = static_cast<const char*>(logits) + static_cast<size_t>(r) * ld * (BF16 ? 2 : 4);
  const int y0 = blk * kBlock, y1 = min(V, y0 + kBlock);
  const bool vec = (reinterpret_cast<uintptr_t>(row) & 15) == 0;
  const int nch = vec ? (y1 - y0) / E : 0;  // whole chunks of this block
  const u32x4* rc = reinterpret_cast<const u32x4*>(row) + y0 / E;
  u32x4 raw[CPL];
#pragma unroll
  for (int j = 0; j < CPL; ++j) {
    const int c = j * PTD_WAVE + lane;
    raw[j] = c < nch ? rc[c] : u32x4{0u, 0u, 0u, 0u};
  }
  float m = -INFINITY;
#pragma unroll
  for (int j = 0; j < CPL; ++j)
    if (j * PTD_WAVE + lane < nch) {
      float x[E];
      chunk_vals<BF16>(raw[j], x);
#pragma unroll
      for (int e = 0; e < E; ++e) m = fmaxf(m, x[e]);
    }
  for (int y = y0 + nch * E + lane; y < y1; y += PTD_WAVE) m = fmaxf(m, logit<BF16>(row, y));
  m = ptd::wave_max(m);
  double z = 0.0;
#pragma unroll
  for (int j = 0; j < CPL; ++j)
    if (j * PTD_WAVE + lane < nch) {
      float x[E];
      chunk_vals<BF16>(raw[j], x);
#pragma unroll
      for (int e = 0; e < E; e += 2)  // pairs added in fp32 (one rounding, 2^-24), then fp64
        z += static_cast<double>(exp_term(x[e], m, c_hi, c_lo) + exp_term(x[e + 1], m, c_hi, c_lo));
    }
  for (int y = y0 + nch * E + lane; y < y1; y += PTD_WAVE)
    z += static_cast<double>(exp_term(logit<BF16>(row, y), m, c_hi, c_lo));
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) z += shfl_xor_f64(z, o);
  if (lane == 0) stats[static_cast<size_t>(r) * nblk + blk] = RowStat{static_cast<double>(m), z};
}

// The same statistics with one workgroup per (block, row), one or two chunks
// per thread: the shorter latency per block where the blocks of a call are
// few (a single sequence's rows).
template <bool BF16>
__global__ void __launch_bounds__(kStatThreads)
k_block_stats_wg(const void* __restrict__ logits, int V, long long ld, int nblk, float c_hi,
              float c_lo, RowStat* __restrict__ stats) {
  constexpr int E = BF16 ? 8 : 4;
  constexpr int NW = kStatThreads / PTD_WAVE;
  constexpr int CPT = kBlock / E / kStatThreads;  // chunks per thread: 1 (bf16) or 2
  __shared__ float s_max[NW];
  __shared__ double s_sum[NW];
  const int blk = blockIdx.x, r = blockIdx.y, tid = threadIdx.x, lane = tid & 63,
            wave = tid >> 6;
  const char* row = static_cast<const char*>(logits) + static_cast<size_t>(r) * ld * (BF16 ? 2 : 4);
  const int y0 = blk * kBlock, y1 = min(V, y0 + kBlock);
  const bool vec = (reinterpret_cast<uintptr_t>(row) & 15) == 0;
  const int nch = vec ? (y1 - y0) / E : 0;  // whole chunks of this block
  const u32x4* rc = reinterpret_cast<const u32x4*>(row) + y0 / E;
  float x[CPT][E];
  bool have[CPT];
#pragma unroll
  for (int j = 0; j < CPT; ++j) {
    const int c = tid + j * kStatThreads;
    have[j] = c < nch;
    if (have[j]) chunk_vals<BF16>(rc[c], x[j]);
  }
  float m = -INFINITY;
#pragma unroll
  for (int j = 0; j < CPT; ++j)
    if (have[j])
#pragma unroll
      for (int e = 0; e < E; ++e) m = fmaxf(m, x[j][e]);
  for (int y = y0 + nch * E + tid; y < y1; y += kStatThreads) m = fmaxf(m, logit<BF16>(row, y));
  m = ptd::wave_max(m);
  if (lane == 0) s_max[wave] = m;
  __syncthreads();
#pragma unroll
  for (int w = 0; w < NW; ++w) m = fmaxf(m, s_max[w]);
  double z = 0.0;
#pragma unroll
  for (int j = 0; j < CPT; ++j)
    if (have[j])
#pragma unroll
      for (int e = 0; e < E; e += 2)  // pairs added in fp32 (one rounding, 2^-24), then fp64
        z += static_cast<double>(exp_term(x[j][e], m, c_hi, c_lo) + exp_term(x[j][e + 1], m, c_hi, c_lo));
  for (int y = y0 + nch * E + tid; y < y1; y += kStatThreads)
    z += static_cast<double>(exp_term(logit<BF16>(row, y), m, c_hi, c_lo));
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) z += shfl_xor_f64(z, o);
  if (lane == 0) s_sum[wave] = z;
  __syncthreads();
  if (tid == 0) {
    double t = 0.0;
    for (int w = 0; w < NW; ++w) t += s_sum[w];
    stats[static_cast<size_t>(r) * nblk + blk] = RowStat{static_cast<double>(m), t};
  }
}

struct SampleArgs {
  const void* logits;
  long long ld;
  int V, T;
  const int32_t* tokens;    // [B][T]
  const int32_t* parent;    // [B][T]
  const int32_t* tree_len;  // [B] or null
  const double* u_node;     // [B][T]
  const double* u_bonus;    // [B][T+1]
  const RowStat* stats;     // [B*(T+1)][nblk] block statistics
  int nblk;
  double inv_temp;          // 1 / temperature
  float c_hi, c_lo;         // log2(e) / temperature = c_hi + c_lo
  int32_t* accept_len;
  int32_t* accept_nodes;
  int32_t* out_tokens;
  int32_t* dev_status;
};

struct WalkLds {
  int par[PTD_MAX_T], tok[PTD_MAX_T], kids[PTD_MAX_T], path[PTD_MAX_T], rej[PTD_MAX_T];
  double p[PTD_MAX_T], u[PTD_MAX_T];
  float rm[PTD_MAX_T + 1];   // row maxima
  double rz[PTD_MAX_T + 1];  // row normalizers
  uint32_t bits[kMaxVocab / 32];
  double res[kMaxBlocks];    // residual block sums of the terminal's row
  float bscale[kMaxBlocks];  // e^((m_b - m)/t) of the terminal's row
  float bm[kMaxBlocks];      // its block maxima
  int wcount[kWalkWaves];
  double wsum[kWalkWaves];
  int nkids, next, depth, nrej, xblk;
  double before, target;
};

// WIDE: rows of more than 32 blocks, whose statistics are combined one wave
// per row and whose bonus block is found by wave scans; narrower rows take
// one thread per row and one thread for the search (shorter code, measured
// faster there).
template <bool BF16, bool WIDE>
__global__ void __launch_bounds__(kWalkThreads) k_verify_sample(SampleArgs a) {
  __shared__ WalkLds L;
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int T = a.T, V = a.V;
  int n = T;
  if (a.tree_len) {
    n = a.tree_len[b];
    n = n < 0 ? 0 : (n > T ? T : n);
  }
  const size_t row0 = static_cast<size_t>(b) * (T + 1);
  auto row_ptr = [&](int r) {
    return static_cast<const char*>(a.logits) + (row0 + r) * a.ld * (BF16 ? 2 : 4);
  };
  int32_t* an = a.accept_nodes + static_cast<size_t>(b) * T;
  int32_t* ot = a.out_tokens + row0;

  // stage the tree and the uniforms; every row's maximum and normalizer from
  // its blocks (loads of both issued together); each node's logit under its
  // parent's row is gathered as soon as the node's own entries have landed
  bool bad = false;
  int my_par = -1, my_tok = -1;
  float my_l = 0.f;
  if (tid < n) {
    my_par = a.parent[static_cast<size_t>(b) * T + tid];
    my_tok = a.tokens[static_cast<size_t>(b) * T + tid];
    L.u[tid] = a.u_node[static_cast<size_t>(b) * T + tid];
  }
  if constexpr (WIDE) {
  // one wave per row, a lane per block (two above 64 blocks), the loads of
  // four rows issued before any is used
  static_assert(kMaxBlocks <= 2 * PTD_WAVE, "two blocks per lane");
  constexpr int kRowsAtOnce = 4;
  for (int r0 = wave; r0 <= T; r0 += kRowsAtOnce * kWalkWaves) {
    RowStat st[kRowsAtOnce][2];
#pragma unroll
    for (int j = 0; j < kRowsAtOnce; ++j) {
      const int r = r0 + j * kWalkWaves;
      const RowStat* bs = a.stats + (row0 + min(r, T)) * a.nblk;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int k = lane + h * PTD_WAVE;
        st[j][h] = (r <= T && k < a.nblk) ? bs[k] : RowStat{-INFINITY, 0.0};
      }
    }
#pragma unroll
    for (int j = 0; j < kRowsAtOnce; ++j) {
      const int r = r0 + j * kWalkWaves;
      if (r > T) break;  // uniform
      const float m = ptd::wave_max(fmaxf(static_cast<float>(st[j][0].m), static_cast<float>(st[j][1].m)));
      double z = 0.0;
#pragma unroll
      for (int h = 0; h < 2; ++h)
        if (lane + h * PTD_WAVE < a.nblk)
          z += st[j][h].z * static_cast<double>(exp_term(static_cast<float>(st[j][h].m), m, a.c_hi, a.c_lo));
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) z += shfl_xor_f64(z, o);
      if (lane == 0) {
        L.rm[r] = m;
        L.rz[r] = z;
      }
    }
  }
  } else {
  for (int r = tid; r <= T; r += kWalkThreads) {
    const RowStat* bs = a.stats + (row0 + r) * a.nblk;
    float m = -INFINITY;
#pragma unroll 8
    for (int k = 0; k < a.nblk; ++k) m = fmaxf(m, static_cast<float>(bs[k].m));
    double z = 0.0;
#pragma unroll 8
    for (int k = 0; k < a.nblk; ++k) {
      const RowStat st = bs[k];
      z += st.z * static_cast<double>(exp_term(static_cast<float>(st.m), m, a.c_hi, a.c_lo));
    }
    L.rm[r] = m;
    L.rz[r] = z;
  }
  }
  if (tid < n) {
    bad = my_par < -1 || my_par >= tid;
    L.par[tid] = my_par;
    L.tok[tid] = my_tok;
    if (!bad && my_tok >= 0 && my_tok < V) my_l = logit<BF16>(row_ptr(my_par + 1), my_tok);
  }
  for (int w = tid; w < (V + 31) / 32; w += kWalkThreads) L.bits[w] = 0u;
  if (__syncthreads_or(bad)) {
    if (tid == 0) ptd::report(a.dev_status, PTD_ERR_BAD_TREE);
    for (int i = tid; i <= T; i += kWalkThreads) {
      if (i < T) an[i] = -1;
      ot[i] = -1;
    }
    if (tid == 0) a.accept_len[b] = 0;
    return;
  }
  if (tid < n) {
    const int r = my_par + 1;
    L.p[tid] = (my_tok >= 0 && my_tok < V)
                   ? exp((static_cast<double>(my_l) - static_cast<double>(L.rm[r])) * a.inv_temp) /
                         L.rz[r]
                   : 0.0;
  }
  if (tid == 0) {
    L.depth = 0;
    L.nrej = 0;
  }
  __syncthreads();

  // the walk, by wave 0 alone.  At node v the children (nodes c > v with
  // parent v) are listed 64 at a time in index order by a ballot; the
  // decisions then run over them in order with wave-uniform values (token,
  // probability and uniform broadcast from the child's lane): a token
  // already rejected at v counts with p = 0, the child is accepted iff
  // u < p / S, else S -= p and its token is rejected (kept in L.rej and
  // marked in the bitmap, cleared when the walk moves on).
  if (wave == 0) {
    int v = -1, depth = 0, nrej = 0;
    for (;;) {
      double S = 1.0;
      int next = -1;
      for (int c0 = v + 1; c0 < n && next < 0; c0 += PTD_WAVE) {
        const int c = c0 + lane;
        const bool kid = c < n && L.par[c] == v;
        uint64_t kb = __ballot(kid);
        const int t_l = kid ? L.tok[c] : -1;
        const double p_l = kid ? L.p[c] : 0.0;
        const double u_l = kid ? L.u[c] : 2.0;
        while (kb) {  // uniform
          const int src = __builtin_ctzll(kb);
          kb &= kb - 1ull;
          const int t = __builtin_amdgcn_readlane(t_l, src);
          const double p0 = readlane_f64(p_l, src), u = readlane_f64(u_l, src);
          const bool valid = t >= 0 && t < V;
          const bool dup = valid && ((L.bits[t >> 5] >> (t & 31)) & 1u);
          const double p = dup ? 0.0 : p0;
          const double thr = S > 0.0 ? p / S : 0.0;
          if (u < thr) {
            next = c0 + src;
            break;
          }
          S -= p;
          if (valid && !dup) {
            if (lane == 0) {
              L.bits[t >> 5] |= 1u << (t & 31);
              L.rej[nrej] = t;
            }
            ++nrej;
          }
        }
      }
      if (next < 0) break;
      // accepted: clear this node's rejections, move to the child
      for (int j = lane; j < nrej; j += PTD_WAVE) {
        const int t = L.rej[j];
        atomicAnd(&L.bits[t >> 5], ~(1u << (t & 31)));
      }
      nrej = 0;
      if (lane == 0) L.path[depth] = next;
      ++depth;
      v = next;
    }
    if (lane == 0) {
      L.depth = depth;
      L.nrej = nrej;
      L.next = v;
    }
  }
  __syncthreads();
  const int v = L.next;

  // the bonus token: inverse CDF of the residual distribution of row v + 1.
  // term(y) = exp_term(l_y, m_b) * e^((m_b - m)/t) for y in block b, exactly
  // as the block sums were formed; the residual block sums (block sum less
  // the rejected terms) locate the block, whose terms are then scanned.
  const int r = v + 1;
  const float m = L.rm[r];
  const RowStat* bs = a.stats + (row0 + r) * a.nblk;
  const char* rowp = row_ptr(r);
  // block maxima, scales and sums, and the rejected tokens' terms (their
  // loads issued together, one thread per block / per rejected token)
  const int nrej_t = L.nrej;
  for (int k = tid; k < a.nblk; k += kWalkThreads) {
    const RowStat st = bs[k];
    const float f = exp_term(static_cast<float>(st.m), m, a.c_hi, a.c_lo);
    L.bm[k] = static_cast<float>(st.m);
    L.bscale[k] = f;
    L.res[k] = st.z * static_cast<double>(f);
  }
  if (tid < nrej_t) {
    const int t = L.rej[tid], k = t / kBlock;
    const float f = exp_term(static_cast<float>(bs[k].m), m, a.c_hi, a.c_lo);
    L.p[tid] = static_cast<double>(exp_term(logit<BF16>(rowp, t), static_cast<float>(bs[k].m),
                                            a.c_hi, a.c_lo)) *
               static_cast<double>(f);
  }
  __syncthreads();
  auto term = [&](int y) -> double {
    const int k = y / kBlock;
    return static_cast<double>(exp_term(logit<BF16>(rowp, y), L.bm[k], a.c_hi, a.c_lo)) *
           static_cast<double>(L.bscale[k]);
  };
  if constexpr (WIDE) {
  if (wave == 0) {
    if (lane == 0)
      for (int j = 0; j < nrej_t; ++j)  // the rejected tokens' terms leave their blocks
        L.res[L.rej[j] / kBlock] -= L.p[j];
    // running totals over the blocks (fp64 wave scans, two blocks per lane:
    // k = lane and k = 64 + lane); the first block with residual mass whose
    // running total passes the target; if rounding leaves none, the last
    // block with residual mass
    const double r0 = lane < a.nblk ? L.res[lane] : 0.0;
    const double r1 = lane + PTD_WAVE < a.nblk ? L.res[lane + PTD_WAVE] : 0.0;
    const double i0 = wave_incl_scan_f64(r0);
    const double t0 = readlane_f64(i0, PTD_WAVE - 1);
    const double i1 = t0 + wave_incl_scan_f64(r1);
    const double total = readlane_f64(i1, PTD_WAVE - 1);
    const double target = a.u_bonus[row0 + r] * total;
    const uint64_t h0 = __ballot(r0 > 0.0 && i0 > target), h1 = __ballot(r1 > 0.0 && i1 > target);
    const uint64_t m0 = __ballot(r0 > 0.0), m1 = __ballot(r1 > 0.0);
    int xb;
    if (h0 | h1) xb = h0 ? __builtin_ctzll(h0) : PTD_WAVE + __builtin_ctzll(h1);
    else if (m1 | m0) xb = m1 ? 2 * PTD_WAVE - 1 - __builtin_clzll(m1) : PTD_WAVE - 1 - __builtin_clzll(m0);
    else xb = -1;
    // the running total before block xb: the scans' exclusive values (the
    // shuffles run on every lane; lane 0's results are replaced afterwards)
    double e0 = shfl_up_f64(i0, 1);
    double e1 = shfl_up_f64(i1, 1);
    if (lane == 0) {
      e0 = 0.0;
      e1 = t0;
    }
    const int xl = xb < 0 ? 0 : xb & (PTD_WAVE - 1);
    const double b0 = readlane_f64(e0, xl), b1 = readlane_f64(e1, xl);
    if (lane == 0) {
      L.xblk = total > 0.0 ? xb : -1;
      L.before = xb >= PTD_WAVE ? b1 : b0;
      L.target = target;
    }
  }
  __syncthreads();
  } else {
  if (tid == 0) {
    for (int j = 0; j < nrej_t; ++j)  // the rejected tokens' terms leave their blocks
      L.res[L.rej[j] / kBlock] -= L.p[j];
    double total = 0.0;
    for (int k = 0; k < a.nblk; ++k) total += L.res[k];
    const double target = a.u_bonus[row0 + r] * total;
    // the first block whose running total passes the target; if rounding
    // leaves none, the last block with residual mass
    int xb = -1, lastb = -1;
    double run = 0.0, before = 0.0, before_last = 0.0;
    for (int k = 0; k < a.nblk; ++k) {
      const double rk = L.res[k];
      if (rk > 0.0) {
        if (xb < 0 && run + rk > target) {
          xb = k;
          before = run;
        }
        lastb = k;
        before_last = run;
      }
      run += rk;
    }
    if (xb < 0) {
      xb = lastb;
      before = before_last;
    }
    L.xblk = total > 0.0 ? xb : -1;
    L.before = before;
    L.target = target;
  }
  __syncthreads();
  }
  const int xb = L.xblk;
  if (xb < 0) {  // no residual mass: every token was rejected
    if (tid == 0) ot[L.depth] = -1;
  } else {
    // the block's terms, two consecutive entries per thread, in index order
    const int ya = xb * kBlock + 2 * tid, yb = ya + 1;
    const bool in_a = ya < V && !((L.bits[ya >> 5] >> (ya & 31)) & 1u);
    const bool in_b = yb < V && !((L.bits[yb >> 5] >> (yb & 31)) & 1u);
    const double ea = in_a ? term(ya) : 0.0, eb = in_b ? term(yb) : 0.0;
    const double own = ea + eb;
    const double incl = wave_incl_scan_f64(own);
    double excl = shfl_up_f64(incl, 1);
    if (lane == 0) excl = 0.0;
    if (lane == 63) L.wsum[wave] = incl;
    if (tid == 0) L.nkids = kWalkThreads;
    __syncthreads();
    double start = L.before;
    for (int w = 0; w < wave; ++w) start += L.wsum[w];
    const double target = L.target;
    if (own > 0.0 && start + incl > target) atomicMin(&L.nkids, tid);
    __syncthreads();
    bool fallback = false;
    if (L.nkids == kWalkThreads) {  // rounding: the last thread with mass
      fallback = true;
      if (tid == 0) L.nkids = -1;
      __syncthreads();
      if (own > 0.0) atomicMax(&L.nkids, tid);
      __syncthreads();
    }
    if (tid == L.nkids) {
      const double cum = start + excl;
      int x;
      if (ea > 0.0 && (!fallback && cum + ea > target)) x = ya;
      else x = eb > 0.0 ? yb : ya;
      ot[L.depth] = x;
    }
  }
  const int depth = L.depth;
  for (int i = tid; i <= T; i += kWalkThreads) {
    if (i < T) an[i] = i < depth ? L.path[i] : -1;
    if (i < depth) ot[i] = L.tok[L.path[i]];
    else if (i > depth) ot[i] = -1;
  }
  if (tid == 0) a.accept_len[b] = depth;
}

}  // namespace

extern "C" size_t ptd_verify_sample_workspace_bytes(int32_t B, int32_t T, int32_t V) {
  if (B < 1 || T < 1 || T > PTD_MAX_T || V < 1 || V > kMaxVocab) return 0;
  const int nblk = (V + kBlock - 1) / kBlock;
  const size_t n = static_cast<size_t>(B) * (T + 1) * nblk * sizeof(RowStat);
  return (n + 255) & ~static_cast<size_t>(255);
}

extern "C" int ptd_verify_sample(const void* logits, ptd_dtype dtype, int32_t V, int64_t ld,
                                 const int32_t* draft_tokens, const int32_t* parent,
                                 const int32_t* tree_len, int32_t B, int32_t T,
                                 double temperature, const double* u_node,
                                 const double* u_bonus, int32_t* accept_len,
                                 int32_t* accept_nodes, int32_t* out_tokens, void* workspace,
                                 size_t workspace_bytes, int32_t* dev_status, void* stream) {
  PTD_RETURN_IF(!logits || !draft_tokens || !parent || !u_node || !u_bonus || !accept_len ||
                    !accept_nodes || !out_tokens,
                PTD_ERR_NULL);
  PTD_RETURN_IF(dtype != PTD_BF16 && dtype != PTD_F32, PTD_ERR_DTYPE);
  PTD_RETURN_IF(B < 1 || T < 1 || T > PTD_MAX_T || V < 1 || V > kMaxVocab || ld < V,
                PTD_ERR_SHAPE);
  PTD_RETURN_IF(!(temperature > 0.0 && temperature < INFINITY), PTD_ERR_SHAPE);
  PTD_RETURN_IF(static_cast<long long>(B) * (T + 1) > 65535, PTD_ERR_SHAPE);  // grid rows
  const size_t need = ptd_verify_sample_workspace_bytes(B, T, V);
  PTD_RETURN_IF(!workspace || workspace_bytes < need, PTD_ERR_WORKSPACE);
  PTD_RETURN_IF(!ptd_aligned(workspace, 16), PTD_ERR_ALIGN);
  hipStream_t st = static_cast<hipStream_t>(stream);
  RowStat* stats = static_cast<RowStat*>(workspace);
  const double c = 1.4426950408889634 / temperature;
  const float c_hi = static_cast<float>(c);
  const float c_lo = static_cast<float>(c - static_cast<double>(c_hi));
  const int R = B * (T + 1);
  const int nblk = (V + kBlock - 1) / kBlock;
  SampleArgs a{logits, ld, V, T, draft_tokens, parent, tree_len, u_node, u_bonus, stats, nblk,
               1.0 / temperature, c_hi, c_lo, accept_len, accept_nodes, out_tokens, dev_status};
  // statistics: one wave per block when the call has many blocks (a batch
  // of sequences: 1040 rows x 63 blocks, 63.6 against 85 us), else one
  // workgroup per block (a single sequence's 65-97 rows: 0.8 us shorter)
  const bool wave_stats = static_cast<long long>(R) * nblk >= 8192;
  const dim3 sgrid = wave_stats
      ? dim3((nblk + kStatThreads / PTD_WAVE - 1) / (kStatThreads / PTD_WAVE), R)
      : dim3(nblk, R);
  const bool wide = nblk > 32;
#define PTD_STATS(bf_)                                                                        \
  if (wave_stats)                                                                             \
    hipLaunchKernelGGL(k_block_stats<bf_>, sgrid, dim3(kStatThreads), 0, st, logits, V, ld,   \
                       nblk, c_hi, c_lo, stats);                                              \
  else                                                                                        \
    hipLaunchKernelGGL(k_block_stats_wg<bf_>, sgrid, dim3(kStatThreads), 0, st, logits, V,    \
                       ld, nblk, c_hi, c_lo, stats);                                          \
  if (wide) hipLaunchKernelGGL((k_verify_sample<bf_, true>), dim3(B), dim3(kWalkThreads), 0, st, a); \
  else hipLaunchKernelGGL((k_verify_sample<bf_, false>), dim3(B), dim3(kWalkThreads), 0, st, a);
  if (dtype == PTD_BF16) {
    PTD_STATS(true)
  } else {
    PTD_STATS(false)
  }
#undef PTD_STATS
  return ptd_launch_status();
}
