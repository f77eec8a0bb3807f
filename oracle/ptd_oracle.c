/*
 * Plain fp64 CPU oracle for one Progressive Tree Drafting step.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, includes
 * or calls this file; only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark load it.  It shares no code with the GPU path.
 *
 * Every function is the plain definition of its result, written for a reader
 * to check against the paper by eye: no blocking, no fusion, no reordering.
 * Floating point is fp64 throughout; bf16/fp32 inputs are widened exactly.
 *
 *   oracle_tree_mask       Sec. 3.1 "Tree Construction": pi(v) = {v} u pi(P(v)),
 *                          position from |pi(v)|.
 *   oracle_attention_row   Sec. 3.1 + Sec. 3.2: a node attends to the committed
 *   oracle_tree_attention  prefix X and to its own ancestors only (softmax of
 *                          scaled dot products, plain two-pass form).
 *   oracle_topk            Sec. 3.2 greedy verification tokens (argmax), App. A
 *                          top-k candidates; order (value desc, index asc).
 *   oracle_verify          Sec. 3.2 eligible edges I and accepted sequence X';
 *                          Alg. 1 step 5-6.
 *   oracle_expand          Sec. 3.1 "Progressive Expansion" (V^t, E^t) with the
 *                          width limit of "Overhead Constraints", top-k children.
 *   oracle_tree_rope       Sec. 3.1 position |pi(v)| of a tree node, continuing
 *                          the committed positions; rotary embedding of its
 *                          query and key at that position (RoFormer rotation).
 *   oracle_kv_commit       Sec. 3.2 accepted sequence X': the accepted nodes'
 *                          keys and values become the next committed rows.
 *   oracle_e4m3_decode     value of an OCP FP8 E4M3 code (keys and values
 *                          cached in 8 bits, a serving format: not in the paper).
 *   oracle_verify_sample   Sec. 3.2 sampling decoding strategy; App. E
 *                          recursive candidate-tree sampling, normalized as in
 *                          the proof of App. F.
 *
 * Error returns: 0 = ok, 7 = malformed tree (parent[i] outside [-1, i)),
 * 2 = bad sizes, 8 = kv_len outside [0, L_cap - T], 9 = accepted path not
 * strictly increasing node ids in [0, T) (or its length outside [0, T]).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_OK 0
#define ORC_BAD_SIZE 2
#define ORC_BAD_TREE 7
#define ORC_BAD_KV_LEN 8
#define ORC_BAD_PATH 9

/* element widening: dtype 0 = fp32, 1 = bf16 (upper half of an fp32),
 * 2 = fp64 */
static double load_elem(const void* base, int dtype, size_t idx) {
  if (dtype == 2) return ((const double*)base)[idx];
  if (dtype == 1) {
    uint16_t h = ((const uint16_t*)base)[idx];
    uint32_t u = ((uint32_t)h) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
  }
  return (double)((const float*)base)[idx];
}

static int node_count(const int32_t* tree_len, int b, int T) {
  if (!tree_len) return T;
  int n = tree_len[b];
  return n < 0 ? 0 : (n > T ? T : n);
}

static int tree_is_valid(const int32_t* par, int n) {
  for (int i = 0; i < n; ++i)
    if (par[i] < -1 || par[i] >= i) return 0;
  return 1;
}

/* ---------------------------------------------------------------------------
 * Ancestor sets.  Sec. 3.1: pi(v) = {v} u pi(P(v)); a root's parent is the last
 * committed token, which is outside the tree.  Bit j of row i lives in word
 * j/64, bit j%64.  depth[i] = |pi(i)|.  Rows at or beyond tree_len are zero.
 * ------------------------------------------------------------------------- */
int oracle_tree_mask(const int32_t* parent, const int32_t* tree_len, int B, int T,
                     uint64_t* mask, int32_t* depth) {
  if (B < 0 || T < 1) return ORC_BAD_SIZE;
  const int W = (T + 63) / 64;
  int status = ORC_OK;
  for (int b = 0; b < B; ++b) {
    const int32_t* par = parent + (size_t)b * T;
    const int n = node_count(tree_len, b, T);
    memset(mask + (size_t)b * T * W, 0, sizeof(uint64_t) * (size_t)T * W);
    memset(depth + (size_t)b * T, 0, sizeof(int32_t) * (size_t)T);
    if (!tree_is_valid(par, n)) { status = ORC_BAD_TREE; continue; }
    for (int i = 0; i < n; ++i) {
      uint64_t* row = mask + ((size_t)b * T + i) * W;
      int count = 0;
      for (int a = i; a != -1; a = par[a]) {  /* v, then P(v), then P(P(v)) ... */
        row[a / 64] |= (uint64_t)1 << (a % 64);
        ++count;
      }
      depth[(size_t)b * T + i] = count;
    }
  }
  return status;
}

/* ---------------------------------------------------------------------------
 * Tree attention for one (sequence b, query head h, node i).
 * Keys: every committed position j in [0, kv_len[b]) and the cache row
 * kv_len[b] + a of every a in pi(i).  KV head g = h / (Hq / Hkv).
 *   s_j = scale * <q, k_j>;  m = max_j s_j;  p_j = exp(s_j - m);
 *   out = sum_j p_j v_j / sum_j p_j.
 * Layouts: q [B][T][Hq][D], caches [B][Hkv][L_cap][D], out row of D doubles.
 * tree_len (NULL: every node live) gives each sequence its own tree size
 * n_b = clamp(tree_len[b], 0, T) inside the padded batch: nodes at index
 * >= n_b are padding, whose parents, queries and cache rows are not read,
 * and whose outputs are zero.  Only n_b cache rows follow the committed ones.
 * ------------------------------------------------------------------------- */
int oracle_attention_row(const void* q, const void* k_cache, const void* v_cache,
                         int dtype, const int32_t* kv_len, const int32_t* parent,
                         const int32_t* tree_len, int B, int T, int Hq, int Hkv, int D,
                         int L_cap, double scale, int b, int h, int i, double* out) {
  if (b < 0 || b >= B || h < 0 || h >= Hq || i < 0 || i >= T || Hkv <= 0 ||
      Hq % Hkv)
    return ORC_BAD_SIZE;
  int nt = T;
  if (tree_len) nt = tree_len[b] < 0 ? 0 : (tree_len[b] > T ? T : tree_len[b]);
  const int32_t* par = parent + (size_t)b * T;
  if (!tree_is_valid(par, nt)) return ORC_BAD_TREE;
  const int n = kv_len[b];
  if (n < 0 || n + nt > L_cap) return ORC_BAD_SIZE;
  if (i >= nt) {  /* padding node */
    for (int d = 0; d < D; ++d) out[d] = 0.0;
    return ORC_OK;
  }
  const int g = h / (Hq / Hkv);

  /* the key rows node i may see */
  int nkeys = n;
  for (int a = i; a != -1; a = par[a]) ++nkeys;
  int* rows = (int*)malloc(sizeof(int) * (size_t)nkeys);
  double* s = (double*)malloc(sizeof(double) * (size_t)nkeys);
  if (!rows || !s) { free(rows); free(s); return ORC_BAD_SIZE; }
  int c = 0;
  for (int j = 0; j < n; ++j) rows[c++] = j;
  for (int a = i; a != -1; a = par[a]) rows[c++] = n + a;

  const size_t qoff = (((size_t)b * T + i) * Hq + h) * D;
  const size_t kvoff = ((size_t)b * Hkv + g) * L_cap;
  for (int j = 0; j < nkeys; ++j) {
    double dot = 0.0;
    for (int d = 0; d < D; ++d)
      dot += load_elem(q, dtype, qoff + d) *
             load_elem(k_cache, dtype, (kvoff + rows[j]) * D + d);
    s[j] = scale * dot;
  }
  double m = s[0];
  for (int j = 1; j < nkeys; ++j)
    if (s[j] > m) m = s[j];
  double denom = 0.0;
  for (int j = 0; j < nkeys; ++j) {
    s[j] = exp(s[j] - m);
    denom += s[j];
  }
  for (int d = 0; d < D; ++d) {
    double acc = 0.0;
    for (int j = 0; j < nkeys; ++j)
      acc += s[j] * load_elem(v_cache, dtype, (kvoff + rows[j]) * D + d);
    out[d] = acc / denom;
  }
  free(rows);
  free(s);
  return ORC_OK;
}

/* All rows; out is [B][T][Hq][D] doubles. */
int oracle_tree_attention(const void* q, const void* k_cache, const void* v_cache,
                          int dtype, const int32_t* kv_len, const int32_t* parent,
                          const int32_t* tree_len, int B, int T, int Hq, int Hkv, int D,
                          int L_cap, double scale, double* out) {
  for (int b = 0; b < B; ++b)
    for (int i = 0; i < T; ++i)
      for (int h = 0; h < Hq; ++h) {
        int st = oracle_attention_row(q, k_cache, v_cache, dtype, kv_len, parent, tree_len,
                                      B, T, Hq, Hkv, D, L_cap, scale, b, h, i,
                                      out + (((size_t)b * T + i) * Hq + h) * D);
        if (st) return st;
      }
  return ORC_OK;
}

/* ---------------------------------------------------------------------------
 * OCP 8-bit floating point E4M3 ("e4m3fn"): bit 7 sign, bits 6..3 exponent e
 * (bias 7), bits 2..0 mantissa m.  e > 0: (1 + m/8) * 2^(e-7); e = 0:
 * (m/8) * 2^-6 (subnormals, and +-0); e = 15 with m = 7 is NaN (the format
 * has no infinities, so e = 15 with m < 7 is a normal number, up to 448).
 * ------------------------------------------------------------------------- */
static double e4m3_value(uint8_t c) {
  const int sgn = c >> 7, e = (c >> 3) & 15, m = c & 7;
  double v;
  if (e == 15 && m == 7) return NAN;
  if (e == 0) v = ldexp((double)m / 8.0, -6);
  else v = ldexp(1.0 + (double)m / 8.0, e - 7);
  return sgn ? -v : v;
}

int oracle_e4m3_decode(const uint8_t* codes, long long n, double* out) {
  if (n < 0) return ORC_BAD_SIZE;
  for (long long i = 0; i < n; ++i) out[i] = e4m3_value(codes[i]);
  return ORC_OK;
}

/* ---------------------------------------------------------------------------
 * Top-k / argmax per row: sort positions by value descending, ties by the
 * lower position (values compared as fp64, so -0.0 and +0.0 are equal).
 * idx/val may be NULL; val receives the row's own values.
 * ------------------------------------------------------------------------- */
typedef struct { double v; int32_t i; } orc_entry;

static int orc_cmp(const void* pa, const void* pb) {
  const orc_entry* a = (const orc_entry*)pa;
  const orc_entry* b = (const orc_entry*)pb;
  if (a->v > b->v) return -1;
  if (a->v < b->v) return 1;
  return (a->i > b->i) - (a->i < b->i);
}

int oracle_topk(const void* logits, int dtype, int R, int V, long long ld, int k,
                int32_t* argmax, int32_t* idx, double* val) {
  if (R < 0 || V < 1 || k < 1 || k > V || ld < V) return ORC_BAD_SIZE;
  orc_entry* e = (orc_entry*)malloc(sizeof(orc_entry) * (size_t)V);
  if (!e) return ORC_BAD_SIZE;
  for (int r = 0; r < R; ++r) {
    for (int j = 0; j < V; ++j) {
      e[j].v = load_elem(logits, dtype, (size_t)r * (size_t)ld + j);
      e[j].i = j;
    }
    qsort(e, (size_t)V, sizeof(orc_entry), orc_cmp);
    if (argmax) argmax[r] = e[0].i;
    for (int t = 0; t < k; ++t) {
      if (idx) idx[(size_t)r * k + t] = e[t].i;
      if (val) val[(size_t)r * k + t] = e[t].v;
    }
  }
  free(e);
  return ORC_OK;
}

/* ---------------------------------------------------------------------------
 * Greedy verification (Sec. 3.2).  Verification token of node n is the argmax
 * of its logits row (row n+1; row 0 belongs to the last committed token, the
 * parent of every root).  Edge (P(c), c) is eligible iff the parent's
 * verification token equals token[c].  A node is accepted iff every edge on
 * its root path is eligible.  The accepted length k is the largest depth of an
 * accepted node; the terminal is the lowest-index accepted node of that depth.
 * X' = tokens of the terminal's root path (shallowest first) followed by the
 * terminal's verification token (argmax[0] when nothing is accepted).
 * accept_nodes [B][T] and out_tokens [B][T+1] are padded with -1.
 * ------------------------------------------------------------------------- */
int oracle_verify(const int32_t* argmax, const int32_t* tokens,
                  const int32_t* parent, const int32_t* tree_len, int B, int T,
                  int32_t* accept_len, int32_t* accept_nodes, int32_t* out_tokens) {
  if (B < 0 || T < 1) return ORC_BAD_SIZE;
  int status = ORC_OK;
  int* ok = (int*)malloc(sizeof(int) * (size_t)T);
  int* dep = (int*)malloc(sizeof(int) * (size_t)T);
  if (!ok || !dep) { free(ok); free(dep); return ORC_BAD_SIZE; }
  for (int b = 0; b < B; ++b) {
    const int32_t* par = parent + (size_t)b * T;
    const int32_t* tok = tokens + (size_t)b * T;
    const int32_t* am = argmax + (size_t)b * (T + 1);
    int32_t* an = accept_nodes + (size_t)b * T;
    int32_t* ot = out_tokens + (size_t)b * (T + 1);
    for (int i = 0; i < T; ++i) an[i] = -1;
    for (int i = 0; i <= T; ++i) ot[i] = -1;
    accept_len[b] = 0;
    const int n = node_count(tree_len, b, T);
    if (!tree_is_valid(par, n)) { status = ORC_BAD_TREE; continue; }

    int best = -1;
    for (int i = 0; i < n; ++i) {
      /* accepted iff every edge from the committed token down to i is eligible */
      int acc = 1, d = 0;
      for (int c = i; c != -1; c = par[c]) {
        if (tok[c] != am[par[c] + 1]) acc = 0;
        ++d;
      }
      ok[i] = acc;
      dep[i] = d;
      if (acc && (best < 0 || d > dep[best])) best = i;
    }
    if (best < 0) {
      ot[0] = am[0];
      continue;
    }
    const int k = dep[best];
    accept_len[b] = k;
    int pos = k - 1;
    for (int c = best; c != -1; c = par[c]) {
      an[pos] = c;
      ot[pos] = tok[c];
      --pos;
    }
    ot[k] = am[best + 1];
  }
  free(ok);
  free(dep);
  return status;
}

/* ---------------------------------------------------------------------------
 * Progressive expansion with top-k children (Sec. 3.1; App. A top-k).
 *   1. Node v (index order) offers topk_idx[v+1][0..k-1] as children.
 *      A node at depth d only grows if d + 1 <= d_max; it stops once it has
 *      width_sched[d] children (existing ones included).  A candidate equal to
 *      the token of a child v already has (old or just added) is the same node
 *      and is skipped.  The committed token (row 0) is not expanded.
 *   2. The grown tree is renumbered breadth-first: by depth; within a depth,
 *      by the new number of the parent; within a parent, old children in old
 *      index order, then new children in candidate order.  Roots keep their
 *      old relative order.
 *   3. The first T_max nodes are kept (a breadth-first prefix keeps every
 *      kept node's parent).  Slots beyond tree_len_next hold -1.
 * width_sched has d_max entries (entry 0 would be the number of roots and is
 * not used here).
 * ------------------------------------------------------------------------- */
int oracle_expand(const int32_t* parent, const int32_t* tokens,
                  const int32_t* tree_len, int B, int T, const int32_t* topk_idx,
                  int k, const int32_t* width_sched, int d_max, int T_max,
                  int32_t* parent_next, int32_t* tokens_next,
                  int32_t* tree_len_next) {
  if (B < 0 || T < 1 || k < 1 || d_max < 1 || T_max < 1) return ORC_BAD_SIZE;
  int status = ORC_OK;
  const int cap = T * (k + 1);
  /* grown tree: old nodes 0..n-1, then new nodes */
  int* gpar = (int*)malloc(sizeof(int) * (size_t)cap);
  int* gtok = (int*)malloc(sizeof(int) * (size_t)cap);
  int* gdep = (int*)malloc(sizeof(int) * (size_t)cap);
  int* newid = (int*)malloc(sizeof(int) * (size_t)cap);
  int* order = (int*)malloc(sizeof(int) * (size_t)cap);
  if (!gpar || !gtok || !gdep || !newid || !order) {
    free(gpar); free(gtok); free(gdep); free(newid); free(order);
    return ORC_BAD_SIZE;
  }
  for (int b = 0; b < B; ++b) {
    const int32_t* par = parent + (size_t)b * T;
    const int32_t* tok = tokens + (size_t)b * T;
    int32_t* pn = parent_next + (size_t)b * T_max;
    int32_t* tn = tokens_next + (size_t)b * T_max;
    for (int i = 0; i < T_max; ++i) { pn[i] = -1; tn[i] = -1; }
    tree_len_next[b] = 0;
    const int n = node_count(tree_len, b, T);
    if (!tree_is_valid(par, n)) { status = ORC_BAD_TREE; continue; }

    int total = 0;
    for (int i = 0; i < n; ++i) {
      gpar[total] = par[i];
      gtok[total] = tok[i];
      gdep[total] = (par[i] < 0) ? 1 : gdep[par[i]] + 1;
      ++total;
    }
    /* step 1: candidate children */
    for (int v = 0; v < n; ++v) {
      const int d = gdep[v];
      if (d + 1 > d_max) continue;
      int nchild = 0;
      for (int c = 0; c < total; ++c)
        if (gpar[c] == v) ++nchild;
      for (int r = 0; r < k; ++r) {
        if (nchild >= width_sched[d]) break;
        const int cand = topk_idx[((size_t)b * (T + 1) + v + 1) * k + r];
        int dup = 0;
        for (int c = 0; c < total; ++c)
          if (gpar[c] == v && gtok[c] == cand) dup = 1;
        if (dup) continue;
        gpar[total] = v;
        gtok[total] = cand;
        gdep[total] = d + 1;
        ++total;
        ++nchild;
      }
    }
    /* step 2: breadth-first renumbering.  Grown-tree ids of a parent's
     * children increase in exactly the stated order (old children have
     * ids < n in index order, new ones follow in candidate order), so a stable
     * pass over ids in increasing order per parent gives the order. */
    int cnt = 0;
    for (int c = 0; c < total; ++c)
      if (gpar[c] == -1) { order[cnt] = c; newid[c] = cnt; ++cnt; }
    for (int head = 0; head < cnt; ++head) {
      const int p = order[head];
      for (int c = 0; c < total; ++c)
        if (gpar[c] == p) { order[cnt] = c; newid[c] = cnt; ++cnt; }
    }
    /* step 3: keep the first T_max */
    const int keep = cnt < T_max ? cnt : T_max;
    for (int t = 0; t < keep; ++t) {
      const int c = order[t];
      pn[t] = gpar[c] < 0 ? -1 : newid[gpar[c]];
      tn[t] = gtok[c];
    }
    tree_len_next[b] = keep;
  }
  free(gpar); free(gtok); free(gdep); free(newid); free(order);
  return status;
}

/* ---------------------------------------------------------------------------
 * Positions and rotary embedding of the tree rows.
 * Sec. 3.1 "Tree Construction": the position of node v is given by |pi(v)|.
 * A root's parent is the last committed token, at position kv_len[b] - 1, so
 * node i of sequence b sits at
 *     pos(i) = kv_len[b] + |pi(i)| - 1,
 * which is where a chain of accepted nodes lands once committed.
 * The model turns queries and keys by their positions with the rotary
 * embedding of Su et al. (RoFormer, 2021): dimension pair p (0 <= p < D/2)
 * is rotated by the angle a = pos * inv_freq[p],
 *     (x_a, x_b) -> (x_a cos a - x_b sin a,  x_a sin a + x_b cos a),
 * where pair p is (x[p], x[p + D/2]) for pairing 0 ("half" layout) or
 * (x[2p], x[2p + 1]) for pairing 1 ("interleaved" layout).
 * In:  q [B][T][Hq][D]; keys are rows kv_len[b] + i of k_cache
 *      [B][Hkv][L_cap][D]; inv_freq [D/2].
 * Out (fp64): q_out [B][T][Hq][D], k_out [B][Hkv][T][D] (the tree rows),
 *      pos [B][T].  A sequence with a malformed tree or kv_len outside
 *      [0, L_cap - T] is skipped (outputs zero) and reported.
 * ------------------------------------------------------------------------- */
static void rope_vector(const void* src, int dtype, size_t base, int D, double pos,
                        const double* inv_freq, int pairing, double* dst) {
  for (int p = 0; p < D / 2; ++p) {
    const int ia = pairing == 0 ? p : 2 * p;
    const int ib = pairing == 0 ? p + D / 2 : 2 * p + 1;
    const double xa = load_elem(src, dtype, base + (size_t)ia);
    const double xb = load_elem(src, dtype, base + (size_t)ib);
    const double a = pos * inv_freq[p];
    dst[ia] = xa * cos(a) - xb * sin(a);
    dst[ib] = xa * sin(a) + xb * cos(a);
  }
}

int oracle_tree_rope(const void* q, const void* k_cache, int dtype, const int32_t* kv_len,
                     const int32_t* parent, int B, int T, int Hq, int Hkv, int D, int L_cap,
                     const double* inv_freq, int pairing, double* q_out, double* k_out,
                     int32_t* pos) {
  if (B < 0 || T < 1 || Hq < 1 || Hkv < 1 || D < 2 || D % 2 != 0 || L_cap < 1 ||
      (pairing != 0 && pairing != 1))
    return ORC_BAD_SIZE;
  int status = ORC_OK;
  for (int b = 0; b < B; ++b) {
    const int32_t* par = parent + (size_t)b * T;
    memset(q_out + (size_t)b * T * Hq * D, 0, sizeof(double) * (size_t)T * Hq * D);
    memset(k_out + (size_t)b * Hkv * T * D, 0, sizeof(double) * (size_t)Hkv * T * D);
    memset(pos + (size_t)b * T, 0, sizeof(int32_t) * (size_t)T);
    if (!tree_is_valid(par, T)) { status = ORC_BAD_TREE; continue; }
    if (kv_len[b] < 0 || (long long)kv_len[b] + T > L_cap) {
      if (status == ORC_OK) status = ORC_BAD_KV_LEN;
      continue;
    }
    for (int i = 0; i < T; ++i) {
      int size = 0;                                 /* |pi(i)| */
      for (int a = i; a != -1; a = par[a]) ++size;
      const int p_i = kv_len[b] + size - 1;
      pos[(size_t)b * T + i] = p_i;
      for (int h = 0; h < Hq; ++h) {
        const size_t off = (((size_t)b * T + i) * Hq + h) * D;
        rope_vector(q, dtype, off, D, (double)p_i, inv_freq, pairing, q_out + off);
      }
      for (int g = 0; g < Hkv; ++g) {
        const size_t src = (((size_t)b * Hkv + g) * L_cap + kv_len[b] + i) * D;
        const size_t dst = (((size_t)b * Hkv + g) * T + i) * D;
        rope_vector(k_cache, dtype, src, D, (double)p_i, inv_freq, pairing, k_out + dst);
      }
    }
  }
  return status;
}

/* ---------------------------------------------------------------------------
 * Commit of the accepted path (Sec. 3.2).  The step accepts
 * X' = (n_0, n_1, ..., n_k, V_{n_k}): n_0 is the last committed token, and
 * n_1 .. n_k (accept_nodes[b][0 .. k-1], k = accept_len[b], shallowest
 * first) are draft nodes whose keys and values the forward pass wrote at
 * cache rows kv_len[b] + n_j.  They become committed tokens: node n_j
 * (j = 1 .. k) is copied to row kv_len[b] + j - 1 in every KV head, and the
 * committed length becomes kv_len[b] + k.  Every other row keeps its content.
 * The bonus token V_{n_k} is the next step's input; it has no key or value yet.
 * The k source rows are read before any destination row is written, so a
 * destination that is also an earlier node's source is copied correctly.
 * Caches [B][Hkv][L_cap][D] (dtype 0 fp32, 1 bf16) are updated in place.
 * A sequence with kv_len outside [0, L_cap - T], or a path that is not
 * strictly increasing node ids in [0, T) with 0 <= k <= T, is left unchanged
 * (kv_len_next = kv_len) and reported.
 * ------------------------------------------------------------------------- */
int oracle_kv_commit(void* k_cache, void* v_cache, int dtype, const int32_t* kv_len,
                     const int32_t* accept_len, const int32_t* accept_nodes, int B, int T,
                     int Hkv, int D, int L_cap, int32_t* kv_len_next) {
  if (B < 0 || T < 1 || Hkv < 1 || D < 1 || L_cap < 1) return ORC_BAD_SIZE;
  const size_t es = dtype == 1 ? 2 : 4;
  const size_t row = es * (size_t)D;
  unsigned char* tmp = (unsigned char*)malloc(row * (size_t)T);
  if (!tmp) return ORC_BAD_SIZE;
  int status = ORC_OK;
  for (int b = 0; b < B; ++b) {
    const int32_t* nodes = accept_nodes + (size_t)b * T;
    const int k = accept_len[b];
    kv_len_next[b] = kv_len[b];
    if (kv_len[b] < 0 || (long long)kv_len[b] + T > L_cap) {
      if (status == ORC_OK) status = ORC_BAD_KV_LEN;
      continue;
    }
    int path_ok = k >= 0 && k <= T;
    for (int j = 0; path_ok && j < k; ++j)
      if (nodes[j] < 0 || nodes[j] >= T || (j > 0 && nodes[j] <= nodes[j - 1])) path_ok = 0;
    if (!path_ok) {
      if (status == ORC_OK) status = ORC_BAD_PATH;
      continue;
    }
    for (int c = 0; c < 2; ++c) {
      unsigned char* cache = (unsigned char*)(c == 0 ? k_cache : v_cache);
      for (int g = 0; g < Hkv; ++g) {
        unsigned char* head = cache + ((size_t)b * Hkv + g) * (size_t)L_cap * row;
        for (int j = 0; j < k; ++j)              /* read every source row ... */
          memcpy(tmp + (size_t)j * row, head + (size_t)(kv_len[b] + nodes[j]) * row, row);
        for (int j = 0; j < k; ++j)              /* ... then write the destinations */
          memcpy(head + (size_t)(kv_len[b] + j) * row, tmp + (size_t)j * row, row);
      }
    }
    kv_len_next[b] = kv_len[b] + k;
  }
  free(tmp);
  return status;
}

/* ---------------------------------------------------------------------------
 * Sampling verification (Sec. 3.2 "sampling decoding strategy"; App. E,
 * recursive candidate-tree sampling; App. F, distributional consistency).
 * P_v = softmax(logits row of v / temperature) over the vocabulary; row 0 is
 * the last committed token n_0 (the parent of every root), row v + 1 is
 * node v.  Starting at n_0, the children of the current node v are examined
 * in index order.  Child n (token t_n) is accepted iff
 *     u_node[n] < P_v[t_n] / S,
 * where S is the mass of P_v not yet rejected at v (S = 1 before the first
 * child; App. F divides by it).  A rejected child's token gets probability 0
 * (S drops by its old value), so a later sibling with the same token is never
 * accepted.  On acceptance the walk moves to n; when every child of v is
 * rejected, v is the terminal and the bonus token is drawn from the residual
 * distribution (P_v with the rejected tokens removed) by inverse CDF in index
 * order: the smallest x with  sum_{y <= x} P'_y > u_bonus[row of v] * W,
 * W = sum_y P'_y (the last token with P'_y > 0 if rounding leaves none; -1 if
 * W = 0).  Outputs as oracle_verify.  margin[b] (nullable) is the smallest
 * distance, over the sequence's decisions, between a uniform and the value
 * it was compared with (normalized units); a result whose margin is below
 * the rounding of another implementation may legitimately differ.
 * u_node [B][T], u_bonus [B][T+1], logits rows [B*(T+1)] of stride ld.
 * ------------------------------------------------------------------------- */
int oracle_verify_sample(const void* logits, int dtype, long long ld, int V,
                         const int32_t* tokens, const int32_t* parent, const int32_t* tree_len,
                         int B, int T, double temperature, const double* u_node,
                         const double* u_bonus, int32_t* accept_len, int32_t* accept_nodes,
                         int32_t* out_tokens, double* margin) {
  if (B < 0 || T < 1 || V < 1 || ld < V || !(temperature > 0.0)) return ORC_BAD_SIZE;
  const size_t es = dtype == 1 ? 2 : 4;
  int status = ORC_OK;
  double* prob = (double*)malloc(sizeof(double) * (size_t)V);   /* P_v, rejected tokens zeroed */
  if (!prob) return ORC_BAD_SIZE;
  for (int b = 0; b < B; ++b) {
    const int32_t* par = parent + (size_t)b * T;
    const int32_t* tok = tokens + (size_t)b * T;
    int32_t* an = accept_nodes + (size_t)b * T;
    int32_t* ot = out_tokens + (size_t)b * (T + 1);
    double mg = INFINITY;
    for (int i = 0; i < T; ++i) an[i] = -1;
    for (int i = 0; i <= T; ++i) ot[i] = -1;
    accept_len[b] = 0;
    if (margin) margin[b] = INFINITY;
    const int n = node_count(tree_len, b, T);
    if (!tree_is_valid(par, n)) { status = ORC_BAD_TREE; continue; }

    int v = -1, depth = 0;                   /* current node (-1: n_0) */
    for (;;) {
      const char* row = (const char*)logits + ((size_t)b * (T + 1) + (size_t)(v + 1)) * (size_t)ld * es;
      /* P_v = softmax(row / temperature), then the children in index order */
      double m = -INFINITY, z = 0.0;
      for (int y = 0; y < V; ++y) { const double l = load_elem(row, dtype, (size_t)y); if (l > m) m = l; }
      for (int y = 0; y < V; ++y) z += exp((load_elem(row, dtype, (size_t)y) - m) / temperature);
      for (int y = 0; y < V; ++y) prob[y] = exp((load_elem(row, dtype, (size_t)y) - m) / temperature) / z;
      double S = 1.0;
      int next = -1;
      for (int c = v + 1; c < n; ++c) {
        if (par[c] != v) continue;
        const int t = tok[c];
        const double p = (t >= 0 && t < V) ? prob[t] : 0.0;
        const double thr = S > 0.0 ? p / S : 0.0;
        const double d = fabs(u_node[(size_t)b * T + c] - thr);
        if (d < mg) mg = d;
        if (u_node[(size_t)b * T + c] < thr) { next = c; break; }
        S -= p;
        if (t >= 0 && t < V) prob[t] = 0.0;
      }
      if (next >= 0) {
        an[depth] = next;
        ot[depth] = tok[next];
        ++depth;
        v = next;
        continue;
      }
      /* terminal: inverse CDF of the residual distribution */
      double W = 0.0;
      for (int y = 0; y < V; ++y) W += prob[y];
      int x = -1;
      if (W > 0.0) {
        const double target = u_bonus[(size_t)b * (T + 1) + (size_t)(v + 1)] * W;
        double cum = 0.0;
        for (int y = 0; y < V; ++y) {
          if (prob[y] <= 0.0) continue;
          const double before = cum;
          cum += prob[y];
          x = y;
          if (cum > target) {
            const double d = fmin(target - before, cum - target) / W;
            if (d < mg) mg = d;
            break;
          }
        }
      }
      ot[depth] = x;
      accept_len[b] = depth;
      break;
    }
    if (margin) margin[b] = mg;
  }
  free(prob);
  return status;
}

/* ---------------------------------------------------------------------------
 * Stepping: depth control of the draft tree (Sec. 3.1 "Overhead Constraints",
 * Stepping Mechanism; Alg. 1 step 3).  When a sub-tree (the tree under one
 * root of the forest) is deeper than d_max, its earliest-added child and that
 * child's descendants become the sub-tree and every other branch is pruned.
 * Depth of a sub-tree = number of nodes on its longest root path.  The
 * earliest-added child of a node is its lowest-index child (breadth-first
 * numbering puts old children before new ones, and new ones in candidate
 * order).  Stepping repeats until the depth is at most d_max, so a chain
 * keeps its last d_max nodes (a sliding window).  The kept forest is
 * renumbered breadth-first -- by depth; by the parent's new index; siblings
 * in old index order; roots in the order of the roots they replace -- and cut
 * to T_max nodes; slots from tree_len_next on hold -1.
 * ------------------------------------------------------------------------- */
int oracle_step_prune(const int32_t* parent, const int32_t* tokens, const int32_t* tree_len,
                      int B, int T, int d_max, int T_max, int32_t* parent_next,
                      int32_t* tokens_next, int32_t* tree_len_next) {
  if (B < 0 || T < 1 || d_max < 1 || T_max < 1) return ORC_BAD_SIZE;
  int status = ORC_OK;
  int* h = (int*)malloc(sizeof(int) * (size_t)T);       /* depth of the sub-tree under v */
  int* fc = (int*)malloc(sizeof(int) * (size_t)T);      /* lowest-index child */
  int* keep = (int*)malloc(sizeof(int) * (size_t)T);
  int* order = (int*)malloc(sizeof(int) * (size_t)T);
  int* newid = (int*)malloc(sizeof(int) * (size_t)T);
  if (!h || !fc || !keep || !order || !newid) {
    free(h); free(fc); free(keep); free(order); free(newid);
    return ORC_BAD_SIZE;
  }
  for (int b = 0; b < B; ++b) {
    const int32_t* par = parent + (size_t)b * T;
    const int32_t* tok = tokens + (size_t)b * T;
    int32_t* pn = parent_next + (size_t)b * T_max;
    int32_t* tn = tokens_next + (size_t)b * T_max;
    for (int i = 0; i < T_max; ++i) { pn[i] = -1; tn[i] = -1; }
    tree_len_next[b] = 0;
    const int n = node_count(tree_len, b, T);
    if (!tree_is_valid(par, n)) { status = ORC_BAD_TREE; continue; }
    for (int v = 0; v < n; ++v) { h[v] = 1; fc[v] = -1; keep[v] = 0; }
    for (int v = n - 1; v >= 0; --v)          /* children have larger indices */
      if (par[v] >= 0 && h[v] + 1 > h[par[v]]) h[par[v]] = h[v] + 1;
    for (int v = 0; v < n; ++v)
      if (par[v] >= 0 && fc[par[v]] < 0) fc[par[v]] = v;
    /* the new root of each sub-tree, in the order of the old roots */
    int nroots = 0;
    for (int r = 0; r < n; ++r) {
      if (par[r] != -1) continue;
      int x = r;
      while (h[x] > d_max) x = fc[x];         /* h > 1 means a child exists */
      keep[x] = 2;                            /* 2: a root of the kept forest */
      order[nroots++] = x;
    }
    for (int v = 0; v < n; ++v)
      if (!keep[v] && par[v] >= 0 && keep[par[v]]) keep[v] = 1;
    /* breadth-first renumbering of the kept forest */
    int cnt = nroots;
    for (int i = 0; i < nroots; ++i) newid[order[i]] = i;
    for (int head = 0; head < cnt; ++head) {
      const int p = order[head];
      for (int c = p + 1; c < n; ++c)
        if (keep[c] == 1 && par[c] == p) { newid[c] = cnt; order[cnt++] = c; }
    }
    const int out = cnt < T_max ? cnt : T_max;
    for (int t = 0; t < out; ++t) {
      const int c = order[t];
      pn[t] = keep[c] == 2 ? -1 : newid[par[c]];
      tn[t] = tok[c];
    }
    tree_len_next[b] = out;
  }
  free(h); free(fc); free(keep); free(order); free(newid);
  return status;
}

/* ---------------------------------------------------------------------------
 * Candidate pool (Sec. 3.1 "Draft Extraction via Merging"; Alg. 1 steps 1
 * and 4).  Per sequence: candidate trees of tokens keyed by their root's
 * token.
 * Merge of a draft tree: for every node u (index order), the sub-tree of u --
 * u and its descendants, a tree rooted at token(u) -- is merged by M into the
 * pool tree keyed token(u) (created with a lone root if absent): a child of
 * the draft node whose token is not among the children of the matching pool
 * node is added, one whose token is there is merged into it, recursively.
 * The sub-tree's nodes are taken in index order (each after its parent),
 * which fixes the insertion order.  Bounds: a pool
 * tree holds at most n_cap nodes (its root included), a sequence at most
 * e_max trees; an insertion beyond either bound is skipped together with the
 * sub-tree it would carry.
 * Retrieve: the pool tree keyed by the last committed token, without its
 * root, as a packed draft tree: breadth first (by depth; by the parent's
 * output index; siblings in insertion order), the root's children with
 * parent -1, cut to T_max nodes; tree_len 0 if there is no such tree.
 * The state is this file's own (struct OraclePool); callers hold an opaque
 * pointer.
 * ------------------------------------------------------------------------- */
typedef struct {
  int B, e_max, n_cap;
  int* ntrees;   /* [B] */
  int* key;      /* [B][e_max] */
  int* count;    /* [B][e_max] */
  int* tok;      /* [B][e_max][n_cap] */
  int* par;      /* [B][e_max][n_cap]: index of the parent in the same tree, -1 at the root */
} OraclePool;

void* oracle_pool_new(int B, int e_max, int n_cap) {
  if (B < 1 || e_max < 1 || n_cap < 1) return NULL;
  OraclePool* p = (OraclePool*)calloc(1, sizeof(OraclePool));
  if (!p) return NULL;
  p->B = B; p->e_max = e_max; p->n_cap = n_cap;
  p->ntrees = (int*)calloc((size_t)B, sizeof(int));
  p->key = (int*)calloc((size_t)B * e_max, sizeof(int));
  p->count = (int*)calloc((size_t)B * e_max, sizeof(int));
  p->tok = (int*)calloc((size_t)B * e_max * n_cap, sizeof(int));
  p->par = (int*)calloc((size_t)B * e_max * n_cap, sizeof(int));
  if (!p->ntrees || !p->key || !p->count || !p->tok || !p->par) {
    free(p->ntrees); free(p->key); free(p->count); free(p->tok); free(p->par); free(p);
    return NULL;
  }
  return p;
}

void oracle_pool_free(void* pool) {
  OraclePool* p = (OraclePool*)pool;
  if (!p) return;
  free(p->ntrees); free(p->key); free(p->count); free(p->tok); free(p->par); free(p);
}

/* M(pool tree e, draft sub-tree under draft node u): the sub-tree's nodes in
 * index order (every node after its parent); map[v] = pool node of draft
 * node v, -1 outside the sub-tree or skipped. */
static void pool_merge_subtree(OraclePool* p, int b, int e, const int32_t* par,
                               const int32_t* tok, int n, int u, int* map) {
  int* cnt = &p->count[(size_t)b * p->e_max + e];
  int* ttok = p->tok + ((size_t)b * p->e_max + e) * p->n_cap;
  int* tpar = p->par + ((size_t)b * p->e_max + e) * p->n_cap;
  for (int v = 0; v < n; ++v) map[v] = -1;
  map[u] = 0;                                  /* the pool tree's root */
  for (int c = u + 1; c < n; ++c) {
    const int pn = map[par[c]];
    if (par[c] < u || pn < 0) continue;        /* outside the sub-tree, or skipped */
    int match = -1;
    for (int k = 0; k < *cnt; ++k)
      if (tpar[k] == pn && ttok[k] == tok[c]) { match = k; break; }
    if (match < 0 && *cnt < p->n_cap) {
      match = *cnt;
      ttok[match] = tok[c];
      tpar[match] = pn;
      ++*cnt;
    }
    map[c] = match;                            /* -1: full, c and its sub-tree skipped */
  }
}

int oracle_pool_merge(void* pool, const int32_t* parent, const int32_t* tokens,
                      const int32_t* tree_len, int B, int T) {
  OraclePool* p = (OraclePool*)pool;
  if (!p || B != p->B || T < 1) return ORC_BAD_SIZE;
  int status = ORC_OK;
  int* map = (int*)malloc(sizeof(int) * (size_t)T);
  if (!map) return ORC_BAD_SIZE;
  for (int b = 0; b < B; ++b) {
    const int32_t* par = parent + (size_t)b * T;
    const int32_t* tok = tokens + (size_t)b * T;
    const int n = node_count(tree_len, b, T);
    if (!tree_is_valid(par, n)) { status = ORC_BAD_TREE; continue; }
    for (int u = 0; u < n; ++u) {
      int e = -1;
      for (int k = 0; k < p->ntrees[b]; ++k)
        if (p->key[(size_t)b * p->e_max + k] == tok[u]) { e = k; break; }
      if (e < 0) {
        if (p->ntrees[b] >= p->e_max) continue;  /* no room for another tree */
        e = p->ntrees[b]++;
        p->key[(size_t)b * p->e_max + e] = tok[u];
        p->count[(size_t)b * p->e_max + e] = 1;
        p->tok[((size_t)b * p->e_max + e) * p->n_cap] = tok[u];
        p->par[((size_t)b * p->e_max + e) * p->n_cap] = -1;
      }
      pool_merge_subtree(p, b, e, par, tok, n, u, map);
    }
  }
  free(map);
  return status;
}

int oracle_pool_retrieve(void* pool, const int32_t* last_token, int B, int T_max,
                         int32_t* parent_out, int32_t* tokens_out, int32_t* tree_len_out) {
  OraclePool* p = (OraclePool*)pool;
  if (!p || B != p->B || T_max < 1) return ORC_BAD_SIZE;
  int* order = (int*)malloc(sizeof(int) * (size_t)p->n_cap);
  int* outid = (int*)malloc(sizeof(int) * (size_t)p->n_cap);
  if (!order || !outid) { free(order); free(outid); return ORC_BAD_SIZE; }
  for (int b = 0; b < B; ++b) {
    int32_t* po = parent_out + (size_t)b * T_max;
    int32_t* to = tokens_out + (size_t)b * T_max;
    for (int i = 0; i < T_max; ++i) { po[i] = -1; to[i] = -1; }
    tree_len_out[b] = 0;
    int e = -1;
    for (int k = 0; k < p->ntrees[b]; ++k)
      if (p->key[(size_t)b * p->e_max + k] == last_token[b]) { e = k; break; }
    if (e < 0) continue;
    const int cnt = p->count[(size_t)b * p->e_max + e];
    const int* ttok = p->tok + ((size_t)b * p->e_max + e) * p->n_cap;
    const int* tpar = p->par + ((size_t)b * p->e_max + e) * p->n_cap;
    /* breadth first from the root (node 0); children in insertion order */
    int q = 0;
    order[q++] = 0;
    outid[0] = -1;
    for (int head = 0; head < q; ++head) {
      const int x = order[head];
      for (int k = 0; k < cnt; ++k)
        if (tpar[k] == x) { outid[k] = q - 1; order[q++] = k; }
    }
    const int len = (q - 1) < T_max ? (q - 1) : T_max;
    for (int i = 0; i < len; ++i) {
      const int k = order[i + 1];
      to[i] = ttok[k];
      po[i] = outid[tpar[k]];
    }
    tree_len_out[b] = len;
  }
  free(order); free(outid);
  return ORC_OK;
}

/* ---------------------------------------------------------------------------
 * Paged key/value caches: a storage layout of the committed cache and the
 * tree rows (the attention they feed is oracle_tree_attention's).  Row r of
 * sequence b and KV head g is row r % page_size of page
 * page_table[b][r / page_size]:
 *     cache[b][g][r][:] = pages[page_table[b][r / page_size]][g][r % page_size][:]
 * for r < max_pages * page_size.  Elements are copied as they are (dtype
 * only sets their size: 1 = bf16, 0 = fp32).  Returns 10 if a page id is
 * outside [0, num_pages) (that row is left zero).
 * ------------------------------------------------------------------------- */
int oracle_gather_pages(const void* pages, int dtype, const int32_t* page_table, int B, int Hkv,
                        int D, int page_size, int max_pages, int num_pages, void* cache) {
  if (B < 1 || Hkv < 1 || D < 1 || page_size < 1 || max_pages < 1 || num_pages < 1)
    return ORC_BAD_SIZE;
  const size_t es = dtype == 1 ? 2 : 4;
  const size_t row = es * (size_t)D;
  const size_t L = (size_t)max_pages * page_size;
  int status = ORC_OK;
  memset(cache, 0, row * L * (size_t)Hkv * (size_t)B);
  for (int b = 0; b < B; ++b)
    for (int g = 0; g < Hkv; ++g)
      for (size_t r = 0; r < L; ++r) {
        const int pg = page_table[(size_t)b * max_pages + r / (size_t)page_size];
        if (pg < 0 || pg >= num_pages) { status = 10; continue; }
        const size_t src = (((size_t)pg * Hkv + g) * page_size + r % (size_t)page_size) * row;
        const size_t dst = (((size_t)b * Hkv + g) * L + r) * row;
        memcpy((char*)cache + dst, (const char*)pages + src, row);
      }
  return status;
}
