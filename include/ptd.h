/*
 * ptd.h -- C ABI of the Progressive Tree Drafting hot path on MI355X (gfx950).
 *
 * One decoding step of Progressive Tree Drafting (PTD) packs a token tree
 * after the committed prefix and runs the target model once over it (Sec. 3.1,
 * Sec. 3.2, Alg. 1 step 2).  This library provides the data-parallel part of
 * that step, as hand-written HIP kernels:
 *
 *   ptd_build_tree_mask  ancestor-or-self bitmasks and depths of the tree
 *   ptd_tree_attention   tree-masked attention over committed KV + ancestors
 *                        (ptd_tree_attention_ragged: trees of different sizes
 *                        in one padded batch; ptd_tree_attention_paged: the
 *                        same on paged caches; ptd_tree_attention_fp8kv: on
 *                        8-bit E4M3 key/value caches; _paged_fp8kv: both)
 *   ptd_topk_argmax      per-row argmax / top-k of the verification logits
 *   ptd_verify           greedy longest accepted path (+ bonus token)
 *   ptd_expand           progressive expansion with top-k children
 *   ptd_verify_expand    the two above in one launch
 *   ptd_tree_rope        positions of the tree nodes; rotary embedding of
 *                        their queries and keys at those positions
 *   ptd_kv_commit        the accepted path's keys/values become committed rows
 *   ptd_verify_sample    sampling verification (recursive candidate-tree
 *                        sampling) with caller-drawn uniforms
 *   ptd_step_prune       stepping: depth control of the draft forest
 *   ptd_pool_*           the value-keyed candidate pool: merge of every
 *                        draft sub-tree, retrieval by the last token
 *
 * Conventions shared by every entry point
 *   - Array arguments are DEVICE pointers owned by the caller (stream-ordered;
 *     the library keeps no pointer after the call returns).  Exceptions are
 *     marked "host".
 *   - Calls are asynchronous on `stream` (a hipStream_t passed as void*; NULL
 *     means the default stream).  No entry point synchronizes the stream or
 *     allocates device memory; scratch memory comes from a caller workspace.
 *   - The return value is a ptd_status.  Host-detectable errors (null pointers,
 *     sizes, alignment, workspace size) are returned before anything is
 *     launched.  A failed launch returns PTD_ERR_HIP.  Data-dependent errors
 *     that only the device can see (a malformed parent array, a KV length that
 *     does not fit the cache) are written to *dev_status (device int32,
 *     nullable) with first-error-wins semantics; the caller zeroes it.  After
 *     a device-reported error the outputs are unspecified.
 *   - Outputs are bitwise reproducible run to run (no float atomics; partial
 *     results are combined in a fixed order).
 *   - Tree arrays: node i of a sequence has parent[i] in [-1, i) (topological
 *     order); -1 means the node's parent is the last committed token.  The tree
 *     may be a forest.  Sec. 3.1 "Tree Construction".
 */
#ifndef PTD_H
#define PTD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PTD_F32 = 0,  /* IEEE binary32 */
  PTD_BF16 = 1  /* bfloat16 (upper half of binary32) */
} ptd_dtype;

typedef enum {
  PTD_OK = 0,
  PTD_ERR_NULL = 1,      /* a required pointer is NULL */
  PTD_ERR_SHAPE = 2,     /* a size is out of range or inconsistent */
  PTD_ERR_DTYPE = 3,     /* unsupported dtype combination */
  PTD_ERR_ALIGN = 4,     /* a pointer or leading dimension is misaligned */
  PTD_ERR_WORKSPACE = 5, /* workspace missing or too small */
  PTD_ERR_HIP = 6,       /* a HIP runtime call or kernel launch failed */
  PTD_ERR_BAD_TREE = 7,  /* device-detected: parent[i] outside [-1, i) */
  PTD_ERR_KV_LEN = 8,    /* device-detected: kv_len < 0 or kv_len + T > L_cap */
  PTD_ERR_BAD_PATH = 9,  /* device-detected: accepted path not strictly increasing
                            node ids in [0, T), or its length outside [0, T] */
  PTD_ERR_PAGE = 10,     /* device-detected: a page id outside [0, num_pages) */
  PTD_ERR_SCRATCH = 11   /* the problem needs more scratch than the fixed array of
                            ptd_tree_attention_noalloc (PTD_NOALLOC_SCRATCH_BYTES) */
} ptd_status;

/* Dimension pairs turned together by the rotary embedding. */
typedef enum {
  PTD_ROPE_HALF = 0,        /* pair p = (x[p], x[p + D/2]) */
  PTD_ROPE_INTERLEAVED = 1  /* pair p = (x[2p], x[2p + 1]) */
} ptd_rope_pairing;

#define PTD_MAX_T 1024   /* tree nodes per sequence */
#define PTD_MAX_K 16     /* top-k */
#define PTD_MAX_DEPTH 64 /* entries of a width schedule */
#define PTD_NOALLOC_SCRATCH_BYTES (64u << 20) /* device scratch of ptd_tree_attention_noalloc */

/* Attention problem description (host struct, read during the call only). */
typedef struct {
  int32_t B;          /* sequences, >= 1 */
  int32_t Hq;         /* query heads, >= 1 */
  int32_t Hkv;        /* key/value heads; Hq % Hkv == 0 (GQA group Hq/Hkv) */
  int32_t D;          /* head dim: 64 or 128 */
  int32_t L_cap;      /* rows per (sequence, KV head) in the caches */
  ptd_dtype in_dtype; /* dtype of q, k_cache, v_cache */
  ptd_dtype out_dtype;/* dtype of out */
  float scale;        /* softmax scale; 0 selects 1/sqrt(D) */
} ptd_attn_shape;

/* Human-readable name of a status code (static string, never NULL). */
const char* ptd_status_string(int status);

/* Library version as MAJOR*10000 + MINOR*100 + PATCH. */
int ptd_version(void);

/*
 * ptd_build_tree_mask -- ancestor sets pi(v) = {v} u pi(P(v)) and positions
 * |pi(v)| (Sec. 3.1 "Tree Construction").
 *   parent    int32 [B][T]
 *   tree_len  int32 [B] or NULL (NULL: all T nodes are live).  Nodes at index
 *             >= tree_len[b] are padding: their mask rows and depths are 0.
 *   mask      uint64 [B][T][W], W = ceil(T/64): bit j of word j/64 of row i is
 *             set iff node j is i or an ancestor of i.
 *   depth     int32 [B][T]: |pi(i)| (1 for a root).
 *   dev_status  PTD_ERR_BAD_TREE if some live parent[i] is outside [-1, i).
 * Errors: PTD_ERR_NULL, PTD_ERR_SHAPE (B < 1, T < 1 or T > PTD_MAX_T).
 */
int ptd_build_tree_mask(const int32_t* parent, const int32_t* tree_len, int32_t B,
                        int32_t T, uint64_t* mask, int32_t* depth,
                        int32_t* dev_status, void* stream);

/*
 * Workspace bytes ptd_tree_attention needs for this shape and tree size
 * (split-KV partial results, plus room for the masks when they are read from
 * memory -- fp32 inputs, or T > 128 -- and mask == NULL).  The workspace needs
 * no initialisation; calls sharing one workspace must not overlap.
 * shape->L_cap may be below T (for ptd_tree_attention_ragged).
 * Returns 0 on invalid arguments.
 */
size_t ptd_tree_attention_workspace_bytes(const ptd_attn_shape* shape, int32_t T);

/*
 * ptd_tree_attention -- each tree node attends to the committed prefix and to
 * its own ancestors only (Sec. 3.1 "Tree Construction"; the joint forward over
 * [X; T; C_X] of Sec. 3.2 uses the same mask):
 *   for sequence b, query head h (KV head g = h / (Hq/Hkv)) and node i,
 *     keys  S = { rows 0 .. kv_len[b]-1 } u { row kv_len[b] + a : a in pi(i) }
 *     out[b][i][h] = sum_{j in S} softmax_j(scale * q . k_j) v_j
 *   q        [B][T][Hq][D]           in_dtype
 *   k_cache  [B][Hkv][L_cap][D]      in_dtype; tree node i's key is row kv_len[b]+i
 *   v_cache  [B][Hkv][L_cap][D]      in_dtype; likewise
 *   kv_len   int32 [B]               committed length; needs kv_len+T <= L_cap
 *                                    (L_cap < T is rejected up front)
 *   parent   int32 [B][T]            tree (all T nodes live)
 *   T        nodes per sequence, 1 .. PTD_MAX_T
 *   out      [B][T][Hq][D]           out_dtype (fp32 accumulation inside)
 *   shape    host struct above
 *   mask     uint64 [B][T][ceil(T/64)] from ptd_build_tree_mask, or NULL to
 *            have it built into the workspace.  Read only by the fp32 path
 *            and for T > 128: with bf16 inputs and T <= 128 the kernel derives
 *            every row's ancestor words from parent itself (mask ignored).
 *   workspace, workspace_bytes: device scratch of at least
 *            ptd_tree_attention_workspace_bytes(shape, T) bytes, 256-byte aligned
 * Pointers to q/k/v/out must be 16-byte aligned.  in_dtype bf16 runs on MFMA
 * (v_mfma_f32_16x16x32_bf16); fp32 inputs run on the vector ALUs.
 * dev_status: PTD_ERR_BAD_TREE, PTD_ERR_KV_LEN.
 * Errors: PTD_ERR_NULL, PTD_ERR_SHAPE, PTD_ERR_DTYPE, PTD_ERR_ALIGN,
 * PTD_ERR_WORKSPACE, PTD_ERR_HIP.
 */
int ptd_tree_attention(const void* q, const void* k_cache, const void* v_cache,
                       const int32_t* kv_len, const int32_t* parent, int32_t T,
                       void* out, const ptd_attn_shape* shape,
                       const uint64_t* mask, void* workspace,
                       size_t workspace_bytes, int32_t* dev_status, void* stream);

/*
 * ptd_tree_attention_ragged -- ptd_tree_attention over a padded batch of
 * trees of different sizes (the attention of Sec. 3.1, with a batch of
 * sequences that each carry their own draft tree, as a server holds them):
 *   tree_len  int32 [B] device, or NULL (all T nodes live).  Sequence b has
 *             n_b = min(max(tree_len[b], 0), T) live nodes 0 .. n_b-1; the
 *             slots n_b .. T-1 are padding.
 * Live node i attends exactly as in ptd_tree_attention (its ancestors are
 * live nodes); the rows of padding nodes in out are zero.  Parents, queries
 * and cache rows of padding nodes are not read, and a sequence's cache needs
 * only kv_len[b] + n_b <= L_cap rows.  mask (if given) must come from
 * ptd_build_tree_mask with the same tree_len.  Other arguments, workspace,
 * dev_status and errors as ptd_tree_attention.
 */
int ptd_tree_attention_ragged(const void* q, const void* k_cache, const void* v_cache,
                              const int32_t* kv_len, const int32_t* tree_len,
                              const int32_t* parent, int32_t T, void* out,
                              const ptd_attn_shape* shape, const uint64_t* mask,
                              void* workspace, size_t workspace_bytes,
                              int32_t* dev_status, void* stream);

/*
 * ptd_tree_attention_fp8kv -- ptd_tree_attention_ragged on key/value caches
 * stored as OCP FP8 E4M3 codes (1 byte per element, half the bytes of bf16;
 * a serving format, not in the paper) with one fp32 scale per KV head:
 *   key row j of head g = e4m3(k_cache[b][g][j][:]) * k_scale[g], values likewise
 *   k_cache, v_cache  uint8 [B][Hkv][L_cap][D] E4M3 codes (no NaN codes)
 *   k_scale, v_scale  fp32 [Hkv] device, or NULL for 1
 *   q                 bf16 [B][T][Hq][D]: shape->in_dtype must be PTD_BF16
 * D = 128 only.  Codes are widened to bf16 exactly inside the kernel, the key
 * scale joins the softmax scale and the value scale the output, so the
 * arithmetic is that of the bf16 path on the decoded caches.  tree_len may be
 * NULL; masks are derived or built as for ptd_tree_attention (no mask
 * argument).  Workspace: ptd_tree_attention_workspace_bytes(shape, T).
 * dev_status and errors as ptd_tree_attention; PTD_ERR_DTYPE for non-bf16
 * queries, PTD_ERR_SHAPE for D != 128, PTD_ERR_ALIGN for scales that are not
 * 4-byte aligned.
 */
int ptd_tree_attention_fp8kv(const void* q, const void* k_cache, const void* v_cache,
                             const float* k_scale, const float* v_scale,
                             const int32_t* kv_len, const int32_t* tree_len,
                             const int32_t* parent, int32_t T, void* out,
                             const ptd_attn_shape* shape, void* workspace,
                             size_t workspace_bytes, int32_t* dev_status, void* stream);

/*
 * ptd_tree_attention_noalloc -- ptd_tree_attention_ragged for callers that
 * cannot allocate device memory or pass a workspace (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation).  Same
 * operation, arguments (tree_len may be NULL), results and dev_status codes
 * as ptd_tree_attention_ragged, without the workspace arguments: the split
 * partials and, when needed, the ancestor masks go to a fixed device array of
 * PTD_NOALLOC_SCRATCH_BYTES (64 MiB) that the library holds on each GPU it
 * runs on until the process ends.  The call allocates nothing and clears
 * nothing (the scratch needs no initialisation).  Every call on one GPU
 * shares that GPU's array: calls that overlap on one GPU (several streams or
 * host threads) race and their outputs are unspecified; calls ordered on one
 * stream are safe.  ptd_tree_attention_workspace_bytes(shape, T) is the
 * scratch a problem needs (the masks' share only with T > 128 or fp32
 * inputs, when mask is NULL).
 * Errors: those of ptd_tree_attention_ragged except PTD_ERR_WORKSPACE;
 * PTD_ERR_SCRATCH if the problem needs more than PTD_NOALLOC_SCRATCH_BYTES;
 * PTD_ERR_HIP if the array's device address cannot be obtained.
 */
int ptd_tree_attention_noalloc(const void* q, const void* k_cache, const void* v_cache,
                               const int32_t* kv_len, const int32_t* tree_len,
                               const int32_t* parent, int32_t T, void* out,
                               const ptd_attn_shape* shape, const uint64_t* mask,
                               int32_t* dev_status, void* stream);

/* Paged key/value caches (host struct, read during the call only). */
typedef struct {
  const void* k_pages;        /* [num_pages][Hkv][page_size][D] in_dtype */
  const void* v_pages;        /* likewise */
  const int32_t* page_table;  /* [B][max_pages]: row r of sequence b lives in
                                 page page_table[b][r / page_size], at
                                 r % page_size */
  int32_t page_size;          /* rows per page: a power of two >= 32 */
  int32_t max_pages;          /* page-table entries per sequence */
  int32_t num_pages;          /* pages in k_pages / v_pages */
} ptd_kv_pages;

/*
 * ptd_tree_attention_paged -- ptd_tree_attention_ragged on paged caches: the
 * same operation, arguments and workspace (tree_len may be NULL), with
 * sequence b's cache row r (committed rows, then tree node i at row
 * kv_len[b] + i) read from page page_table[b][r / page_size].  shape->L_cap
 * must equal max_pages * page_size; bf16 inputs only (the MFMA path).
 * Entries of the page table past a sequence's kv_len + n_b rows are not read.
 * A page id outside [0, num_pages) is reported and page 0 is read in its
 * place.
 * dev_status: PTD_ERR_BAD_TREE, PTD_ERR_KV_LEN, PTD_ERR_PAGE.
 * Errors: as ptd_tree_attention; PTD_ERR_DTYPE for fp32 inputs.
 */
int ptd_tree_attention_paged(const void* q, const ptd_kv_pages* kv, const int32_t* kv_len,
                             const int32_t* tree_len, const int32_t* parent, int32_t T, void* out,
                             const ptd_attn_shape* shape, const uint64_t* mask,
                             void* workspace, size_t workspace_bytes, int32_t* dev_status,
                             void* stream);

/*
 * ptd_tree_attention_paged_fp8kv -- ptd_tree_attention_fp8kv on paged caches:
 * kv->k_pages / v_pages hold E4M3 codes, [num_pages][Hkv][page_size][D]
 * bytes, addressed through the page table as in ptd_tree_attention_paged;
 * k_scale / v_scale as in ptd_tree_attention_fp8kv.  Errors: the union of the
 * two calls' checks.
 */
int ptd_tree_attention_paged_fp8kv(const void* q, const ptd_kv_pages* kv, const float* k_scale,
                                   const float* v_scale, const int32_t* kv_len,
                                   const int32_t* tree_len, const int32_t* parent, int32_t T,
                                   void* out, const ptd_attn_shape* shape, void* workspace,
                                   size_t workspace_bytes, int32_t* dev_status, void* stream);

/* Workspace bytes ptd_topk_argmax needs (0 on invalid arguments). */
size_t ptd_topk_workspace_bytes(int32_t R, int32_t V, int32_t k);

/*
 * ptd_topk_argmax -- greedy verification tokens (the highest-probability
 * prediction of every node, Sec. 3.2) and the top-k candidates used for child
 * expansion (App. A), per row of logits.
 *   logits    [R][ld] of dtype; row r's entries are logits[r*ld .. r*ld+V-1]
 *   R         rows (B*(T+1) for a step: row 0 of each sequence is the last
 *             committed token, row i+1 is node i)
 *   V, ld     vocabulary size (1 .. 2^31-1) and row stride in elements (>= V)
 *   k         1 .. PTD_MAX_K, k <= V
 *   argmax    int32 [R]            (required)
 *   topk_idx  int32 [R][k]         (nullable)
 *   topk_val  float [R][k]         (nullable) the selected entries' own values,
 *                                  widened exactly to fp32
 * Order: value descending; equal values by the lower index; -0.0 equals +0.0.
 * Logits are expected non-NaN (NaN ordering is unspecified); +-inf are ordered.
 * A workspace is needed when a row is split over several workgroups, that is
 * when V exceeds one workgroup's slice (32768 bf16 or 16384 fp32 values, 1.5
 * times that when R times the slices of a row would exceed 256);
 * ptd_topk_workspace_bytes gives its size (the larger of the bf16 and fp32
 * needs), 0 when none is needed.  It needs no initialisation, and calls
 * sharing one must not overlap.
 * Errors: PTD_ERR_NULL, PTD_ERR_SHAPE, PTD_ERR_DTYPE, PTD_ERR_WORKSPACE,
 * PTD_ERR_HIP.
 */
int ptd_topk_argmax(const void* logits, ptd_dtype dtype, int32_t R, int32_t V,
                    int64_t ld, int32_t k, int32_t* argmax, int32_t* topk_idx,
                    float* topk_val, void* workspace, size_t workspace_bytes,
                    void* stream);

/*
 * ptd_verify -- greedy verification (Sec. 3.2; Alg. 1 steps 5-6).  The edge
 * (P(c), c) is eligible iff the verification token of P(c) -- argmax row
 * P(c)+1, row 0 for a root -- equals draft_tokens[c].  A node is accepted iff
 * all edges on its root path are eligible.  accept_len = largest depth of an
 * accepted node (0 if none); the terminal is the lowest-index accepted node of
 * that depth.  X' = the draft tokens of the terminal's root path, shallowest
 * first, then the bonus token argmax[terminal+1] (argmax[0] if nothing is
 * accepted).
 *   argmax        int32 [B][T+1]
 *   draft_tokens  int32 [B][T]
 *   parent        int32 [B][T]
 *   tree_len      int32 [B] or NULL (nodes >= tree_len[b] are ignored)
 *   accept_len    int32 [B]
 *   accept_nodes  int32 [B][T]   node ids of the path, -1 padded
 *   out_tokens    int32 [B][T+1] X' without n_0, -1 padded
 * dev_status: PTD_ERR_BAD_TREE.
 * Errors: PTD_ERR_NULL, PTD_ERR_SHAPE, PTD_ERR_HIP.
 */
int ptd_verify(const int32_t* argmax, const int32_t* draft_tokens,
               const int32_t* parent, const int32_t* tree_len, int32_t B,
               int32_t T, int32_t* accept_len, int32_t* accept_nodes,
               int32_t* out_tokens, int32_t* dev_status, void* stream);

/*
 * ptd_expand -- progressive expansion V^t = V^{t-1} u {d_v} with top-k
 * children (Sec. 3.1 "Progressive Expansion" and "Overhead Constraints";
 * App. A):
 *   1. node v (index order) offers topk_idx[b][v+1][0..k-1] as children; a
 *      node of depth d grows only if d+1 <= d_max, and stops once it has
 *      width_sched[d] children counting existing ones; a candidate equal to
 *      the token of one of v's children (existing or just added) is skipped
 *      (same node, as in the merge of Sec. 3.1 "Draft Extraction").  The
 *      committed token (row 0) is not expanded.
 *   2. breadth-first renumbering: by depth, then by the parent's new index,
 *      then old children in index order before new children in candidate
 *      order; roots keep their relative order.
 *   3. the first T_max nodes are kept; slots >= tree_len_next[b] hold -1.
 *   parent, tokens  int32 [B][T];  tree_len int32 [B] or NULL
 *   topk_idx        int32 [B][T+1][k] (as written by ptd_topk_argmax)
 *   width_sched     HOST int32 [d_max]; entry 0 (number of roots) is unused
 *   d_max           1 .. PTD_MAX_DEPTH;  T_max 1 .. PTD_MAX_T;
 *                   T*(k+1) <= 16384
 *   parent_next, tokens_next  int32 [B][T_max];  tree_len_next int32 [B]
 * dev_status: PTD_ERR_BAD_TREE.
 * Errors: PTD_ERR_NULL, PTD_ERR_SHAPE, PTD_ERR_HIP.
 */
int ptd_expand(const int32_t* parent, const int32_t* tokens,
               const int32_t* tree_len, int32_t B, int32_t T,
               const int32_t* topk_idx, int32_t k, const int32_t* width_sched,
               int32_t d_max, int32_t T_max, int32_t* parent_next,
               int32_t* tokens_next, int32_t* tree_len_next,
               int32_t* dev_status, void* stream);

/*
 * ptd_verify_expand -- ptd_verify followed by ptd_expand on the same tree in
 * one launch (the tree is staged on chip once); outputs are identical to the
 * two calls in sequence.  Arguments have the meaning given above; both groups
 * of outputs are written.  Sec. 3.2 and Sec. 3.1 as cited there.
 * dev_status: PTD_ERR_BAD_TREE.  Errors: PTD_ERR_NULL, PTD_ERR_SHAPE,
 * PTD_ERR_HIP.
 */
int ptd_verify_expand(const int32_t* argmax, const int32_t* draft_tokens,
                      const int32_t* parent, const int32_t* tree_len, int32_t B,
                      int32_t T, const int32_t* topk_idx, int32_t k,
                      const int32_t* width_sched, int32_t d_max, int32_t T_max,
                      int32_t* accept_len, int32_t* accept_nodes, int32_t* out_tokens,
                      int32_t* parent_next, int32_t* tokens_next,
                      int32_t* tree_len_next, int32_t* dev_status, void* stream);

/*
 * ptd_tree_rope -- positions of the tree nodes and the rotary embedding of
 * their queries and keys.  Sec. 3.1 "Tree Construction": the position of node
 * v is given by |pi(v)|; a root's parent is the last committed token (at
 * position kv_len[b] - 1), so
 *     pos[b][i] = kv_len[b] + |pi(i)| - 1.
 * The rotary embedding (Su et al., RoFormer) turns dimension pair p,
 * 0 <= p < D/2, by the angle a = pos * inv_freq[p]:
 *     (x_a, x_b) -> (x_a cos a - x_b sin a, x_a sin a + x_b cos a).
 *   q          [B][T][Hq][D] in_dtype, turned in place; NULL to skip queries
 *   k_cache    [B][Hkv][L_cap][D] in_dtype: the tree rows kv_len[b] + i,
 *              i < T, are turned in place (no other row is touched); NULL to
 *              skip keys
 *   kv_len, parent, T   as for ptd_tree_attention (all T nodes live); kv_len
 *              needs 0 <= kv_len, and kv_len + T <= L_cap when k_cache is
 *              given (kv_len + T <= INT32_MAX otherwise)
 *   shape      B, Hq, Hkv, D (64 or 128), L_cap and in_dtype; out_dtype and
 *              scale are not used
 *   theta      base of the default frequencies inv_freq[p] = theta^(-2p/D)
 *              (finite, > 0; ignored when inv_freq is given)
 *   inv_freq   HOST double [D/2] or NULL: explicit frequencies (for scaled
 *              variants of the embedding)
 *   pairing    a ptd_rope_pairing
 *   pos_out    int32 [B][T] or NULL: the positions
 * Angles and their sine and cosine are computed in fp64, the rotation in
 * fp32, and results are rounded to in_dtype (nearest even).  q and k_cache
 * must be 16-byte aligned.  A sequence whose tree or kv_len is rejected is
 * left untouched.
 * dev_status: PTD_ERR_BAD_TREE, PTD_ERR_KV_LEN.
 * Errors: PTD_ERR_NULL (shape, kv_len or parent NULL, or all of q, k_cache,
 * pos_out NULL), PTD_ERR_SHAPE, PTD_ERR_DTYPE, PTD_ERR_ALIGN, PTD_ERR_HIP.
 */
int ptd_tree_rope(void* q, void* k_cache, const int32_t* kv_len, const int32_t* parent,
                  int32_t T, const ptd_attn_shape* shape, double theta,
                  const double* inv_freq, int32_t pairing, int32_t* pos_out,
                  int32_t* dev_status, void* stream);

/*
 * ptd_kv_commit -- commit of the accepted path (Sec. 3.2: the accepted
 * sequence X' = (n_0, n_1, ..., n_k, V_{n_k})).  The draft nodes n_1..n_k,
 * whose keys and values the forward pass wrote at cache rows kv_len[b] + n_j,
 * become committed tokens: for j = 1..k, row kv_len[b] + n_j moves to row
 * kv_len[b] + j - 1 in every KV head of both caches, and
 * kv_len_next[b] = kv_len[b] + k.  Other rows keep their content.  The bonus
 * token V_{n_k} is the next step's input and has no key or value yet.  With
 * ptd_tree_rope's positions, a node of depth j was rotated at
 * kv_len[b] + j - 1, its committed row.
 *   k_cache, v_cache  [B][Hkv][L_cap][D] in_dtype, updated in place, 16-byte
 *                     aligned
 *   kv_len            int32 [B]; needs 0 <= kv_len and kv_len + T <= L_cap
 *   accept_len        int32 [B]: k, 0 .. T
 *   accept_nodes      int32 [B][T]: n_1 .. n_k first (as written by
 *                     ptd_verify), strictly increasing in [0, T); entries
 *                     from k on are not read
 *   T                 tree rows per sequence, 1 .. PTD_MAX_T
 *   shape             B, Hkv, D (64 or 128), L_cap and in_dtype are used
 *   kv_len_next       int32 [B]; must not be the kv_len buffer
 * A sequence whose kv_len or path is rejected keeps its caches and gets
 * kv_len_next = kv_len.
 * dev_status: PTD_ERR_KV_LEN, PTD_ERR_BAD_PATH.
 * Errors: PTD_ERR_NULL, PTD_ERR_SHAPE, PTD_ERR_DTYPE, PTD_ERR_ALIGN, PTD_ERR_HIP.
 */
int ptd_kv_commit(void* k_cache, void* v_cache, const int32_t* kv_len,
                  const int32_t* accept_len, const int32_t* accept_nodes, int32_t T,
                  const ptd_attn_shape* shape, int32_t* kv_len_next, int32_t* dev_status,
                  void* stream);

/* Workspace bytes ptd_verify_sample needs: a (maximum, normalizer) pair of
 * doubles per block of 2048 vocabulary entries per logits row, 256-byte
 * rounded (0 on invalid arguments).  The workspace needs no initialisation;
 * calls sharing one must not overlap. */
size_t ptd_verify_sample_workspace_bytes(int32_t B, int32_t T, int32_t V);

/*
 * ptd_verify_sample -- sampling verification of the tree (Sec. 3.2 "sampling
 * decoding strategy"; App. E recursive candidate-tree sampling; App. F proof
 * of distributional consistency).  P_v = softmax(row of v / temperature),
 * row 0 being the last committed token n_0 and row v+1 node v.  From n_0 the
 * children of the current node v are examined in index order; child n with
 * token t is accepted iff u_node[b][n] < P_v[t] / S, S = mass of P_v not yet
 * rejected at v (1 before the first child).  A rejected token's probability
 * becomes 0 (S drops by it), so a later sibling with the same token is
 * rejected.  The walk moves to an accepted child; when all children of v are
 * rejected, v is the terminal and the bonus token is the smallest x with
 * sum_{y<=x} P'_y > u_bonus[b][row of v] * W, P' being P_v with the rejected
 * tokens removed and W its total (the last token with P'_y > 0 if rounding
 * leaves none; -1 if W = 0).
 *   logits        [B*(T+1)][ld] of dtype, finite; V entries per row
 *   V             1 .. 262144;  ld >= V (elements)
 *   draft_tokens, parent  int32 [B][T];  tree_len int32 [B] or NULL
 *   temperature   finite, > 0
 *   u_node        double [B][T]   the draw made when node n is examined
 *   u_bonus       double [B][T+1] the draw for the bonus token at each row
 *                 (uniforms in [0, 1), drawn by the caller)
 *   accept_len, accept_nodes, out_tokens  as for ptd_verify
 *   workspace     >= ptd_verify_sample_workspace_bytes(B, T, V), 16-byte aligned
 *   B*(T+1)       at most 65535 rows
 * Precision: the normalizer is a fp64 sum of fp32 exponentials taken per
 * block of 2048 entries relative to the block maximum and rescaled to the
 * row maximum (each factor ~1.2e-7 relative, argument rounding compensated);
 * the examined children's numerators are fp64; the bonus CDF sums the same
 * terms in fp64.  A uniform within ~5e-7 of the probability or cumulative
 * probability it is compared with may decide differently from an exact
 * computation.
 * dev_status: PTD_ERR_BAD_TREE.
 * Errors: PTD_ERR_NULL, PTD_ERR_SHAPE, PTD_ERR_DTYPE, PTD_ERR_WORKSPACE,
 * PTD_ERR_ALIGN, PTD_ERR_HIP.
 */
int ptd_verify_sample(const void* logits, ptd_dtype dtype, int32_t V, int64_t ld,
                      const int32_t* draft_tokens, const int32_t* parent,
                      const int32_t* tree_len, int32_t B, int32_t T, double temperature,
                      const double* u_node, const double* u_bonus, int32_t* accept_len,
                      int32_t* accept_nodes, int32_t* out_tokens, void* workspace,
                      size_t workspace_bytes, int32_t* dev_status, void* stream);

/*
 * ptd_step_prune -- stepping, the depth control of the draft tree (Sec. 3.1
 * "Overhead Constraints", Stepping Mechanism; Alg. 1 step 3).  A sub-tree
 * (the tree under one root of the forest) deeper than d_max is replaced by
 * the sub-tree of its earliest-added child -- the lowest-index child -- and
 * its other branches are pruned, repeatedly, so a chain keeps its last d_max
 * nodes.  Depth = number of nodes on the longest root path.  The kept forest
 * is renumbered breadth first (by depth; by the parent's new index; siblings
 * in old index order; roots in the order of the roots they replace) and cut
 * to T_max nodes; slots from tree_len_next on hold -1.
 *   parent, tokens  int32 [B][T], T 1 .. 128;  tree_len int32 [B] or NULL
 *   d_max           >= 1;  T_max 1 .. PTD_MAX_T
 *   parent_next, tokens_next  int32 [B][T_max];  tree_len_next int32 [B]
 * dev_status: PTD_ERR_BAD_TREE (that sequence's output is empty).
 * Errors: PTD_ERR_NULL, PTD_ERR_SHAPE, PTD_ERR_HIP.
 */
int ptd_step_prune(const int32_t* parent, const int32_t* tokens, const int32_t* tree_len,
                   int32_t B, int32_t T, int32_t d_max, int32_t T_max, int32_t* parent_next,
                   int32_t* tokens_next, int32_t* tree_len_next, int32_t* dev_status,
                   void* stream);

/*
 * Candidate pool (Sec. 3.1 "Draft Extraction via Merging"; Alg. 1 steps 1
 * and 4): per sequence, trees of tokens keyed by the token of their root, at
 * most e_max trees (1 .. 2048) of at most n_cap nodes (1 .. 129, root
 * included, so that a retrieved tree can fill 128 draft slots).  The pool is a caller-owned device buffer of ptd_pool_bytes
 * bytes, 256-byte aligned, set up once by ptd_pool_init; every call that
 * names it must pass the same B, e_max and n_cap.  Calls on one pool must not
 * overlap.  Returns 0 from ptd_pool_bytes on invalid arguments.
 */
size_t ptd_pool_bytes(int32_t B, int32_t e_max, int32_t n_cap);
int ptd_pool_init(void* pool, size_t pool_bytes, int32_t B, int32_t e_max, int32_t n_cap,
                  void* stream);

/*
 * ptd_pool_merge -- for every node u of the draft tree (index order), the
 * sub-tree of u (u and its descendants, a tree rooted at token(u)) is merged
 * by M into the pool tree keyed token(u), which is created with a lone root
 * if absent: a child whose token is not among the matching pool node's
 * children is added, one whose token is there is merged into it.  A
 * sub-tree's nodes are taken in index order (each after its parent), which
 * fixes the insertion order.  An insertion beyond n_cap nodes, or a new tree
 * beyond e_max trees, is skipped together with what it would carry.
 *   parent, tokens  int32 [B][T], T 1 .. 128;  tree_len int32 [B] or NULL
 * dev_status: PTD_ERR_BAD_TREE (that sequence's pool is left unchanged).
 * Errors: PTD_ERR_NULL, PTD_ERR_SHAPE, PTD_ERR_WORKSPACE (pool_bytes too
 * small), PTD_ERR_ALIGN, PTD_ERR_HIP.
 */
int ptd_pool_merge(void* pool, size_t pool_bytes, int32_t B, int32_t e_max, int32_t n_cap,
                   const int32_t* parent, const int32_t* tokens, const int32_t* tree_len,
                   int32_t T, int32_t* dev_status, void* stream);

/*
 * ptd_pool_retrieve -- the candidate tree C_X of the next step: the pool tree
 * keyed by last_token[b] (the last committed token), without its root, as a
 * packed tree: breadth first (by depth; by the parent's output index;
 * siblings in insertion order), the root's children with parent -1, cut to
 * T_max nodes; slots from tree_len_out on hold -1; tree_len_out 0 if there is
 * no such tree.
 *   last_token      int32 [B]
 *   parent_out, tokens_out  int32 [B][T_max], T_max 1 .. PTD_MAX_T;
 *   tree_len_out    int32 [B]
 * Errors: PTD_ERR_NULL, PTD_ERR_SHAPE, PTD_ERR_WORKSPACE, PTD_ERR_ALIGN,
 * PTD_ERR_HIP.
 */
int ptd_pool_retrieve(const void* pool, size_t pool_bytes, int32_t B, int32_t e_max,
                      int32_t n_cap, const int32_t* last_token, int32_t T_max,
                      int32_t* parent_out, int32_t* tokens_out, int32_t* tree_len_out,
                      void* stream);

#ifdef __cplusplus
}
#endif

#endif /* PTD_H */
