/*
 * proxyattn.h - C ABI of the ProxyAttn prefill path on MI355X (gfx950).
 *
 * ProxyAttn ("Guided Sparse Attention via Representative Heads",
 * arXiv 2509.24745) speeds up long-context prefill in three steps:
 *
 *   1. proxyattn_estimate        proxy-head block scoring (Sec. 3.1, Eq. 1-2)
 *                                and the per-head last-block attention mass
 *                                the budget is read from (Alg. 1, first two
 *                                steps);
 *   2. proxyattn_select_budget   block-aware dynamic per-head budget (Alg. 1,
 *                                last two steps) and per-head Top-K block
 *                                lists (Sec. 3.2, Eq. 3);
 *   3. proxyattn_block_sparse_prefill
 *                                causal block-sparse attention over the
 *                                selected blocks only (Sec. 3.2, last
 *                                paragraph).
 *
 * proxyattn_dense_prefill runs the same attention kernel over every causal
 * block; it is the dense baseline the sparse path is measured against.
 *
 * One sequence, one attention layer, prefill.  Notation: N tokens, Hq query
 * heads, Hkv key/value heads (GQA: query head i reads KV head i/(Hq/Hkv)),
 * head dim d, block size b, G proxy groups (contiguous runs of Hq/G query
 * heads), stride s, Mq = Nk = ceil(N/b) blocks, N' = ceil(N/s) strided tokens.
 *
 * Conventions shared by every entry point:
 *  - Tensor pointers are DEVICE pointers owned by the caller, 16-byte aligned.
 *    Problem descriptors and scalars are host values.
 *  - The library never allocates device memory and never synchronises.  Every
 *    call validates all of its arguments first; a call that returns
 *    PROXYATTN_E_INVALID, PROXYATTN_E_UNSUPPORTED or PROXYATTN_E_WORKSPACE has
 *    enqueued nothing.  PROXYATTN_E_HIP means that one of the call's launches
 *    failed; kernels the call launched before it stay enqueued, and the
 *    outputs are then unspecified.  A call that returns PROXYATTN_OK has enqueued its
 *    kernels, in order, on `stream` (a hipStream_t; NULL = the default stream)
 *    and returns without waiting.  Faults inside kernels surface at the
 *    caller's next synchronisation.
 *  - Calls are stateless and thread-safe.  Calls that share a workspace must
 *    be ordered (same stream, or synchronised by the caller).
 *  - Results are bitwise deterministic (no floating-point atomics).
 *  - N == 0 is a valid empty problem: nothing is enqueued.
 *  - Inputs must be finite; non-finite inputs give unspecified outputs.
 */
#ifndef PROXYATTN_H
#define PROXYATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes. */
#define PROXYATTN_OK 0
#define PROXYATTN_E_INVALID 1     /* null pointer, negative size, gamma out of (0,1], ... */
#define PROXYATTN_E_UNSUPPORTED 2 /* a shape or dtype the library does not implement */
#define PROXYATTN_E_WORKSPACE 3   /* workspace smaller than proxyattn_workspace_size */
#define PROXYATTN_E_HIP 4         /* a kernel launch failed (see proxyattn_last_error) */

/* Element types of Q, K, V and O. */
#define PROXYATTN_BF16 0
#define PROXYATTN_F32 1

/*
 * Problem descriptor.  Q is [N][Hq][d], K and V are [N][Hkv][d], O is
 * [N][Hq][d]; the innermost dimension d is contiguous.  Token and head
 * strides are in ELEMENTS; 0 selects the packed default (tok = H*d,
 * head = d).  Every row start (token*tok_stride + head*head_stride) must be
 * 16-byte aligned.
 *
 * Supported: d in {64, 128}; b in {64, 128}; s in {1, 2, 4} with b/s >= 16;
 * Hq <= 4096; Hq % Hkv == 0; Hq % G == 0; Nk <= 8192.  bf16 problems compute products on
 * bf16 MFMA with fp32 accumulation; fp32 problems on fp32 MFMA.
 */
typedef struct proxyattn_problem {
    uint32_t struct_size;      /* = sizeof(proxyattn_problem) */
    int32_t seq_len;           /* N >= 0 */
    int32_t num_q_heads;       /* Hq */
    int32_t num_kv_heads;      /* Hkv */
    int32_t head_dim;          /* d */
    int32_t block_size;        /* b */
    int32_t num_proxy_groups;  /* G */
    int32_t stride;            /* s: keep tokens t with t % s == 0 (Sec. 3.1) */
    int32_t dtype;             /* PROXYATTN_BF16 or PROXYATTN_F32 */
    float softmax_scale;       /* <= 0 selects 1/sqrt(d) */
    int64_t q_tok_stride, q_head_stride;
    int64_t kv_tok_stride, kv_head_stride; /* shared by K and V */
    int64_t o_tok_stride, o_head_stride;
    /* Order in which the attention kernel takes its work items (a tuning
     * knob: results are bitwise the same under every setting).
     * attn_order: 0 selects by kernel and problem size; 1 longest block rows
     * first, heads fastest; 2 chunks of R block rows x all query heads; 3
     * chunks of R block rows x the query heads of one KV head, KV head by KV
     * head, for the rows m >= M0, then the rows m < M0 of every head, longest
     * first (M0 = Nk / 8, or Nk / 4 where the re-blocked K/V is small).
     * attn_chunk_rows: R in [1, 8192]; 0 selects by problem size.  Values
     * outside these ranges make every call fail with PROXYATTN_E_INVALID. */
    int32_t attn_order;
    int32_t attn_chunk_rows;
} proxyattn_problem;

/*
 * Bytes of device workspace that proxyattn_estimate and the two prefill
 * entry points need (the largest of their needs; one buffer serves all).
 * Returns PROXYATTN_OK and writes *bytes, or an error for a bad problem.
 *
 * The regions (each rounded up to 256 bytes; esz = element size, b' = b/s,
 * C = key chunks of the block scoring, at most ceil(N'/4096)):
 *   pooled Q^g and K^g      2 * G * N' * d * esz
 *   row (max, sum) pairs    G * C * N' * 8
 *   per-(row, block) maxima G * P * b' * 4
 *   last-block pairs        Hq * b * Mq * 8, plus Hq * b * 4
 *   blocked K/V copy        Hkv * Mq * 2 * b * d * esz
 *   work-queue counters     1024
 * P is the number of lower-triangular block pairs (m, n <= m) of one group
 * of block rows.  The estimation produces and reduces the per-(row, block)
 * maxima one group at a time; a group is a run of consecutive bands of 128
 * strided rows, grown while G * P * b' * 4 stays within 512 MiB (a single
 * band always forms one).  Up to N = 131072 with G = 4 and b' = 32 one group
 * covers every row (P = Mq(Mq+1)/2, 268 MB); longer problems take several
 * groups, and the region stays near 512 MiB instead of growing with the
 * square of the sequence length.
 */
int proxyattn_workspace_size(const proxyattn_problem* p, size_t* bytes);

/*
 * Where proxyattn_estimate leaves the pooled proxy heads inside the
 * workspace: Q^g at workspace+*qg_offset and K^g at workspace+*kg_offset,
 * each [G][N'][d] in the problem's dtype (packed).  For inspection and tests.
 */
int proxyattn_workspace_layout(const proxyattn_problem* p, size_t* qg_offset, size_t* kg_offset);

/*
 * Step 1: block scoring (Sec. 3.1) and last-block mass (Alg. 1).
 *
 *  block_logscore [G][Mq][Nk] fp32 (out): natural log of Eq. 1's
 *      A^g = maxpool(softmax(Q^g K^g^T / sqrt d)) where Q^g, K^g are the
 *      group means of Eq. 2 taken on the tokens t % s == 0, rounded to the
 *      problem dtype; the softmax of strided row t' runs over the strided
 *      causal keys u' <= t'; the max-pool of block (m, n) runs over its
 *      strided rows and causal keys.  Entries with n > m are -inf.
 *  lastblk_mass [Hq][Nk] fp32 (out): per query head i, the attention
 *      probabilities of the last min(b, N) query tokens over all causal keys,
 *      computed with the head's own Q and its KV head's K at full
 *      resolution, summed over those rows and over the keys of each block
 *      (each row of the output sums to min(b, N)).
 *  workspace: device buffer of at least proxyattn_workspace_size bytes.
 */
int proxyattn_estimate(const proxyattn_problem* p, const void* q, const void* k,
                       float* block_logscore, float* lastblk_mass, void* workspace,
                       size_t workspace_bytes, void* stream);

/*
 * Step 2: per-head budget (Alg. 1) and block lists (Eq. 3).
 *
 *  gamma in (0, 1]: cumulative-probability threshold.  Per head, the masses
 *      are normalised to sum 1, sorted descending, and the budget is the
 *      smallest count of leading blocks whose sum reaches gamma (Nk if none;
 *      Nk for gamma == 1).
 *  min_budget_tokens >= 0: the count is raised to ceil(min_budget_tokens/b)
 *      and capped at Nk.
 *  head_count [Hq] int32 (out): the per-head budget in blocks.
 *  block_count [Hq][Mq] int32 (out): min(head_count[i], m+1).
 *  block_index [Hq][Mq][Nk] int32 (out): for head i and block row m, the
 *      block_count[i][m] causal blocks n <= m with the highest
 *      block_logscore[g(i)][m][n] (ties to the lower n), listed from the
 *      highest score down, then -1 up to Nk.  In this order the lists of the
 *      heads of one proxy group are prefixes of one another, which lets the
 *      attention step fetch shared key/value blocks once for all of them.
 *      The same sets listed by ascending block index come from
 *      proxyattn_budget followed by proxyattn_select_topk with mode
 *      PROXYATTN_TOPK_CONSTANT | PROXYATTN_LIST_ASCENDING.
 */
int proxyattn_select_budget(const proxyattn_problem* p, const float* block_logscore,
                            const float* lastblk_mass, float gamma, int32_t min_budget_tokens,
                            int32_t* head_count, int32_t* block_count, int32_t* block_index,
                            void* stream);

/*
 * Step 2 in two calls (budget variants; proxyattn_select_budget is
 * proxyattn_budget followed by proxyattn_select_topk in constant mode: with
 * up to 128 key blocks it runs both in one launch, with the same counts and
 * lists for masses without NaN).
 *
 * proxyattn_budget: Alg. 1's per-head budget alone; arguments as for
 *     proxyattn_select_budget, head_count [Hq] int32 (out).
 *
 * proxyattn_select_topk: Eq. 3 with per-head budgets supplied by the caller
 *     (device array head_count [Hq] int32, in; values outside [0, Nk] are
 *     clamped to it), e.g. the output of proxyattn_budget, or one value for
 *     every head (the static Top-K allocation the paper compares against in
 *     its analysis of dynamic budgets, Sec. 5).  `mode` is one reading of
 *     Eq. 3's K = b_i N (b_i = head_count[i] / Nk), optionally OR-ed with
 *     PROXYATTN_LIST_ASCENDING:
 *       PROXYATTN_TOPK_CONSTANT   N = Nk: every block row m keeps
 *                                 min(head_count[i], m+1) blocks (the reading
 *                                 proxyattn_select_budget uses);
 *       PROXYATTN_TOPK_ROW_RATIO  N = m+1, the row's causal blocks: row m
 *                                 keeps ceil(head_count[i] (m+1) / Nk) blocks;
 *       PROXYATTN_LIST_ASCENDING  list each row's blocks by ascending block
 *                                 index instead of from the highest score
 *                                 down (the same set of blocks; -1 padded).
 *     Other outputs as for proxyattn_select_budget.  Any other bit in mode:
 *     PROXYATTN_E_INVALID.
 */
#define PROXYATTN_TOPK_CONSTANT 0
#define PROXYATTN_TOPK_ROW_RATIO 1
#define PROXYATTN_LIST_ASCENDING 2

int proxyattn_budget(const proxyattn_problem* p, const float* lastblk_mass, float gamma,
                     int32_t min_budget_tokens, int32_t* head_count, void* stream);

int proxyattn_select_topk(const proxyattn_problem* p, const float* block_logscore,
                          const int32_t* head_count, int32_t mode, int32_t* block_count,
                          int32_t* block_index, void* stream);

/*
 * Step 3: block-sparse causal attention.  For query token t in block m and
 * head i, out[t][i] = softmax_u(c * <q_t, k_u>) v_u over the keys u <= t of
 * the blocks block_index[i][m][0 .. block_count[i][m]).  Lists may be in any
 * order but must hold distinct blocks within 0..m, with 1 <= count <= m+1
 * (the lists proxyattn_select_budget writes satisfy this; a row with count 0
 * gets out = 0 and lse = -inf; out-of-range entries are clamped, never read
 * out of bounds).  Blocks are accumulated in list order.
 *  out: [N][Hq][d] in the problem's dtype (o strides).
 *  lse: [Hq][N] fp32 natural-log row log-sum-exp, or NULL.
 *  workspace: as for proxyattn_estimate.  The call first copies K and V into
 *      the blocked layout of proxyattn_prepare_kv inside the workspace, then
 *      runs proxyattn_block_sparse_prefill_blocked on that copy.
 */
int proxyattn_block_sparse_prefill(const proxyattn_problem* p, const void* q, const void* k,
                                   const void* v, const int32_t* block_count,
                                   const int32_t* block_index, void* out, float* lse,
                                   void* workspace, size_t workspace_bytes, void* stream);

/*
 * The attention kernels read K and V from a blocked copy made once per K/V:
 * for every KV head and key block, its keys and its values transposed, cut
 * into sub-blocks of 64 keys that are each one contiguous chunk (rows past N
 * are zero).  Callers that run several attention calls on the same K and V
 * (the sparse path and its dense baseline, several thresholds) make the copy
 * once with proxyattn_prepare_kv and pass it to the _blocked calls below.
 * The layout is private to the library; only its size is part of the ABI.
 *
 * proxyattn_kv_blocked_size: bytes of the copy,
 *     Hkv * ceil(N/b) * 2 * b * d * sizeof(element).
 * proxyattn_prepare_kv: writes the copy of k and v (problem strides) to
 *     kv_blocked (device, 16-byte aligned, at least proxyattn_kv_blocked_size
 *     bytes, else PROXYATTN_E_WORKSPACE).
 * proxyattn_blocked_workspace_size: bytes of workspace the _blocked calls
 *     need (the attention kernel's work-queue counters; a small constant).
 * proxyattn_block_sparse_prefill_blocked / proxyattn_dense_prefill_blocked:
 *     as proxyattn_block_sparse_prefill / proxyattn_dense_prefill, reading K
 *     and V from kv_blocked (written by proxyattn_prepare_kv for the same
 *     problem; kv_blocked_bytes as above).  workspace: at least
 *     proxyattn_blocked_workspace_size bytes; calls that share it must be
 *     ordered.
 */
int proxyattn_kv_blocked_size(const proxyattn_problem* p, size_t* bytes);
int proxyattn_prepare_kv(const proxyattn_problem* p, const void* k, const void* v,
                         void* kv_blocked, size_t kv_blocked_bytes, void* stream);
int proxyattn_blocked_workspace_size(const proxyattn_problem* p, size_t* bytes);
int proxyattn_block_sparse_prefill_blocked(const proxyattn_problem* p, const void* q,
                                           const void* kv_blocked, size_t kv_blocked_bytes,
                                           const int32_t* block_count,
                                           const int32_t* block_index, void* out, float* lse,
                                           void* workspace, size_t workspace_bytes,
                                           void* stream);
int proxyattn_dense_prefill_blocked(const proxyattn_problem* p, const void* q,
                                    const void* kv_blocked, size_t kv_blocked_bytes, void* out,
                                    float* lse, void* workspace, size_t workspace_bytes,
                                    void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * block-sparse attention of proxyattn_block_sparse_prefill_blocked with no
 * workspace argument.  Arguments as there; results bitwise the same.  Its
 * only scratch, the attention kernel's work-queue counters (1 KiB, whatever
 * the problem size), lives in a static device array of 1 KiB that the
 * library holds on every GPU it runs on until the process ends; a need
 * beyond that size would fail with PROXYATTN_E_UNSUPPORTED.  The call
 * allocates and frees nothing; its first call on a device looks the array's
 * address up (a failure there returns PROXYATTN_E_HIP).  Every call on one
 * GPU shares that GPU's array and clears it before use: calls that overlap
 * on one GPU (concurrent streams, or threads without ordering) race and give
 * wrong results; calls ordered on one stream are safe.
 */
int proxyattn_block_sparse_prefill_blocked_noalloc(const proxyattn_problem* p, const void* q,
                                                   const void* kv_blocked,
                                                   size_t kv_blocked_bytes,
                                                   const int32_t* block_count,
                                                   const int32_t* block_index, void* out,
                                                   float* lse, void* stream);

/*
 * Checks caller-made lists against what proxyattn_block_sparse_prefill
 * accepts: the lists of Eq. 3 (Sec. 3.2) select distinct causal key blocks
 * n <= m of query block m.  For every head i and block row m writes
 * status[i][m] (device [Hq][Mq] int32, out): 0 when
 * 1 <= block_count[i][m] <= m+1 and the first block_count[i][m] entries of
 * block_index[i][m] are distinct and lie in 0..m; otherwise the OR of
 *   PROXYATTN_LIST_BAD_COUNT  count outside [1, m+1];
 *   PROXYATTN_LIST_BAD_INDEX  an entry outside [0, m];
 *   PROXYATTN_LIST_DUPLICATE  a block listed twice,
 * where the entries examined are the first min(max(count, 0), Nk).  Reads
 * nothing beyond those entries; deterministic; no workspace.
 */
#define PROXYATTN_LIST_BAD_COUNT 1
#define PROXYATTN_LIST_BAD_INDEX 2
#define PROXYATTN_LIST_DUPLICATE 4
int proxyattn_check_lists(const proxyattn_problem* p, const int32_t* block_count,
                          const int32_t* block_index, int32_t* status, void* stream);

/* Dense causal attention with the same kernels (every block n <= m); the
 * workspace holds the blocked K/V copy as for the sparse call. */
int proxyattn_dense_prefill(const proxyattn_problem* p, const void* q, const void* k,
                            const void* v, void* out, float* lse, void* workspace,
                            size_t workspace_bytes, void* stream);

/*
 * Head-similarity diagnostic (not on the prefill path): the overlap scores
 * of Eq. 4 (the paper's sink-token analysis) for query token t =
 * query_token, on every head's own full-resolution causal attention
 * A[i][u] = softmax_u(c <q_t,i , k_u,kv(i)>), u <= t:
 *     scores[i][j] = sum of A[j][u] over the topk tokens u with the largest
 *                    A[i][u] (ties to the lower token; all t+1 tokens when
 *                    topk > t+1).
 *  sink_tokens in [0, query_token]: the attention to tokens u < sink_tokens
 *      is set to zero first; renormalize (0 or 1): each head's remaining
 *      attention is then rescaled to sum 1 (all zero if nothing remains).
 *  scores: [Hq][Hq] fp32 device output.  workspace: as for
 *  proxyattn_estimate (holds the probabilities).  Deterministic.
 */
int proxyattn_head_overlap(const proxyattn_problem* p, const void* q, const void* k,
                           int32_t query_token, int32_t topk, int32_t sink_tokens,
                           int32_t renormalize, float* scores, void* workspace,
                           size_t workspace_bytes, void* stream);

/* Static text for a return code. */
const char* proxyattn_error_string(int code);

/* Text of the last error raised on the calling thread ("" if none). */
const char* proxyattn_last_error(void);

/* Library version, e.g. "0.1.0". */
const char* proxyattn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* PROXYATTN_H */
