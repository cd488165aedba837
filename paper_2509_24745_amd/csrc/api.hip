// C ABI of the ProxyAttn prefill path: argument validation, workspace
// layout and kernel sequencing.  Every entry point validates all of its
// arguments before enqueuing anything, never allocates and never
// synchronises.
#include <algorithm>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "proxyattn.h"
#include "internal.h"

namespace pa {

static thread_local char g_last_error[512] = "";

static int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
static int fail(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return code;
}

static int hip_fail(hipError_t e, const char* where) {
    return fail(PROXYATTN_E_HIP, "%s: %s", where, hipGetErrorString(e));
}

static size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Validates the descriptor and resolves it into a Shape.
static int resolve(const proxyattn_problem* p, Shape* sh) {
    if (!p) return fail(PROXYATTN_E_INVALID, "problem is NULL");
    if (p->struct_size != sizeof(proxyattn_problem))
        return fail(PROXYATTN_E_INVALID, "struct_size %u != %zu", p->struct_size,
                    sizeof(proxyattn_problem));
    if (p->seq_len < 0) return fail(PROXYATTN_E_INVALID, "seq_len %d < 0", p->seq_len);
    if (p->num_q_heads <= 0 || p->num_kv_heads <= 0 || p->num_proxy_groups <= 0)
        return fail(PROXYATTN_E_INVALID, "head and group counts must be positive");
    if (p->head_dim <= 0 || p->block_size <= 0 || p->stride <= 0)
        return fail(PROXYATTN_E_INVALID, "head_dim, block_size and stride must be positive");
    // grid y/z dimensions carry head and group counts, and the attention
    // kernel's item numbers (about Hq * (Nk + 8R)) must fit an int
    if (p->num_q_heads > 4096)
        return fail(PROXYATTN_E_UNSUPPORTED, "num_q_heads %d > 4096", p->num_q_heads);
    if (p->num_q_heads % p->num_kv_heads)
        return fail(PROXYATTN_E_UNSUPPORTED, "num_q_heads %% num_kv_heads != 0");
    if (p->num_q_heads % p->num_proxy_groups)
        return fail(PROXYATTN_E_UNSUPPORTED, "num_q_heads %% num_proxy_groups != 0");
    if (p->head_dim != 64 && p->head_dim != 128)
        return fail(PROXYATTN_E_UNSUPPORTED, "head_dim %d not in {64, 128}", p->head_dim);
    if (p->block_size != 64 && p->block_size != 128)
        return fail(PROXYATTN_E_UNSUPPORTED, "block_size %d not in {64, 128}", p->block_size);
    if (p->stride != 1 && p->stride != 2 && p->stride != 4)
        return fail(PROXYATTN_E_UNSUPPORTED, "stride %d not in {1, 2, 4}", p->stride);
    if (p->block_size % p->stride || p->block_size / p->stride < 16)
        return fail(PROXYATTN_E_UNSUPPORTED, "block_size / stride must be an integer >= 16");
    if (p->dtype != PROXYATTN_BF16 && p->dtype != PROXYATTN_F32)
        return fail(PROXYATTN_E_UNSUPPORTED, "dtype %d", p->dtype);
    if (!(p->softmax_scale == p->softmax_scale) || isinf(p->softmax_scale))
        return fail(PROXYATTN_E_INVALID, "softmax_scale is not finite");
    const int64_t mq = ((int64_t)p->seq_len + p->block_size - 1) / p->block_size;
    if (mq > 8192) return fail(PROXYATTN_E_UNSUPPORTED, "ceil(N/b) = %lld > 8192", (long long)mq);
    const int esz = p->dtype == PROXYATTN_BF16 ? 2 : 4;
    const int64_t d = p->head_dim;
    Shape s{};
    s.n = p->seq_len;
    s.hq = p->num_q_heads;
    s.hkv = p->num_kv_heads;
    s.d = p->head_dim;
    s.b = p->block_size;
    s.g = p->num_proxy_groups;
    s.s = p->stride;
    s.dtype = p->dtype;
    s.mq = (int)mq;
    s.np = (p->seq_len + p->stride - 1) / p->stride;
    s.bp = p->block_size / p->stride;
    s.rep = p->num_q_heads / p->num_kv_heads;
    s.gsize = p->num_q_heads / p->num_proxy_groups;
    // Key loops of the estimation kernels: chunks of at most kMassChunk keys
    // (mass) and kEstMaxTiles 32-key tiles (block scoring), split further
    // while a launch would have fewer than kFillGroups workgroups, so that
    // short sequences do not leave most CUs idle behind a few long chains.
    {
        int mc = kMassChunk;
        while (mc > s.b && (int64_t)s.hq * ((s.n + mc - 1) / mc) < kFillGroups) mc /= 2;
        s.mass_chunk = mc;
        s.nchunks = (s.n + mc - 1) / mc;
        const int nrb = (s.np + 127) / 128, ntiles = (s.np + 31) / 32;
        // workgroups of est_rowmax with kc tiles per chunk (counting stops at
        // the target)
        auto groups = [&](int kc) {
            int64_t t = 0;
            for (int x = 0; x < nrb && t * s.g < kFillGroups; ++x)
                t += (std::min(x * 128 + 127, s.np - 1) / 32) / kc + 1;
            return t * s.g;
        };
        int kc = std::max(4, std::min((ntiles + 3) / 4 * 4, kEstMaxTiles));
        while (kc > 4 && groups(kc) < kFillGroups) kc = std::max(4, (kc / 2 + 3) / 4 * 4);
        s.est_kc = kc;
        s.est_nc = std::max(1, (ntiles + kc - 1) / kc);
    }
    s.scale = p->softmax_scale > 0.f ? p->softmax_scale : (float)(1.0 / sqrt((double)p->head_dim));
    s.scale2 = s.scale * 1.4426950408889634f;
    s.inv_gsize = 1.0f / (float)s.gsize;
    s.q_tok = p->q_tok_stride ? p->q_tok_stride : (int64_t)p->num_q_heads * d;
    s.q_head = p->q_head_stride ? p->q_head_stride : d;
    s.kv_tok = p->kv_tok_stride ? p->kv_tok_stride : (int64_t)p->num_kv_heads * d;
    s.kv_head = p->kv_head_stride ? p->kv_head_stride : d;
    s.o_tok = p->o_tok_stride ? p->o_tok_stride : (int64_t)p->num_q_heads * d;
    s.o_head = p->o_head_stride ? p->o_head_stride : d;
    // attention work order (tuning knob).  Defaults: the sparse kernel takes
    // KV-head-major chunks followed by the short rows at every size (against
    // row chunks of 2 rows, 0.5-2 % faster from 8K to 64K with 8 KV heads;
    // ending on the short rows keeps the workgroups' finishing times close).
    // Chunks hold 4 rows when the re-blocked K/V takes more than 3/4 of the
    // MALL (which the queries, lists and outputs stream through as well), so
    // that the whole GPU works on one KV head's K/V at a time and it stays in
    // the MALL (measured -2 % at 64K, -3 % at 128K, -10 % at 256K with 8 KV
    // heads, against row chunks), else 2 rows.  The dense kernel, whose rows
    // grow with m, keeps row chunks below that size (KV-head-major is 1.5 %
    // slower at 32K and 5.6 % at 8K there) and KV-head-major above it.
    {
        // the item arithmetic multiplies R by head counts in int
        if (p->attn_order < 0 || p->attn_order > 3)
            return fail(PROXYATTN_E_INVALID, "attn_order %d not in [0, 3]", p->attn_order);
        if (p->attn_chunk_rows < 0 || p->attn_chunk_rows > 8192)
            return fail(PROXYATTN_E_INVALID, "attn_chunk_rows %d not in [0, 8192]",
                        p->attn_chunk_rows);
        const size_t kvb_bytes = (size_t)s.hkv * s.mq * 2 * s.b * s.d * esz;
        const bool big = kvb_bytes * 4 > kMallBytes * 3;
        s.attn_order = p->attn_order ? p->attn_order - 1 : 2;
        s.attn_order_dense = p->attn_order ? p->attn_order - 1 : (big ? 2 : 1);
        s.attn_chunk_rows = p->attn_chunk_rows ? p->attn_chunk_rows : (big ? 4 : 2);
        // the KV-head-major order ends on the rows m < Nk / 8 (Nk / 4 below
        // the MALL rule, where the K/V of those rows is small: 8K -4.7 %, 32K
        // -0.9 % against Nk / 8; from 64K up Nk / 8 is 0.2 % faster)
        s.attn_short_rows = s.mq / (big ? 8 : 4);
    }
    const int64_t strides[6] = {s.q_tok, s.q_head, s.kv_tok, s.kv_head, s.o_tok, s.o_head};
    for (int j = 0; j < 6; ++j) {
        if (strides[j] < 0) return fail(PROXYATTN_E_INVALID, "negative stride");
        if ((strides[j] * esz) % 16)
            return fail(PROXYATTN_E_UNSUPPORTED, "strides must keep rows 16-byte aligned");
    }
    *sh = s;
    return PROXYATTN_OK;
}

// Band groups: consecutive 128-row bands (128 / b' block rows each) whose
// block rows' lower-triangular pairs, over all proxy groups, fit
// kRbmMaxBytes (a single band always forms a group).  Greedy from the first
// band.
static int rbm_walk(const Shape& sh, int want, RbmGroup* out, int64_t* max_pairs) {
    const int nbands = (sh.np + 127) / 128;
    const int rpb = 128 / sh.bp;
    const int64_t cap = (int64_t)(kRbmMaxBytes / ((size_t)sh.g * sh.bp * 4));
    auto pairs = [&](int xb0, int xb1) {
        const int64_t m0 = (int64_t)xb0 * rpb, m1 = std::min((int64_t)xb1 * rpb, (int64_t)sh.mq);
        return m1 * (m1 + 1) / 2 - m0 * (m0 + 1) / 2;
    };
    int k = 0, xb0 = 0;
    int64_t mx = 0;
    while (xb0 < nbands) {
        int xb1 = xb0 + 1;
        while (xb1 < nbands && pairs(xb0, xb1 + 1) <= cap) ++xb1;
        mx = std::max(mx, pairs(xb0, xb1));
        if (k == want && out) { out->xb0 = xb0; out->xb1 = xb1; }
        ++k;
        xb0 = xb1;
    }
    if (max_pairs) *max_pairs = mx;
    return k;
}

int rbm_groups(const Shape& sh, int64_t* max_pairs) { return rbm_walk(sh, -1, nullptr, max_pairs); }

void rbm_group(const Shape& sh, int k, RbmGroup* out) { rbm_walk(sh, k, out, nullptr); }

size_t kv_blocked_bytes(const Shape& sh) {
    const size_t esz = sh.dtype == PROXYATTN_BF16 ? 2 : 4;
    return (size_t)sh.hkv * sh.mq * 2 * sh.d * sh.b * esz;
}

WsLayout ws_layout(const Shape& sh) {
    const size_t esz = sh.dtype == PROXYATTN_BF16 ? 2 : 4;
    WsLayout L{};
    size_t off = 0;
    L.qg = off;   off = align_up(off + (size_t)sh.g * sh.np * sh.d * esz);
    L.kg = off;   off = align_up(off + (size_t)sh.g * sh.np * sh.d * esz);
    L.rowpart = off; off = align_up(off + (size_t)sh.g * sh.est_nc * sh.np * 8);
    int64_t pairs = 0;
    rbm_groups(sh, &pairs);
    L.rbm = off;  off = align_up(off + (size_t)sh.g * (size_t)pairs * sh.bp * 4);
    L.part = off; off = align_up(off + (size_t)sh.hq * sh.b * sh.mq * 8);
    L.lnorm = off; off = align_up(off + (size_t)sh.hq * sh.b * 4);
    L.kvb = off;  off = align_up(off + kv_blocked_bytes(sh));
    L.queue = off; off = align_up(off + kQueueBytes);
    // the diagnostic reuses the re-blocked K/V region (never live at the same time)
    L.diag = L.kvb;
    const size_t diag_end = L.diag + align_up((size_t)sh.hq * sh.n * 4) + align_up((size_t)sh.hq * 8);
    L.total = off > diag_end ? off : diag_end;
    return L;
}

static int check_ws(const Shape& sh, const void* ws, size_t bytes, WsLayout* L) {
    *L = ws_layout(sh);
    if (!ws) return fail(PROXYATTN_E_INVALID, "workspace is NULL");
    if (!aligned16(ws)) return fail(PROXYATTN_E_INVALID, "workspace not 16-byte aligned");
    if (bytes < L->total)
        return fail(PROXYATTN_E_WORKSPACE, "workspace %zu bytes < %zu needed", bytes, L->total);
    return PROXYATTN_OK;
}

static int check_ptr(const void* p, const char* name) {
    if (!p) return fail(PROXYATTN_E_INVALID, "%s is NULL", name);
    if (!aligned16(p)) return fail(PROXYATTN_E_INVALID, "%s not 16-byte aligned", name);
    return PROXYATTN_OK;
}

#define PA_TRY(expr)                         \
    do {                                     \
        const int rc_ = (expr);              \
        if (rc_ != PROXYATTN_OK) return rc_; \
    } while (0)

#define PA_LAUNCH(expr, where)                        \
    do {                                              \
        const hipError_t e_ = (expr);                 \
        if (e_ != hipSuccess) return hip_fail(e_, where); \
    } while (0)

}  // namespace pa

using namespace pa;

extern "C" {

int proxyattn_workspace_size(const proxyattn_problem* p, size_t* bytes) {
    g_last_error[0] = 0;
    Shape sh;
    PA_TRY(resolve(p, &sh));
    if (!bytes) return fail(PROXYATTN_E_INVALID, "bytes is NULL");
    *bytes = sh.n == 0 ? 0 : ws_layout(sh).total;
    return PROXYATTN_OK;
}

int proxyattn_workspace_layout(const proxyattn_problem* p, size_t* qg_offset, size_t* kg_offset) {
    g_last_error[0] = 0;
    Shape sh;
    PA_TRY(resolve(p, &sh));
    if (!qg_offset || !kg_offset) return fail(PROXYATTN_E_INVALID, "offset pointer is NULL");
    const WsLayout L = ws_layout(sh);
    *qg_offset = L.qg;
    *kg_offset = L.kg;
    return PROXYATTN_OK;
}

int proxyattn_estimate(const proxyattn_problem* p, const void* q, const void* k,
                       float* block_logscore, float* lastblk_mass, void* workspace,
                       size_t workspace_bytes, void* stream) {
    g_last_error[0] = 0;
    Shape sh;
    PA_TRY(resolve(p, &sh));
    if (sh.n == 0) return PROXYATTN_OK;
    PA_TRY(check_ptr(q, "q"));
    PA_TRY(check_ptr(k, "k"));
    PA_TRY(check_ptr(block_logscore, "block_logscore"));
    PA_TRY(check_ptr(lastblk_mass, "lastblk_mass"));
    WsLayout L;
    PA_TRY(check_ws(sh, workspace, workspace_bytes, &L));
    hipStream_t st = (hipStream_t)stream;
    char* ws = (char*)workspace;
    const EstWs w{ws + L.qg, ws + L.kg, (float*)(ws + L.rbm), (float2*)(ws + L.rowpart),
                  (float2*)(ws + L.part), (float*)(ws + L.lnorm)};
    PA_LAUNCH(launch_estimate(sh, q, k, w, block_logscore, lastblk_mass, st), "estimate");
    return PROXYATTN_OK;
}

int proxyattn_select_budget(const proxyattn_problem* p, const float* block_logscore,
                            const float* lastblk_mass, float gamma, int32_t min_budget_tokens,
                            int32_t* head_count, int32_t* block_count, int32_t* block_index,
                            void* stream) {
    g_last_error[0] = 0;
    Shape sh;
    PA_TRY(resolve(p, &sh));
    if (!(gamma > 0.f && gamma <= 1.f))
        return fail(PROXYATTN_E_INVALID, "gamma must lie in (0, 1]");
    if (min_budget_tokens < 0) return fail(PROXYATTN_E_INVALID, "min_budget_tokens < 0");
    if (sh.n == 0) return PROXYATTN_OK;
    PA_TRY(check_ptr(block_logscore, "block_logscore"));
    PA_TRY(check_ptr(lastblk_mass, "lastblk_mass"));
    PA_TRY(check_ptr(head_count, "head_count"));
    PA_TRY(check_ptr(block_count, "block_count"));
    PA_TRY(check_ptr(block_index, "block_index"));
    const int64_t min_blocks64 = ((int64_t)min_budget_tokens + sh.b - 1) / sh.b;
    const int min_blocks = (int)(min_blocks64 > sh.mq ? sh.mq : min_blocks64);
    hipStream_t st = (hipStream_t)stream;
    PA_LAUNCH(launch_budget_select(sh, lastblk_mass, gamma, min_blocks, head_count, block_logscore,
                                   block_count, block_index, st),
              "budget_select");
    return PROXYATTN_OK;
}

int proxyattn_budget(const proxyattn_problem* p, const float* lastblk_mass, float gamma,
                     int32_t min_budget_tokens, int32_t* head_count, void* stream) {
    g_last_error[0] = 0;
    Shape sh;
    PA_TRY(resolve(p, &sh));
    if (!(gamma > 0.f && gamma <= 1.f))
        return fail(PROXYATTN_E_INVALID, "gamma must lie in (0, 1]");
    if (min_budget_tokens < 0) return fail(PROXYATTN_E_INVALID, "min_budget_tokens < 0");
    if (sh.n == 0) return PROXYATTN_OK;
    PA_TRY(check_ptr(lastblk_mass, "lastblk_mass"));
    PA_TRY(check_ptr(head_count, "head_count"));
    const int64_t min_blocks64 = ((int64_t)min_budget_tokens + sh.b - 1) / sh.b;
    const int min_blocks = (int)(min_blocks64 > sh.mq ? sh.mq : min_blocks64);
    PA_LAUNCH(launch_budget(sh, lastblk_mass, gamma, min_blocks, head_count, (hipStream_t)stream),
              "budget");
    return PROXYATTN_OK;
}

int proxyattn_select_topk(const proxyattn_problem* p, const float* block_logscore,
                          const int32_t* head_count, int32_t mode, int32_t* block_count,
                          int32_t* block_index, void* stream) {
    g_last_error[0] = 0;
    Shape sh;
    PA_TRY(resolve(p, &sh));
    if (mode & ~(PROXYATTN_TOPK_ROW_RATIO | PROXYATTN_LIST_ASCENDING))
        return fail(PROXYATTN_E_INVALID, "unknown top-k mode %d", (int)mode);
    if (sh.n == 0) return PROXYATTN_OK;
    PA_TRY(check_ptr(block_logscore, "block_logscore"));
    PA_TRY(check_ptr(head_count, "head_count"));
    PA_TRY(check_ptr(block_count, "block_count"));
    PA_TRY(check_ptr(block_index, "block_index"));
    PA_LAUNCH(launch_select(sh, block_logscore, head_count, (mode & PROXYATTN_TOPK_ROW_RATIO) != 0,
                            (mode & PROXYATTN_LIST_ASCENDING) != 0, block_count, block_index,
                            (hipStream_t)stream),
              "select");
    return PROXYATTN_OK;
}

int proxyattn_check_lists(const proxyattn_problem* p, const int32_t* block_count,
                          const int32_t* block_index, int32_t* status, void* stream) {
    g_last_error[0] = 0;
    Shape sh;
    PA_TRY(resolve(p, &sh));
    if (sh.n == 0) return PROXYATTN_OK;
    PA_TRY(check_ptr(block_count, "block_count"));
    PA_TRY(check_ptr(block_index, "block_index"));
    PA_TRY(check_ptr(status, "status"));
    PA_LAUNCH(launch_check_lists(sh, block_count, block_index, status, (hipStream_t)stream),
              "check_lists");
    return PROXYATTN_OK;
}

static int check_kvb(const Shape& sh, const void* kvb, size_t bytes) {
    PA_TRY(check_ptr(kvb, "kv_blocked"));
    const size_t need = kv_blocked_bytes(sh);
    if (bytes < need)
        return fail(PROXYATTN_E_WORKSPACE, "kv_blocked %zu bytes < %zu needed", bytes, need);
    return PROXYATTN_OK;
}

static int check_attn_args(const Shape& sh, const void* q, const int32_t* block_count,
                           const int32_t* block_index, void* out, float* lse, bool dense) {
    PA_TRY(check_ptr(q, "q"));
    PA_TRY(check_ptr(out, "out"));
    if (!dense) {
        PA_TRY(check_ptr(block_count, "block_count"));
        PA_TRY(check_ptr(block_index, "block_index"));
    }
    if (lse && ((uintptr_t)lse & 3u)) return fail(PROXYATTN_E_INVALID, "lse not 4-byte aligned");
    return PROXYATTN_OK;
}

static int prefill_common(const proxyattn_problem* p, const void* q, const void* k,
                          const void* v, const int32_t* block_count, const int32_t* block_index,
                          void* out, float* lse, void* workspace, size_t workspace_bytes,
                          void* stream, bool dense) {
    g_last_error[0] = 0;
    Shape sh;
    PA_TRY(resolve(p, &sh));
    if (sh.n == 0) return PROXYATTN_OK;
    PA_TRY(check_ptr(k, "k"));
    PA_TRY(check_ptr(v, "v"));
    PA_TRY(check_attn_args(sh, q, block_count, block_index, out, lse, dense));
    WsLayout L;
    PA_TRY(check_ws(sh, workspace, workspace_bytes, &L));
    hipStream_t st = (hipStream_t)stream;
    char* ws = (char*)workspace;
    int* queue = (int*)(ws + L.queue);
    // the re-blocking kernel also clears the work-queue counters
    PA_LAUNCH(launch_kv_block(sh, k, v, ws + L.kvb, queue, st), "kv_block");
    PA_LAUNCH(launch_attention(sh, dense, q, ws + L.kvb, block_count, block_index, out, lse, queue,
                               st),
              "attention");
    return PROXYATTN_OK;
}

static int prefill_blocked_common(const proxyattn_problem* p, const void* q, const void* kvb,
                                  size_t kvb_bytes, const int32_t* block_count,
                                  const int32_t* block_index, void* out, float* lse,
                                  void* workspace, size_t workspace_bytes, void* stream,
                                  bool dense) {
    g_last_error[0] = 0;
    Shape sh;
    PA_TRY(resolve(p, &sh));
    if (sh.n == 0) return PROXYATTN_OK;
    PA_TRY(check_kvb(sh, kvb, kvb_bytes));
    PA_TRY(check_attn_args(sh, q, block_count, block_index, out, lse, dense));
    if (!workspace) return fail(PROXYATTN_E_INVALID, "workspace is NULL");
    if (!aligned16(workspace)) return fail(PROXYATTN_E_INVALID, "workspace not 16-byte aligned");
    if (workspace_bytes < kQueueBytes)
        return fail(PROXYATTN_E_WORKSPACE, "workspace %zu bytes < %zu needed", workspace_bytes,
                    kQueueBytes);
    hipStream_t st = (hipStream_t)stream;
    int* queue = (int*)workspace;
    PA_LAUNCH(launch_queue_reset(queue, st), "queue_reset");
    PA_LAUNCH(launch_attention(sh, dense, q, kvb, block_count, block_index, out, lse, queue, st),
              "attention");
    return PROXYATTN_OK;
}

int proxyattn_block_sparse_prefill(const proxyattn_problem* p, const void* q, const void* k,
                                   const void* v, const int32_t* block_count,
                                   const int32_t* block_index, void* out, float* lse,
                                   void* workspace, size_t workspace_bytes, void* stream) {
    return prefill_common(p, q, k, v, block_count, block_index, out, lse, workspace,
                          workspace_bytes, stream, false);
}

int proxyattn_dense_prefill(const proxyattn_problem* p, const void* q, const void* k,
                            const void* v, void* out, float* lse, void* workspace,
                            size_t workspace_bytes, void* stream) {
    return prefill_common(p, q, k, v, nullptr, nullptr, out, lse, workspace, workspace_bytes,
                          stream, true);
}

int proxyattn_block_sparse_prefill_blocked_noalloc(const proxyattn_problem* p, const void* q,
                                                   const void* kv_blocked,
                                                   size_t kv_blocked_bytes_,
                                                   const int32_t* block_count,
                                                   const int32_t* block_index, void* out,
                                                   float* lse, void* stream) {
    g_last_error[0] = 0;
    Shape sh;
    PA_TRY(resolve(p, &sh));
    if (sh.n == 0) return PROXYATTN_OK;
    PA_TRY(check_kvb(sh, kv_blocked, kv_blocked_bytes_));
    PA_TRY(check_attn_args(sh, q, block_count, block_index, out, lse, false));
    // the scratch this call needs (the work-queue counters) against the
    // static array's size; the queues do not grow with the problem
    if (kQueueBytes > kScratchBytes)
        return fail(PROXYATTN_E_UNSUPPORTED, "scratch of %zu bytes needed, %zu available",
                    kQueueBytes, kScratchBytes);
    int* queue = nullptr;
    PA_LAUNCH(scratch_address(&queue), "scratch address");
    hipStream_t st = (hipStream_t)stream;
    PA_LAUNCH(launch_queue_reset(queue, st), "queue_reset");
    PA_LAUNCH(launch_attention(sh, false, q, kv_blocked, block_count, block_index, out, lse, queue,
                               st),
              "attention");
    return PROXYATTN_OK;
}

int proxyattn_kv_blocked_size(const proxyattn_problem* p, size_t* bytes) {
    g_last_error[0] = 0;
    Shape sh;
    PA_TRY(resolve(p, &sh));
    if (!bytes) return fail(PROXYATTN_E_INVALID, "bytes is NULL");
    *bytes = kv_blocked_bytes(sh);
    return PROXYATTN_OK;
}

int proxyattn_prepare_kv(const proxyattn_problem* p, const void* k, const void* v,
                         void* kv_blocked, size_t kv_blocked_bytes_, void* stream) {
    g_last_error[0] = 0;
    Shape sh;
    PA_TRY(resolve(p, &sh));
    if (sh.n == 0) return PROXYATTN_OK;
    PA_TRY(check_ptr(k, "k"));
    PA_TRY(check_ptr(v, "v"));
    PA_TRY(check_kvb(sh, kv_blocked, kv_blocked_bytes_));
    PA_LAUNCH(launch_kv_block(sh, k, v, kv_blocked, nullptr, (hipStream_t)stream), "kv_block");
    return PROXYATTN_OK;
}

int proxyattn_blocked_workspace_size(const proxyattn_problem* p, size_t* bytes) {
    g_last_error[0] = 0;
    Shape sh;
    PA_TRY(resolve(p, &sh));
    if (!bytes) return fail(PROXYATTN_E_INVALID, "bytes is NULL");
    *bytes = sh.n == 0 ? 0 : kQueueBytes;
    return PROXYATTN_OK;
}

int proxyattn_block_sparse_prefill_blocked(const proxyattn_problem* p, const void* q,
                                           const void* kv_blocked, size_t kv_blocked_bytes_,
                                           const int32_t* block_count,
                                           const int32_t* block_index, void* out, float* lse,
                                           void* workspace, size_t workspace_bytes,
                                           void* stream) {
    return prefill_blocked_common(p, q, kv_blocked, kv_blocked_bytes_, block_count, block_index,
                                  out, lse, workspace, workspace_bytes, stream, false);
}

int proxyattn_dense_prefill_blocked(const proxyattn_problem* p, const void* q,
                                    const void* kv_blocked, size_t kv_blocked_bytes_, void* out,
                                    float* lse, void* workspace, size_t workspace_bytes,
                                    void* stream) {
    return prefill_blocked_common(p, q, kv_blocked, kv_blocked_bytes_, nullptr, nullptr, out, lse,
                                  workspace, workspace_bytes, stream, true);
}

const char* proxyattn_error_string(int code) {
    switch (code) {
        case PROXYATTN_OK: return "ok";
        case PROXYATTN_E_INVALID: return "invalid argument";
        case PROXYATTN_E_UNSUPPORTED: return "unsupported problem";
        case PROXYATTN_E_WORKSPACE: return "workspace too small";
        case PROXYATTN_E_HIP: return "HIP launch failure";
        default: return "unknown error";
    }
}

const char* proxyattn_last_error(void) { return g_last_error; }

const char* proxyattn_version(void) { return "0.1.0"; }

int proxyattn_head_overlap(const proxyattn_problem* p, const void* q, const void* k,
                           int32_t query_token, int32_t topk, int32_t sink_tokens,
                           int32_t renormalize, float* scores, void* workspace,
                           size_t workspace_bytes, void* stream) {
    g_last_error[0] = 0;
    Shape sh;
    PA_TRY(resolve(p, &sh));
    if (query_token < 0 || query_token >= sh.n)
        return fail(PROXYATTN_E_INVALID, "query_token %d outside [0, %d)", (int)query_token, sh.n);
    if (topk < 1) return fail(PROXYATTN_E_INVALID, "topk %d < 1", (int)topk);
    if (sink_tokens < 0 || sink_tokens > query_token)
        return fail(PROXYATTN_E_INVALID, "sink_tokens %d outside [0, query_token]", (int)sink_tokens);
    if (renormalize != 0 && renormalize != 1)
        return fail(PROXYATTN_E_INVALID, "renormalize must be 0 or 1");
    PA_TRY(check_ptr(q, "q"));
    PA_TRY(check_ptr(k, "k"));
    PA_TRY(check_ptr(scores, "scores"));
    WsLayout L;
    PA_TRY(check_ws(sh, workspace, workspace_bytes, &L));
    char* ws = (char*)workspace;
    float* z = (float*)(ws + L.diag);
    uint64_t* kth = (uint64_t*)(ws + L.diag + align_up((size_t)sh.hq * sh.n * 4));
    PA_LAUNCH(launch_head_overlap(sh, q, k, query_token, topk, sink_tokens, renormalize, z, kth,
                                  scores, (hipStream_t)stream),
              "head_overlap");
    return PROXYATTN_OK;
}

}  // extern "C"

