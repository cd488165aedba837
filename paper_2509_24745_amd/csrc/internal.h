// Host-side declarations shared by the C-ABI entry points and the kernel
// launchers.  Not part of the public interface.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pa {

// A validated problem with every derived size resolved.  Passed to kernels
// by value.
struct Shape {
    int n;        // N tokens
    int hq, hkv;  // query / KV heads
    int d;        // head dim
    int b;        // block size
    int g;        // proxy groups
    int s;        // stride
    int dtype;    // PROXYATTN_BF16 / PROXYATTN_F32
    int mq;       // ceil(N / b) = Nk
    int np;       // ceil(N / s) strided tokens
    int bp;       // b / s strided tokens per block
    int rep;      // Hq / Hkv
    int gsize;    // Hq / G
    int mass_chunk;  // keys per chunk of the last-block mass kernels
    int nchunks;     // ceil(N / mass_chunk)
    int est_kc;      // key tiles (32 keys) per chunk of est_rowmax, a multiple of 4
    int est_nc;      // chunks of the longest row: ceil(ceil(N' / 32) / est_kc)
    float scale;  // softmax scale c
    float scale2; // c * log2(e)
    float inv_gsize;  // fl32(1 / |G|)
    int64_t q_tok, q_head, kv_tok, kv_head, o_tok, o_head;  // element strides
    // attention work order (see attn_item): 0 plain, 1 row chunks, 2
    // KV-head-major chunks, then the short rows; the dense kernel's order;
    // rows per chunk
    int attn_order;
    int attn_order_dense;
    int attn_chunk_rows;
    int attn_short_rows;   // order 2 ends on the block rows m < attn_short_rows
};

// Number of XCDs workgroups are dealt to round-robin on MI355X.
constexpr int kNumXcd = 8;

// MI355X's last-level memory-side cache (Infinity Cache / MALL), shared by all
// XCDs.
constexpr size_t kMallBytes = (size_t)256 << 20;

// The attention kernel is persistent: its workgroups pull work items from
// kNumXcd queues (one int32 counter per queue, each on its own 128-byte line).
constexpr int kQueueStride = 32;
constexpr size_t kQueueBytes = (size_t)kNumXcd * kQueueStride * 4;

// Size of the static device scratch array that the entry point which
// allocates nothing uses instead of a workspace (it holds the work queues).
constexpr size_t kScratchBytes = 1024;

// Largest key chunk of the last-block mass kernels (a multiple of every
// block size); shorter sequences halve it down to one block.
constexpr int kMassChunk = 2048;

// Workgroups a launch of an estimation kernel should reach before its key
// loops stop being split: 256 CUs x 2 resident workgroups x 2.
constexpr int kFillGroups = 1024;

// Longest key chunk of est_rowmax, in 32-key tiles: on long sequences every
// workgroup is resident from the start, and without a cap the last row
// band's chain of tiles (up to N'/32) would set the kernel's time.
constexpr int kEstMaxTiles = 128;

// Largest region of per-(row, key block) maxima the estimation keeps at once:
// longer problems produce and reduce them one group of row bands at a time.
constexpr size_t kRbmMaxBytes = (size_t)512 << 20;

// A group of est_rowmax's 128-strided-row bands [xb0, xb1).
struct RbmGroup {
    int xb0, xb1;
};
// Number of band groups (and, if max_pairs is not NULL, the largest group's
// lower-triangular block pairs per proxy group); rbm_group gives group k.
int rbm_groups(const Shape& sh, int64_t* max_pairs);
void rbm_group(const Shape& sh, int k, RbmGroup* out);

// Byte offsets of the workspace regions (each 256-byte aligned).
struct WsLayout {
    size_t qg, kg;   // pooled proxy heads [G][N'][d] (problem dtype)
    size_t rowpart;  // proxy rows' per-chunk (max, sum of exp2) [G][est_nc][N'] float2
    size_t rbm;      // per-(row, key block) max of the scaled proxy logits of one band
                     // group, [G][pairs][b'] fp32 (lower-triangular block pairs
                     // of the group's block rows)
    size_t part;     // last-block (max, sum) per (head, row, key block) [Hq][b][Mq] float2
    size_t lnorm;    // last-block rows' log2-sum-exp [Hq][b] fp32
    size_t kvb;      // re-blocked K and V^T [Hkv][Mq][2 b d] (problem dtype)
    size_t queue;    // attention work-queue counters [kNumXcd][kQueueStride] int32
    size_t diag;     // head-overlap diagnostic: probabilities [Hq][N] fp32, then the
                     // per-head k-th keys [Hq] uint64 (overlaps kvb)
    size_t total;
};

WsLayout ws_layout(const Shape& sh);

// Bytes of the blocked K/V copy: [Hkv][Mq][2 b d] elements.
size_t kv_blocked_bytes(const Shape& sh);

// Workspace regions the estimation launches use.
struct EstWs {
    void* qg;          // pooled proxy queries
    void* kg;          // pooled proxy keys
    float* rbm;        // per-(row, key block) maxima
    float2* rowpart;   // per-(row, key chunk) (max, sum)
    float2* part;      // last-block (max, sum) per (head, row, key block)
    float* lnorm;      // last-block rows' log2-sum-exp
};
// Pooling, proxy block scores (logA [G][Mq][Nk]) and last-block masses
// (mass [Hq][Nk]) in three launches.
hipError_t launch_estimate(const Shape& sh, const void* q, const void* k, const EstWs& w,
                           float* logA, float* mass, hipStream_t st);
hipError_t launch_budget(const Shape& sh, const float* mass, float gamma, int min_blocks,
                         int* head_count, hipStream_t st);
hipError_t launch_select(const Shape& sh, const float* logA, const int* head_count,
                         int row_ratio, int ascending, int* block_count, int* block_index,
                         hipStream_t st);
// launch_budget then launch_select (rank order, constant K), as one launch
// when Nk <= 128; the counts and lists are the same either way.
hipError_t launch_budget_select(const Shape& sh, const float* mass, float gamma, int min_blocks,
                                int* head_count, const float* logA, int* block_count,
                                int* block_index, hipStream_t st);
hipError_t launch_check_lists(const Shape& sh, const int* block_count, const int* block_index,
                              int* status, hipStream_t st);
// launch_kv_block also resets the attention work queues when `queue` is not
// NULL; launch_queue_reset resets them alone.  Either must precede every
// launch_attention on the same stream.
hipError_t launch_kv_block(const Shape& sh, const void* k, const void* v, void* kvb, int* queue,
                           hipStream_t st);
hipError_t launch_queue_reset(int* queue, hipStream_t st);
// Device address of the current device's static scratch array (looked up on
// the first call per device).
hipError_t scratch_address(int** out);
hipError_t launch_head_overlap(const Shape& sh, const void* q, const void* k, int t, int topk,
                               int sink, int renorm, float* z, uint64_t* kth, float* score,
                               hipStream_t st);
hipError_t launch_attention(const Shape& sh, bool dense, const void* q, const void* kvb,
                            const int* block_count, const int* block_index, void* out, float* lse,
                            int* queue, hipStream_t st);

}  // namespace pa
