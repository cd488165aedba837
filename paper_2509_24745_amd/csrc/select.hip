// Block-aware budget (Alg. 1, last two steps) and per-head Top-K block
// lists (Sec. 3.2, Eq. 3).
//
// budget: one workgroup per query head.  The head's last-block masses are
//   normalised to sum 1 (Alg. 1 normalises the pooled block scores), sorted
//   descending in LDS (bitonic), prefix-summed with a wavefront scan, and
//   the first prefix reaching gamma gives the count k*+1 (Nk if none, Nk for
//   gamma >= 1), then raised to the minimum budget and capped at Nk.
// select: one workgroup per (proxy group, block row m).  The m+1 causal
//   candidates are sorted by (score descending, index ascending) as 64-bit
//   keys in LDS (bitonic); every head of the group lists the first
//   min(count_i, m+1) of them in that rank order and pads its row with -1
//   (the per-row-ratio reading of Eq. 3 instead lists ceil(count_i (m+1) / Nk),
//   i.e. the same fraction of every row's causal blocks).
//   Rank order makes the lists of a group's heads prefixes of one another,
//   so the attention workgroups of those heads, which run side by side on
//   one XCD, fetch the same K/V blocks in the same order; blocks read close
//   together in time are shared through the L2.  On request the same sets
//   are listed by ascending block index instead (a rank table in LDS and a
//   stream compaction per head).
// check_lists: one workgroup per (block row m, head i); validates a
//   caller-made list against what the attention step accepts.
#include "common.h"
#include "internal.h"

namespace pa {

// In-place bitonic sort of a[0..P) (P a power of two), ascending.
template <typename K>
__device__ void bitonic_sort_asc(K* a, int P, int tid, int nth) {
    for (int size = 2; size <= P; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int t = tid; t < P / 2; t += nth) {
                const int i = 2 * t - (t & (stride - 1));
                const int j = i + stride;
                const bool up = (i & size) == 0;
                const K x = a[i], y = a[j];
                if (up ? (x > y) : (x < y)) { a[i] = y; a[j] = x; }
            }
            __syncthreads();
        }
    }
}

static __host__ __device__ inline int next_pow2(int x) {
    int p = 1;
    while (p < x) p <<= 1;
    return p;
}

// ---------------------------------------------------------------------------
// budget: grid Hq, 1024 threads
// ---------------------------------------------------------------------------
constexpr int kBudgetThreads = 1024;
constexpr int kMaxBlocks = 8192;

__global__ __launch_bounds__(kBudgetThreads) void budget_kernel(Shape sh,
                                                                const float* __restrict__ mass,
                                                                float gamma, int min_blocks,
                                                                int* __restrict__ head_count) {
    __shared__ float a[kMaxBlocks];
    __shared__ float wtot[kBudgetThreads / 64];
    __shared__ int hit;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int i = blockIdx.x, nk = sh.mq;
    const int P = next_pow2(nk);
    const float* mrow = mass + (int64_t)i * nk;

    // total mass (fixed-order reduction)
    float part = 0.f;
    for (int n = tid; n < nk; n += kBudgetThreads) part += mrow[n];
    part = wave_sum(part);
    if (lane == 0) wtot[w] = part;
    if (tid == 0) hit = nk;
    __syncthreads();
    float total = 0.f;
    for (int j = 0; j < kBudgetThreads / 64; ++j) total += wtot[j];
    // normalised block shares, padded with -1 (sorted to the end)
    for (int n = tid; n < P; n += kBudgetThreads) a[n] = n < nk ? mrow[n] / total : -1.f;
    __syncthreads();
    // descending order = ascending order of the negated values
    for (int n = tid; n < P; n += kBudgetThreads) a[n] = -a[n];
    __syncthreads();
    bitonic_sort_asc<float>(a, P, tid, kBudgetThreads);
    // inclusive prefix sums: each thread owns E consecutive entries
    const int E = (P + kBudgetThreads - 1) / kBudgetThreads;
    const int e0 = tid * E;
    float own = 0.f;
    for (int e = 0; e < E; ++e) {
        const int n = e0 + e;
        if (n < nk) own += -a[n];
    }
    float incl = own;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const float y = __shfl_up(incl, o);
        if (lane >= o) incl += y;
    }
    float excl_w = __shfl_up(incl, 1);
    if (lane == 0) excl_w = 0.f;
    __syncthreads();
    if (lane == 63) wtot[w] = incl;
    __syncthreads();
    float base = 0.f;
    for (int j = 0; j < w; ++j) base += wtot[j];
    float run = base + excl_w;
    if (gamma < 1.f) {
        for (int e = 0; e < E; ++e) {
            const int n = e0 + e;
            if (n >= nk) break;
            run += -a[n];
            if (run >= gamma) { atomicMin(&hit, n); break; }
        }
    }
    __syncthreads();
    if (tid == 0) {
        int c = (gamma < 1.f && hit < nk) ? hit + 1 : nk;
        c = max(c, min_blocks);
        c = min(c, nk);
        head_count[i] = c;
    }
}

// ---------------------------------------------------------------------------
// select: grid (Mq, G), 256 threads, dynamic LDS = P * 8 bytes (+ P * 4 for
// ascending lists)
// ---------------------------------------------------------------------------
constexpr int kSelectThreads = 256;

__global__ __launch_bounds__(kSelectThreads) void select_kernel(Shape sh,
                                                                const float* __restrict__ logA,
                                                                const int* __restrict__ head_count,
                                                                int row_ratio, int ascending,
                                                                int* __restrict__ block_count,
                                                                int* __restrict__ block_index) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
    __shared__ int wsum[kSelectThreads / 64];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int m = blockIdx.x, g = blockIdx.y, nk = sh.mq;
    const int ncand = m + 1;
    const int P = next_pow2(ncand);
    uint64_t* key = reinterpret_cast<uint64_t*>(smem_raw);
    const float* srow = logA + ((int64_t)g * sh.mq + m) * nk;
    // key: (order of -score) << 32 | index  -> ascending = score desc, index asc
    for (int n = tid; n < P; n += kSelectThreads) {
        uint64_t kk = ~0ull;
        if (n < ncand) kk = ((uint64_t)(~float_order_key(srow[n])) << 32) | (uint32_t)n;
        key[n] = kk;
    }
    __syncthreads();
    bitonic_sort_asc<uint64_t>(key, P, tid, kSelectThreads);
    // ascending lists: rank[n] = position of block n in the rank order; each
    // thread owns E consecutive candidates
    int* rank = reinterpret_cast<int*>(key + P);
    const int E = (ncand + kSelectThreads - 1) / kSelectThreads;
    const int n0 = min(tid * E, ncand), n1 = min(n0 + E, ncand);
    if (ascending) {
        for (int p = tid; p < ncand; p += kSelectThreads) rank[(int)(key[p] & 0xffffffffu)] = p;
        __syncthreads();
    }
    // the sorted keys are the candidates in rank order: a head's set is the
    // first min(count, m+1) of them (sets of one group are prefixes of each
    // other); it is listed in that order, or by ascending block index
    for (int i = g * sh.gsize; i < (g + 1) * sh.gsize; ++i) {
        // counts outside [0, Nk] (caller-supplied) are clamped
        const int c = min(max(head_count[i], 0), nk);
        // per-row ratio: ceil(c (m+1) / Nk), exact in integers (< 2^26)
        const int kk = row_ratio ? min((c * ncand + nk - 1) / nk, ncand) : min(c, ncand);
        int* out = block_index + ((int64_t)i * sh.mq + m) * nk;
        if (!ascending) {
            for (int p = tid; p < nk; p += kSelectThreads)
                out[p] = p < kk ? (int)(key[p] & 0xffffffffu) : -1;
        } else {
            // stream compaction of the blocks with rank < kk, in index order:
            // a thread's own count, then an exclusive scan over the workgroup
            int own = 0;
            for (int n = n0; n < n1; ++n) own += rank[n] < kk;
            int incl = own;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const int y = __shfl_up(incl, o);
                if (lane >= o) incl += y;
            }
            if (lane == 63) wsum[w] = incl;
            __syncthreads();
            int pos = incl - own;
            for (int j = 0; j < w; ++j) pos += wsum[j];
            for (int n = n0; n < n1; ++n)
                if (rank[n] < kk) out[pos++] = n;
            for (int p = kk + tid; p < nk; p += kSelectThreads) out[p] = -1;
            __syncthreads();   // wsum is reused by the next head
        }
        if (tid == 0) block_count[(int64_t)i * sh.mq + m] = kk;
    }
}

// Status of list (i, m): bit 0 = count outside [1, m+1]; bit 1 = one of the
// first min(max(count, 0), Nk) entries outside [0, m]; bit 2 = a block listed
// twice among them.  A bitmap of the row's m+1 causal blocks in LDS finds
// the duplicates (integer LDS atomics: the result does not depend on which
// thread sees the second copy).
constexpr int kCheckThreads = 256;

__global__ __launch_bounds__(kCheckThreads) void check_lists_kernel(
    Shape sh, const int* __restrict__ block_count, const int* __restrict__ block_index,
    int* __restrict__ status) {
    __shared__ unsigned seen[8192 / 32];
    __shared__ int flags;
    const int m = blockIdx.x, i = blockIdx.y, tid = threadIdx.x, nk = sh.mq;
    for (int wd = tid; wd < (m + 32) / 32; wd += kCheckThreads) seen[wd] = 0u;
    if (tid == 0) flags = 0;
    __syncthreads();
    const int64_t row = (int64_t)i * sh.mq + m;
    const int cnt = block_count[row];
    const int n = min(max(cnt, 0), nk);
    const int* list = block_index + row * nk;
    int f = (cnt < 1 || cnt > m + 1) ? 1 : 0;
    for (int p = tid; p < n; p += kCheckThreads) {
        const int v = list[p];
        if (v < 0 || v > m) {
            f |= 2;
        } else {
            const unsigned bit = 1u << (v & 31);
            if (atomicOr(&seen[v >> 5], bit) & bit) f |= 4;
        }
    }
    if (f) atomicOr(&flags, f);
    __syncthreads();
    if (tid == 0) status[row] = flags;
}

hipError_t launch_check_lists(const Shape& sh, const int* block_count, const int* block_index,
                              int* status, hipStream_t st) {
    hipLaunchKernelGGL(check_lists_kernel, dim3(sh.mq, sh.hq), dim3(kCheckThreads), 0, st, sh,
                       block_count, block_index, status);
    return hipGetLastError();
}

hipError_t launch_budget(const Shape& sh, const float* mass, float gamma, int min_blocks,
                         int* head_count, hipStream_t st) {
    hipLaunchKernelGGL(budget_kernel, dim3(sh.hq), dim3(kBudgetThreads), 0, st, sh, mass, gamma,
                       min_blocks, head_count);
    return hipGetLastError();
}

hipError_t launch_select(const Shape& sh, const float* logA, const int* head_count,
                         int row_ratio, int ascending, int* block_count, int* block_index,
                         hipStream_t st) {
    const size_t P = (size_t)next_pow2(sh.mq);
    const size_t smem = P * 8 + (ascending ? P * 4 : 0);
    if (smem > 65536) {
        hipError_t e = hipFuncSetAttribute((const void*)select_kernel,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(select_kernel, dim3(sh.mq, sh.g), dim3(kSelectThreads), smem, st, sh, logA,
                       head_count, row_ratio, ascending, block_count, block_index);
    return hipGetLastError();
}

}  // namespace pa
