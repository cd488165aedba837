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
// budget + select in one launch (Nk <= 128, rank order): in every select
//   workgroup, wave 0 sorts the row's candidates in registers (one or two
//   per lane) while waves 1-3 derive the budgets of the group's heads, three
//   heads at a time per wave with one or two blocks per lane, by the budget
//   workgroup's own arithmetic (the same sums in the same order, the same
//   sorting network over the same padded shares, the same prefix sums), so
//   the counts and lists are those of the two launches for masses without
//   NaN; the workgroups of block row 0 write the counts out.  Lane
//   exchanges go through DPP where the pattern allows.  On short sequences
//   the second launch, its dependent wait and the LDS sort's barriers are
//   most of the selection time.
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

// Lane exchange x[l ^ O] for a compile-time O: DPP for O < 16 (quad
// permutations; O = 4 as the quad reversal followed by the half-row mirror,
// since (7 - l) ^ 3 = l ^ 4 within 8 lanes; O = 8 as the row rotation by 8),
// an LDS permute for 16, v_permlane32_swap for 32.
template <int O>
__device__ __forceinline__ uint32_t lane_xor(uint32_t x) {
    if constexpr (O == 1) {
        return __builtin_amdgcn_update_dpp(0, x, 0xB1, 0xF, 0xF, false);   // quad_perm [1,0,3,2]
    } else if constexpr (O == 2) {
        return __builtin_amdgcn_update_dpp(0, x, 0x4E, 0xF, 0xF, false);   // quad_perm [2,3,0,1]
    } else if constexpr (O == 4) {
        const uint32_t y = __builtin_amdgcn_update_dpp(0, x, 0x1B, 0xF, 0xF, false);  // [3,2,1,0]
        return __builtin_amdgcn_update_dpp(0, y, 0x141, 0xF, 0xF, false);  // row_half_mirror
    } else if constexpr (O == 8) {
        return __builtin_amdgcn_update_dpp(0, x, 0x128, 0xF, 0xF, false);  // row_ror:8
    } else if constexpr (O == 16) {
        return (uint32_t)__shfl_xor((int)x, 16);
    } else {
        static_assert(O == 32, "lane_xor: O in {1, 2, 4, 8, 16, 32}");
        const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
        return (__lane_id() & 32) ? r[0] : r[1];
    }
}
template <int O>
__device__ __forceinline__ float lane_xor_f(float x) {
    return __uint_as_float(lane_xor<O>(__float_as_uint(x)));
}

// The bitonic network over E * 64 entries held E per lane: entry
// e = lane + 64 r sits in register r of the lane.  One compare-exchange
// stage pairs e with e ^ STRIDE (between lanes for STRIDE < 64, between two
// registers of the lane otherwise) with bitonic_sort_asc's rule: the pair
// swaps when its lower entry is greater (rising runs, bit SIZE of e clear)
// or smaller (falling runs).
template <int STRIDE>
__device__ __forceinline__ float xor_of(float a) { return lane_xor_f<STRIDE>(a); }
template <int STRIDE>
__device__ __forceinline__ uint64_t xor_of(uint64_t a) {
    return ((uint64_t)lane_xor<STRIDE>((uint32_t)(a >> 32)) << 32) | lane_xor<STRIDE>((uint32_t)a);
}

template <int SIZE, int STRIDE, int E, typename K>
__device__ __forceinline__ void bitonic_stage(K (&a)[E], int lane) {
    if constexpr (STRIDE >= 64) {
        constexpr int RS = STRIDE / 64;
#pragma unroll
        for (int r = 0; r < E; ++r) {
            if ((r & RS) == 0) {
                const K xi = a[r], xj = a[r | RS];
                const bool up = ((lane + 64 * r) & SIZE) == 0;
                if (up ? (xi > xj) : (xi < xj)) {
                    a[r] = xj;
                    a[r | RS] = xi;
                }
            }
        }
    } else {
#pragma unroll
        for (int r = 0; r < E; ++r) {
            const K y = xor_of<STRIDE>(a[r]);
            const bool lower = (lane & STRIDE) == 0;
            const K xi = lower ? a[r] : y, xj = lower ? y : a[r];
            const bool up = ((lane + 64 * r) & SIZE) == 0;
            a[r] = (up ? (xi > xj) : (xi < xj)) ? y : a[r];
        }
    }
}
// The stages of run size SIZE, strides SIZE/2 .. 1.
template <int SIZE, int STRIDE, int E, typename K>
__device__ __forceinline__ void bitonic_merge(K (&a)[E], int lane) {
    bitonic_stage<SIZE, STRIDE>(a, lane);
    if constexpr (STRIDE > 1) bitonic_merge<SIZE, STRIDE / 2>(a, lane);
}
// The run sizes 2 .. LIMIT that do not exceed P (uniform over the wave): the
// network of P entries.
template <int SIZE, int LIMIT, int E, typename K>
__device__ __forceinline__ void bitonic_sort_regs(K (&a)[E], int lane, int P) {
    if (SIZE <= P) bitonic_merge<SIZE, SIZE / 2>(a, lane);
    if constexpr (SIZE < LIMIT) bitonic_sort_regs<SIZE * 2, LIMIT>(a, lane, P);
}

// The budgets of H heads with Nk <= 64 E in one wave, interleaved: lane l
// holds the masses x[h][r] of blocks l + 64 r (0 beyond Nk).  budget_kernel
// keeps block n in thread n (waves 0 .. E-1 with these Nk); this repeats its
// operations on the same values: each of its waves' sums of the masses,
// added in wave order (the other waves' totals are zero); the shares
// negated and padded with +1 up to P = next_pow2(Nk); the bitonic network
// over those P entries (entries >= P, held at +inf, are never paired with
// entries < P); each wave's inclusive scan, offset by the totals of the
// waves before it; and the first prefix reaching gamma.
template <int H, int E>
__device__ __forceinline__ void wave_budgets(const float (&x)[H][E], int nk, float gamma,
                                             int min_blocks, int lane, int (&c)[H]) {
    const int P = next_pow2(nk);
    float a[H][E];
#pragma unroll
    for (int h = 0; h < H; ++h) {
        float total = 0.f;
#pragma unroll
        for (int r = 0; r < E; ++r) {
            const int e = lane + 64 * r;
            float t = e < nk ? 0.f + x[h][r] : 0.f;
            t += lane_xor_f<32>(t);
            t += lane_xor_f<16>(t);
            t += lane_xor_f<8>(t);
            t += lane_xor_f<4>(t);
            t += lane_xor_f<2>(t);
            t += lane_xor_f<1>(t);
            total += t;
        }
#pragma unroll
        for (int r = 0; r < E; ++r) {
            const int e = lane + 64 * r;
            a[h][r] = e < nk ? -(x[h][r] / total) : (e < P ? 1.f : __builtin_inff());
        }
    }
#pragma unroll
    for (int h = 0; h < H; ++h) bitonic_sort_regs<2, 64 * E>(a[h], lane, P);
#pragma unroll
    for (int h = 0; h < H; ++h) {
        float base = 0.f;
        int hit = nk;
#pragma unroll
        for (int r = 0; r < E; ++r) {
            const int e = lane + 64 * r;
            float own = 0.f;
            if (e < nk) own += -a[h][r];
            float incl = own;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const float y = __shfl_up(incl, o);
                if (lane >= o) incl += y;
            }
            float excl = __shfl_up(incl, 1);
            if (lane == 0) excl = 0.f;
            float run = base + excl;
            run += -a[h][r];
            const uint64_t hits = __ballot(gamma < 1.f && e < nk && run >= gamma);
            if (hit == nk && hits) hit = 64 * r + __builtin_ctzll(hits);
            base += __shfl(incl, 63);
        }
        int cc = (gamma < 1.f && hit < nk) ? hit + 1 : nk;
        cc = max(cc, min_blocks);
        c[h] = min(cc, nk);
    }
}
// Up to 128 blocks (two entries per lane) one launch is faster than two;
// with 256 (four per lane) the one wave's sorts take longer than the second
// launch saves (measured: 30 against 24 us at 24K tokens).
constexpr int kFusedMaxBlocks = 128;
constexpr int kFusedHeads = 3;         // heads per wave and round

// ---------------------------------------------------------------------------
// select: grid (Mq, G), 256 threads, dynamic LDS = P * 8 bytes (+ P * 4 for
// ascending lists; + 4 per head of the group when fused)
// ---------------------------------------------------------------------------
constexpr int kSelectThreads = 256;

// FE > 0 (fused, Nk <= 64 FE): the counts are derived from `mass` (see
// wave_budgets) and written to head_count by block row 0; FE = 0: they are
// read from head_count.
template <int FE>
__global__ __launch_bounds__(kSelectThreads) void select_kernel(Shape sh,
                                                                const float* __restrict__ logA,
                                                                int* __restrict__ head_count,
                                                                const float* __restrict__ mass,
                                                                float gamma, int min_blocks,
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
    int* cnt = reinterpret_cast<int*>(key + P) + (ascending ? P : 0);
    if constexpr (FE > 0) {
        // wave 0 sorts the row's candidates in registers (FE per lane; the
        // keys are distinct, so any sorting network gives the same order)
        // while waves 1-3 derive the group's budgets, kFusedHeads heads per
        // wave and round
        if (w == 0) {
            uint64_t kk[FE];
#pragma unroll
            for (int r = 0; r < FE; ++r) {
                const int e = lane + 64 * r;
                kk[r] = e < ncand ? ((uint64_t)(~float_order_key(srow[e])) << 32) | (uint32_t)e
                                  : ~0ull;
            }
            bitonic_sort_regs<2, 64 * FE>(kk, lane, P);
#pragma unroll
            for (int r = 0; r < FE; ++r)
                if (lane + 64 * r < P) key[lane + 64 * r] = kk[r];
        } else {
            const int i0 = g * sh.gsize, i1 = i0 + sh.gsize;
            for (int ib = i0 + kFusedHeads * (w - 1); ib < i1; ib += 3 * kFusedHeads) {
                float x[kFusedHeads][FE];
                int c[kFusedHeads];
#pragma unroll
                for (int h = 0; h < kFusedHeads; ++h)
#pragma unroll
                    for (int r = 0; r < FE; ++r) {
                        const int e = lane + 64 * r;
                        x[h][r] = (ib + h < i1 && e < nk) ? mass[(int64_t)(ib + h) * nk + e] : 0.f;
                    }
                wave_budgets<kFusedHeads, FE>(x, nk, gamma, min_blocks, lane, c);
                if (lane == 0) {
#pragma unroll
                    for (int h = 0; h < kFusedHeads; ++h) {
                        if (ib + h < i1) {
                            cnt[ib + h - i0] = c[h];
                            if (m == 0) head_count[ib + h] = c[h];
                        }
                    }
                }
            }
        }
        __syncthreads();
    } else {
        // key: (order of -score) << 32 | index  -> ascending = score desc, index asc
        for (int n = tid; n < P; n += kSelectThreads) {
            uint64_t kk = ~0ull;
            if (n < ncand) kk = ((uint64_t)(~float_order_key(srow[n])) << 32) | (uint32_t)n;
            key[n] = kk;
        }
        __syncthreads();
        bitonic_sort_asc<uint64_t>(key, P, tid, kSelectThreads);
    }
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
        const int c = min(max(FE > 0 ? cnt[i - g * sh.gsize] : head_count[i], 0), nk);
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
        hipError_t e = hipFuncSetAttribute((const void*)select_kernel<0>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
        if (e != hipSuccess) return e;
    }
    // the kernel only reads head_count when not fused
    hipLaunchKernelGGL(select_kernel<0>, dim3(sh.mq, sh.g), dim3(kSelectThreads), smem, st, sh,
                       logA, const_cast<int*>(head_count), nullptr, 0.f, 0, row_ratio, ascending,
                       block_count, block_index);
    return hipGetLastError();
}

template <int FE>
static hipError_t launch_fused(const Shape& sh, const float* mass, float gamma, int min_blocks,
                               int* head_count, const float* logA, int* block_count,
                               int* block_index, hipStream_t st) {
    const size_t smem = (size_t)next_pow2(sh.mq) * 8 + (size_t)sh.gsize * 4;
    if (smem > 65536) {
        hipError_t e = hipFuncSetAttribute((const void*)select_kernel<FE>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(select_kernel<FE>, dim3(sh.mq, sh.g), dim3(kSelectThreads), smem, st, sh,
                       logA, head_count, mass, gamma, min_blocks, 0, 0, block_count, block_index);
    return hipGetLastError();
}

hipError_t launch_budget_select(const Shape& sh, const float* mass, float gamma, int min_blocks,
                                int* head_count, const float* logA, int* block_count,
                                int* block_index, hipStream_t st) {
    if (sh.mq <= 64)
        return launch_fused<1>(sh, mass, gamma, min_blocks, head_count, logA, block_count,
                               block_index, st);
    if (sh.mq <= kFusedMaxBlocks)
        return launch_fused<2>(sh, mass, gamma, min_blocks, head_count, logA, block_count,
                               block_index, st);
    hipError_t e = launch_budget(sh, mass, gamma, min_blocks, head_count, st);
    if (e != hipSuccess) return e;
    return launch_select(sh, logA, head_count, 0, 0, block_count, block_index, st);
}

}  // namespace pa
