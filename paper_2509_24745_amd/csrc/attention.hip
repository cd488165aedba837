// Causal block-sparse attention over the selected blocks (Sec. 3.2, last
// paragraph) and its dense baseline (every causal block).
//
// Work item = (query head i, query block m): b query rows, one wave per 32
// rows.  The item walks its list of key blocks in sub-blocks of 64 keys; for
// each sub-block it computes
//   S^T = K Q^T            (32x32x16 bf16 MFMA; K from LDS, Q in registers)
//   online softmax          (lane-local per query + one half-wave exchange)
//   O^T += V^T P^T          (P^T straight from the S^T accumulators)
// Each lane owns one query column of every tile, so the probabilities in
// S^T's accumulators are already laid out as the B operand of the PV
// product: a 32-key tile's 16 accumulator slots of lane half h cover keys
// 8(r/4) + 4h + r%4, and the V^T operand is read in that key order.
//
// A pre-pass re-blocks K and V once per call into
//   kvb[h][n][sub] = { K rows of the sub-block (64 x d, row-major),
//                      V^T of the sub-block (d x 64, keys permuted: bits 2
//                      and 3 of the offset in each 32-key tile swapped) }
// so that every sub-block is one contiguous 16*d*8-byte chunk (spread over
// all HBM channels whatever KV head is being read), the 8 keys a lane needs
// for one PV step are contiguous (one 16-byte LDS read), and rows past N are
// zero.
//
// Pipeline (one barrier per 64-key step j; two workgroups share a CU):
//   - sub-tiles are copied global -> LDS with global_load_lds (no staging
//     registers); K and V^T have separate double buffers, K one step ahead:
//     during step j the copies of K(j+2) and V(j+1) run while the wave reads
//     K(j+1) and V(j);
//   - the scores of step j+1 (MFMA) are interleaved instruction by
//     instruction with the softmax of step j (VALU), then PV of step j runs,
//     as one explicit software pipeline in which every LDS fragment read is
//     issued two MFMAs ahead of its use;
//   - the probability sum of step j and the row maxima of step j+1 are
//     computed inside the PV segments (held there by empty asm operands, so
//     that the optimizer cannot sink them past the masking branch); a masked
//     sub-tile (the diagonal block or a ragged end) takes its maxima again
//     after masking, and the rare rescale branch stays outside the block.
#include <algorithm>
#include <mutex>
#include <vector>

#include "common.h"
#include "internal.h"
#include "work_order.h"

namespace pa {

__device__ __forceinline__ int swap_bits23(int x) {
    return (x & ~12) | ((x & 4) << 1) | ((x & 8) >> 1);
}

// ---------------------------------------------------------------------------
// K, V -> kvb.  grid (Mq, Hkv), 256 threads.  Rows >= N are zero.  Also
// zeroes the attention work-queue counters.
// ---------------------------------------------------------------------------
constexpr int kSubKeys = 64;  // keys per attention sub-block

template <typename T, int D, int B>
__global__ __launch_bounds__(256) void kv_block_kernel(Shape sh, const T* __restrict__ k,
                                                       const T* __restrict__ v,
                                                       T* __restrict__ kvb,
                                                       int* __restrict__ queue) {
    static_assert(kNumXcd * kQueueStride <= 256, "one thread per queue word");
    if (queue && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x < kNumXcd * kQueueStride)
        queue[threadIdx.x] = 0;
    constexpr int V = Vec16<T>::n;
    constexpr int LDR = D + V;
    constexpr int KT = kSubKeys < B ? kSubKeys : B;
    constexpr int SUB = 2 * KT * D;
    __shared__ __attribute__((aligned(16))) T tile[B * LDR];
    const int blk = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
    const T* ksrc = k + (int64_t)h * sh.kv_head;
    const T* vsrc = v + (int64_t)h * sh.kv_head;
    T* dst = kvb + ((int64_t)h * sh.mq + blk) * (2 * B * D);
    for (int vi = tid; vi < B * D / V; vi += 256) {
        const int row = vi / (D / V), col = (vi % (D / V)) * V;
        const int tok = blk * B + row;
        u32x4 xk = zero_u32x4(), xv = zero_u32x4();
        if (tok < sh.n) {
            xk = *reinterpret_cast<const u32x4*>(ksrc + (int64_t)tok * sh.kv_tok + col);
            xv = *reinterpret_cast<const u32x4*>(vsrc + (int64_t)tok * sh.kv_tok + col);
        }
        // K rows go straight to their sub-block
        T* kd = dst + (row / KT) * SUB + (row % KT) * D + col;
        *reinterpret_cast<u32x4*>(kd) = xk;
        *reinterpret_cast<u32x4*>(tile + row * LDR + col) = xv;
    }
    __syncthreads();
    // V^T: row d of sub-block `sub` holds its KT keys in permuted order
    for (int ov = tid; ov < D * B / V; ov += 256) {
        const int sub = ov / (D * KT / V);
        const int rem = ov % (D * KT / V);
        const int d = rem / (KT / V), p0 = (rem % (KT / V)) * V;
        u32x4 x = zero_u32x4();
#pragma unroll
        for (int e = 0; e < V; ++e) {
            const int p = p0 + e;
            const int key = sub * KT + ((p & ~31) | swap_bits23(p & 31));
            put_elem<T>(x, e, tile[key * LDR + d]);
        }
        *reinterpret_cast<u32x4*>(dst + sub * SUB + KT * D + d * KT + p0) = x;
    }
}

// Clears the attention work-queue counters (a fill kernel rather than a
// memset, so that the sequence stays correct when a caller records it in a
// graph).
__global__ __launch_bounds__(256) void queue_reset_kernel(int* __restrict__ queue) {
    if (threadIdx.x < kNumXcd * kQueueStride) queue[threadIdx.x] = 0;
}

hipError_t launch_queue_reset(int* queue, hipStream_t st) {
    hipLaunchKernelGGL(queue_reset_kernel, dim3(1), dim3(256), 0, st, queue);
    return hipGetLastError();
}

// Scratch of the entry point that allocates nothing: the work-queue counters
// live in this file-scope device array, one copy per GPU, for the life of
// the process.  Host code never passes the array's name to a kernel (on the
// host it is only a stand-in for the symbol); it uses the device address
// that hipGetSymbolAddress returns, looked up once per device with that
// device current and kept in scratch_ptr[].
static __device__ __align__(256) int scratch[kScratchBytes / sizeof(int)];
static_assert(kQueueBytes <= kScratchBytes, "the work queues fit the scratch array");

constexpr int kMaxDevices = 64;
static std::mutex scratch_mu;
static int* scratch_ptr[kMaxDevices];

hipError_t scratch_address(int** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(scratch_mu);
    if (!scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        scratch_ptr[dev] = (int*)p;
    }
    *out = scratch_ptr[dev];
    return hipSuccess;
}

// ---------------------------------------------------------------------------
// attention.  Persistent grid (one workgroup per resident slot), 2B threads (B/32
// waves), 2 workgroups per CU.
// ---------------------------------------------------------------------------
template <typename T> __device__ __forceinline__ T cvt_p(float p);
template <> __device__ __forceinline__ bf16 cvt_p<bf16>(float p) { return (bf16)p; }
template <> __device__ __forceinline__ float cvt_p<float>(float p) { return p; }

// Slack (log2 units) by which a row max may exceed the running reference max
// before the accumulators are rescaled.
constexpr float kRescaleSlack = 8.f;

template <typename T, int D, int B>
struct AttnCfg {
    static constexpr int V = Vec16<T>::n;
    static constexpr int NTH = 2 * B;                  // B/32 waves
    static constexpr int KT = kSubKeys < B ? kSubKeys : B;  // keys per sub-block
    static constexpr int NSUB = B / KT;                // sub-blocks per block
    static constexpr int NT = KT / 32;                 // 32-key tiles per sub-block
    static constexpr int SUB = 2 * KT * D;             // elements of a kvb sub-block
    static constexpr int KPAD = D + V;                 // padded K row in LDS (elements)
    static constexpr int VPAD = KT + V;                // padded V^T row in LDS
    static constexpr int K_ELEMS = KT * KPAD;
    static constexpr int V_ELEMS = D * VPAD;
    static constexpr int STAGE = K_ELEMS + V_ELEMS;
    static constexpr int VPT = SUB / V / NTH;          // 16-byte vectors per thread per sub-block
    // Waves per SIMD the LDS of one CU (160 KiB) leaves room for, capped at
    // 2: the kernel's register budget.  d = 128 with b = 64 (two-wave
    // workgroups), and fp32 at d = 128, are held to one wave per SIMD by LDS.
    static constexpr int LDS_BYTES = 2 * STAGE * (int)sizeof(T) + 16;
    static constexpr int WAVES_PER_SIMD_LDS = (160 * 1024 / LDS_BYTES) * (NTH / 64) / 4;
    static constexpr int MIN_WAVES = WAVES_PER_SIMD_LDS < 1 ? 1 : (WAVES_PER_SIMD_LDS > 2 ? 2 : WAVES_PER_SIMD_LDS);
};

// Direct global -> LDS copy of one kvb sub-block (K rows, then V^T rows)
// into the padded LDS layout.  One buffer_load_dwordx4 ... lds moves 64
// consecutive 16-byte LDS slots (slot = lane); the padded layout has one
// spare slot per row, which loads a harmless duplicate of the row's first
// chunk.  The buffer descriptor spans exactly the sub-block (built in SGPRs
// per copy), so each lane needs one 32-bit offset per instruction, computed
// once, and the hardware range check keeps every read inside the sub-block.
// Instructions are dealt to the waves round-robin.
template <typename T, int D, int KT, int NW>
struct SubTileDma {
    static constexpr int V = Vec16<T>::n;
    static constexpr int KSR = D / V + 1;              // slots per padded K row
    static constexpr int VSR = KT / V + 1;             // slots per padded V^T row
    static constexpr int K_INS = KT * KSR / 64;        // wave instructions, K part
    static constexpr int V_INS = D * VSR / 64;         // wave instructions, V^T part
    static constexpr int KJ = (K_INS + NW - 1) / NW;   // per wave (upper bound)
    static constexpr int VJ = (V_INS + NW - 1) / NW;
    static constexpr int SUB_BYTES = 2 * KT * D * (int)sizeof(T);
    static_assert(KT * KSR % 64 == 0 && D * VSR % 64 == 0, "whole wave instructions");

    uint32_t koff[KJ], voff[VJ];   // byte offsets inside a sub-block
    int w;

    __device__ __forceinline__ SubTileDma(int w_, int lane) : w(w_) {
#pragma unroll
        for (int j = 0; j < KJ; ++j) {
            const int slot = (w + j * NW) * 64 + lane;
            const int row = slot / KSR, ch = slot % KSR;
            koff[j] = (uint32_t)((row * D + (ch == KSR - 1 ? 0 : ch * V)) * sizeof(T));
        }
#pragma unroll
        for (int j = 0; j < VJ; ++j) {
            const int slot = (w + j * NW) * 64 + lane;
            const int row = slot / VSR, ch = slot % VSR;
            voff[j] = (uint32_t)((KT * D + row * KT + (ch == VSR - 1 ? 0 : ch * V)) * sizeof(T));
        }
    }
    static __device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const T* sub) {
        // raw buffer, 32-bit dword format (CDNA descriptor word 3)
        return __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(sub), 0, SUB_BYTES, 0x00020000);
    }
    __device__ __forceinline__ void issue_k(const T* sub, T* k_lds) const {
        const __amdgpu_buffer_rsrc_t r = rsrc(sub);
#pragma unroll
        for (int j = 0; j < KJ; ++j) {
            const int ins = w + j * NW;
            if (KJ * NW == K_INS || ins < K_INS)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    r, (__attribute__((address_space(3))) void*)(k_lds + ins * 64 * V), 16, koff[j],
                    0, 0, 0);
        }
    }
    __device__ __forceinline__ void issue_v(const T* sub, T* v_lds) const {
        const __amdgpu_buffer_rsrc_t r = rsrc(sub);
#pragma unroll
        for (int j = 0; j < VJ; ++j) {
            const int ins = w + j * NW;
            if (VJ * NW == V_INS || ins < V_INS)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    r, (__attribute__((address_space(3))) void*)(v_lds + ins * 64 * V), 16, voff[j],
                    0, 0, 0);
        }
    }
};

// The two K and two V^T tiles in LDS.  They are four separate variables so
// that each has an alias scope of its own: the compiler then sees that the
// reads of one slot do not depend on the copy in flight into another, and
// does not make them wait for it.
template <typename T>
struct LdsSlots {
    T* k0;
    T* k1;
    T* v0;
    T* v1;
    __device__ __forceinline__ T* k(int p) const { return p ? k1 : k0; }
    __device__ __forceinline__ T* v(int p) const { return p ? v1 : v0; }
};

// Waits for this wave's global -> LDS copies (they count in vmcnt, like any
// vector-memory load).  A copy's data is in LDS only once its wave has
// waited; the barrier after this wait then hands the tiles to the other
// waves.  (s_waitcnt fields: vmcnt 0, expcnt and lgkmcnt left at their
// maxima.)
__device__ __forceinline__ void wait_copies() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// MFMAs between the LDS read of an operand fragment and the MFMA that uses it
// (bf16 attention loop).  With the probabilities formed in the PV segments,
// 3 is 0.3-0.7 % faster than 2 (8K to 128K, sparse and dense; 2 was the
// better lead while the QK segments carried the softmax).
constexpr int kReadLead = 3;
// Largest sum of one lane's probabilities in a step that certainly leaves the
// lazily rescaled reference in place: every bf16 probability is then at most
// 2^7, so its exponent is below log2(2^7 (1 + 2^-8)) < kRescaleSlack.
constexpr float kLazySum = 128.f;

// Causal / ragged mask of one 64-key sub-tile: keys past `lim` (offset of
// the last visible key inside the sub-tile) become -inf.  A key's offset is
// 32 kt + 8 (r/4) + (r%4) + 4 h; the compile-time part is compared with the
// per-lane limit lim - 4h.
template <int NT>
__device__ __forceinline__ void mask_tail(f32x16* s, int lim, int h) {
    const int lim_h = lim - 4 * h;
#pragma unroll
    for (int kt = 0; kt < NT; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            s[kt][r] = (32 * kt + 8 * (r >> 2) + (r & 3) <= lim_h) ? s[kt][r] : kNegInf;
}

// Max of a lane's raw scores over the sub-tile, then over both wave halves
// (four independent chains instead of one serial one).
template <int NT>
__device__ __forceinline__ float tile_max(const f32x16* s) {
    float c[4] = {kNegInf, kNegInf, kNegInf, kNegInf};
#pragma unroll
    for (int kt = 0; kt < NT; ++kt)
#pragma unroll
        for (int r = 0; r < 16; r += 2) c[(r >> 1) & 3] = fmaxf(c[(r >> 1) & 3], fmaxf(s[kt][r], s[kt][r + 1]));
    return halves_max(fmaxf(fmaxf(c[0], c[1]), fmaxf(c[2], c[3])));
}

// Sum of the probabilities a lane feeds to the PV product.  bf16: two per
// v_dot2_f32_bf16 (the sum then matches the rounded P the MFMA consumes).
template <typename T, int NT>
__device__ __forceinline__ float prob_sum(const typename FragOf<T>::type (*pf)[2]);

template <>
__device__ __forceinline__ float prob_sum<bf16, 2>(const bf16x8 (*pf)[2]) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int e = 0; e < 2; ++e)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const bf16x2 pr = {pf[kt][e][2 * j], pf[kt][e][2 * j + 1]};
                acc[j] = __builtin_amdgcn_fdot2_f32_bf16(pr, one, acc[j], false);
            }
    return (acc[0] + acc[1]) + (acc[2] + acc[3]);
}

template <>
__device__ __forceinline__ float prob_sum<float, 2>(const f32x8 (*pf)[2]) {
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int e = 0; e < 2; ++e)
#pragma unroll
            for (int j = 0; j < 8; ++j) acc[j & 3] += pf[kt][e][j];
    return (acc[0] + acc[1]) + (acc[2] + acc[3]);
}

// One work item: query block m of query head i.  Every wave of the
// workgroup calls it with the same (m, i); it starts and ends with no copy
// in flight, and the caller's barrier separates it from the previous item's
// LDS reads.
template <typename T, int D, int B, bool DENSE>
__device__ __forceinline__ void attn_one(const Shape& sh, const T* __restrict__ q,
                                         const T* __restrict__ kvb,
                                         const int* __restrict__ block_count,
                                         const int* __restrict__ block_index,
                                         T* __restrict__ out, float* __restrict__ lse,
                                         const int m, const int i,
                                         const LdsSlots<T>& slot) {
    typedef AttnCfg<T, D, B> C;
    typedef typename FragOf<T>::type Frag;
    typedef SubTileDma<T, D, C::KT, C::NTH / 64> Dma;
    static_assert(C::KPAD == Dma::KSR * C::V && C::VPAD == Dma::VSR * C::V, "padded pitches");
    constexpr int NT = C::NT;
    constexpr int DT = D / 32;   // output tiles along d
    constexpr int KS = D / 16;   // k steps of Q K^T
    static_assert(NT == 2, "64-key sub-tiles");

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, h = lane >> 5, lc = lane & 31;
    const int kvh = i / sh.rep;
    const int n_tok = sh.n;
    // counts and indices are clamped to the causal range, so malformed caller
    // lists give wrong values but never an out-of-bounds access
    const int cnt = DENSE ? (m + 1) : min(block_count[(int64_t)i * sh.mq + m], m + 1);
    const int* list = DENSE ? nullptr : block_index + ((int64_t)i * sh.mq + m) * sh.mq;
    const int qtok = m * B + 32 * w + lc;
    const bool qvalid = qtok < n_tok;
    const int qlim = min(qtok, n_tok - 1);   // last key this row may see

    if (cnt <= 0) {
        if (qvalid) {
            T* orow = out + (int64_t)qtok * sh.o_tok + (int64_t)i * sh.o_head;
            // lane half h zeroes elements [h D/2, (h+1) D/2); a rolled loop,
            // so that no per-lane address stays live across work items
            u32x4* o4 = reinterpret_cast<u32x4*>(orow + h * (D / 2));
#pragma unroll 1
            for (int e = 0; e < D / 2 / Vec16<T>::n; ++e) o4[e] = zero_u32x4();
            if (lse && h == 0) lse[(int64_t)i * n_tok + qtok] = kNegInf;
        }
        return;
    }

    Frag qf[KS];
    {
        const T* qrow = q + (int64_t)min(qtok, n_tok - 1) * sh.q_tok + (int64_t)i * sh.q_head;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) qf[ks] = load_frag<T>(qrow + 16 * ks + 8 * h);
    }

    const T* kvbase = kvb + (int64_t)kvh * sh.mq * (2 * B * D);
    // step j = sub-block (j % NSUB) of listed block (j / NSUB).  List entries
    // arrive 64 at a time, one per lane, through a vector load, and are picked
    // with v_readlane: no scalar-memory load in the loop, whose out-of-order
    // return would force every LDS wait to drain completely.
    int lst_base = -64, lst = 0;
    auto block_of = [&](int it) -> int {
        if (DENSE) return it;
        const int c0 = it & ~63;
        if (c0 != lst_base) {
            lst_base = c0;
            lst = (c0 + lane < cnt) ? list[c0 + lane] : 0;
        }
        return min(max(__builtin_amdgcn_readlane(lst, it & 63), 0), m);
    };
    auto sub_src = [&](int nb, int sub) { return kvbase + (int64_t)nb * (2 * B * D) + sub * C::SUB; };
    auto needs_mask = [&](int nb) { return nb == m || (nb + 1) * B > n_tok; };
    auto qk = [&](f32x16* acc, const T* kt_) {
#pragma unroll
        for (int kt = 0; kt < NT; ++kt) {
            acc[kt] = zero16();
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                mma(acc[kt], load_frag<T>(kt_ + (32 * kt + lc) * C::KPAD + 16 * ks + 8 * h), qf[ks]);
        }
    };

    float m_run = kNegInf, l_run = 0.f;
    f32x16 o[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[dt] = zero16();

    const int steps = cnt * C::NSUB;
    auto nb_of_step = [&](int j, int nb_prev) {
        return (j % C::NSUB == 0) ? block_of(j / C::NSUB) : nb_prev;
    };
    // prologue: K of steps 0 and 1, V of step 0; scores and max of step 0
    int nb0 = block_of(0);
    int nb1 = steps > 1 ? nb_of_step(1, nb0) : nb0;
    const Dma dma(w, lane);
    dma.issue_k(sub_src(nb0, 0), slot.k(0));
    dma.issue_v(sub_src(nb0, 0), slot.v(0));
    if (steps > 1) dma.issue_k(sub_src(nb1, 1 % C::NSUB), slot.k(1));
    wait_copies();
    __syncthreads();
    f32x16 s_cur[NT];
    qk(s_cur, slot.k(0));
    if (needs_mask(nb0)) mask_tail<NT>(s_cur, qlim - nb0 * B, h);
    float mx = tile_max<NT>(s_cur) * sh.scale2;

    // probabilities of the step the PV MFMAs consume next, from its scores
    Frag pf[NT][2];
    auto form_p = [&](const f32x16* s, float nm) {
#pragma unroll
        for (int kt = 0; kt < NT; ++kt)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                pf[kt][r >> 3][r & 7] = cvt_p<T>(fast_exp2(fmaf(s[kt][r], sh.scale2, nm)));
    };
    // the reference moves only when some row's max exceeds it by more than
    // kRescaleSlack (probabilities stay < 2^8)
    auto rescale_to = [&](float mxs) {
        const float m_new = fmaxf(m_run, mxs);
        const float alpha = (m_run == kNegInf) ? 0.f : fast_exp2(m_run - m_new);
        l_run *= alpha;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[dt] *= alpha;
        m_run = m_new;
    };
    // a row whose keys so far are all masked keeps m_run = -inf: its
    // probabilities are exp2(-inf) = 0
    auto neg_ref = [&]() { return (m_run == kNegInf) ? 0.f : -m_run; };
    if constexpr (sizeof(T) == 2) {
        // bf16: the first step's reference and probabilities here; later
        // steps form theirs in the PV segments of the step before
        if (__builtin_amdgcn_ballot_w64(mx > m_run + kRescaleSlack)) rescale_to(mx);
        form_p(s_cur, neg_ref());
    }

    // One 64-key step.  `sc` holds the scores of step st, `sn` receives those
    // of step st+1 (two distinct register sets, used alternately, so the next
    // scores never wait for the current softmax to free its registers; bf16
    // keeps `sc` only for the step's rescale check).
    auto step = [&](f32x16* sc, f32x16* sn, int st) {
        if constexpr (sizeof(T) == 2) {
            // a masked sub-tile (the diagonal or a ragged end, rare): its
            // probabilities formed again from its masked scores
            if (st > 0 && needs_mask(nb0)) {
                mask_tail<NT>(sc, qlim - nb0 * B - (st % C::NSUB) * C::KT, h);
                form_p(sc, neg_ref());
            }
        }
        // K(st+1) and V(st) have landed; every wave is done with step st-1,
        // whose slots (K(st), V(st-1)) the next copies overwrite
        wait_copies();
        __syncthreads();
        int nb2 = nb1;
        if (st + 2 < steps) {
            nb2 = nb_of_step(st + 2, nb1);
            dma.issue_k(sub_src(nb2, (st + 2) % C::NSUB), slot.k(st & 1));
        }
        if (st + 1 < steps) dma.issue_v(sub_src(nb1, (st + 1) % C::NSUB), slot.v((st + 1) & 1));

        if constexpr (sizeof(T) == 2) {
            // Lazy rescaling checked after the fact.  The step's
            // probabilities were formed against the reference of the step
            // before (a masked sub-tile, rare, forms them again from its
            // masked scores).  A lane whose probabilities sum to at most
            // kLazySum holds none above it, so its row max exceeds the
            // reference by less than kRescaleSlack and the reference stays,
            // as the max itself would decide; otherwise (rare, and always on
            // overflow or while a row has no reference) the row max is taken
            // and, where the reference moves, the probabilities formed
            // again: the same decisions and values as taking the max first.
            float ps = prob_sum<T, NT>(pf);
            if (__builtin_amdgcn_ballot_w64(!(ps <= kLazySum) || m_run == kNegInf)) {
                const float mxs = tile_max<NT>(sc) * sh.scale2;
                if (__builtin_amdgcn_ballot_w64(mxs > m_run + kRescaleSlack)) {
                    rescale_to(mxs);
                    form_p(sc, neg_ref());
                    ps = prob_sum<T, NT>(pf);
                }
            }
            l_run += ps;
        } else {
            if (__builtin_amdgcn_ballot_w64(mx > m_run + kRescaleSlack)) rescale_to(mx);
        }
        const float neg_m = neg_ref();

        // --- scores of step st+1 (MFMA), then PV of step st (MFMA); bf16
        // forms step st+1's probabilities (VALU) beside the PV MFMAs, fp32
        // forms step st's beside the QK MFMAs.  On the last step the scores
        // (and the probabilities formed from them) come from a stale slot
        // and are discarded.
        if constexpr (sizeof(T) == 2) {
            // An explicit software pipeline over the NF = NQ + NP MFMAs of the
            // step: segment j issues MFMA j, the LDS read of the fragment that
            // MFMA j + kReadLead consumes and, in the PV half, a slice of the
            // next step's probabilities; sched_barrier keeps every segment in
            // place, so each fragment
            // arrives kReadLead MFMAs after its read was issued.  (Left to
            // itself the scheduler, short of registers, reads each fragment
            // right before its MFMA, which then waits out a whole LDS round
            // trip.)  QK MFMAs alternate between the two 32-key tiles and PV
            // MFMAs between the DT output tiles, so consecutive MFMAs never
            // feed each other; every accumulator still sums in the same order.
            // The probabilities of step st+1 are VALU work for the PV
            // segments: group g (pf[g / 2][g % 2], 8 keys of one 32-key tile)
            // is formed from the scores of step st+1 in the DT segments after
            // the last PV MFMA that reads group g of step st, the last group
            // after the loop.  The QK segments carry no VALU work.  The row
            // maxima the reference needs are no longer taken every step (the
            // check at the next step's start, above); against taking them in
            // the PV segments and forming the probabilities beside the QK
            // MFMAs, this is -2.8 % at 128K and -2.7 % at 32K (dense -2.6 %),
            // with bitwise the same output.  The check placed before the
            // step's copies are issued instead was slower than the old way.
            constexpr int NQ = NT * KS, NP = NT * 2 * DT, NF = NQ + NP;
            constexpr int EPP = 8 / DT;   // probabilities per PV segment
            static_assert(EPP * DT == 8 && NP == 2 * NT * DT, "probability groups");
            const T* kb = slot.k((st + 1) & 1);
            const T* vb = slot.v(st & 1);
            auto frag = [&](int j) -> Frag {
                if (j < NQ)
                    return load_frag<T>(kb + (32 * (j % NT) + lc) * C::KPAD + 16 * (j / NT) + 8 * h);
                const int p = j - NQ, kt = p / (2 * DT), e = (p / DT) % 2, dt = p % DT;
                return load_frag<T>(vb + (32 * dt + lc) * C::VPAD + 32 * kt + 16 * e + 8 * h);
            };
            Frag f[NF];
#pragma unroll
            for (int kt = 0; kt < NT; ++kt) sn[kt] = zero16();
#pragma unroll
            for (int j = 0; j < kReadLead; ++j) f[j] = frag(j);
            __builtin_amdgcn_sched_barrier(0);
            // While a wave issues its MFMA pipeline it takes precedence over
            // the other workgroup's wave on the same SIMD when that one is at
            // its step boundary (copy wait, barrier, copy issue, rescale
            // check), so the matrix pipe is fed first: -0.5 to -0.7 % of the
            // attention time at 32K and 128K against equal priorities.
            __builtin_amdgcn_s_setprio(3);
#pragma unroll
            for (int j = 0; j < NF; ++j) {
                if (j < NQ) {
                    mma(sn[j % NT], f[j], qf[j / NT]);
                } else {
                    const int p = j - NQ;
                    mma(o[p % DT], f[j], pf[p / (2 * DT)][(p / DT) % 2]);
                }
                if (j + kReadLead < NF) f[j + kReadLead] = frag(j + kReadLead);
                if (j >= NQ + DT) {
                    const int p = j - NQ, g = p / DT - 1;
                    if (g < 2 * NT - 1) {
#pragma unroll
                        for (int u = 0; u < EPP; ++u) {
                            const int r = 8 * (g % 2) + EPP * (p % DT) + u;
                            pf[g / 2][g % 2][r & 7] =
                                cvt_p<T>(fast_exp2(fmaf(sn[g / 2][r], sh.scale2, neg_m)));
                        }
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
            }
            __builtin_amdgcn_s_setprio(0);
            // the last group of step st+1's probabilities (with its scores
            // from a stale slot on the last step: formed and discarded)
#pragma unroll
            for (int r = 8; r < 16; ++r)
                pf[NT - 1][1][r & 7] = cvt_p<T>(fast_exp2(fmaf(sn[NT - 1][r], sh.scale2, neg_m)));
        } else {
            qk(sn, slot.k((st + 1) & 1));
#pragma unroll
            for (int kt = 0; kt < NT; ++kt)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    pf[kt][r >> 3][r & 7] = cvt_p<T>(fast_exp2(fmaf(sc[kt][r], sh.scale2, neg_m)));
            l_run += prob_sum<T, NT>(pf);
            const T* vt_ = slot.v(st & 1);
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
#pragma unroll
                for (int kt = 0; kt < NT; ++kt)
#pragma unroll
                    for (int e = 0; e < 2; ++e)
                        mma(o[dt], load_frag<T>(vt_ + (32 * dt + lc) * C::VPAD + 32 * kt + 16 * e + 8 * h),
                            pf[kt][e]);
        }
        // --- mask and max of step st+1 (fp32; bf16 masks at the start of the
        // next step and checks its probabilities there)
        if constexpr (sizeof(T) != 2) {
            if (st + 1 < steps && needs_mask(nb1))
                mask_tail<NT>(sn, qlim - nb1 * B - ((st + 1) % C::NSUB) * C::KT, h);
            mx = tile_max<NT>(sn) * sh.scale2;
        }
        nb0 = nb1;
        nb1 = nb2;
    };
    f32x16 s_alt[NT];
    for (int st = 0; st < steps; st += 2) {
        step(s_cur, s_alt, st);
        if (st + 1 < steps) step(s_alt, s_cur, st + 1);
    }

    const float l_tot = halves_sum(l_run);
    const float inv = 1.f / l_tot;
    if constexpr (sizeof(T) == 2 && D == 128 && B == 128) {
        // O through LDS: the wave's 32 x D tile is written to the K slots
        // (free once every wave is done with the last step) and read back as
        // 16-byte row chunks, so that each store writes whole 128-byte lines
        constexpr int OP = D + 8;
        static_assert(2 * 32 * OP <= C::K_ELEMS, "two waves' O tiles per K slot");
        __syncthreads();
        T* ot = (w < 2 ? slot.k(0) : slot.k(1)) + (w & 1) * 32 * OP;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int rg = 0; rg < 4; ++rg) {
                const int d0 = 32 * dt + 8 * rg + 4 * h;
                const float v0 = o[dt][4 * rg + 0] * inv, v1 = o[dt][4 * rg + 1] * inv;
                const float v2 = o[dt][4 * rg + 2] * inv, v3 = o[dt][4 * rg + 3] * inv;
                *reinterpret_cast<uint2*>(ot + lc * OP + d0) = make_uint2(pack_bf16x2(v0, v1),
                                                                          pack_bf16x2(v2, v3));
            }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
        for (int it = 0; it < 8; ++it) {
            const int r = 4 * it + (lane >> 4), c = (lane & 15) * 8;
            const u32x4 val = *reinterpret_cast<const u32x4*>(ot + r * OP + c);
            const int tok = m * B + 32 * w + r;
            if (tok < n_tok)
                *reinterpret_cast<u32x4*>(out + (int64_t)tok * sh.o_tok + (int64_t)i * sh.o_head + c) = val;
        }
        if (qvalid && lse && h == 0) lse[(int64_t)i * n_tok + qtok] = (m_run + log2f(l_tot)) * kLn2;
        return;
    }
    if (qvalid) {
        T* orow = out + (int64_t)qtok * sh.o_tok + (int64_t)i * sh.o_head;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
            for (int rg = 0; rg < 4; ++rg) {
                const int d0 = 32 * dt + 8 * rg + 4 * h;
                const float v0 = o[dt][4 * rg + 0] * inv, v1 = o[dt][4 * rg + 1] * inv;
                const float v2 = o[dt][4 * rg + 2] * inv, v3 = o[dt][4 * rg + 3] * inv;
                if constexpr (sizeof(T) == 2) {
                    *reinterpret_cast<uint2*>(orow + d0) = make_uint2(pack_bf16x2(v0, v1),
                                                                      pack_bf16x2(v2, v3));
                } else {
                    *reinterpret_cast<float4*>(orow + d0) = make_float4(v0, v1, v2, v3);
                }
            }
        }
        if (lse && h == 0) lse[(int64_t)i * n_tok + qtok] = (m_run + log2f(l_tot)) * kLn2;
    }
}

// Persistent kernel: one resident workgroup per slot (2B threads, B/32
// waves); workgroup w takes the next item of queue w % 8 until the queue is
// empty, then helps drain the other queues.  Taking work dynamically keeps
// every slot busy whatever the mix of list lengths: the hardware dispatcher
// hands workgroups to the shader engines of an XCD in a fixed rotation, so a
// grid of one workgroup per item lets the engines that receive the long items
// hold back all the others.
template <typename T, int D, int B, bool DENSE>
__global__ __launch_bounds__(2 * B, (AttnCfg<T, D, B>::MIN_WAVES)) void attn_kernel(Shape sh, const T* __restrict__ q,
                                                        const T* __restrict__ kvb,
                                                        const int* __restrict__ block_count,
                                                        const int* __restrict__ block_index,
                                                        T* __restrict__ out,
                                                        float* __restrict__ lse,
                                                        int* __restrict__ queue) {
    typedef AttnCfg<T, D, B> C;
    __shared__ __attribute__((aligned(16))) T ks0[C::K_ELEMS];
    __shared__ __attribute__((aligned(16))) T ks1[C::K_ELEMS];
    __shared__ __attribute__((aligned(16))) T vs0[C::V_ELEMS];
    __shared__ __attribute__((aligned(16))) T vs1[C::V_ELEMS];
    const LdsSlots<T> slot{ks0, ks1, vs0, vs1};
    __shared__ int next_item;
    const int per_queue = attn_items(sh) / kNumXcd;
    // own XCD's queue first; once it is empty, the other queues in turn
    // (their remaining items are their shortest), so no XCD idles while
    // another still has work.  Every probe of an empty queue moves on, so the
    // loop ends after at most kNumXcd of them.
    int x = blockIdx.x % kNumXcd, empty = 0;
    for (;;) {
        // the barrier also keeps the previous item's LDS reads ahead of the
        // next item's copies
        if (threadIdx.x == 0) next_item = atomicAdd(queue + x * kQueueStride, 1);
        __syncthreads();
        const int pos = next_item;
        __syncthreads();
        if (pos >= per_queue) {
            if (++empty == kNumXcd) break;
            x = (x + 1) % kNumXcd;
            continue;
        }
        int m, i;
        if (!attn_item(sh, x + kNumXcd * pos, &m, &i)) continue;
        attn_one<T, D, B, DENSE>(sh, q, kvb, block_count, block_index, out, lse, m, i, slot);
    }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
template <typename T, int D, int B>
static hipError_t kvb_t(const Shape& sh, const void* k, const void* v, void* kvb, int* queue,
                        hipStream_t st) {
    hipLaunchKernelGGL((kv_block_kernel<T, D, B>), dim3(sh.mq, sh.hkv), dim3(256), 0, st, sh,
                       (const T*)k, (const T*)v, (T*)kvb, queue);
    return hipGetLastError();
}

hipError_t launch_kv_block(const Shape& sh, const void* k, const void* v, void* kvb, int* queue,
                           hipStream_t st) {
    if (sh.dtype == 0) {
        if (sh.d == 64) return sh.b == 64 ? kvb_t<bf16, 64, 64>(sh, k, v, kvb, queue, st) : kvb_t<bf16, 64, 128>(sh, k, v, kvb, queue, st);
        return sh.b == 64 ? kvb_t<bf16, 128, 64>(sh, k, v, kvb, queue, st) : kvb_t<bf16, 128, 128>(sh, k, v, kvb, queue, st);
    }
    if (sh.d == 64) return sh.b == 64 ? kvb_t<float, 64, 64>(sh, k, v, kvb, queue, st) : kvb_t<float, 64, 128>(sh, k, v, kvb, queue, st);
    return sh.b == 64 ? kvb_t<float, 128, 64>(sh, k, v, kvb, queue, st) : kvb_t<float, 128, 128>(sh, k, v, kvb, queue, st);
}

// Workgroups of `fn` (with `threads` threads) resident on the current device
// at once, rounded down to a multiple of kNumXcd (at least kNumXcd, so that
// every queue has a workgroup).  Cached per (device, kernel).
static int resident_grid(const void* fn, int threads, int* grid) {
    struct Entry { int dev; const void* fn; int grid; };
    static std::mutex mu;
    static std::vector<Entry> cache;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return (int)e;
    {
        std::lock_guard<std::mutex> lk(mu);
        for (const Entry& c : cache)
            if (c.dev == dev && c.fn == fn) { *grid = c.grid; return 0; }
    }
    int cus = 0, per_cu = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return (int)e;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, threads, 0);
    if (e != hipSuccess) return (int)e;
    const int g = per_cu * cus / kNumXcd * kNumXcd;
    *grid = g < kNumXcd ? kNumXcd : g;
    std::lock_guard<std::mutex> lk(mu);
    cache.push_back({dev, fn, *grid});
    return 0;
}

template <typename T, int D, int B>
static hipError_t attn_t(const Shape& sh, bool dense, const void* q, const void* kvb,
                         const int* bc, const int* bi, void* out, float* lse, int* queue,
                         hipStream_t st) {
    const void* fn = dense ? (const void*)attn_kernel<T, D, B, true>
                           : (const void*)attn_kernel<T, D, B, false>;
    int g = 0;
    const int e = resident_grid(fn, 2 * B, &g);
    if (e) return (hipError_t)e;
    Shape s = sh;
    if (dense) s.attn_order = sh.attn_order_dense;
    const dim3 grid((unsigned)std::min(g, attn_items(s)));
    if (dense)
        hipLaunchKernelGGL((attn_kernel<T, D, B, true>), grid, dim3(2 * B), 0, st, s,
                           (const T*)q, (const T*)kvb, bc, bi, (T*)out, lse, queue);
    else
        hipLaunchKernelGGL((attn_kernel<T, D, B, false>), grid, dim3(2 * B), 0, st, s,
                           (const T*)q, (const T*)kvb, bc, bi, (T*)out, lse, queue);
    return hipGetLastError();
}

hipError_t launch_attention(const Shape& sh, bool dense, const void* q, const void* kvb,
                            const int* bc, const int* bi, void* out, float* lse, int* queue,
                            hipStream_t st) {
    if (sh.dtype == 0) {
        if (sh.d == 64) return sh.b == 64 ? attn_t<bf16, 64, 64>(sh, dense, q, kvb, bc, bi, out, lse, queue, st)
                                          : attn_t<bf16, 64, 128>(sh, dense, q, kvb, bc, bi, out, lse, queue, st);
        return sh.b == 64 ? attn_t<bf16, 128, 64>(sh, dense, q, kvb, bc, bi, out, lse, queue, st)
                          : attn_t<bf16, 128, 128>(sh, dense, q, kvb, bc, bi, out, lse, queue, st);
    }
    if (sh.d == 64) return sh.b == 64 ? attn_t<float, 64, 64>(sh, dense, q, kvb, bc, bi, out, lse, queue, st)
                                      : attn_t<float, 64, 128>(sh, dense, q, kvb, bc, bi, out, lse, queue, st);
    return sh.b == 64 ? attn_t<float, 128, 64>(sh, dense, q, kvb, bc, bi, out, lse, queue, st)
                      : attn_t<float, 128, 128>(sh, dense, q, kvb, bc, bi, out, lse, queue, st);
}

}  // namespace pa
