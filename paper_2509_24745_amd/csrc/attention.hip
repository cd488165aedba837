// Causal block-sparse attention over the selected blocks (Sec. 3.2, last
// paragraph) and its dense baseline (every causal block).
//
// Work item = (query head i, query block m): b query rows, one wave per 32
// rows.  The item walks its list of key blocks; for each block it computes
//   S^T = K Q^T            (32x32x16 bf16 MFMA; K from LDS, Q in registers)
//   online softmax          (lane-local per query + one half-wave exchange)
//   O^T += V^T P^T          (P^T straight from the S^T accumulators)
// Each lane owns one query column of every tile, so the probabilities of
// S^T's accumulators are already laid out as the B operand of the PV
// product: a 32-key tile's 16 accumulator slots of lane half h cover keys
// 8(r/4) + 4h + r%4, and the V^T operand is read with the same key order.
// That order is baked into a blocked copy of V made once per call:
//   vt[h][n][d][p],  p = key-in-block with bits 2 and 3 of its offset in
//   the 32-key tile swapped,
// so that the 8 keys a lane needs for one PV step are contiguous (one 16-byte
// LDS read), and staging a V^T block is a contiguous 16-byte-per-thread copy.
//
// K and V^T tiles of the next listed block are fetched into registers while
// the current block is computed, then written to the other LDS buffer
// (double buffered; single buffered when two stages do not fit in LDS).
#include "common.h"
#include "internal.h"

namespace pa {

__device__ __forceinline__ int swap_bits23(int x) {
    return (x & ~12) | ((x & 4) << 1) | ((x & 8) >> 1);
}

// ---------------------------------------------------------------------------
// V -> blocked V^T.  grid (Mq, Hkv), 256 threads.  Keys >= N are zero.
// ---------------------------------------------------------------------------
template <typename T, int D, int B>
__global__ __launch_bounds__(256) void vt_kernel(Shape sh, const T* __restrict__ v,
                                                 T* __restrict__ vt) {
    constexpr int V = Vec16<T>::n;
    constexpr int LDR = D + V;
    __shared__ __attribute__((aligned(16))) T tile[B * LDR];
    const int blk = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
    const T* src = v + (int64_t)h * sh.kv_head;
    for (int vi = tid; vi < B * D / V; vi += 256) {
        const int row = vi / (D / V), col = (vi % (D / V)) * V;
        const int tok = blk * B + row;
        uint4 x = make_uint4(0, 0, 0, 0);
        if (tok < sh.n) x = *reinterpret_cast<const uint4*>(src + (int64_t)tok * sh.kv_tok + col);
        *reinterpret_cast<uint4*>(tile + row * LDR + col) = x;
    }
    __syncthreads();
    T* dst = vt + ((int64_t)h * sh.mq + blk) * (D * B);
    for (int ov = tid; ov < D * B / V; ov += 256) {
        const int d = ov / (B / V), p0 = (ov % (B / V)) * V;
        uint4 x;
        T* xe = reinterpret_cast<T*>(&x);
#pragma unroll
        for (int e = 0; e < V; ++e) {
            const int p = p0 + e;
            const int key = (p & ~31) | swap_bits23(p & 31);
            xe[e] = tile[key * LDR + d];
        }
        *reinterpret_cast<uint4*>(dst + (int64_t)d * B + p0) = x;
    }
}

// ---------------------------------------------------------------------------
// attention.  grid Hq*Mq, 2B threads.
// ---------------------------------------------------------------------------
template <typename T> __device__ __forceinline__ T cvt_p(float p);
template <> __device__ __forceinline__ bf16 cvt_p<bf16>(float p) { return (bf16)p; }
template <> __device__ __forceinline__ float cvt_p<float>(float p) { return p; }

template <typename T, int D, int B>
struct AttnCfg {
    static constexpr int V = Vec16<T>::n;
    static constexpr int NTH = 2 * B;          // B/32 waves
    static constexpr int KPAD = D + V;         // padded K row (elements)
    static constexpr int VPAD = B + V;         // padded V^T row
    static constexpr int K_ELEMS = B * KPAD;
    static constexpr int V_ELEMS = D * VPAD;
    static constexpr int STAGE = K_ELEMS + V_ELEMS;
    static constexpr int STAGES = (2 * STAGE * (int)sizeof(T) <= 160 * 1024) ? 2 : 1;
    static constexpr int VPT = (B * D / V) / NTH;  // 16-byte vectors per thread per tile
};

template <typename T, int D, int B, bool DENSE>
__global__ __launch_bounds__(2 * B, 1) void attn_kernel(Shape sh, const T* __restrict__ q,
                                                        const T* __restrict__ k,
                                                        const T* __restrict__ vt,
                                                        const int* __restrict__ block_count,
                                                        const int* __restrict__ block_index,
                                                        T* __restrict__ out,
                                                        float* __restrict__ lse) {
    typedef AttnCfg<T, D, B> C;
    typedef typename FragOf<T>::type Frag;
    constexpr int NT = B / 32;   // key tiles per block
    constexpr int DT = D / 32;   // output tiles along d
    constexpr int KS = D / 16;   // k steps of Q K^T
    constexpr int V = C::V;
    __shared__ __attribute__((aligned(16))) T smem[C::STAGES * C::STAGE];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, h = lane >> 5, lc = lane & 31;
    const int item = blockIdx.x;
    const int m = sh.mq - 1 - item / sh.hq;     // longest rows first
    const int i = item % sh.hq;
    const int kvh = i / sh.rep;
    const int n_tok = sh.n;
    // counts and indices are clamped to the causal range, so malformed caller
    // lists give wrong values but never an out-of-bounds access
    const int cnt = DENSE ? (m + 1) : min(block_count[(int64_t)i * sh.mq + m], m + 1);
    const int* list = DENSE ? nullptr : block_index + ((int64_t)i * sh.mq + m) * sh.mq;
    const int qtok = m * B + 32 * w + lc;
    const bool qvalid = qtok < n_tok;

    if (cnt <= 0) {
        if (qvalid) {
            T* orow = out + (int64_t)qtok * sh.o_tok + (int64_t)i * sh.o_head;
            for (int e = h; e < D; e += 2) orow[e] = from_f32_rne<T>(0.f);
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

    const T* kbase = k + (int64_t)kvh * sh.kv_head;
    const T* vbase = vt + (int64_t)kvh * sh.mq * (D * B);
    u32x4 kreg[C::VPT], vreg[C::VPT];
    auto fetch = [&](int nb) {
        const T* kb = kbase + (int64_t)nb * B * sh.kv_tok;
        const T* vb = vbase + (int64_t)nb * (D * B);
#pragma unroll
        for (int c = 0; c < C::VPT; ++c) {
            const int vi = tid + c * C::NTH;
            const int row = vi / (D / V), col = (vi % (D / V)) * V;
            kreg[c] = (nb * B + row < n_tok)
                          ? *reinterpret_cast<const u32x4*>(kb + (int64_t)row * sh.kv_tok + col)
                          : zero_u32x4();
            vreg[c] = *reinterpret_cast<const u32x4*>(vb + (int64_t)vi * V);
        }
    };
    auto stash = [&](int buf) {
        T* ks_ = smem + buf * C::STAGE;
        T* vs_ = ks_ + C::K_ELEMS;
#pragma unroll
        for (int c = 0; c < C::VPT; ++c) {
            const int vi = tid + c * C::NTH;
            const int row = vi / (D / V), col = (vi % (D / V)) * V;
            *reinterpret_cast<u32x4*>(ks_ + row * C::KPAD + col) = kreg[c];
            const int vrow = vi / (B / V), vcol = (vi % (B / V)) * V;
            *reinterpret_cast<u32x4*>(vs_ + vrow * C::VPAD + vcol) = vreg[c];
        }
    };

    float m_run = kNegInf, l_run = 0.f;
    f32x16 o[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[dt] = zero16();

    int n_cur = DENSE ? 0 : min(max(list[0], 0), m);
    fetch(n_cur);
    stash(0);
    __syncthreads();
    for (int it = 0; it < cnt; ++it) {
        const int buf = (C::STAGES == 2) ? (it & 1) : 0;
        int n_next = -1;
        if (it + 1 < cnt) {
            n_next = DENSE ? it + 1 : min(max(list[it + 1], 0), m);
            fetch(n_next);
        }
        const T* ks_ = smem + buf * C::STAGE;
        const T* vs_ = ks_ + C::K_ELEMS;

        f32x16 s[NT];
#pragma unroll
        for (int kt = 0; kt < NT; ++kt) {
            s[kt] = zero16();
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                mma(s[kt], load_frag<T>(ks_ + (32 * kt + lc) * C::KPAD + 16 * ks + 8 * h), qf[ks]);
        }
        const bool need_mask = (n_cur == m) || ((n_cur + 1) * B > n_tok);
        float mx = kNegInf;
#pragma unroll
        for (int kt = 0; kt < NT; ++kt) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                float x = s[kt][r] * sh.scale2;
                if (need_mask) {
                    const int key = n_cur * B + 32 * kt + c_row(r, h);
                    if (key > qtok || key >= n_tok) x = kNegInf;
                }
                s[kt][r] = x;
                mx = fmaxf(mx, x);
            }
        }
        mx = fmaxf(mx, swap_halves(mx));
        const float m_new = fmaxf(m_run, mx);
        const float m_use = (m_new == kNegInf) ? 0.f : m_new;
        const float alpha = exp2f(m_run - m_use);
        float psum = 0.f;
        Frag pf[NT][2];
#pragma unroll
        for (int kt = 0; kt < NT; ++kt) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const float p = exp2f(s[kt][r] - m_use);
                psum += p;
                pf[kt][r >> 3][r & 7] = cvt_p<T>(p);
            }
        }
        l_run = l_run * alpha + psum;
        m_run = m_new;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[dt] *= alpha;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
            for (int kt = 0; kt < NT; ++kt) {
#pragma unroll
                for (int e = 0; e < 2; ++e)
                    mma(o[dt], load_frag<T>(vs_ + (32 * dt + lc) * C::VPAD + 32 * kt + 16 * e + 8 * h),
                        pf[kt][e]);
            }
        }
        if (it + 1 < cnt) {
            if (C::STAGES == 1) __syncthreads();
            stash(C::STAGES == 2 ? (buf ^ 1) : 0);
        }
        __syncthreads();
        n_cur = n_next;
    }

    const float l_tot = l_run + swap_halves(l_run);
    const float inv = 1.f / l_tot;
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

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
template <typename T, int D, int B>
static hipError_t vt_t(const Shape& sh, const void* v, void* vt, hipStream_t st) {
    hipLaunchKernelGGL((vt_kernel<T, D, B>), dim3(sh.mq, sh.hkv), dim3(256), 0, st, sh,
                       (const T*)v, (T*)vt);
    return hipGetLastError();
}

hipError_t launch_vt(const Shape& sh, const void* v, void* vt, hipStream_t st) {
    if (sh.dtype == 0) {
        if (sh.d == 64) return sh.b == 64 ? vt_t<bf16, 64, 64>(sh, v, vt, st) : vt_t<bf16, 64, 128>(sh, v, vt, st);
        return sh.b == 64 ? vt_t<bf16, 128, 64>(sh, v, vt, st) : vt_t<bf16, 128, 128>(sh, v, vt, st);
    }
    if (sh.d == 64) return sh.b == 64 ? vt_t<float, 64, 64>(sh, v, vt, st) : vt_t<float, 64, 128>(sh, v, vt, st);
    return sh.b == 64 ? vt_t<float, 128, 64>(sh, v, vt, st) : vt_t<float, 128, 128>(sh, v, vt, st);
}

template <typename T, int D, int B>
static hipError_t attn_t(const Shape& sh, bool dense, const void* q, const void* k, const void* vt,
                         const int* bc, const int* bi, void* out, float* lse, hipStream_t st) {
    const dim3 grid((unsigned)(sh.hq * sh.mq));
    if (dense)
        hipLaunchKernelGGL((attn_kernel<T, D, B, true>), grid, dim3(2 * B), 0, st, sh, (const T*)q,
                           (const T*)k, (const T*)vt, bc, bi, (T*)out, lse);
    else
        hipLaunchKernelGGL((attn_kernel<T, D, B, false>), grid, dim3(2 * B), 0, st, sh, (const T*)q,
                           (const T*)k, (const T*)vt, bc, bi, (T*)out, lse);
    return hipGetLastError();
}

hipError_t launch_attention(const Shape& sh, bool dense, const void* q, const void* k,
                            const void* vt, const int* bc, const int* bi, void* out, float* lse,
                            hipStream_t st) {
    if (sh.dtype == 0) {
        if (sh.d == 64) return sh.b == 64 ? attn_t<bf16, 64, 64>(sh, dense, q, k, vt, bc, bi, out, lse, st)
                                          : attn_t<bf16, 64, 128>(sh, dense, q, k, vt, bc, bi, out, lse, st);
        return sh.b == 64 ? attn_t<bf16, 128, 64>(sh, dense, q, k, vt, bc, bi, out, lse, st)
                          : attn_t<bf16, 128, 128>(sh, dense, q, k, vt, bc, bi, out, lse, st);
    }
    if (sh.d == 64) return sh.b == 64 ? attn_t<float, 64, 64>(sh, dense, q, k, vt, bc, bi, out, lse, st)
                                      : attn_t<float, 64, 128>(sh, dense, q, k, vt, bc, bi, out, lse, st);
    return sh.b == 64 ? attn_t<float, 128, 64>(sh, dense, q, k, vt, bc, bi, out, lse, st)
                      : attn_t<float, 128, 128>(sh, dense, q, k, vt, bc, bi, out, lse, st);
}

}  // namespace pa
