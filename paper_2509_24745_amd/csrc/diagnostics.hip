// Head-similarity diagnostic: the overlap scores of Eq. 4 (the sink-token
// analysis) for one query token t, on the heads' own full-resolution
// attention.
//
//   ovl_logits:  z[h][u] = c log2(e) <q_t,h , k_u,kv(h)> for u <= t
//   ovl_select:  one workgroup per head: the softmax of z (fixed-order
//                reductions), sink tokens zeroed and the rest renormalised on
//                request, then the k-th smallest 64-bit key
//                (~order(p) << 32 | u: score descending, token ascending) by
//                an 8-pass radix select, so the head's top-k set is exactly
//                {u : key(u) <= kth}, ties going to the lower token
//   ovl_score:   Score[i][j] = sum of p_j over head i's top-k set (fixed-order
//                reduction), one workgroup per (i, j)
//
// Bandwidth-bound and small (Hq x (t+1) values); not on the prefill path.
#include "common.h"
#include "internal.h"

namespace pa {

constexpr int kOvlThreads = 1024;

// Fixed-order block reduction of one float per thread (sum or max).
template <bool MAX>
__device__ float block_reduce(float x, float* red) {
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, nw = blockDim.x >> 6;
    x = MAX ? wave_max(x) : wave_sum(x);
    __syncthreads();
    if (lane == 0) red[w] = x;
    __syncthreads();
    float r = MAX ? kNegInf : 0.f;
    for (int j = 0; j < nw; ++j) r = MAX ? fmaxf(r, red[j]) : r + red[j];
    return r;
}

template <typename T>
__global__ __launch_bounds__(256) void ovl_logits_kernel(Shape sh, const T* __restrict__ q,
                                                         const T* __restrict__ k, int t,
                                                         float* __restrict__ z) {
    __shared__ float qs[128];
    const int h = blockIdx.y, tid = threadIdx.x, kvh = h / sh.rep;
    const T* qrow = q + (int64_t)t * sh.q_tok + (int64_t)h * sh.q_head;
    for (int e = tid; e < sh.d; e += 256) qs[e] = to_f32(qrow[e]);
    __syncthreads();
    const int u = blockIdx.x * 256 + tid;
    if (u > t) return;
    const T* krow = k + (int64_t)u * sh.kv_tok + (int64_t)kvh * sh.kv_head;
    constexpr int V = Vec16<T>::n;
    float acc = 0.f;
    for (int e = 0; e < sh.d; e += V) {
        const u32x4 x = *reinterpret_cast<const u32x4*>(krow + e);
#pragma unroll
        for (int j = 0; j < V; ++j) acc = fmaf(qs[e + j], get_elem<T>(x, j), acc);
    }
    z[(int64_t)h * sh.n + u] = acc * sh.scale2;
}

__global__ __launch_bounds__(kOvlThreads) void ovl_select_kernel(Shape sh, int t, int topk,
                                                                 int sink, int renorm,
                                                                 float* __restrict__ z,
                                                                 uint64_t* __restrict__ kth) {
    __shared__ float red[kOvlThreads / 64];
    __shared__ int hist[256];
    __shared__ int digit_sh, remaining_sh;
    const int h = blockIdx.x, tid = threadIdx.x;
    const int n1 = t + 1;
    float* p = z + (int64_t)h * sh.n;

    float mx = kNegInf;
    for (int u = tid; u < n1; u += kOvlThreads) mx = fmaxf(mx, p[u]);
    mx = block_reduce<true>(mx, red);
    float s = 0.f;
    for (int u = tid; u < n1; u += kOvlThreads) s += fast_exp2(p[u] - mx);
    s = block_reduce<false>(s, red);
    const float inv = 1.f / s;
    float s2 = 0.f;
    for (int u = tid; u < n1; u += kOvlThreads) {
        const float v = (u < sink) ? 0.f : fast_exp2(p[u] - mx) * inv;
        p[u] = v;
        s2 += v;
    }
    if (renorm) {
        s2 = block_reduce<false>(s2, red);
        const float inv2 = s2 > 0.f ? 1.f / s2 : 0.f;
        for (int u = tid; u < n1; u += kOvlThreads) p[u] *= inv2;
    }
    __syncthreads();

    // radix select of the kk-th smallest key, 8 bits per pass from the top
    const int kk = min(topk, n1);
    uint64_t prefix = 0;
    if (tid == 0) remaining_sh = kk;
    for (int pass = 7; pass >= 0; --pass) {
        const int shift = 8 * pass;
        for (int b = tid; b < 256; b += kOvlThreads) hist[b] = 0;
        __syncthreads();
        for (int u = tid; u < n1; u += kOvlThreads) {
            const uint64_t key = ((uint64_t)(~float_order_key(p[u])) << 32) | (uint32_t)u;
            if (pass == 7 || (key >> (shift + 8)) == (prefix >> (shift + 8)))
                atomicAdd(&hist[(key >> shift) & 255], 1);
        }
        __syncthreads();
        if (tid == 0) {
            int cum = 0, b = 0;
            const int rem = remaining_sh;
            for (; b < 255; ++b) {
                if (cum + hist[b] >= rem) break;
                cum += hist[b];
            }
            digit_sh = b;
            remaining_sh = rem - cum;
        }
        __syncthreads();
        prefix |= (uint64_t)digit_sh << shift;
    }
    if (tid == 0) kth[h] = prefix;
}

__global__ __launch_bounds__(256) void ovl_score_kernel(Shape sh, int t,
                                                        const float* __restrict__ z,
                                                        const uint64_t* __restrict__ kth,
                                                        float* __restrict__ score) {
    __shared__ float red[4];
    const int i = blockIdx.x, j = blockIdx.y, tid = threadIdx.x;
    const float* pi = z + (int64_t)i * sh.n;
    const float* pj = z + (int64_t)j * sh.n;
    const uint64_t lim = kth[i];
    float s = 0.f;
    for (int u = tid; u <= t; u += 256) {
        const uint64_t key = ((uint64_t)(~float_order_key(pi[u])) << 32) | (uint32_t)u;
        if (key <= lim) s += pj[u];
    }
    s = block_reduce<false>(s, red);
    if (tid == 0) score[(int64_t)i * sh.hq + j] = s;
}

hipError_t launch_head_overlap(const Shape& sh, const void* q, const void* k, int t, int topk,
                               int sink, int renorm, float* z, uint64_t* kth, float* score,
                               hipStream_t st) {
    const dim3 g1((t + 1 + 255) / 256, sh.hq);
    if (sh.dtype == 0)
        hipLaunchKernelGGL(ovl_logits_kernel<bf16>, g1, dim3(256), 0, st, sh, (const bf16*)q,
                           (const bf16*)k, t, z);
    else
        hipLaunchKernelGGL(ovl_logits_kernel<float>, g1, dim3(256), 0, st, sh, (const float*)q,
                           (const float*)k, t, z);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(ovl_select_kernel, dim3(sh.hq), dim3(kOvlThreads), 0, st, sh, t, topk, sink,
                       renorm, z, kth);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(ovl_score_kernel, dim3(sh.hq, sh.hq), dim3(256), 0, st, sh, t,
                       (const float*)z, (const uint64_t*)kth, score);
    return hipGetLastError();
}

}  // namespace pa
