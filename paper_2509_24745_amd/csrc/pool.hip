// Proxy-head pooling on the strided tokens (Sec. 3.1, Eq. 2 and the strided
// qk-pair dropping that follows it).
//
// Q^g[t'] = fl32(sum_{i in group g, ascending} Q[s t'][i]) * fl32(1/|G|)
// K^g[t'] = fl32(sum_{i in group g, ascending} K[s t'][kv(i)]) * fl32(1/|G|)
// rounded to nearest-even in the problem dtype.  The group's KV keys are
// summed once per query head of the group, so for GQA the pooled key is
// the mean of the KV heads of the group's query heads.
//
// Memory-bound: each thread owns one 16-byte slice of one pooled row.
// Algorithmic bytes per pooled token: |G| (q + k) rows read, 2 rows written.
#include "common.h"
#include "internal.h"

namespace pa {

template <typename T, int D>
__global__ __launch_bounds__(256) void pool_kernel(Shape sh, const T* __restrict__ q,
                                                   const T* __restrict__ k, T* __restrict__ qg,
                                                   T* __restrict__ kg) {
    constexpr int V = Vec16<T>::n;
    constexpr int SLICES = D / V;
    const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t rows = (int64_t)sh.g * sh.np;
    if (gid >= rows * SLICES) return;
    const int slice = (int)(gid % SLICES);
    const int64_t row = gid / SLICES;
    const int g = (int)(row / sh.np);
    const int tp = (int)(row % sh.np);
    const int64_t t = (int64_t)tp * sh.s;
    float aq[V], ak[V];
#pragma unroll
    for (int e = 0; e < V; ++e) { aq[e] = 0.f; ak[e] = 0.f; }
    for (int i = g * sh.gsize; i < (g + 1) * sh.gsize; ++i) {
        const T* qp = q + t * sh.q_tok + (int64_t)i * sh.q_head + slice * V;
        const T* kp = k + t * sh.kv_tok + (int64_t)(i / sh.rep) * sh.kv_head + slice * V;
        const uint4 qv = *reinterpret_cast<const uint4*>(qp);
        const uint4 kv = *reinterpret_cast<const uint4*>(kp);
        const T* qe = reinterpret_cast<const T*>(&qv);
        const T* ke = reinterpret_cast<const T*>(&kv);
#pragma unroll
        for (int e = 0; e < V; ++e) {
            aq[e] = aq[e] + to_f32<T>(qe[e]);
            ak[e] = ak[e] + to_f32<T>(ke[e]);
        }
    }
    uint4 oq, ok;
    T* oqe = reinterpret_cast<T*>(&oq);
    T* oke = reinterpret_cast<T*>(&ok);
#pragma unroll
    for (int e = 0; e < V; ++e) {
        // separate multiply after the sum: no contraction into an fma
        const float mq = __fmul_rn(aq[e], sh.inv_gsize);
        const float mk = __fmul_rn(ak[e], sh.inv_gsize);
        oqe[e] = from_f32_rne<T>(mq);
        oke[e] = from_f32_rne<T>(mk);
    }
    const int64_t o = ((int64_t)g * sh.np + tp) * D + slice * V;
    *reinterpret_cast<uint4*>(qg + o) = oq;
    *reinterpret_cast<uint4*>(kg + o) = ok;
}

template <typename T, int D>
static hipError_t pool_t(const Shape& sh, const void* q, const void* k, void* qg, void* kg,
                         hipStream_t st) {
    constexpr int V = Vec16<T>::n;
    const int64_t threads = (int64_t)sh.g * sh.np * (D / V);
    const int64_t blocks = (threads + 255) / 256;
    hipLaunchKernelGGL((pool_kernel<T, D>), dim3((unsigned)blocks), dim3(256), 0, st, sh,
                       (const T*)q, (const T*)k, (T*)qg, (T*)kg);
    return hipGetLastError();
}

hipError_t launch_pool(const Shape& sh, const void* q, const void* k, void* qg, void* kg,
                       hipStream_t st) {
    if (sh.dtype == 0) {
        return sh.d == 64 ? pool_t<bf16, 64>(sh, q, k, qg, kg, st)
                          : pool_t<bf16, 128>(sh, q, k, qg, kg, st);
    }
    return sh.d == 64 ? pool_t<float, 64>(sh, q, k, qg, kg, st)
                      : pool_t<float, 128>(sh, q, k, qg, kg, st);
}

}  // namespace pa
