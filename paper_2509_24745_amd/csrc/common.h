// Device-side building blocks shared by the ProxyAttn kernels (gfx950).
//
// Matrix products use the 32x32 MFMA tile.  For a product D = A * B with
// A: 32 x 16 and B: 16 x 32, lane l (64 lanes) supplies
//     A[m = l % 32][k-slot (l / 32, j)]   and   B[k-slot (l / 32, j)][n = l % 32]
// for j = 0..7, and receives D[m][n = l % 32] for the 16 rows
//     m = 8 * (r / 4) + 4 * (l / 32) + (r % 4),  r = 0..15.
// Which hardware k index a (half, j) slot maps to does not matter as long as
// both operands use the same slot for the same k; every kernel here fills A
// and B through that one slot convention.
//
// bf16 operands: one v_mfma_f32_32x32x16_bf16 per 16-wide k step.
// fp32 operands: the same 8-slot fragments are consumed by eight
// v_mfma_f32_32x32x2_f32 (slot j of both halves per instruction), so the
// data layout of every kernel is identical for the two element types.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pa {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
// 16 bytes as a native vector: register staging of tiles (HIP's uint4 class
// defeats scalar replacement and ends up on the stack)
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Element e of a 16-byte vector holding 16/sizeof(T) values of T.
template <typename T> __device__ __forceinline__ void put_elem(u32x4& x, int e, T v);
template <> __device__ __forceinline__ void put_elem<float>(u32x4& x, int e, float v) {
    x[e] = __float_as_uint(v);
}
template <> __device__ __forceinline__ void put_elem<__bf16>(u32x4& x, int e, __bf16 v) {
    const uint32_t b = __builtin_bit_cast(uint16_t, v);
    x[e >> 1] |= (e & 1) ? (b << 16) : b;
}

// Element e of such a vector as a float.
template <typename T> __device__ __forceinline__ float get_elem(const u32x4& x, int e);
template <> __device__ __forceinline__ float get_elem<float>(const u32x4& x, int e) {
    return __uint_as_float(x[e]);
}
template <> __device__ __forceinline__ float get_elem<__bf16>(const u32x4& x, int e) {
    const uint32_t w = x[e >> 1];
    return __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
}

__device__ __forceinline__ u32x4 zero_u32x4() {
    u32x4 z = {0u, 0u, 0u, 0u};
    return z;
}

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kNegInf = -__builtin_huge_valf();

template <typename T> struct FragOf;
template <> struct FragOf<bf16> { typedef bf16x8 type; };
template <> struct FragOf<float> { typedef f32x8 type; };

// Elements of T per 16-byte vector load.
template <typename T> struct Vec16 { static constexpr int n = 16 / sizeof(T); };

__device__ __forceinline__ void mma(f32x16& acc, const bf16x8& a, const bf16x8& b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
}

__device__ __forceinline__ void mma(f32x16& acc, const f32x8& a, const f32x8& b) {
#pragma unroll
    for (int j = 0; j < 8; ++j) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[j], b[j], acc, 0, 0, 0);
}

template <typename T>
__device__ __forceinline__ typename FragOf<T>::type load_frag(const T* p) {
    return *reinterpret_cast<const typename FragOf<T>::type*>(p);
}

__device__ __forceinline__ f32x16 zero16() {
    f32x16 z;
#pragma unroll
    for (int i = 0; i < 16; ++i) z[i] = 0.f;
    return z;
}

// Row (within a 32-row C tile) held in accumulator slot r by lane half h.
__device__ __forceinline__ int c_row(int r, int h) { return 8 * (r >> 2) + 4 * h + (r & 3); }

// Round-to-nearest-even fp32 -> bf16 (finite inputs).
__device__ __forceinline__ bf16 f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    uint16_t h = (uint16_t)(u >> 16);
    return __builtin_bit_cast(bf16, h);
}

// Two fp32 values rounded to bf16 (nearest-even) packed low-first in 32 bits.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return (uint32_t)__builtin_bit_cast(uint16_t, f32_to_bf16_rne(lo)) |
           ((uint32_t)__builtin_bit_cast(uint16_t, f32_to_bf16_rne(hi)) << 16);
}

__device__ __forceinline__ float bf16_to_f32(bf16 x) {
    uint16_t h = __builtin_bit_cast(uint16_t, x);
    return __uint_as_float(((uint32_t)h) << 16);
}

template <typename T> __device__ __forceinline__ float to_f32(T x);
template <> __device__ __forceinline__ float to_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ float to_f32<bf16>(bf16 x) { return bf16_to_f32(x); }

template <typename T> __device__ __forceinline__ T from_f32_rne(float x);
template <> __device__ __forceinline__ float from_f32_rne<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32_rne<bf16>(float x) { return f32_to_bf16_rne(x); }

// 2^x on the hardware transcendental unit (v_exp_f32, ~1 ulp; no denormal
// range fix-up, which the softmax does not need).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Exchanges between the two wave halves without LDS: v_permlane32_swap of x
// with itself gives, in every lane l, r[0] = x[l % 32] and r[1] = x[l % 32 + 32].
__device__ __forceinline__ float swap_halves(float x) {   // x of lane l ^ 32
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
    return __uint_as_float((__lane_id() & 32) ? r[0] : r[1]);
}
__device__ __forceinline__ float halves_max(float x) {    // max of lanes l and l ^ 32
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float halves_sum(float x) {    // x[l % 32] + x[l % 32 + 32]
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
    return x;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
    return x;
}

// Monotone map of a float to uint32 (larger float -> larger key).
__device__ __forceinline__ uint32_t float_order_key(float f) {
    uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Index of the lower-triangular pair (m, n), n <= m.
__device__ __forceinline__ int64_t tri_index(int m, int n) {
    return (int64_t)m * (m + 1) / 2 + n;
}

}  // namespace pa
