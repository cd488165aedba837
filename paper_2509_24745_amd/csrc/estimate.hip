// Block scoring (Sec. 3.1, Eq. 1) and the last-block attention mass the
// per-head budget is read from (Alg. 1, first two steps).
//
// All score tiles are computed transposed, S^T = K Q^T, on the 32x32 MFMA
// tile: lane l then owns one query (column l % 32) and 16 keys of it, so row
// statistics (max, sum) are lane-local plus one exchange between the two
// wave halves.  Key tiles of 32 rows are staged through LDS (double
// buffered) and shared by the 4 waves of a workgroup; query fragments stay in
// registers for the whole key loop.
//
// Proxy scores (a2 + a3):
//   est_rowmax: one pass over the strided causal keys per strided query row,
//     giving, for every key block n <= m, the row's largest scaled logit in
//     that block, rbm[m, n][t' - m b'], and the row's (max, sum of exp2)
//     over the keys of each key chunk it covers.
//   est_reduce: combines the chunks' (max, sum) pairs into the row
//     log2-sum-exp L2[t'], then logA[m, n] = ln2 * max_{t' in m}
//     (rbm[m, n][t'] - L2[t']) = log max_{t', u'} softmax(...)  (the
//     max-pool of Eq. 1, log domain).
// A row's key range is cut into chunks of at most kEstMaxTiles 32-key tiles
// (so that no workgroup's chain of tiles sets the kernel's time), and further
// on short sequences so that the launch still fills the chip.
// One MFMA pass instead of two (no recomputation of the tiles to re-derive
// the max-pool after the row normaliser is known); rbm costs
// G * Mq(Mq+1)/2 * b' * 4 bytes of workspace.
//
// Last-block mass (a4): the last min(b, N) query tokens of every head
// against all keys, split into key chunks for parallelism, in one pass.
//   mass_block:  per (head, row, key block) the block's (max, sum of exp2).
//   mass_norm:   each row's normaliser from its blocks.
//   mass_sum:    per key block, the sum over rows of the block's share.
#include "common.h"
#include "internal.h"

namespace pa {

// Stages a tile of 32 consecutive key rows [row0, row0 + 32) x D (row-major,
// `ld` elements between rows, rows >= nrows read as zero) through registers
// into an LDS tile with rows padded by 16 bytes.
template <typename T, int D, int NTH>
struct KeyTile {
    static constexpr int V = Vec16<T>::n;
    static constexpr int LDT = D + V;
    static constexpr int VECS = 32 * D / V;
    static constexpr int PER = (VECS + NTH - 1) / NTH;
    u32x4 reg[PER];

    __device__ __forceinline__ void load(const T* base, int64_t ld, int row0, int nrows, int tid) {
#pragma unroll
        for (int c = 0; c < PER; ++c) {
            const int vi = tid + c * NTH;
            if (PER * NTH == VECS || vi < VECS) {
                const int row = vi / (D / V), col = (vi % (D / V)) * V;
                if (row0 + row < nrows)
                    reg[c] = *reinterpret_cast<const u32x4*>(base + (int64_t)(row0 + row) * ld + col);
                else
                    reg[c] = zero_u32x4();
            }
        }
    }
    __device__ __forceinline__ void store(T* lds, int tid) const {
#pragma unroll
        for (int c = 0; c < PER; ++c) {
            const int vi = tid + c * NTH;
            if (PER * NTH == VECS || vi < VECS) {
                const int row = vi / (D / V), col = (vi % (D / V)) * V;
                *reinterpret_cast<u32x4*>(lds + row * LDT + col) = reg[c];
            }
        }
    }
};

// S^T tile (32 keys x 32 queries) of one wave: keys from an LDS tile,
// queries from register fragments.  Lane (lc, h) receives the 16 keys
// c_row(r, h) of query lc.
template <typename T, int D>
__device__ __forceinline__ f32x16 st_tile(const T* lds_tile, const typename FragOf<T>::type* qf,
                                          int lc, int h) {
    constexpr int LDT = D + Vec16<T>::n;
    f32x16 acc = zero16();
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks)
        mma(acc, load_frag<T>(lds_tile + lc * LDT + 16 * ks + 8 * h), qf[ks]);
    return acc;
}

// ---------------------------------------------------------------------------
// a2: per-(row, key block) max and per-(row, key chunk) (max, sum)
// grid (ceil(N'/128), est_nc, G), 256 threads; workgroup (x, c) takes the
// strided rows R0 = (gridDim.x - 1 - x) * 128 .. +127 (longest rows first),
// wave w rows R0+32w..+31, against key tiles [c est_kc, (c+1) est_kc) of the
// causal range (chunks past it exit at once).  Only the wave's diagonal key
// tile needs the causal mask.
// ---------------------------------------------------------------------------
template <typename T, int D, int BP>
__global__ __launch_bounds__(256, 2) void est_rowmax_kernel(Shape sh, const T* __restrict__ qg,
                                                            const T* __restrict__ kg,
                                                            float* __restrict__ rbm,
                                                            float2* __restrict__ rowpart) {
    typedef typename FragOf<T>::type Frag;
    constexpr int KS = D / 16;
    __shared__ __attribute__((aligned(16))) T tiles[2][32 * KeyTile<T, D, 256>::LDT];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, h = lane >> 5, lc = lane & 31;
    const int c = blockIdx.y, g = blockIdx.z;
    const int np = sh.np;
    const int R0 = (gridDim.x - 1 - blockIdx.x) * 128;
    const int kt_begin = c * sh.est_kc;
    const T* qbase = qg + (int64_t)g * np * D;
    const T* kbase = kg + (int64_t)g * np * D;
    const int row = R0 + 32 * w + lc;
    const bool wave_on = R0 + 32 * w < np;
    const int diag_tile = (R0 + 32 * w) / 32;   // the wave's rows all lie in this key tile
    const int wave_last_tile = wave_on ? diag_tile : -1;
    const int last_row_tile = min(R0 + 127, np - 1) / 32;
    if (kt_begin > last_row_tile) return;   // the whole workgroup: no barrier skipped
    const int last_tile = min(last_row_tile, kt_begin + sh.est_kc - 1);
    const float scale2 = sh.scale2;

    Frag qf[KS];
    {
        const T* qrow = qbase + (int64_t)min(row, np - 1) * D;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) qf[ks] = load_frag<T>(qrow + 16 * ks + 8 * h);
    }
    const int64_t tri_total = (int64_t)sh.mq * (sh.mq + 1) / 2;
    float* rbm_g = rbm + (int64_t)g * tri_total * BP;

    // running max m (scaled, log2 units) and sum l of exp2(c' s - m)
    float m = kNegInf, l = 0.f, bm = kNegInf;
    KeyTile<T, D, 256> kt_ld;
    kt_ld.load(kbase, D, kt_begin * 32, np, tid);
    kt_ld.store(tiles[kt_begin & 1], tid);
    __syncthreads();
    for (int kt = kt_begin; kt <= last_tile; ++kt) {
        if (kt < last_tile) kt_ld.load(kbase, D, (kt + 1) * 32, np, tid);
        if (kt <= wave_last_tile) {
            f32x16 acc = st_tile<T, D>(tiles[kt & 1], qf, lc, h);
            if (kt == diag_tile) {
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    acc[r] = (kt * 32 + c_row(r, h) <= row) ? acc[r] : kNegInf;
            }
            // raw maxima (the scale is positive, so it commutes with max)
            float c4[4];
#pragma unroll
            for (int j = 0; j < 4; ++j)
                c4[j] = fmaxf(fmaxf(acc[4 * j], acc[4 * j + 1]), fmaxf(acc[4 * j + 2], acc[4 * j + 3]));
            const float tm = fmaxf(fmaxf(c4[0], c4[1]), fmaxf(c4[2], c4[3])) * scale2;
            // a lane half can have all of its keys masked so far (mn = -inf):
            // it then adds exp2(-inf) = 0 and keeps l = 0
            const float mn = fmaxf(m, tm);
            const float neg = (mn == kNegInf) ? 0.f : -mn;
            const float alpha = (m == kNegInf) ? 0.f : fast_exp2(m - mn);
            float sp[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int r = 0; r < 16; ++r) sp[r & 3] += fast_exp2(fmaf(acc[r], scale2, neg));
            l = fmaf(l, alpha, (sp[0] + sp[1]) + (sp[2] + sp[3]));
            m = mn;
            if constexpr (BP == 16) {
                // one 32-key tile holds two key blocks: slots r < 8 and r >= 8
                const float s0 = halves_max(fmaxf(c4[0], c4[1]) * scale2);
                const float s1 = halves_max(fmaxf(c4[2], c4[3]) * scale2);
                if (h == 0 && row < np) {
                    const int mr = row / 16, j = row % 16, n0 = 2 * kt;
                    if (n0 <= mr) rbm_g[tri_index(mr, n0) * 16 + j] = s0;
                    if (n0 + 1 <= mr) rbm_g[tri_index(mr, n0 + 1) * 16 + j] = s1;
                }
            } else {
                constexpr int TPB = BP / 32;  // key tiles per block
                const float sm = halves_max(tm);
                bm = (kt % TPB == 0) ? sm : fmaxf(bm, sm);
                if ((kt % TPB == TPB - 1 || kt == wave_last_tile) && h == 0 && row < np) {
                    const int mr = row / BP, j = row % BP, n = kt / TPB;
                    rbm_g[tri_index(mr, n) * BP + j] = bm;
                }
            }
        }
        if (kt < last_tile) kt_ld.store(tiles[(kt + 1) & 1], tid);
        __syncthreads();
    }
    const float mo = swap_halves(m), lo = swap_halves(l);
    const float mm = fmaxf(m, mo);
    if (h == 0 && row < np) {
        // a half with m = -inf has l = 0; a row with no visible key in this
        // chunk writes (-inf, 0)
        const float ll = (m == kNegInf ? 0.f : l * fast_exp2(m - mm)) +
                         (mo == kNegInf ? 0.f : lo * fast_exp2(mo - mm));
        rowpart[((int64_t)g * sh.est_nc + c) * np + row] = make_float2(mm, ll);
    }
}

// ---------------------------------------------------------------------------
// a3: row normalisers and the block max-pool in the log domain.
// grid (Mq, G), 256 threads.
// ---------------------------------------------------------------------------
template <int BP>
__global__ __launch_bounds__(256) void est_reduce_kernel(Shape sh, const float* __restrict__ rbm,
                                                         const float2* __restrict__ rowpart,
                                                         float* __restrict__ logA) {
    __shared__ float L[BP];
    const int m = blockIdx.x, g = blockIdx.y, tid = threadIdx.x;
    const int r0 = m * BP;
    const int nr = min(BP, sh.np - r0);
    // the block's rows lie in one 128-row band of est_rowmax (BP divides
    // 128), which wrote chunks 0 .. nck-1 for them
    const int nck = (min((r0 / 128) * 128 + 127, sh.np - 1) / 32) / sh.est_kc + 1;
    for (int j = tid; j < BP; j += 256) {
        float v = 0.f;
        if (j < nr) {
            const float2* pp = rowpart + (int64_t)g * sh.est_nc * sh.np + r0 + j;
            float mx = kNegInf;
            for (int cc = 0; cc < nck; ++cc) mx = fmaxf(mx, pp[(int64_t)cc * sh.np].x);
            // mx is finite: key 0 (chunk 0) is visible to every row
            float sum = 0.f;
            for (int cc = 0; cc < nck; ++cc) {
                const float2 x = pp[(int64_t)cc * sh.np];
                if (x.x != kNegInf) sum += x.y * fast_exp2(x.x - mx);
            }
            v = mx + log2f(sum);
        }
        L[j] = v;
    }
    __syncthreads();
    const int64_t tri_total = (int64_t)sh.mq * (sh.mq + 1) / 2;
    const float* base = rbm + ((int64_t)g * tri_total + tri_index(m, 0)) * BP;
    float* out = logA + ((int64_t)g * sh.mq + m) * sh.mq;
    for (int n = tid; n < sh.mq; n += 256) {
        float v = kNegInf;
        if (n <= m) {
            const float* p = base + (int64_t)n * BP;
            if (nr == BP) {
#pragma unroll
                for (int j = 0; j < BP; j += 4) {
                    const f32x4 x = *reinterpret_cast<const f32x4*>(p + j);
                    v = fmaxf(v, fmaxf(fmaxf(x[0] - L[j], x[1] - L[j + 1]),
                                       fmaxf(x[2] - L[j + 2], x[3] - L[j + 3])));
                }
            } else {
                for (int j = 0; j < nr; ++j) v = fmaxf(v, p[j] - L[j]);
            }
            v *= kLn2;
        }
        out[n] = v;
    }
}

// ---------------------------------------------------------------------------
// a4: last-block mass, one pass over the keys.
// mass_block: grid (nchunks, Hq), B*2 threads (B/32 waves, 32 last-block rows
//   each).  For every (row, key block) of its key chunk: the block's largest
//   scaled logit m and the sum of exp2(logit - m) over the block's visible
//   keys, written to part[i][row][block] (float2).
// mass_norm, mass_sum: each row's log2-sum-exp over its visible blocks, then
//   mass[i][n] = sum over rows of s * exp2(m - L) in a fixed order.
// ---------------------------------------------------------------------------
template <typename T, int D, int B>
__global__ __launch_bounds__(B * 2, 2) void mass_block_kernel(Shape sh, const T* __restrict__ q,
                                                          const T* __restrict__ k,
                                                          float2* __restrict__ part) {
    typedef typename FragOf<T>::type Frag;
    constexpr int NTH = B * 2;
    __shared__ __attribute__((aligned(16))) T tiles[2][32 * KeyTile<T, D, NTH>::LDT];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, h = lane >> 5, lc = lane & 31;
    const int c = blockIdx.x, i = blockIdx.y, kvh = i / sh.rep;
    const int n = sh.n;
    const int nrows = min(B, n), t0 = n - nrows;
    const int rl = 32 * w + lc, t = t0 + rl;
    const bool wave_on = 32 * w < nrows;
    const int wave_first_t = t0 + 32 * w;
    const int wave_last_t = t0 + min(32 * w + 31, nrows - 1);
    const int key0 = c * sh.mass_chunk, key1 = min(key0 + sh.mass_chunk, n);
    const int kt0 = key0 / 32, kt1 = (key1 - 1) / 32;
    const T* kbase = k + (int64_t)kvh * sh.kv_head;

    Frag qf[D / 16];
    {
        const T* qrow = q + (int64_t)min(t, n - 1) * sh.q_tok + (int64_t)i * sh.q_head;
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks) qf[ks] = load_frag<T>(qrow + 16 * ks + 8 * h);
    }
    // this lane's running (max, sum of exp2) over its keys of the current block
    float bm = kNegInf, bs = 0.f;
    KeyTile<T, D, NTH> ld;
    ld.load(kbase, sh.kv_tok, kt0 * 32, n, tid);
    ld.store(tiles[0], tid);
    __syncthreads();
    for (int kt = kt0; kt <= kt1; ++kt) {
        const int buf = (kt - kt0) & 1;
        if (kt < kt1) ld.load(kbase, sh.kv_tok, (kt + 1) * 32, n, tid);
        if (wave_on && kt * 32 <= wave_last_t) {
            f32x16 acc = st_tile<T, D>(tiles[buf], qf, lc, h);
            // only tiles reaching past the wave's first row need the causal mask
            if (kt * 32 + 31 > wave_first_t) {
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    acc[r] = (kt * 32 + c_row(r, h) <= t) ? acc[r] : kNegInf;
            }
            float c4[4];
#pragma unroll
            for (int j = 0; j < 4; ++j)
                c4[j] = fmaxf(fmaxf(acc[4 * j], acc[4 * j + 1]), fmaxf(acc[4 * j + 2], acc[4 * j + 3]));
            const float tm = fmaxf(fmaxf(c4[0], c4[1]), fmaxf(c4[2], c4[3])) * sh.scale2;
            const float mn = fmaxf(bm, tm);
            if (mn != kNegInf) {
                const float neg = -mn;
                float sp[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int r = 0; r < 16; ++r) sp[r & 3] += fast_exp2(fmaf(acc[r], sh.scale2, neg));
                bs = fmaf(bs, bm == kNegInf ? 0.f : fast_exp2(bm - mn), (sp[0] + sp[1]) + (sp[2] + sp[3]));
                bm = mn;
            }
        }
        if (((kt + 1) * 32) % B == 0 || kt == kt1) {
            // block done: combine the two lane halves (one row) and store
            const float mo = swap_halves(bm), so = swap_halves(bs);
            const float mm = fmaxf(bm, mo);
            const float ss = (bm == kNegInf ? 0.f : bs * fast_exp2(bm - mm)) +
                             (mo == kNegInf ? 0.f : so * fast_exp2(mo - mm));
            if (wave_on && h == 0 && rl < nrows)
                part[((int64_t)i * B + rl) * sh.mq + (kt * 32) / B] = make_float2(mm, ss);
            bm = kNegInf;
            bs = 0.f;
        }
        if (kt < kt1) ld.store(tiles[buf ^ 1], tid);
        __syncthreads();
    }
}

constexpr int kMassReduceThreads = 1024;   // 16 waves

// Row normalisers: grid (Hq, ceil(rows / 16)), one wave per last-block row:
// the row's log2-sum-exp over its visible blocks n <= t / b (block n holds
// key n b <= t, so every one of them was written).
__global__ __launch_bounds__(kMassReduceThreads) void mass_norm_kernel(Shape sh,
                                                                      const float2* __restrict__ part,
                                                                      float* __restrict__ lnorm) {
    constexpr int NW = kMassReduceThreads / 64;
    const int i = blockIdx.x, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int b = sh.b, mq = sh.mq;
    const int nrows = min(b, sh.n), t0 = sh.n - nrows;
    const int r = blockIdx.y * NW + w;
    if (r >= nrows) return;   // whole waves; no barrier follows
    const int nmax = (t0 + r) / b;
    const float2* pr = part + ((int64_t)i * b + r) * mq;
    float m = kNegInf, s = 0.f;
    for (int nb = lane; nb <= nmax; nb += 64) {
        const float2 x = pr[nb];
        if (x.x != kNegInf) {
            const float mn = fmaxf(m, x.x);
            s = (m == kNegInf ? 0.f : s * fast_exp2(m - mn)) + x.y * fast_exp2(x.x - mn);
            m = mn;
        }
    }
    const float M = wave_max(m);   // finite: block 0 is visible to every row
    const float sv = wave_sum(m == kNegInf ? 0.f : s * fast_exp2(m - M));
    if (lane == 0) lnorm[(int64_t)i * b + r] = M + log2f(sv);
}

// Block masses: grid (Hq, ceil(Nk / 64)), 64 blocks per workgroup, one per
// lane; wave w sums rows w, w + 16, ... and wave 0 adds the 16 partial sums in
// order (a fixed-order sum).
__global__ __launch_bounds__(kMassReduceThreads) void mass_sum_kernel(Shape sh,
                                                                     const float2* __restrict__ part,
                                                                     const float* __restrict__ lnorm,
                                                                     float* __restrict__ mass) {
    constexpr int NW = kMassReduceThreads / 64;
    __shared__ float L[128];
    __shared__ float ps[NW][64];
    const int i = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int b = sh.b, mq = sh.mq;
    const int nrows = min(b, sh.n), t0 = sh.n - nrows;
    for (int r = tid; r < nrows; r += kMassReduceThreads) L[r] = lnorm[(int64_t)i * b + r];
    __syncthreads();
    const float2* base = part + (int64_t)i * b * mq;
    const int nb = blockIdx.y * 64 + lane;
    float acc = 0.f;
    if (nb < mq) {
        for (int r = w; r < nrows; r += NW) {
            if (nb * b <= t0 + r) {
                const float2 x = base[(int64_t)r * mq + nb];
                if (x.x != kNegInf) acc += x.y * fast_exp2(x.x - L[r]);
            }
        }
    }
    ps[w][lane] = acc;
    __syncthreads();
    if (w == 0 && nb < mq) {
        float sum = 0.f;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) sum += ps[ww][lane];
        mass[(int64_t)i * mq + nb] = sum;
    }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
template <typename T, int D>
static hipError_t rowmax_t(const Shape& sh, const void* qg, const void* kg, float* rbm,
                           float2* rowpart, hipStream_t st) {
    dim3 grid((sh.np + 127) / 128, sh.est_nc, sh.g);
    switch (sh.bp) {
        case 16: hipLaunchKernelGGL((est_rowmax_kernel<T, D, 16>), grid, dim3(256), 0, st, sh, (const T*)qg, (const T*)kg, rbm, rowpart); break;
        case 32: hipLaunchKernelGGL((est_rowmax_kernel<T, D, 32>), grid, dim3(256), 0, st, sh, (const T*)qg, (const T*)kg, rbm, rowpart); break;
        case 64: hipLaunchKernelGGL((est_rowmax_kernel<T, D, 64>), grid, dim3(256), 0, st, sh, (const T*)qg, (const T*)kg, rbm, rowpart); break;
        case 128: hipLaunchKernelGGL((est_rowmax_kernel<T, D, 128>), grid, dim3(256), 0, st, sh, (const T*)qg, (const T*)kg, rbm, rowpart); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_est_rowmax(const Shape& sh, const void* qg, const void* kg, float* rbm,
                             float2* rowpart, hipStream_t st) {
    if (sh.dtype == 0)
        return sh.d == 64 ? rowmax_t<bf16, 64>(sh, qg, kg, rbm, rowpart, st)
                          : rowmax_t<bf16, 128>(sh, qg, kg, rbm, rowpart, st);
    return sh.d == 64 ? rowmax_t<float, 64>(sh, qg, kg, rbm, rowpart, st)
                      : rowmax_t<float, 128>(sh, qg, kg, rbm, rowpart, st);
}

hipError_t launch_est_reduce(const Shape& sh, const float* rbm, const float2* rowpart,
                             float* logA, hipStream_t st) {
    dim3 grid(sh.mq, sh.g);
    switch (sh.bp) {
        case 16: hipLaunchKernelGGL((est_reduce_kernel<16>), grid, dim3(256), 0, st, sh, rbm, rowpart, logA); break;
        case 32: hipLaunchKernelGGL((est_reduce_kernel<32>), grid, dim3(256), 0, st, sh, rbm, rowpart, logA); break;
        case 64: hipLaunchKernelGGL((est_reduce_kernel<64>), grid, dim3(256), 0, st, sh, rbm, rowpart, logA); break;
        case 128: hipLaunchKernelGGL((est_reduce_kernel<128>), grid, dim3(256), 0, st, sh, rbm, rowpart, logA); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <typename T, int D, int B>
static hipError_t mass_t(const Shape& sh, const void* q, const void* k, float2* part, float* lnorm,
                         float* mass, hipStream_t st) {
    hipLaunchKernelGGL((mass_block_kernel<T, D, B>), dim3(sh.nchunks, sh.hq), dim3(B * 2), 0, st, sh,
                       (const T*)q, (const T*)k, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    constexpr int NW = kMassReduceThreads / 64;
    hipLaunchKernelGGL(mass_norm_kernel, dim3(sh.hq, (min(sh.b, sh.n) + NW - 1) / NW),
                       dim3(kMassReduceThreads), 0, st, sh, (const float2*)part, lnorm);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(mass_sum_kernel, dim3(sh.hq, (sh.mq + 63) / 64), dim3(kMassReduceThreads), 0,
                       st, sh, (const float2*)part, (const float*)lnorm, mass);
    return hipGetLastError();
}

hipError_t launch_mass(const Shape& sh, const void* q, const void* k, float2* part, float* lnorm,
                       float* mass, hipStream_t st) {
    if (sh.dtype == 0) {
        if (sh.d == 64) return sh.b == 64 ? mass_t<bf16, 64, 64>(sh, q, k, part, lnorm, mass, st)
                                          : mass_t<bf16, 64, 128>(sh, q, k, part, lnorm, mass, st);
        return sh.b == 64 ? mass_t<bf16, 128, 64>(sh, q, k, part, lnorm, mass, st)
                          : mass_t<bf16, 128, 128>(sh, q, k, part, lnorm, mass, st);
    }
    if (sh.d == 64) return sh.b == 64 ? mass_t<float, 64, 64>(sh, q, k, part, lnorm, mass, st)
                                      : mass_t<float, 64, 128>(sh, q, k, part, lnorm, mass, st);
    return sh.b == 64 ? mass_t<float, 128, 64>(sh, q, k, part, lnorm, mass, st)
                      : mass_t<float, 128, 128>(sh, q, k, part, lnorm, mass, st);
}

}  // namespace pa
