// Block scoring (Sec. 3.1, Eq. 1-2) and the last-block attention mass the
// per-head budget is read from (Alg. 1, first two steps).
//
// Proxy-head pooling (Sec. 3.1, Eq. 2 and the strided qk-pair dropping that
// follows it):
//   Q^g[t'] = fl32(sum_{i in group g, ascending} Q[s t'][i]) * fl32(1/|G|)
//   K^g[t'] = fl32(sum_{i in group g, ascending} K[s t'][kv(i)]) * fl32(1/|G|)
// rounded to nearest-even in the problem dtype.  The group's KV keys are
// summed once per query head of the group, so for GQA the pooled key is the
// mean of the KV heads of the group's query heads.  Memory-bound: each thread
// owns one 16-byte slice of one pooled row.
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
//
// Launches.  The two chains (pool -> est_rowmax -> est_reduce and
// mass_block -> mass_norm -> mass_sum) do not depend on each other, so each
// launch runs one stage of both, the workgroups of the two roles side by side
// in one grid (horizontal fusion: three launches instead of six, which on
// short sequences is most of the estimation time; the arithmetic of every
// output is that of the stage alone):
//   est_stage1:  pool      + mass_block
//   est_stage2:  est_rowmax + mass_norm
//   est_stage3:  est_reduce + mass_sum
// On long sequences stages 2 and 3 repeat per group of row bands, so that
// the per-(row, block) maxima they pass on need a bounded region (the mass
// stages run with the first group).
#include <algorithm>

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
// a1: pooling.  One 256-thread workgroup per 256 (pooled row, 16-byte slice)
// pairs; `blk` is the workgroup's index among the pooling workgroups.
// ---------------------------------------------------------------------------
template <typename T, int D>
__device__ __forceinline__ void pool_body(const Shape& sh, const T* __restrict__ q,
                                          const T* __restrict__ k, T* __restrict__ qg,
                                          T* __restrict__ kg, int64_t blk) {
    constexpr int V = Vec16<T>::n;
    constexpr int SLICES = D / V;
    const int64_t gid = blk * 256 + threadIdx.x;
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
    // the heads' slices are loaded kPoolBatch at a time (all in flight
    // together; a batch past the group's last head re-reads that head and
    // discards it), then added in ascending head order
    constexpr int kPoolBatch = 4;
    const int i0 = g * sh.gsize, i1 = i0 + sh.gsize;
    for (int ib = i0; ib < i1; ib += kPoolBatch) {
        uint4 qv[kPoolBatch], kv[kPoolBatch];
#pragma unroll
        for (int u = 0; u < kPoolBatch; ++u) {
            const int i = min(ib + u, i1 - 1);
            qv[u] = *reinterpret_cast<const uint4*>(q + t * sh.q_tok + (int64_t)i * sh.q_head +
                                                    slice * V);
            kv[u] = *reinterpret_cast<const uint4*>(k + t * sh.kv_tok +
                                                    (int64_t)(i / sh.rep) * sh.kv_head + slice * V);
        }
#pragma unroll
        for (int u = 0; u < kPoolBatch; ++u) {
            if (ib + u < i1) {
                const T* qe = reinterpret_cast<const T*>(&qv[u]);
                const T* ke = reinterpret_cast<const T*>(&kv[u]);
#pragma unroll
                for (int e = 0; e < V; ++e) {
                    aq[e] = aq[e] + to_f32<T>(qe[e]);
                    ak[e] = ak[e] + to_f32<T>(ke[e]);
                }
            }
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

// ---------------------------------------------------------------------------
// a2: per-(row, key block) max and per-(row, key chunk) (max, sum)
// One 256-thread workgroup per (128-row band, key chunk c, group g): it
// takes the strided rows R0 .. R0+127, wave w rows R0+32w..+31, against key
// tiles [c est_kc, (c+1) est_kc) of the causal range (chunks past it exit at
// once).  Only the wave's diagonal key tile needs the causal mask.  The
// per-(row, key block) maxima go to the current band group's rbm region:
// lower-triangular pairs (m, n) at tri_index(m, n) - tri_base, tri_count
// pairs per proxy group.
// ---------------------------------------------------------------------------
template <typename T, int D, int BP>
__device__ __forceinline__ void est_rowmax_body(const Shape& sh, const T* __restrict__ qg,
                                                const T* __restrict__ kg,
                                                float* __restrict__ rbm,
                                                float2* __restrict__ rowpart, int R0, int c, int g,
                                                int64_t tri_base, int64_t tri_count) {
    typedef typename FragOf<T>::type Frag;
    constexpr int KS = D / 16;
    __shared__ __attribute__((aligned(16))) T tiles[2][32 * KeyTile<T, D, 256>::LDT];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, h = lane >> 5, lc = lane & 31;
    const int np = sh.np;
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
    float* rbm_g = rbm + ((int64_t)g * tri_count - tri_base) * BP;

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
// One 256-thread workgroup per (block row m, group g).
// ---------------------------------------------------------------------------
template <int BP>
__device__ __forceinline__ void est_reduce_body(const Shape& sh, const float* __restrict__ rbm,
                                                const float2* __restrict__ rowpart,
                                                float* __restrict__ logA, int m, int g,
                                                int64_t tri_base, int64_t tri_count) {
    __shared__ float L[BP];
    const int tid = threadIdx.x;
    const int r0 = m * BP;
    const int nr = min(BP, sh.np - r0);
    // the block's rows lie in one 128-row band of est_rowmax (BP divides
    // 128), which wrote chunks 0 .. nck-1 for them
    const int nck = (min((r0 / 128) * 128 + 127, sh.np - 1) / 32) / sh.est_kc + 1;
    // the chunk pairs are read kChunkBatch at a time, all in flight together
    // (a batch past the last chunk re-reads it: the max is unchanged and the
    // sum skips it); the sum runs over the chunks in increasing order
    constexpr int kChunkBatch = 8;
    for (int j = tid; j < BP; j += 256) {
        float v = 0.f;
        if (j < nr) {
            const float2* pp = rowpart + (int64_t)g * sh.est_nc * sh.np + r0 + j;
            float mx = kNegInf;
            for (int c0 = 0; c0 < nck; c0 += kChunkBatch) {
                float xs[kChunkBatch];
#pragma unroll
                for (int u = 0; u < kChunkBatch; ++u)
                    xs[u] = pp[(int64_t)min(c0 + u, nck - 1) * sh.np].x;
#pragma unroll
                for (int u = 0; u < kChunkBatch; ++u) mx = fmaxf(mx, xs[u]);
            }
            // mx is finite: key 0 (chunk 0) is visible to every row
            float sum = 0.f;
            for (int c0 = 0; c0 < nck; c0 += kChunkBatch) {
                float2 xs[kChunkBatch];
#pragma unroll
                for (int u = 0; u < kChunkBatch; ++u)
                    xs[u] = pp[(int64_t)min(c0 + u, nck - 1) * sh.np];
#pragma unroll
                for (int u = 0; u < kChunkBatch; ++u) {
                    // a select, not a branch, so that both halves of the
                    // pair are loaded with the one 8-byte load
                    const bool use = c0 + u < nck && xs[u].x != kNegInf;
                    sum = use ? fmaf(xs[u].y, fast_exp2(xs[u].x - mx), sum) : sum;
                }
            }
            v = mx + log2f(sum);
        }
        L[j] = v;
    }
    __syncthreads();
    const float* base = rbm + ((int64_t)g * tri_count + tri_index(m, 0) - tri_base) * BP;
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
// mass_block: one 256-thread workgroup per (key chunk c, head i); wave w
//   takes last-block rows 32w..32w+31 (b = 64: waves 2 and 3 only help to
//   stage the key tiles).  For every (row, key block) of its key chunk: the
//   block's largest scaled logit m and the sum of exp2(logit - m) over the
//   block's visible keys, written to part[i][row][block] (float2).
// mass_norm, mass_sum: each row's log2-sum-exp over its visible blocks, then
//   mass[i][n] = sum over rows of s * exp2(m - L) in a fixed order.
// ---------------------------------------------------------------------------
template <typename T, int D, int B>
__device__ __forceinline__ void mass_block_body(const Shape& sh, const T* __restrict__ q,
                                                const T* __restrict__ k,
                                                float2* __restrict__ part, int c, int i) {
    typedef typename FragOf<T>::type Frag;
    constexpr int NTH = 256;
    static_assert(B <= 128, "at most 4 waves of 32 last-block rows");
    __shared__ __attribute__((aligned(16))) T tiles[2][32 * KeyTile<T, D, NTH>::LDT];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, h = lane >> 5, lc = lane & 31;
    const int kvh = i / sh.rep;
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

// Row normalisers: one wave per last-block row, 4 rows per 256-thread
// workgroup (`rg`: the workgroup's index among the head's): the row's
// log2-sum-exp over its visible blocks n <= t / b (block n holds key n b <= t,
// so every one of them was written).
__device__ __forceinline__ void mass_norm_body(const Shape& sh, const float2* __restrict__ part,
                                               float* __restrict__ lnorm, int i, int rg) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int b = sh.b, mq = sh.mq;
    const int nrows = min(b, sh.n), t0 = sh.n - nrows;
    const int r = rg * 4 + w;
    if (r >= nrows) return;   // whole waves; no barrier follows
    const int nmax = (t0 + r) / b;
    const float2* pr = part + ((int64_t)i * b + r) * mq;
    // a lane's blocks nb = lane, lane + 64, ... in increasing order, read
    // kNormBatch at a time (all in flight together); selects, not branches,
    // so that each pair is one 8-byte load
    constexpr int kNormBatch = 4;
    float m = kNegInf, s = 0.f;
    for (int nb0 = lane; nb0 <= nmax; nb0 += 64 * kNormBatch) {
        float2 xs[kNormBatch];
#pragma unroll
        for (int u = 0; u < kNormBatch; ++u) {
            const int nb = nb0 + 64 * u;
            xs[u] = pr[min(nb, nmax)];
        }
#pragma unroll
        for (int u = 0; u < kNormBatch; ++u) {
            const float2 x = xs[u];
            const bool use = nb0 + 64 * u <= nmax && x.x != kNegInf;
            const float mn = fmaxf(m, x.x);
            const float sn = (m == kNegInf ? 0.f : s * fast_exp2(m - mn)) + x.y * fast_exp2(x.x - mn);
            s = use ? sn : s;
            m = use ? mn : m;
        }
    }
    const float M = wave_max(m);   // finite: block 0 is visible to every row
    const float sv = wave_sum(m == kNegInf ? 0.f : s * fast_exp2(m - M));
    if (lane == 0) lnorm[(int64_t)i * b + r] = M + log2f(sv);
}

// Block masses: 64 blocks per 256-thread workgroup (`chunk`), one per lane.
// The fixed-order sum: partial p (p = 0..15) adds rows p, p + 16, ... in
// increasing order (wave w computes partials w, w + 4, w + 8, w + 12), then
// the 16 partials are added in order.
constexpr int kMassPartials = 16;

__device__ __forceinline__ void mass_sum_body(const Shape& sh, const float2* __restrict__ part,
                                              const float* __restrict__ lnorm,
                                              float* __restrict__ mass, int i, int chunk) {
    __shared__ float L[128];
    __shared__ float ps[kMassPartials][64];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int b = sh.b, mq = sh.mq;
    const int nrows = min(b, sh.n), t0 = sh.n - nrows;
    for (int r = tid; r < nrows; r += 256) L[r] = lnorm[(int64_t)i * b + r];
    __syncthreads();
    const float2* base = part + (int64_t)i * b * mq;
    const int nb = chunk * 64 + lane;
    // a partial's rows (at most 128 / kMassPartials) are read together, all
    // in flight at once, then accumulated (one fma each) in increasing order;
    // an invisible block or a row past the last reads as (-inf, 0) and is
    // skipped (a select, not a branch, so that each pair is one 8-byte load)
    constexpr int kRowsPerPartial = 128 / kMassPartials;
#pragma unroll
    for (int pp = 0; pp < kMassPartials / 4; ++pp) {
        const int p = w + 4 * pp;
        float2 xs[kRowsPerPartial];
#pragma unroll
        for (int u = 0; u < kRowsPerPartial; ++u) {
            const int r = p + kMassPartials * u;
            xs[u] = (nb < mq && r < nrows && nb * b <= t0 + r) ? base[(int64_t)r * mq + nb]
                                                              : make_float2(kNegInf, 0.f);
        }
        float acc = 0.f;
#pragma unroll
        for (int u = 0; u < kRowsPerPartial; ++u) {
            const int r = min(p + kMassPartials * u, nrows - 1);
            acc = xs[u].x != kNegInf ? fmaf(xs[u].y, fast_exp2(xs[u].x - L[r]), acc) : acc;
        }
        ps[p][lane] = acc;
    }
    __syncthreads();
    if (w == 0 && nb < mq) {
        float sum = 0.f;
#pragma unroll
        for (int p = 0; p < kMassPartials; ++p) sum += ps[p][lane];
        mass[(int64_t)i * mq + nb] = sum;
    }
}

// ---------------------------------------------------------------------------
// The three fused launches (1-D grids of 256-thread workgroups; the
// workgroups of the longer role come first).
// ---------------------------------------------------------------------------
struct EstGrid {
    int pool;      // pooling workgroups
    int mblock;    // mass_block workgroups: nchunks x Hq
    int rowmax;    // est_rowmax workgroups: nbx x est_nc x G (of the band group)
    int nbx;       // 128-row bands of est_rowmax in the band group
    int xb1;       // one past the group's last band (bands run longest first)
    int norm;      // mass_norm workgroups: Hq x ceil(rows / 4) (first group only)
    int norm_per;  // per head
    int reduce;    // est_reduce workgroups: the group's block rows x G
    int m0, nm;    // the group's block rows [m0, m0 + nm)
    int msum;      // mass_sum workgroups: Hq x ceil(Nk / 64) (first group only)
    int msum_per;  // per head
    int64_t tri_base;   // tri_index(m0, 0)
    int64_t tri_count;  // lower-triangular pairs of the group's block rows
};

template <typename T, int D, int B>
__global__ __launch_bounds__(256, 2) void est_stage1_kernel(Shape sh, EstGrid eg,
                                                            const T* __restrict__ q,
                                                            const T* __restrict__ k,
                                                            T* __restrict__ qg, T* __restrict__ kg,
                                                            float2* __restrict__ part) {
    const int j = blockIdx.x;
    if (j < eg.mblock) {
        mass_block_body<T, D, B>(sh, q, k, part, j % sh.nchunks, j / sh.nchunks);
        return;
    }
    pool_body<T, D>(sh, q, k, qg, kg, j - eg.mblock);
}

template <typename T, int D, int BP>
__global__ __launch_bounds__(256, 2) void est_stage2_kernel(Shape sh, EstGrid eg,
                                                            const T* __restrict__ qg,
                                                            const T* __restrict__ kg,
                                                            float* __restrict__ rbm,
                                                            float2* __restrict__ rowpart,
                                                            const float2* __restrict__ part,
                                                            float* __restrict__ lnorm) {
    const int j = blockIdx.x;
    if (j < eg.rowmax) {
        const int bx = j % eg.nbx, c = (j / eg.nbx) % sh.est_nc, g = j / (eg.nbx * sh.est_nc);
        est_rowmax_body<T, D, BP>(sh, qg, kg, rbm, rowpart, (eg.xb1 - 1 - bx) * 128, c, g,
                                  eg.tri_base, eg.tri_count);
        return;
    }
    const int jn = j - eg.rowmax;
    mass_norm_body(sh, part, lnorm, jn / eg.norm_per, jn % eg.norm_per);
}

template <int BP>
__global__ __launch_bounds__(256) void est_stage3_kernel(Shape sh, EstGrid eg,
                                                         const float* __restrict__ rbm,
                                                         const float2* __restrict__ rowpart,
                                                         float* __restrict__ logA,
                                                         const float2* __restrict__ part,
                                                         const float* __restrict__ lnorm,
                                                         float* __restrict__ mass) {
    const int j = blockIdx.x;
    if (j < eg.reduce) {
        est_reduce_body<BP>(sh, rbm, rowpart, logA, eg.m0 + j % eg.nm, j / eg.nm, eg.tri_base,
                            eg.tri_count);
        return;
    }
    const int jm = j - eg.reduce;
    mass_sum_body(sh, part, lnorm, mass, jm / eg.msum_per, jm % eg.msum_per);
}

// ---------------------------------------------------------------------------
// launcher
// ---------------------------------------------------------------------------
static EstGrid est_grid(const Shape& sh) {
    EstGrid e{};
    constexpr int kVec = 16;   // bytes per pooled slice
    const int esz = sh.dtype == 0 ? 2 : 4;
    const int64_t slices = (int64_t)sh.g * sh.np * (sh.d * esz / kVec);
    e.pool = (int)((slices + 255) / 256);
    e.mblock = sh.nchunks * sh.hq;
    e.norm_per = (std::min(sh.b, sh.n) + 3) / 4;
    e.norm = sh.hq * e.norm_per;
    e.msum_per = (sh.mq + 63) / 64;
    e.msum = sh.hq * e.msum_per;
    return e;
}

// Band group k of est_rowmax / est_reduce (see rbm_groups): bands [xb0, xb1)
// of 128 strided rows, block rows [m0, m1).
static void set_group(const Shape& sh, const RbmGroup& gr, bool first, EstGrid* e) {
    const int rows_per_band = 128 / sh.bp;   // block rows per 128-row band
    e->xb1 = gr.xb1;
    e->nbx = gr.xb1 - gr.xb0;
    e->rowmax = e->nbx * sh.est_nc * sh.g;
    e->m0 = gr.xb0 * rows_per_band;
    const int m1 = std::min(gr.xb1 * rows_per_band, sh.mq);
    e->nm = m1 - e->m0;
    e->reduce = e->nm * sh.g;
    e->tri_base = (int64_t)e->m0 * (e->m0 + 1) / 2;
    e->tri_count = (int64_t)m1 * (m1 + 1) / 2 - e->tri_base;
    if (!first) e->norm = e->msum = 0;
}

template <typename T, int D, int B, int BP>
static hipError_t est_t(const Shape& sh, const void* q, const void* k, const EstWs& w,
                        float* logA, float* mass, hipStream_t st) {
    EstGrid eg = est_grid(sh);
    hipLaunchKernelGGL((est_stage1_kernel<T, D, B>), dim3(eg.mblock + eg.pool), dim3(256), 0, st, sh,
                       eg, (const T*)q, (const T*)k, (T*)w.qg, (T*)w.kg, w.part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // est_rowmax writes and est_reduce reads the per-(row, block) maxima one
    // band group at a time, so that their region stays bounded (one group,
    // the whole range, unless it would exceed kRbmMaxBytes); the mass
    // stages ride along with the first group
    const int ngroups = rbm_groups(sh, nullptr);
    for (int k = 0; k < ngroups; ++k) {
        RbmGroup gr;
        rbm_group(sh, k, &gr);
        set_group(sh, gr, k == 0, &eg);
        hipLaunchKernelGGL((est_stage2_kernel<T, D, BP>), dim3(eg.rowmax + eg.norm), dim3(256), 0,
                           st, sh, eg, (const T*)w.qg, (const T*)w.kg, w.rbm, w.rowpart,
                           (const float2*)w.part, w.lnorm);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL((est_stage3_kernel<BP>), dim3(eg.reduce + eg.msum), dim3(256), 0, st, sh,
                           eg, (const float*)w.rbm, (const float2*)w.rowpart, logA,
                           (const float2*)w.part, (const float*)w.lnorm, mass);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

template <typename T, int D, int B>
static hipError_t est_bp(const Shape& sh, const void* q, const void* k, const EstWs& w,
                         float* logA, float* mass, hipStream_t st) {
    switch (sh.bp) {
        case 16: return est_t<T, D, B, 16>(sh, q, k, w, logA, mass, st);
        case 32: return est_t<T, D, B, 32>(sh, q, k, w, logA, mass, st);
        case 64: return est_t<T, D, B, 64>(sh, q, k, w, logA, mass, st);
        case 128: return est_t<T, D, B, 128>(sh, q, k, w, logA, mass, st);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_estimate(const Shape& sh, const void* q, const void* k, const EstWs& w,
                           float* logA, float* mass, hipStream_t st) {
    if (sh.dtype == 0) {
        if (sh.d == 64) return sh.b == 64 ? est_bp<bf16, 64, 64>(sh, q, k, w, logA, mass, st)
                                          : est_bp<bf16, 64, 128>(sh, q, k, w, logA, mass, st);
        return sh.b == 64 ? est_bp<bf16, 128, 64>(sh, q, k, w, logA, mass, st)
                          : est_bp<bf16, 128, 128>(sh, q, k, w, logA, mass, st);
    }
    if (sh.d == 64) return sh.b == 64 ? est_bp<float, 64, 64>(sh, q, k, w, logA, mass, st)
                                      : est_bp<float, 64, 128>(sh, q, k, w, logA, mass, st);
    return sh.b == 64 ? est_bp<float, 128, 64>(sh, q, k, w, logA, mass, st)
                      : est_bp<float, 128, 128>(sh, q, k, w, logA, mass, st);
}

}  // namespace pa
