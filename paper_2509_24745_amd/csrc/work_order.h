// The attention kernel's work-item order: which (query head, block row)
// item each ticket of the persistent workgroups' queues stands for.  Plain
// integer arithmetic on the problem's sizes, callable on the host as well
// (a host test enumerates it).  Not part of the public interface.
#pragma once

#include "internal.h"

namespace pa {

// Order 2 ends on the block rows m < attn_short_rows (see attn_item).
__host__ __device__ __forceinline__ int short_rows(const Shape& sh) {
    return sh.attn_short_rows < 0 ? 0 : (sh.attn_short_rows > sh.mq ? sh.mq : sh.attn_short_rows);
}
// Order 2: work-item numbers per queue in its first phase (KV-head-major
// chunks of the rows m >= short_rows).
__host__ __device__ __forceinline__ int kv_major_per_queue(const Shape& sh) {
    const int R = sh.attn_chunk_rows;
    const int chunks = sh.hkv * ((sh.mq - short_rows(sh) + R - 1) / R);
    return ((chunks + kNumXcd - 1) / kNumXcd) * sh.rep * R;
}

// Work item number `b` (b % 8 = queue, b / 8 = position in that queue).  The
// queues are drained by the persistent workgroups of one XCD each (workgroup
// w serves queue w % 8: workgroups are dealt to the XCDs round-robin), so
// queue x is XCD x's work in the order it is taken.
// Order 0: longest block rows first, heads fastest.
// Order 1 (row chunks): chunks of R consecutive block rows (longest first)
//   x all query heads, KV heads outermost inside a chunk; chunk c runs on
//   XCD c % 8.  Inside an XCD the query heads of one KV head on neighbouring
//   rows are adjacent, so the K/V sub-blocks they fetch are shared through
//   the XCD's L2; chunks dealt in turn balance the XCDs.
// Order 2 (KV-head-major chunks, then the short rows): first the rows
//   m >= M0 = attn_short_rows (mq / 8 or mq / 4) in chunks of R rows x the
//   query heads of ONE KV head, ordered KV head by KV head; chunk L runs on
//   XCD L % 8.  At any time the
//   whole GPU reads the K/V of about one KV head, which stays resident in the
//   MALL.  Then the rows m < M0 of every head, longest first, the query heads
//   of one KV head together (group g on XCD g % 8).  A row sees at most m + 1
//   blocks, so the queues end on short items and the workgroups finish close
//   together (ending on the last KV head's rows instead left slots idle for
//   up to a long item's time); these rows read only the first M0 key blocks
//   of each KV head, which the MALL holds together.
// Returns false for padding workgroups.
__host__ __device__ __forceinline__ bool attn_item(const Shape& sh, int b, int* m_out, int* i_out) {
    const int R = sh.attn_chunk_rows;
    if (sh.attn_order == 0 || R <= 0) {
        if (b >= sh.hq * sh.mq) return false;
        *m_out = sh.mq - 1 - b / sh.hq;
        *i_out = b % sh.hq;
        return true;
    }
    const int x = b % kNumXcd, slot = b / kNumXcd;
    if (sh.attn_order == 1) {
        const int chunk_items = sh.hq * R;
        const int c = x + kNumXcd * (slot / chunk_items);
        const int within = slot % chunk_items;
        const int kv = within / (R * sh.rep);
        const int r = (within / sh.rep) % R;
        const int m = sh.mq - 1 - (c * R + r);
        if (m < 0) return false;
        *m_out = m;
        *i_out = kv * sh.rep + within % sh.rep;
        return true;
    }
    const int m0 = short_rows(sh), first = kv_major_per_queue(sh);
    if (slot < first) {
        const int chunk_items = sh.rep * R;
        const int chunks_per_kv = (sh.mq - m0 + R - 1) / R;
        const int L = x + kNumXcd * (slot / chunk_items);
        if (L >= sh.hkv * chunks_per_kv) return false;
        const int kv = L / chunks_per_kv, c = L % chunks_per_kv;
        const int within = slot % chunk_items;
        const int m = sh.mq - 1 - (c * R + within / sh.rep);
        if (m < m0) return false;
        *m_out = m;
        *i_out = kv * sh.rep + within % sh.rep;
        return true;
    }
    const int t = slot - first;
    const int g = x + kNumXcd * (t / sh.rep);
    if (g >= m0 * sh.hkv) return false;
    *m_out = m0 - 1 - g / sh.hkv;
    *i_out = (g % sh.hkv) * sh.rep + t % sh.rep;
    return true;
}

// Number of work-item numbers (a multiple of kNumXcd; some are padding).
__host__ __device__ __forceinline__ int attn_items(const Shape& sh) {
    const int R = sh.attn_chunk_rows;
    if (sh.attn_order == 0 || R <= 0) return kNumXcd * ((sh.hq * sh.mq + kNumXcd - 1) / kNumXcd);
    if (sh.attn_order == 1) {
        const int chunks = (sh.mq + R - 1) / R;
        return kNumXcd * ((chunks + kNumXcd - 1) / kNumXcd) * sh.hq * R;
    }
    const int groups = short_rows(sh) * sh.hkv;
    return kNumXcd * (kv_major_per_queue(sh) + ((groups + kNumXcd - 1) / kNumXcd) * sh.rep);
}

}  // namespace pa
