// Host-side enumeration of the attention kernel's work-item order (built by
// tests/test_work_order.py with the host C++ compiler): for every order,
// chunk size, count of short rows that the KV-head-major order ends on and
// a range of shapes, every ticket number maps to a valid
// (block row, query head) or to padding, every item is reached exactly once,
// and the number of ticket numbers is a multiple of the queue count.
// Prints "<cases> cases, <bad> bad" and exits non-zero on any failure.
#include <cstdio>
#include <utility>
#include <vector>

#include "work_order.h"

int main() {
    long bad = 0, cases = 0;
    const std::pair<int, int> heads[] = {{32, 8}, {28, 4}, {8, 2}, {12, 3}, {4, 4}, {16, 1}, {64, 8}, {6, 6}};
    for (int mq : {1, 2, 3, 7, 8, 9, 15, 16, 17, 33, 64, 100, 127, 128, 129, 255, 512, 1024, 2048})
        for (const auto& hh : heads)
            for (int order = 0; order <= 2; ++order)
                for (int R : {1, 2, 3, 4, 7, 16, 64, 8192})
                for (int sd : {0, 1, 2, 4, 8, -1}) {
                    if (order != 2 && sd != 8) continue;   // only order 2 reads it
                    pa::Shape sh{};
                    sh.mq = mq;
                    sh.hq = hh.first;
                    sh.hkv = hh.second;
                    sh.rep = sh.hq / sh.hkv;
                    sh.attn_order = order;
                    sh.attn_chunk_rows = R;
                    // short rows: none, all, mq / 2, mq / 4, mq / 8, or out of range
                    sh.attn_short_rows = sd == 0 ? 0 : sd == -1 ? mq + 5 : mq / sd;
                    ++cases;
                    const int n = pa::attn_items(sh);
                    if (n % pa::kNumXcd != 0) {
                        ++bad;
                        std::printf("mq %d hq %d hkv %d order %d R %d: %d items, not a multiple of %d\n",
                                    mq, sh.hq, sh.hkv, order, R, n, pa::kNumXcd);
                        continue;
                    }
                    std::vector<int> seen((size_t)mq * sh.hq, 0);
                    bool ok = true;
                    for (int b = 0; b < n && ok; ++b) {
                        int m = -1, i = -1;
                        if (!pa::attn_item(sh, b, &m, &i)) continue;
                        if (m < 0 || m >= mq || i < 0 || i >= sh.hq) {
                            std::printf("mq %d hq %d hkv %d order %d R %d short %d: ticket %d -> (%d, %d)\n",
                                        mq, sh.hq, sh.hkv, order, R, sh.attn_short_rows, b, m, i);
                            ok = false;
                        } else {
                            ++seen[(size_t)m * sh.hq + i];
                        }
                    }
                    for (size_t j = 0; j < seen.size() && ok; ++j)
                        if (seen[j] != 1) {
                            std::printf("mq %d hq %d hkv %d order %d R %d short %d: row %zu head %zu taken %d times\n",
                                        mq, sh.hq, sh.hkv, order, R, sh.attn_short_rows, j / sh.hq,
                                        j % sh.hq, seen[j]);
                            ok = false;
                        }
                    bad += !ok;
                }
    std::printf("%ld cases, %ld bad\n", cases, bad);
    return bad != 0;
}
