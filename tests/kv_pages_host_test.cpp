// Host unit test of the paged-KV bookkeeping (paper_2505_17218_amd/csrc/kv_pages.h),
// built with g++ under the address and undefined-behaviour sanitizers and bounds-checked
// standard containers (tests/test_kv_pages_host.py).  Exercises allocation order, the
// group fork (shared full pages, copied partial page), growth, release with reference
// counts, capacity checks, and a seeded random sequence of operations with the book's
// consistency check after every step.
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "kv_pages.h"

using dash::PageBook;

static int g_fail = 0;
#define EXPECT(c)                                                        \
    do {                                                                 \
        if (!(c)) {                                                      \
            std::fprintf(stderr, "%s:%d: expected %s\n", __FILE__, __LINE__, #c); \
            ++g_fail;                                                    \
        }                                                                \
    } while (0)
#define CONSISTENT(b)                                                    \
    do {                                                                 \
        const std::string e_ = (b).check();                              \
        if (!e_.empty()) {                                               \
            std::fprintf(stderr, "%s:%d: inconsistent: %s\n", __FILE__, __LINE__, e_.c_str()); \
            ++g_fail;                                                    \
        }                                                                \
    } while (0)

static void fork_and_release() {
    PageBook b;
    b.init(10, 6, 4, 32);  // 10 pages, 6 slots of up to 4 pages (128 positions), page size 32
    EXPECT(b.free_pages() == 10);
    CONSISTENT(b);
    // 2 prompts of 40 positions, groups of 3: per prompt one full page + a partial page per sample
    EXPECT(b.fork_need(2, 40, 3) == 8);
    const int32_t slots[6] = {0, 1, 2, 3, 4, 5};
    std::vector<int32_t> pairs;
    b.fork(slots, 2, 40, 3, pairs);
    CONSISTENT(b);
    EXPECT(b.free_pages() == 2);
    // pages are handed out 0, 1, 2, ...: prompt 0 owns 0 (full) and 1 (partial), its
    // samples 1 and 2 share page 0 and copy page 1 into pages 2 and 3
    EXPECT(b.at(0, 0) == 0 && b.at(0, 1) == 1);
    EXPECT(b.at(1, 0) == 0 && b.at(1, 1) == 2);
    EXPECT(b.at(2, 0) == 0 && b.at(2, 1) == 3);
    EXPECT(b.at(3, 0) == 4 && b.at(3, 1) == 5 && b.at(4, 1) == 6 && b.at(5, 1) == 7 && b.at(5, 0) == 4);
    EXPECT(b.refc[0] == 3 && b.refc[4] == 3 && b.refc[1] == 1 && b.refc[7] == 1);
    const std::vector<int32_t> want_pairs = {1, 2, 1, 3, 5, 6, 5, 7};
    EXPECT(pairs == want_pairs);
    for (int s = 0; s < 6; ++s) EXPECT(b.len[s] == 40 && b.npages[s] == 2);
    // slot 0 grows to 65 positions: one more page
    const int32_t s0[1] = {0};
    EXPECT(b.grow_need(s0, 1, 65) == 1);
    EXPECT(b.grow(0, 65));
    EXPECT(b.at(0, 2) == 8 && b.len[0] == 65 && b.free_pages() == 1);
    EXPECT(!b.grow(0, 60));          // already backed: nothing mapped, length kept
    EXPECT(b.len[0] == 65);
    CONSISTENT(b);
    // slots 1 and 2 to 65 positions need two pages, one is free: the caller refuses
    const int32_t s12[2] = {1, 2};
    EXPECT(b.grow_need(s12, 2, 65) == 2 && b.grow_need(s12, 2, 65) > b.free_pages());
    // release: the shared page survives until the last sample of its group lets go
    b.release(0);
    CONSISTENT(b);
    EXPECT(b.refc[0] == 2 && b.free_pages() == 3 && b.empty(0));
    b.release(1);
    b.release(2);
    CONSISTENT(b);
    EXPECT(b.refc[0] == 0 && b.free_pages() == 6);
    b.release(2);  // an empty slot: no change
    CONSISTENT(b);
    EXPECT(b.free_pages() == 6);
    for (int s = 3; s < 6; ++s) b.release(s);
    CONSISTENT(b);
    EXPECT(b.free_pages() == 10);
    for (int p = 0; p < 10; ++p) EXPECT(b.refc[p] == 0);
    // a prompt filling whole pages copies nothing
    pairs.clear();
    EXPECT(b.fork_need(1, 64, 3) == 2);
    b.fork(slots, 1, 64, 3, pairs);
    EXPECT(pairs.empty() && b.refc[b.at(0, 0)] == 3 && b.refc[b.at(0, 1)] == 3 && b.free_pages() == 8);
    CONSISTENT(b);
}

static void random_operations(unsigned seed) {
    std::mt19937 rng(seed);
    const int pages = 64, seqs = 24, max_pages = 6, ps = 16;
    PageBook b;
    b.init(pages, seqs, max_pages, ps);
    auto rnd = [&](int n) { return (int)(rng() % (unsigned)n); };
    int refused = 0, ops = 0;
    for (int it = 0; it < 4000; ++it) {
        const int op = rnd(3);
        if (op == 0) {  // fork a group into empty slots
            const int G = 1 + rnd(4), P = 1 + rnd(max_pages * ps - 1);
            std::vector<int32_t> free_slots;
            for (int s = 0; s < seqs; ++s)
                if (b.empty(s)) free_slots.push_back(s);
            if ((int)free_slots.size() < G) continue;
            std::shuffle(free_slots.begin(), free_slots.end(), rng);
            free_slots.resize(G);
            if (b.fork_need(1, P, G) > b.free_pages()) {
                ++refused;
                continue;
            }
            const size_t before = b.free_pages();
            std::vector<int32_t> pairs;
            b.fork(free_slots.data(), 1, P, G, pairs);
            EXPECT(before - b.free_pages() == b.fork_need(1, P, G));
            EXPECT((int)pairs.size() == (P % ps ? 2 * (G - 1) : 0));
        } else if (op == 1) {  // grow a few slots
            std::vector<int32_t> sl;
            for (int k = 0, n = 1 + rnd(4); k < n; ++k) {
                const int s = rnd(seqs);
                if (!b.empty(s) && std::find(sl.begin(), sl.end(), s) == sl.end()) sl.push_back(s);
            }
            if (sl.empty()) continue;
            const int new_len = 1 + rnd(max_pages * ps);
            const size_t need = b.grow_need(sl.data(), (int)sl.size(), new_len);
            if (need > b.free_pages()) {
                ++refused;
                continue;
            }
            const size_t before = b.free_pages();
            for (int s : sl) b.grow(s, new_len);
            EXPECT(before - b.free_pages() == need);
            for (int s : sl) EXPECT(b.len[s] >= new_len);
        } else {  // release a slot
            b.release(rnd(seqs));
        }
        ++ops;
        CONSISTENT(b);
        if (g_fail) return;
    }
    for (int s = 0; s < seqs; ++s) b.release(s);
    CONSISTENT(b);
    EXPECT(b.free_pages() == (size_t)pages);
    std::printf("seed %u: %d operations, %d refused for capacity\n", seed, ops, refused);
}

int main() {
    fork_and_release();
    for (unsigned seed = 1; seed <= 5; ++seed) random_operations(seed);
    if (g_fail) {
        std::fprintf(stderr, "%d failures\n", g_fail);
        return 1;
    }
    std::printf("kv_pages host test ok\n");
    return 0;
}
