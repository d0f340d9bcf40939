// Host bookkeeping of the paged KV cache: the free list of pages, per-page
// reference counts, each slot's page list and length, the group fork and
// release.  No device code and no HIP calls: the library mirrors this state to
// the device page table, and a host unit test builds this header on its own
// under the address and undefined-behaviour sanitizers.
//
// A slot is one sequence's row of the page table.  Sec. 3.4 duplicates every
// prompt into a group of G samples: after the prompt's forward pass the G slots
// of a group reference the prompt's full pages (reference count G), and each
// slot gets a private copy of a partial last prompt page (copy on write, done
// by the caller with the (source, destination) pairs fork() returns).  Pages
// whose count drops to zero go back to the free list.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <string>
#include <vector>

namespace dash {

struct PageBook {
    int n_pages = 0;    // pages in the pool
    int max_seqs = 0;   // slots
    int max_pages = 0;  // page-table row length
    int page_size = 1;  // positions per page
    std::vector<int32_t> table;      // [max_seqs][max_pages], -1 = no page
    std::vector<int32_t> len;        // positions held per slot
    std::vector<int32_t> npages;     // pages mapped per slot
    std::vector<int32_t> refc;       // references per page
    std::vector<int32_t> free_list;  // free pages; the back is handed out first

    void init(int pages, int seqs, int pages_per_slot, int ps) {
        n_pages = pages;
        max_seqs = seqs;
        max_pages = pages_per_slot;
        page_size = ps;
        table.assign((size_t)seqs * pages_per_slot, -1);
        len.assign(seqs, 0);
        npages.assign(seqs, 0);
        refc.assign(pages, 0);
        free_list.resize(pages);
        for (int i = 0; i < pages; ++i) free_list[i] = pages - 1 - i;  // pages 0, 1, 2, ... first
    }

    size_t free_pages() const { return free_list.size(); }
    bool empty(int slot) const { return npages[slot] == 0 && len[slot] == 0; }
    int32_t& at(int slot, int j) { return table[(size_t)slot * max_pages + j]; }
    int32_t at(int slot, int j) const { return table[(size_t)slot * max_pages + j]; }
    int pages_for(int positions) const { return (positions + page_size - 1) / page_size; }

    // A free page with reference count 1.  Precondition: free_pages() > 0.
    int alloc() {
        const int p = free_list.back();
        free_list.pop_back();
        refc[p] = 1;
        return p;
    }

    void unref(int p) {
        if (--refc[p] == 0) free_list.push_back(p);
    }

    // Pages that growing `slots` to new_len positions would map (an over-estimate if a
    // slot is listed twice).
    size_t grow_need(const int32_t* slots, int n, int new_len) const {
        size_t need = 0;
        const int want = pages_for(new_len);
        for (int i = 0; i < n; ++i)
            if (want > npages[slots[i]]) need += want - npages[slots[i]];
        return need;
    }

    // Map pages so that positions [0, new_len) of `slot` are backed and raise its
    // length to new_len.  Returns whether pages were mapped.  The caller has checked
    // capacity (grow_need <= free_pages) and new_len <= max_pages * page_size.
    bool grow(int slot, int new_len) {
        const int want = pages_for(new_len);
        const bool mapped = npages[slot] < want;
        while (npages[slot] < want) {
            at(slot, npages[slot]) = alloc();
            npages[slot]++;
        }
        if (len[slot] < new_len) len[slot] = new_len;
        return mapped;
    }

    // Drop a slot's references; its pages return to the free list when unreferenced.
    void release(int slot) {
        for (int j = 0; j < npages[slot]; ++j) {
            unref(at(slot, j));
            at(slot, j) = -1;
        }
        npages[slot] = 0;
        len[slot] = 0;
    }

    // Pages a group fork of n_prompts prompts of P positions into groups of G maps:
    // the full prompt pages once per prompt, a partial last page once per sample.
    size_t fork_need(int n_prompts, int P, int G) const {
        const size_t full = P / page_size, part = P % page_size ? 1 : 0;
        return (size_t)n_prompts * (full + part * G);
    }

    // Map the prompt pages of slots[p * G + j] (all empty; capacity checked with
    // fork_need): sample 0 of each prompt owns the prompt's pages, samples 1..G-1
    // reference its full pages and get a fresh page for a partial last one; the
    // (source, destination) page pairs to copy are appended to `pairs`.
    void fork(const int32_t* slots, int n_prompts, int P, int G, std::vector<int32_t>& pairs) {
        const int full = P / page_size, part = P % page_size ? 1 : 0;
        for (int p = 0; p < n_prompts; ++p) {
            const int s0 = slots[p * G];
            for (int j = 0; j < full + part; ++j) at(s0, j) = alloc();
            npages[s0] = full + part;
            len[s0] = P;
            for (int g = 1; g < G; ++g) {
                const int s = slots[p * G + g];
                for (int j = 0; j < full; ++j) {
                    const int pg = at(s0, j);
                    at(s, j) = pg;
                    refc[pg]++;
                }
                if (part) {
                    const int pg = alloc();
                    at(s, full) = pg;
                    pairs.push_back(at(s0, full));
                    pairs.push_back(pg);
                }
                npages[s] = full + part;
                len[s] = P;
            }
        }
    }

    // Consistency of the whole book ("" if consistent): every reference count equals
    // the number of table entries naming the page, free pages are exactly the
    // unreferenced ones (each listed once), slots map exactly npages pages that cover
    // their length, and no slot maps a page twice.
    std::string check() const {
        std::vector<int32_t> count(n_pages, 0);
        for (int s = 0; s < max_seqs; ++s) {
            if (npages[s] < 0 || npages[s] > max_pages) return "slot " + std::to_string(s) + ": bad page count";
            if (len[s] < 0 || pages_for(len[s]) > npages[s]) return "slot " + std::to_string(s) + ": length not backed";
            for (int j = 0; j < max_pages; ++j) {
                const int pg = at(s, j);
                if (j >= npages[s]) {
                    if (pg != -1) return "slot " + std::to_string(s) + ": entry past its pages";
                    continue;
                }
                if (pg < 0 || pg >= n_pages) return "slot " + std::to_string(s) + ": page out of range";
                for (int i = 0; i < j; ++i)
                    if (at(s, i) == pg) return "slot " + std::to_string(s) + ": page mapped twice";
                count[pg]++;
            }
        }
        std::vector<char> in_free(n_pages, 0);
        for (int pg : free_list) {
            if (pg < 0 || pg >= n_pages) return "free list: page out of range";
            if (in_free[pg]) return "free list: page " + std::to_string(pg) + " listed twice";
            in_free[pg] = 1;
        }
        for (int pg = 0; pg < n_pages; ++pg) {
            if (refc[pg] != count[pg]) return "page " + std::to_string(pg) + ": reference count mismatch";
            if ((refc[pg] == 0) != (in_free[pg] != 0)) return "page " + std::to_string(pg) + ": free list mismatch";
        }
        return "";
    }
};

}  // namespace dash
